// File-backed lower tier: see bsr_file_tier.h.
#include "bsr_file_tier.h"

#include <dirent.h>
#include <errno.h>
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <thread>

namespace bsr {

namespace {

constexpr char kMagic[8] = {'B', 'S', 'R', 'T', 'I', 'E', 'R', '1'};
constexpr uint32_t kVersion = 1;
constexpr uint32_t kMaxGroups = 8;

struct Header {
  char magic[8];
  uint32_t version;
  uint32_t n_groups;
  uint64_t key;
  uint64_t slot_bytes;
  uint32_t present;
  uint32_t pad;
  uint64_t tags[kMaxGroups];
};
static_assert(sizeof(Header) <= FileTier::kHeaderBytes, "header fits its block");

uint64_t round4k(uint64_t x) { return (x + 4095) / 4096 * 4096; }

uint64_t steady_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

// Reads exactly n bytes; a file that ends early fails with errno = ENODATA.
bool full_pread(int fd, void* buf, uint64_t n, uint64_t off) {
  uint8_t* p = static_cast<uint8_t*>(buf);
  while (n) {
    const ssize_t r = pread(fd, p, n, static_cast<off_t>(off));
    if (r < 0 && errno == EINTR) continue;
    if (r == 0) errno = ENODATA;
    if (r <= 0) return false;
    p += r;
    off += static_cast<uint64_t>(r);
    n -= static_cast<uint64_t>(r);
  }
  return true;
}

bool full_pwrite(int fd, const void* buf, uint64_t n, uint64_t off) {
  const uint8_t* p = static_cast<const uint8_t*>(buf);
  while (n) {
    const ssize_t r = pwrite(fd, p, n, static_cast<off_t>(off));
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    p += r;
    off += static_cast<uint64_t>(r);
    n -= static_cast<uint64_t>(r);
  }
  return true;
}

}  // namespace

std::string FileTier::path_of(uint64_t key) const {
  char name[40];
  std::snprintf(name, sizeof name, "/%016llx.bsr", static_cast<unsigned long long>(key));
  return dir_ + name;
}

int FileTier::open(const std::string& dir, uint32_t n_groups, uint64_t slot_bytes, const uint64_t* offsets,
                   const uint64_t* payload, uint32_t concurrency, uint32_t readahead, bool direct,
                   std::string* err) {
  if (open_) {
    *err = "file tier already open";
    return -1;
  }
  if (n_groups == 0 || n_groups > kMaxGroups) {
    *err = "file tier supports 1..8 groups";
    return -1;
  }
  if (mkdir(dir.c_str(), 0755) != 0 && errno != EEXIST) {
    *err = "cannot create " + dir + ": " + std::strerror(errno);
    return -1;
  }
  dir_ = dir;
  n_groups_ = n_groups;
  slot_bytes_ = slot_bytes;
  file_bytes_ = kHeaderBytes + round4k(slot_bytes);
  offsets_.assign(offsets, offsets + n_groups);
  payload_.assign(payload, payload + n_groups);
  concurrency_ = concurrency ? concurrency : 1;
  readahead_ = readahead ? readahead : 2 * concurrency_;
  if (readahead_ < concurrency_) readahead_ = concurrency_;
  direct_ = direct;
  // index what the directory already holds (the tier outlives processes)
  DIR* d = opendir(dir.c_str());
  if (d) {
    while (dirent* e = readdir(d)) {
      const size_t len = std::strlen(e->d_name);
      if (len < 5 || std::strcmp(e->d_name + len - 4, ".bsr") != 0) continue;
      const std::string p = dir_ + "/" + e->d_name;
      const int fd = ::open(p.c_str(), O_RDONLY);
      if (fd < 0) continue;
      Header h{};
      if (full_pread(fd, &h, sizeof h, 0) && std::memcmp(h.magic, kMagic, 8) == 0 && h.version == kVersion &&
          h.n_groups == n_groups_ && h.slot_bytes == slot_bytes_ && h.present) {
        Meta m;
        m.present = h.present;
        std::memcpy(m.tags, h.tags, sizeof m.tags);
        index_[h.key] = m;
      }
      ::close(fd);
    }
    closedir(d);
  }
  open_ = true;
  return 0;
}

int FileTier::start(int device, std::string* err) {
  if (started_) return 0;
  device_ = device;
  bounce_.assign(readahead_, nullptr);
  bounce_dev_.assign(readahead_, nullptr);
  bounce_ev_.assign(readahead_, nullptr);
  slots_.assign(readahead_, Slot{});
  for (uint32_t b = 0; b < readahead_; ++b) {
    void* p = nullptr;
    const bool ok = hipHostMalloc(&p, file_bytes_, hipHostMallocDefault) == hipSuccess &&
                    hipEventCreateWithFlags(&bounce_ev_[b], hipEventDisableTiming) == hipSuccess;
    bounce_[b] = static_cast<uint8_t*>(p);
    void* dv = nullptr;
    if (ok && hipHostGetDevicePointer(&dv, p, 0) == hipSuccess) bounce_dev_[b] = static_cast<const uint8_t*>(dv);
    else (void)hipGetLastError();
    if (!ok) {
      *err = "file tier: bounce buffers could not be allocated";
      for (uint32_t k = 0; k <= b; ++k) {
        if (bounce_ev_[k]) (void)hipEventDestroy(bounce_ev_[k]);
        if (bounce_[k]) (void)hipHostFree(bounce_[k]);
      }
      bounce_.clear();
      bounce_dev_.clear();
      bounce_ev_.clear();
      return -1;
    }
  }
  stop_ = false;
  for (uint32_t t = 0; t < concurrency_; ++t) workers_.emplace_back(&FileTier::worker, this);
  started_ = true;
  return 0;
}

void FileTier::close() {
  if (started_) {
    drain();
    {
      std::lock_guard<std::mutex> lk(qmu_);
      stop_ = true;
    }
    qcv_.notify_all();
    for (auto& w : workers_) w.join();
    workers_.clear();
    if (device_ >= 0) (void)hipSetDevice(device_);
    for (auto e : bounce_ev_)
      if (e) (void)hipEventDestroy(e);
    for (auto p : bounce_)
      if (p) (void)hipHostFree(p);
    bounce_.clear();
    bounce_dev_.clear();
    bounce_ev_.clear();
    started_ = false;
  }
  open_ = false;
}

bool FileTier::has(uint64_t key, uint32_t g) const {
  std::lock_guard<std::mutex> lk(imu_);
  auto it = index_.find(key);
  return it != index_.end() && ((it->second.present >> g) & 1u);
}

bool FileTier::tag(uint64_t key, uint32_t g, uint64_t* t) const {
  std::lock_guard<std::mutex> lk(imu_);
  auto it = index_.find(key);
  if (it == index_.end() || !((it->second.present >> g) & 1u)) return false;
  *t = it->second.tags[g];
  return true;
}

uint64_t FileTier::n_entries() const {
  std::lock_guard<std::mutex> lk(imu_);
  uint64_t n = 0;
  for (auto& kv : index_) n += __builtin_popcount(kv.second.present);
  return n;
}

int FileTier::write_header(int fd, uint64_t key, uint32_t present, const uint64_t* tags) {
  std::vector<uint8_t> blk(kHeaderBytes, 0);
  Header h{};
  std::memcpy(h.magic, kMagic, 8);
  h.version = kVersion;
  h.n_groups = n_groups_;
  h.key = key;
  h.slot_bytes = slot_bytes_;
  h.present = present;
  std::memcpy(h.tags, tags, sizeof h.tags);
  std::memcpy(blk.data(), &h, sizeof h);
  return full_pwrite(fd, blk.data(), kHeaderBytes, 0) ? 0 : -1;
}

int FileTier::put(uint64_t key, const void* const* payloads, const uint64_t* tags, std::string* err) {
  std::vector<uint8_t> body(file_bytes_ - kHeaderBytes, 0);
  for (uint32_t g = 0; g < n_groups_; ++g) std::memcpy(body.data() + offsets_[g], payloads[g], payload_[g]);
  uint64_t t[kMaxGroups] = {};
  for (uint32_t g = 0; g < n_groups_; ++g) t[g] = tags[g];
  const uint32_t present = (n_groups_ == 32) ? 0xFFFFFFFFu : ((1u << n_groups_) - 1);
  // write a private file, then rename it over the chunk's file: a reader
  // sees the old file or the new one, never a partial one
  const std::string p = path_of(key);
  char suffix[48];
  std::snprintf(suffix, sizeof suffix, ".%llx.tmp", static_cast<unsigned long long>(
                                                        std::hash<std::thread::id>()(std::this_thread::get_id())));
  const std::string tmp = p + suffix;
  const int fd = ::open(tmp.c_str(), O_WRONLY | O_CREAT | O_TRUNC, 0644);
  if (fd < 0) {
    *err = "cannot write " + tmp + ": " + std::strerror(errno);
    return -1;
  }
  const bool ok = write_header(fd, key, present, t) == 0 && full_pwrite(fd, body.data(), body.size(), kHeaderBytes);
  ::close(fd);
  if (!ok || ::rename(tmp.c_str(), p.c_str()) != 0) {
    *err = (ok ? "cannot rename " : "short write to ") + tmp;
    ::unlink(tmp.c_str());
    return -1;
  }
  std::lock_guard<std::mutex> lk(imu_);
  Meta m;
  m.present = present;
  std::memcpy(m.tags, t, sizeof m.tags);
  index_[key] = m;
  return 0;
}

int FileTier::remove(uint64_t key, int32_t group, std::string* err) {
  std::lock_guard<std::mutex> lk(imu_);
  auto it = index_.find(key);
  if (it == index_.end() || (group >= 0 && !((it->second.present >> group) & 1u))) {
    *err = "no such file-tier entry";
    return 1;
  }
  const std::string p = path_of(key);
  const uint32_t left = group < 0 ? 0u : (it->second.present & ~(1u << group));
  if (left == 0) {
    ::unlink(p.c_str());
    index_.erase(it);
    return 0;
  }
  const int fd = ::open(p.c_str(), O_WRONLY);
  if (fd < 0 || write_header(fd, key, left, it->second.tags) != 0) {
    if (fd >= 0) ::close(fd);
    *err = "cannot rewrite header of " + p;
    return -1;
  }
  ::close(fd);
  it->second.present = left;
  return 0;
}

void FileTier::submit(uint32_t b, uint64_t key) {
  {
    std::lock_guard<std::mutex> lk(qmu_);
    Slot& s = slots_[b];
    ++s.gen;
    s.status = kReadPending;
    queue_.push_back(Task{b, key, s.gen});
  }
  qcv_.notify_one();
}

int FileTier::wait(uint32_t b, uint64_t deadline_ns, uint32_t* present_mask, int* os_error) {
  std::unique_lock<std::mutex> lk(qmu_);
  Slot& s = slots_[b];
  while (s.done_gen != s.gen) {
    if (deadline_ns) {
      const uint64_t now = steady_ns();
      if (now >= deadline_ns) return kReadPending;
      dcv_.wait_for(lk, std::chrono::nanoseconds(deadline_ns - now));
    } else {
      dcv_.wait(lk);
    }
  }
  if (present_mask) *present_mask = s.present;
  if (os_error) *os_error = s.err;
  return s.status;
}

void FileTier::drain() {
  std::unique_lock<std::mutex> lk(qmu_);
  dcv_.wait(lk, [&] { return queue_.empty() && running_ == 0; });
}

void FileTier::worker() {
  (void)hipSetDevice(device_);
  // O_DIRECT reads land in an ordinary page-aligned buffer (direct I/O cannot
  // target the driver-mapped pinned memory), then are copied to the bounce
  // buffer; buffered reads go straight to the bounce buffer.
  uint8_t* aligned = nullptr;
  if (direct_) {
    void* p = nullptr;
    if (posix_memalign(&p, 4096, file_bytes_) == 0) aligned = static_cast<uint8_t*>(p);
  }
  for (;;) {
    Task t;
    {
      std::unique_lock<std::mutex> lk(qmu_);
      qcv_.wait(lk, [&] { return stop_ || !queue_.empty(); });
      if (stop_ && queue_.empty()) {
        std::free(aligned);
        return;
      }
      t = queue_.front();
      queue_.pop_front();
      ++running_;
    }
    // the previous device copy out of this bounce buffer must be complete
    (void)hipEventSynchronize(bounce_ev_[t.b]);
    int status = kReadOk, err = 0;
    uint32_t present = 0;
    const std::string p = path_of(t.key);
    uint8_t* land = direct_ ? aligned : bounce_[t.b];
    const int fd = land ? ::open(p.c_str(), O_RDONLY | (direct_ ? O_DIRECT : 0)) : -1;
    if (fd < 0) {
      err = land ? errno : ENOMEM;
      status = err == ENOENT ? kReadMissing : kReadIoError;
    } else {
      if (!full_pread(fd, land, file_bytes_, 0)) {
        err = errno;
        status = err == ENODATA ? kReadMissing : kReadIoError;  // a truncated file holds no complete object
      } else {
        if (land != bounce_[t.b]) std::memcpy(bounce_[t.b], land, file_bytes_);
        Header h{};
        std::memcpy(&h, bounce_[t.b], sizeof h);
        if (std::memcmp(h.magic, kMagic, 8) != 0 || h.key != t.key || h.slot_bytes != slot_bytes_)
          status = kReadMissing;
        else
          present = h.present;
      }
      ::close(fd);
    }
    {
      std::lock_guard<std::mutex> lk(qmu_);
      Slot& s = slots_[t.b];
      if (s.gen == t.gen) {
        s.status = status;
        s.err = err;
        s.present = present;
        s.done_gen = t.gen;
      }
      --running_;
    }
    dcv_.notify_all();
  }
}

}  // namespace bsr
