// A lower external tier backed by files (one file per chunk), read by a
// pool of threads into a bounded pool of pinned bounce buffers.
//
// §4 "System topology" keeps local SSD as a lower reusable tier under the
// remote store, and §4 "Storage-side concurrency is orthogonal" loads a
// window's objects with a configurable number of concurrent readers; §6.5
// shows load concurrency changing throughput, not the restore working set.
// Here the reader count is that load concurrency, and the bounce pool is the
// host-side landing zone between the file and the device ring (its size is
// reported separately from the ring).
//
// File format (little-endian): a 4 KiB header {magic "BSRTIER1", version,
// n_groups, key, slot_bytes, present-group mask, one tag per group}, then
// the chunk's entries laid out like a staging slot, zero-padded to a 4 KiB
// multiple so the whole file can be read with O_DIRECT.
#pragma once

#include <hip/hip_runtime_api.h>

#include <stdint.h>

#include <condition_variable>
#include <deque>
#include <mutex>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

namespace bsr {

class FileTier {
 public:
  enum ReadStatus : int { kReadPending = 0, kReadOk = 1, kReadMissing = 2, kReadIoError = 3 };

  ~FileTier() { close(); }

  // Open (create) the directory and index every valid file already in it.
  int open(const std::string& dir, uint32_t n_groups, uint64_t slot_bytes, const uint64_t* offsets,
           const uint64_t* payload, uint32_t concurrency, uint32_t readahead, bool direct, std::string* err);
  bool is_open() const { return open_; }
  void close();

  bool available = true;

  bool has(uint64_t key, uint32_t g) const;
  bool tag(uint64_t key, uint32_t g, uint64_t* t) const;
  uint64_t n_entries() const;

  // Write (replace) the chunk file of `key`.  tags[g] are stored in the header.
  int put(uint64_t key, const void* const* payloads, const uint64_t* tags, std::string* err);
  // Remove one group (or all when group < 0); the file goes when no group is left.
  int remove(uint64_t key, int32_t group, std::string* err);

  // ---- reads (need a GPU context: pinned bounce buffers, HIP events) ----
  int start(int device, std::string* err);  // allocate the bounce pool and start the readers
  uint32_t pool_size() const { return readahead_; }
  uint64_t bounce_bytes() const { return static_cast<uint64_t>(readahead_) * file_bytes_; }
  const uint8_t* bounce_data(uint32_t b) const { return bounce_[b] + kHeaderBytes; }
  // the whole pinned buffer b (header and body) and the device's view of it
  const uint8_t* bounce_base(uint32_t b) const { return bounce_[b]; }
  const uint8_t* bounce_device(uint32_t b) const { return bounce_dev_[b]; }
  uint64_t file_bytes() const { return file_bytes_; }
  hipEvent_t bounce_event(uint32_t b) const { return bounce_ev_[b]; }
  // Queue a read of key's file into bounce buffer b.  The reader first waits
  // for bounce_event(b), i.e. for the last device copy out of that buffer.
  void submit(uint32_t b, uint64_t key);
  // Wait for the read into b; returns a ReadStatus (kReadPending on deadline).
  // present_mask receives the header's group mask on success.
  int wait(uint32_t b, uint64_t deadline_ns, uint32_t* present_mask, int* os_error = nullptr);
  // Wait until no read is queued or running.
  void drain();

  static constexpr uint64_t kHeaderBytes = 4096;

 private:
  struct Task {
    uint32_t b;
    uint64_t key;
    uint64_t gen;
  };
  struct Slot {
    uint64_t gen = 0;     // generation of the last submitted read
    uint64_t done_gen = 0;
    int status = kReadOk;
    int err = 0;          // errno of a failed open/read
    uint32_t present = 0;
  };
  std::string path_of(uint64_t key) const;
  void worker();
  int write_header(int fd, uint64_t key, uint32_t present, const uint64_t* tags);

  bool open_ = false;
  bool direct_ = false;
  int device_ = -1;
  std::string dir_;
  uint32_t n_groups_ = 0;
  uint64_t slot_bytes_ = 0;
  uint64_t file_bytes_ = 0;  // header + slot, padded to 4 KiB
  std::vector<uint64_t> offsets_, payload_;
  uint32_t concurrency_ = 1, readahead_ = 1;

  mutable std::mutex imu_;  // index
  struct Meta {
    uint32_t present = 0;
    uint64_t tags[8] = {};
  };
  std::unordered_map<uint64_t, Meta> index_;

  std::mutex qmu_;  // queue + slots
  std::condition_variable qcv_, dcv_;
  std::deque<Task> queue_;
  uint32_t running_ = 0;
  bool stop_ = false;
  bool started_ = false;
  std::vector<Slot> slots_;
  std::vector<uint8_t*> bounce_;
  std::vector<const uint8_t*> bounce_dev_;  // device views of the bounce buffers (null: copy engine only)
  std::vector<hipEvent_t> bounce_ev_;
  std::vector<std::thread> workers_;
};

}  // namespace bsr
