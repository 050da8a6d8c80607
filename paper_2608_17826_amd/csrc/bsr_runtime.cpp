// Host runtime of the bounded-window restore: external pinned-host store,
// chunk-key chain and probe, the W-slot staging ring scheduler, and the
// request state machine behind include/bsr.h.
//
// Paper map (arxiv 2608.17826):
//   probe             §3 "Probe globally", §4 probe_only lookup
//   window loop       §2 "Bounded installation" (Eqs. 3-4), §3 "Install
//                     locally", §4 windowed retrieve
//   admission         §3 "Install locally" (one bounded restore at a time),
//                     or §7's global budget B over the bound requests' rings
//   commit/invalidate §3 Eq. 6 and Prop. 2, §4 "vLLM failure integration"
//   force-local       §3 "Recover without re-entering the same fault"
//
// The ring: chunk i is staged in slot i mod W.  Its copy (pinned host ->
// slot, copy stream) waits for the event that released the slot's previous
// chunk; its install (compute stream) waits for the batch's copies.  The
// device therefore never holds more than W staged chunks, whatever N is.
// Copies of chunks adjacent in the arena and in the ring go out together.
// Each bound request has its own session slot (tag partials, verify words,
// events, status mirror), allocated with the context.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "bsr.h"
#include "bsr_device.h"
#include "bsr_file_tier.h"

namespace {

using bsr::FinishParams;
using bsr::GroupGeom;
using bsr::InstallParams;
using bsr::TagPair;
using bsr::VerifyParams;

thread_local std::string g_err;

int fail_with(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

uint64_t now_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(
             std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

constexpr uint64_t kAlign = 256;
// Requests of at most this many chunk bytes are staged on the compute stream
// (Session::one_stream).
constexpr uint64_t kOneStreamBytes = 64ull << 20;
// Install launches whose staged chunks exceed this many bytes walk their
// chunks in alternate directions from one dispatch position to the next
// (InstallHead::serpentine).  Measured on the 512K 4-group layout: launches
// of 28 and 56 chunks (459 and 919 MB) gain 1.5-1.6 points of 8 TB/s; 14
// chunks (230 MB) gain nothing and 7 chunks lose 0.4.  The gain starts
// where a launch outgrows the 256 MiB Infinity Cache in front of HBM.
constexpr uint64_t kSerpentineBytes = 256ull << 20;
constexpr uint32_t kTimingFlags = BSR_FLAG_TIME_INSTALL | BSR_FLAG_TIME_STAGE;
constexpr uint64_t kArenaBlockAlign = 4096;
uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// FNV-1a-64 (FNV specification: XOR the octet, multiply by the FNV prime)
// ---------------------------------------------------------------------------
constexpr uint64_t kFnvBasis = 0xcbf29ce484222325ull;
constexpr uint64_t kFnvPrime = 0x00000100000001b3ull;

uint64_t fnv1a64(const uint8_t* p, size_t n, uint64_t h = kFnvBasis) {
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= kFnvPrime;
  }
  return h;
}

bool host_is_little_endian() {
  const uint32_t one = 1;
  uint8_t b;
  std::memcpy(&b, &one, 1);
  return b == 1;
}

// d_i for every full chunk, data-parallel over chunks for long inputs.
void chunk_digests(const int32_t* tokens, uint64_t n_chunks, uint32_t C, uint64_t* d) {
  const uint64_t bytes = static_cast<uint64_t>(C) * 4;
  auto work = [&](uint64_t lo, uint64_t hi) {
    for (uint64_t i = lo; i < hi; ++i)
      d[i] = fnv1a64(reinterpret_cast<const uint8_t*>(tokens + i * C), bytes);
  };
  const uint64_t total = n_chunks * bytes;
  unsigned nt = std::thread::hardware_concurrency();
  if (nt > 8) nt = 8;
  if (total < (1u << 20) || nt <= 1 || n_chunks < 2 * nt) {
    work(0, n_chunks);
    return;
  }
  std::vector<std::thread> th;
  const uint64_t per = (n_chunks + nt - 1) / nt;
  for (unsigned t = 0; t < nt; ++t) {
    const uint64_t lo = t * per, hi = std::min(n_chunks, lo + per);
    if (lo < hi) th.emplace_back(work, lo, hi);
  }
  for (auto& x : th) x.join();
}

void chain_keys(uint64_t salt, const int32_t* tokens, uint64_t n_chunks, uint32_t C, uint64_t* keys) {
  std::vector<uint64_t> d(n_chunks);
  chunk_digests(tokens, n_chunks, C, d.data());
  uint64_t h = salt;
  for (uint64_t i = 0; i < n_chunks; ++i) {
    uint8_t rec[16];
    std::memcpy(rec, &h, 8);  // little-endian host (checked at entry)
    std::memcpy(rec + 8, &d[i], 8);
    h = fnv1a64(rec, 16);
    keys[i] = h;
  }
}

// (XOR of LE u32 words) << 32 | (sum mod 2^32)
uint64_t tag_of(const uint8_t* p, uint64_t n) {
  uint32_t s = 0, x = 0;
  const uint64_t nw = n / 4;
  for (uint64_t i = 0; i < nw; ++i) {
    uint32_t w;
    std::memcpy(&w, p + 4 * i, 4);
    s += w;
    x ^= w;
  }
  return (static_cast<uint64_t>(x) << 32) | s;
}

// ---------------------------------------------------------------------------
// layout
// ---------------------------------------------------------------------------
struct Geometry {
  bsr_layout L{};
  uint64_t payload[BSR_MAX_GROUPS]{};
  uint64_t offset[BSR_MAX_GROUPS]{};
  uint64_t slot_bytes = 0;
  uint64_t chunk_payload = 0;
  GroupGeom gg[BSR_MAX_GROUPS]{};  // geometry without request pointers
  uint32_t wg_start[BSR_MAX_GROUPS + 1]{};
  uint32_t wg_per_chunk = 0;
  uint32_t lds_bytes = 0;
  uint32_t order[BSR_MAX_GROUPS]{};  // install dispatch order of the groups
  uint32_t order_prefix[BSR_MAX_GROUPS + 1]{};  // workgroups per chunk before each position of that order
};

int check_layout(const bsr_layout* L) {
  if (!L) return fail_with(BSR_E_ARG, "layout is NULL");
  if (L->chunk_tokens == 0) return fail_with(BSR_E_ARG, "chunk_tokens must be >= 1");
  if (L->n_groups == 0 || L->n_groups > BSR_MAX_GROUPS)
    return fail_with(BSR_E_ARG, "n_groups must be in 1..%d", BSR_MAX_GROUPS);
  uint64_t slot = 0;
  for (uint32_t g = 0; g < L->n_groups; ++g) {
    const bsr_group_desc& d = L->groups[g];
    if (d.block_tokens == 0 || d.n_tensors == 0) return fail_with(BSR_E_ARG, "group %u: zero block_tokens/n_tensors", g);
    if (d.record_bytes < 4 || d.record_bytes % 4) return fail_with(BSR_E_ARG, "group %u: record_bytes must be a positive multiple of 4", g);
    if (d.kind != BSR_KIND_CONTIG && d.kind != BSR_KIND_PLANAR) return fail_with(BSR_E_ARG, "group %u: unknown kind %u", g, d.kind);
    if (d.kind == BSR_KIND_PLANAR && (d.split_bytes == 0 || d.split_bytes % 4 || d.split_bytes >= d.record_bytes))
      return fail_with(BSR_E_ARG, "group %u: planar split_bytes must be a multiple of 4 in (0, record_bytes)", g);
    if (static_cast<uint64_t>(d.block_tokens) * d.record_bytes >= (1ull << 31))
      return fail_with(BSR_E_ARG, "group %u: block bytes too large", g);
    slot += align_up(static_cast<uint64_t>(d.n_tensors) * L->chunk_tokens * d.record_bytes, kAlign);
  }
  if (slot >= (1ull << 32)) return fail_with(BSR_E_ARG, "slot bytes %llu exceed 4 GiB", (unsigned long long)slot);
  return BSR_OK;
}

void build_geometry(const bsr_layout* L, Geometry* G) {
  G->L = *L;
  const uint32_t C = L->chunk_tokens;
  uint64_t off = 0;
  uint32_t wg = 0;
  G->lds_bytes = 0;
  for (uint32_t g = 0; g < L->n_groups; ++g) {
    const bsr_group_desc& d = L->groups[g];
    G->payload[g] = static_cast<uint64_t>(d.n_tensors) * C * d.record_bytes;
    G->offset[g] = off;
    off += align_up(G->payload[g], kAlign);
    GroupGeom& q = G->gg[g];
    q = GroupGeom{};
    q.block_tokens = d.block_tokens;
    q.n_tensors = d.n_tensors;
    q.record_bytes = d.record_bytes;
    q.kind = d.kind;
    q.split_bytes = d.kind == BSR_KIND_PLANAR ? d.split_bytes : 0;
    q.staged_off = static_cast<uint32_t>(G->offset[g]);
    const uint32_t B = d.block_tokens;
    // destination blocks one chunk can touch
    if (C % B == 0)
      q.segs_per_chunk = C / B;
    else if (B % C == 0)
      q.segs_per_chunk = 1;
    else
      q.segs_per_chunk = (C + B - 1) / B + 1;
    const uint32_t seg_tokens = std::min(B, C);
    if (d.kind == BSR_KIND_CONTIG) {
      // equal pieces of at most kMaxPieceBytes, each a multiple of 4 KiB
      const uint64_t seg = static_cast<uint64_t>(seg_tokens) * d.record_bytes;
      const uint64_t n = (seg + bsr::kMaxPieceBytes - 1) / bsr::kMaxPieceBytes;
      q.piece_bytes = static_cast<uint32_t>(align_up((seg + n - 1) / n, bsr::kPieceAlign));
      q.pieces_per_seg = static_cast<uint32_t>((seg + q.piece_bytes - 1) / q.piece_bytes);
      q.piece_tokens = 0;
    } else {
      // tokens per LDS piece: fits the LDS budget and keeps pieces 16-byte multiples
      uint32_t step = 16 / std::__gcd(d.record_bytes, 16u);
      uint32_t pt = std::min(seg_tokens, bsr::kLdsCapBytes / d.record_bytes);
      if (pt >= step) pt -= pt % step;
      if (pt == 0) pt = 1;
      q.piece_tokens = pt;
      q.pieces_per_seg = (seg_tokens + pt - 1) / pt;
      q.piece_bytes = 0;
      const uint32_t need = static_cast<uint32_t>(align_up(static_cast<uint64_t>(pt) * d.record_bytes, 16));
      if (need <= bsr::kLdsCapBytes) G->lds_bytes = std::max(G->lds_bytes, need);  // else: 4-byte word path
    }
    G->wg_start[g] = wg;
    wg += d.n_tensors * q.segs_per_chunk * q.pieces_per_seg;
    q.div_pieces = bsr::make_fastdiv(q.pieces_per_seg);
    q.div_segs = bsr::make_fastdiv(q.segs_per_chunk);
    q.div_per_chunk = bsr::make_fastdiv(d.n_tensors * q.segs_per_chunk * q.pieces_per_seg);
    q.div_block = bsr::make_fastdiv(B);
  }
  G->wg_start[L->n_groups] = wg;
  for (uint32_t g = L->n_groups + 1; g <= BSR_MAX_GROUPS; ++g) G->wg_start[g] = wg;
  G->wg_per_chunk = wg;
  // dispatch order: contiguous groups by descending piece size, then
  // descending block size, with the planar (LDS-staged) groups placed just
  // before the last contiguous group, so that planar pieces, the slowest per
  // workgroup, never form a launch's tail.  On the 512K 4-group layout
  // (three contiguous groups of 8 KiB pieces) the block-size tie-break puts
  // the 16 KB-block group last: 76.4% -> 76.8% of 8 TB/s at W = 32, 76.2 ->
  // 78.3% at W = 16, 62.9 -> 67.2% at W = 8, before the serpentine order
  // (kSerpentineBytes) adds its own gain; planar last, with it: 75.2%
  uint32_t contig[BSR_MAX_GROUPS], planar[BSR_MAX_GROUPS], nc = 0, np = 0;
  for (uint32_t g = 0; g < L->n_groups; ++g) (G->gg[g].kind == BSR_KIND_PLANAR ? planar[np++] : contig[nc++]) = g;
  std::stable_sort(contig, contig + nc, [&](uint32_t a, uint32_t b) {
    const GroupGeom &x = G->gg[a], &y = G->gg[b];
    if (x.piece_bytes != y.piece_bytes) return x.piece_bytes > y.piece_bytes;
    return static_cast<uint64_t>(x.block_tokens) * x.record_bytes > static_cast<uint64_t>(y.block_tokens) * y.record_bytes;
  });
  uint32_t pos = 0;
  for (uint32_t i = 0; i + 1 < nc; ++i) G->order[pos++] = contig[i];
  for (uint32_t i = 0; i < np; ++i) G->order[pos++] = planar[i];
  if (nc) G->order[pos++] = contig[nc - 1];
  uint32_t acc = 0;
  for (uint32_t o = 0; o < L->n_groups; ++o) {
    G->order_prefix[o] = acc;
    acc += G->wg_start[G->order[o] + 1] - G->wg_start[G->order[o]];
  }
  for (uint32_t o = L->n_groups; o <= BSR_MAX_GROUPS; ++o) G->order_prefix[o] = acc;
  G->slot_bytes = off;
  G->chunk_payload = 0;
  for (uint32_t g = 0; g < L->n_groups; ++g) G->chunk_payload += G->payload[g];
}

// ---------------------------------------------------------------------------
// store: a pinned arena cut into slot-shaped blocks
// ---------------------------------------------------------------------------
struct Entry {
  uint32_t block;
  uint64_t tag;
};

struct BlockMeta {
  uint32_t live_groups = 0;  // index entries pointing here
  uint32_t refs = 0;         // references held by bound requests
};

struct Store {
  uint8_t* arena = nullptr;
  uint64_t arena_bytes = 0;
  bool owned = false;
  // the device's view of the arena when HIP reports it pinned over its whole
  // range (the staging-copy kernel reads it); null: the copy engine copies
  const uint8_t* arena_dev = nullptr;
  uint64_t block_stride = 0;
  uint32_t n_blocks = 0;
  std::vector<BlockMeta> meta;
  std::vector<uint32_t> free_list;
  uint32_t next_fresh = 0;
  std::vector<std::unordered_map<uint64_t, Entry>> index;  // per group
  uint64_t n_entries = 0;
  uint32_t blocks_in_use = 0;

  uint8_t* block_ptr(uint32_t b) const { return arena + static_cast<uint64_t>(b) * block_stride; }
  bool alloc(uint32_t* b) {
    if (!free_list.empty()) {
      *b = free_list.back();
      free_list.pop_back();
    } else if (next_fresh < n_blocks) {
      *b = next_fresh++;
    } else {
      return false;
    }
    meta[*b] = BlockMeta{};
    ++blocks_in_use;
    return true;
  }
  void maybe_free(uint32_t b) {
    if (meta[b].live_groups == 0 && meta[b].refs == 0) {
      free_list.push_back(b);
      --blocks_in_use;
    }
  }
};

// ---------------------------------------------------------------------------
// requests
// ---------------------------------------------------------------------------
enum class Phase { Probed, Bound, Failed, Done };

constexpr uint8_t kTierPinned = 0;  // the pinned-host store
constexpr uint8_t kTierFile = 1;    // the file-backed lower tier
constexpr uint8_t kTierNone = 0xFF;

struct Request {
  std::vector<uint64_t> keys;
  std::vector<uint8_t> tier;  // per chunk: the tier the probe found it in
  uint32_t n_probe = 0;
  Phase phase = Phase::Probed;
  uint64_t probe_ns = 0;
  bool has_stats = false;  // counters of its last completion
  bsr_stats stats{};
};

struct Inject {
  int32_t kind = BSR_INJECT_NONE;
  uint32_t chunk = 0;
  uint32_t param = 0;
};

// Device and host resources of one session slot, allocated when the context
// is created so that binding a request allocates nothing.
struct SessionRes {
  TagPair* partials = nullptr;            // per-wave tag partials of one install launch
  bsr::VerifyAux* verify_aux = nullptr;   // verify words
  bsr_dev_status* host_status = nullptr;  // pinned mirror of the status block
  std::vector<hipEvent_t> full_ev, free_ev;
  bool in_use = false;
  // A context that allocates nothing: partials and verify words are in the
  // library's static array, and the status mirror is status_buf (plain host
  // memory; the readback waits for the stream anyway).
  bool static_scratch = false;
  bsr_dev_status status_buf{};
};

struct Session {  // one bound request
  uint64_t id = 0;
  uint32_t res = 0;            // session slot
  uint64_t ring_bytes = 0;     // its share of the admission budget
  uint32_t n_hit = 0;
  uint32_t window = 0;  // slots of this request's ring: W, or n_hit in whole-plan mode
  uint32_t next_chunk = 0;
  bool failed = false;
  bool completing = false;  // a commit or end is waiting for its device work
  // A small request is staged on the compute stream itself (copy == compute):
  // stream order then does what the copy and release events do between two
  // streams, without their hand-over latency.
  bool one_stream = false;
  uint32_t batch = 0;       // chunks per install launch
  bool copy_dirty = false;  // the copy stream holds work no compute-stream wait covers yet
  uint32_t time_flags = 0;  // BSR_FLAG_TIME_INSTALL / BSR_FLAG_TIME_STAGE, taken at bind
  int host_fail = BSR_FAIL_NONE;
  uint8_t* staging = nullptr;
  bsr_dev_status* status = nullptr;
  hipStream_t copy = nullptr, compute = nullptr;
  InstallParams ip{};
  FinishParams fp{};
  std::vector<uint32_t> refs;  // arena blocks referenced
  std::vector<int64_t> slot_free_seq;
  int64_t copy_waited_seq = -1;
  int64_t batch_seq = 0;
  uint32_t slots_touched = 0;
  std::vector<uint8_t> slot_used;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> timing;        // install launches
  std::vector<std::pair<hipEvent_t, hipEvent_t>> stage_timing;  // staging-copy launches
  // chunks copied but not yet installed (the current install batch)
  std::vector<uint32_t> pend;
  std::vector<std::array<uint64_t, BSR_MAX_GROUPS>> pend_tags;
  Inject inject;   // armed before this request was bound
  bsr_stats st{};  // this request's counters
};

}  // namespace

struct bsr_ctx {
  Geometry geo;
  bsr_config cfg{};
  uint32_t W = 0;
  uint32_t batch = 0;      // chunks per install launch of a request staged on the copy stream
  uint32_t batch_one = 0;  // ... and of one staged on the compute stream
  int device = -1;
  std::mutex mu;
  Store store;
  std::unordered_map<uint64_t, Request> requests;
  std::unordered_set<uint64_t> force_local;
  bool tier0_available = true;
  bsr::FileTier ftier;
  // admission: the lock (budget 0) or the global budget B
  uint64_t budget = 0;
  std::vector<SessionRes> res;                  // session slots
  std::unordered_map<uint64_t, Session> bound;  // request id -> its session
  uint64_t bound_bytes = 0, peak_bound_bytes = 0;
  uint32_t peak_bound = 0, n_refused = 0;
  uint64_t last_id = 0;   // request most recently bound or completed
  bsr_stats last{};       // its counters when it is no longer bound
  Inject inject;          // armed for the next bind
  uint64_t partials_bytes = 0;  // per session slot
  uint64_t aux_bytes = 0;       // device bytes per session slot
  uint32_t xcd_log2 = 3;        // log2 of the XCDs of the device's partition
  std::vector<hipEvent_t> timing_pool;
  bool static_claimed = false;  // holds its device's static scratch array
  bool kernel_copies = true;    // staging copies by k_stage (else the copy engine)
};

namespace {

int hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return BSR_OK;
  return fail_with(BSR_E_TRANSFER, "%s: %s", what, hipGetErrorString(e));
}

int set_device(bsr_ctx* c) {
  if (c->device < 0) return fail_with(BSR_E_DEVICE, "operation needs a GPU context (hip_device >= 0)");
  return hip_check(hipSetDevice(c->device), "hipSetDevice");
}

hipEvent_t take_timing_event(bsr_ctx* c) {
  if (!c->timing_pool.empty()) {
    hipEvent_t e = c->timing_pool.back();
    c->timing_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void release_refs(bsr_ctx* c, Session& s) {
  for (uint32_t b : s.refs) {
    if (c->store.meta[b].refs) --c->store.meta[b].refs;
    c->store.maybe_free(b);
  }
  s.refs.clear();
}

Session* find_bound(bsr_ctx* c, uint64_t request_id) {
  auto it = c->bound.find(request_id);
  return it == c->bound.end() ? nullptr : &it->second;
}

// The bound request the caller may act on: BSR_E_STATE when it is not bound
// or another call is already completing it.
int find_active(bsr_ctx* c, uint64_t request_id, Session** out) {
  Session* s = find_bound(c, request_id);
  if (!s) return fail_with(BSR_E_STATE, "request %llu is not bound", (unsigned long long)request_id);
  if (s->completing) return fail_with(BSR_E_STATE, "request %llu is being completed", (unsigned long long)request_id);
  *out = s;
  return BSR_OK;
}

// A staging copy of `bytes` from host memory `src` into the ring at `dst`, on
// the copy stream.  When the source lies in a pinned allocation
// [base, base + extent) whose device view is `dev`, k_stage reads it over
// the host link; otherwise (or with BSR_FLAG_SDMA_COPIES) the copy engine
// copies it.  Both ranges are checked here before any kernel is launched:
// the source inside its pinned allocation, the destination inside this
// request's ring.
hipError_t stage_copy(bsr_ctx* c, Session& s, uint8_t* dst, const uint8_t* src, uint64_t bytes, const uint8_t* base,
                      const uint8_t* dev, uint64_t extent) {
  s.copy_dirty = true;
  // With several requests bound, each staging on a copy stream of its own,
  // their k_stage launches would run side by side on the link; the copy
  // engine queues them instead (3 requests of 512K tokens: 56.9 against
  // 56.6 GB/s in aggregate, the installs beside them at 76% of HBM against 67%).
  const bool shared_link = c->bound.size() > 1 && s.copy != s.compute;
  if (!c->kernel_copies || shared_link || !dev || !base)
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s.copy);
  const bool src_in = src >= base && bytes <= extent && static_cast<uint64_t>(src - base) <= extent - bytes;
  const bool dst_in = dst >= s.staging && bytes <= s.ring_bytes &&
                      static_cast<uint64_t>(dst - s.staging) <= s.ring_bytes - bytes;
  if (!src_in || !dst_in) return hipErrorInvalidValue;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  if (s.time_flags & BSR_FLAG_TIME_STAGE) {
    t0 = take_timing_event(c);
    t1 = take_timing_event(c);
    if (!t0 || !t1) {
      if (t0) c->timing_pool.push_back(t0);
      if (t1) c->timing_pool.push_back(t1);
      t0 = t1 = nullptr;
    }
  }
  const hipError_t e = bsr::launch_stage(bsr::StageParams{dev + (src - base), dst, bytes}, s.copy, t0, t1);
  if (e != hipSuccess) {
    if (t0) c->timing_pool.push_back(t0);
    if (t1) c->timing_pool.push_back(t1);
    return e;
  }
  if (t0) s.stage_timing.emplace_back(t0, t1);
  ++s.st.n_stage_launches;
  s.st.stage_bytes += bytes;
  return hipSuccess;
}

// Enqueue install + verify for the chunks staged since the last flush.
int flush_batch(bsr_ctx* c, Session& s) {
  std::vector<uint32_t>& chunks = s.pend;
  std::vector<std::array<uint64_t, BSR_MAX_GROUPS>>& tags = s.pend_tags;
  if (chunks.empty()) return BSR_OK;
  if (chunks.size() > BSR_MAX_INSTALL_BATCH)  // the verify launch holds one expected tag row per chunk
    return fail_with(BSR_E_STATE, "install batch of %zu chunks exceeds %d", chunks.size(), BSR_MAX_INSTALL_BATCH);
  if (s.inject.kind == BSR_INJECT_LAUNCH_ERROR &&
      std::find(chunks.begin(), chunks.end(), s.inject.chunk) != chunks.end()) {
    const uint32_t at = s.inject.chunk;
    s.inject = Inject{};  // one shot: the retry at commit launches normally
    return fail_with(BSR_E_TRANSFER, "injected install launch failure (batch with chunk %u)", at);
  }
  SessionRes& r = c->res[s.res];
  const uint32_t E = static_cast<uint32_t>(r.full_ev.size());
  const int64_t seq = s.batch_seq++;
  hipEvent_t full = r.full_ev[seq % E];
  hipEvent_t freed = r.free_ev[seq % E];
  int rc;
  if (!s.one_stream) {  // on one stream the copies already precede this install
    if ((rc = hip_check(hipEventRecord(full, s.copy), "hipEventRecord(full)"))) return rc;
    if ((rc = hip_check(hipStreamWaitEvent(s.compute, full, 0), "hipStreamWaitEvent(full)"))) return rc;
    s.copy_dirty = false;
  }

  // the kernel takes chunk first_chunk + c to slot first_slot + c, less W
  // once: a launch holds consecutive chunks, at most W of them
  if (chunks.size() > s.window || chunks.back() - chunks.front() + 1 != chunks.size())
    return fail_with(BSR_E_STATE, "install batch of %zu chunks is not a run of at most W = %u", chunks.size(), s.window);
  InstallParams ip = s.ip;
  ip.h.n_chunks = static_cast<uint32_t>(chunks.size());
  ip.h.first_chunk = chunks.front();
  ip.h.first_slot = chunks.front() % s.window;
  for (uint32_t o = 0; o < BSR_MAX_GROUPS; ++o) ip.h.start[o] = ip.h.n_chunks * c->geo.order_prefix[o];
  ip.h.xcd_full = bsr::xcd_remap_bound(ip.h.n_chunks * ip.h.wg_per_chunk, ip.h.xcd_log2);
  ip.h.serpentine = static_cast<uint64_t>(ip.h.n_chunks) * c->geo.slot_bytes > kSerpentineBytes ? 1u : 0u;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  if (s.time_flags & BSR_FLAG_TIME_INSTALL) {
    t0 = take_timing_event(c);
    t1 = take_timing_event(c);
    if (!t0 || !t1) {
      if (t0) c->timing_pool.push_back(t0);
      if (t1) c->timing_pool.push_back(t1);
      t0 = t1 = nullptr;
    }
  }
  if ((rc = hip_check(bsr::launch_install(ip, ip.h.n_chunks * ip.h.wg_per_chunk, s.compute, t0, t1), "install launch"))) {
    if (t0) c->timing_pool.push_back(t0);
    if (t1) c->timing_pool.push_back(t1);
    return rc;
  }
  if (t0 && t1) s.timing.emplace_back(t0, t1);
  // The batch's slots are free once the install has read them: the verify
  // kernel reads only the tag partials, which the next install (later on
  // this stream) overwrites after it.  Releasing here keeps the verify off
  // the copy engine's path to the slots.
  if (!s.one_stream && (rc = hip_check(hipEventRecord(freed, s.compute), "hipEventRecord(free)"))) return rc;
  for (uint32_t ch : chunks) s.slot_free_seq[ch % s.window] = seq;
  VerifyParams vp{};
  vp.partials = r.partials;
  vp.status = s.status;
  vp.aux = r.verify_aux;
  vp.n_chunks = ip.h.n_chunks;
  vp.first_chunk = ip.h.first_chunk;
  vp.n_groups = c->geo.L.n_groups;
  vp.wg_per_chunk = ip.h.wg_per_chunk;
  std::memcpy(vp.wg_start, c->geo.wg_start, sizeof vp.wg_start);
  for (size_t i = 0; i < chunks.size(); ++i)
    for (uint32_t g = 0; g < BSR_MAX_GROUPS; ++g) vp.expected[i][g] = tags[i][g];
  if ((rc = hip_check(bsr::launch_verify(vp, s.compute), "verify launch"))) return rc;
  s.st.n_install_launches++;
  s.st.installed_bytes += static_cast<uint64_t>(chunks.size()) * c->geo.chunk_payload;
  chunks.clear();
  tags.clear();
  return BSR_OK;
}

int enqueue_finish(bsr_ctx* c, Session& s, uint32_t mode, uint32_t reason, uint32_t chunk, uint32_t mask) {
  // chunks still waiting for their install go first (stream order)
  if (int rc = flush_batch(c, s)) return rc;
  FinishParams fp = s.fp;
  fp.mode = mode;
  fp.reason = reason;
  fp.chunk = chunk;
  fp.group_mask = mask;
  return hip_check(bsr::launch_finish(fp, s.compute), "finish launch");
}

// A launch or enqueue failed: the device may not hold what the host
// enqueued, so the request can no longer be exposed.  Commit invalidates it
// (and no further window of it is accepted).
int launch_failed(bsr_ctx* c, Session& s, int code) {
  s.failed = true;
  if (s.host_fail == BSR_FAIL_NONE) s.host_fail = BSR_FAIL_TRANSFER;
  c->force_local.insert(s.id);
  return code;
}

// Host-detected failure: invalidate the whole advertised prefix.
int host_fail(bsr_ctx* c, Session& s, int reason, uint32_t chunk, uint32_t mask, int code) {
  const std::string msg = g_err;
  c->ftier.drain();  // no read of this request may still target a bounce buffer
  int rc = enqueue_finish(c, s, bsr::kFinishInvalidate, static_cast<uint32_t>(reason), chunk, mask);
  s.failed = true;
  if (s.host_fail == BSR_FAIL_NONE) s.host_fail = reason;
  c->force_local.insert(s.id);
  if (rc) return rc;
  g_err = msg;
  return code;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

int32_t bsr_abi_version(void) { return BSR_ABI_VERSION; }

uint64_t bsr_struct_size(int32_t which) {
  switch (which) {
    case BSR_STRUCT_LAYOUT: return sizeof(bsr_layout);
    case BSR_STRUCT_CONFIG: return sizeof(bsr_config);
    case BSR_STRUCT_GROUP_DST: return sizeof(bsr_group_dst);
    case BSR_STRUCT_DEV_STATUS: return sizeof(bsr_dev_status);
    case BSR_STRUCT_STATS: return sizeof(bsr_stats);
    case BSR_STRUCT_ADMISSION: return sizeof(bsr_admission);
    default: return 0;
  }
}

const char* bsr_last_error(void) { return g_err.c_str(); }

uint64_t bsr_slot_bytes(const bsr_layout* layout) {
  if (check_layout(layout)) return 0;
  Geometry G;
  build_geometry(layout, &G);
  return G.slot_bytes;
}

uint64_t bsr_staging_bytes(const bsr_layout* layout, uint32_t window_chunks) {
  if (window_chunks == 0) {
    fail_with(BSR_E_ARG, "W must be >= 1");
    return 0;
  }
  return bsr_slot_bytes(layout) * window_chunks;
}

uint64_t bsr_plan_staging_bytes(bsr_ctx* c, uint32_t n_hit_chunks) {
  if (!c) {
    fail_with(BSR_E_ARG, "ctx is NULL");
    return 0;
  }
  const uint64_t slots = c->W ? c->W : std::max(1u, n_hit_chunks);
  return slots * c->geo.slot_bytes;
}

int bsr_chunk_keys(uint64_t salt, const int32_t* tokens, uint64_t n_tokens, uint32_t chunk_tokens,
                   uint64_t* keys_out) {
  if (!host_is_little_endian()) return fail_with(BSR_E_ARG, "big-endian host unsupported");
  if (chunk_tokens == 0) return fail_with(BSR_E_ARG, "chunk_tokens must be >= 1");
  const uint64_t n = n_tokens / chunk_tokens;
  if (n == 0) return BSR_OK;
  if (!tokens || !keys_out) return fail_with(BSR_E_ARG, "tokens/keys_out is NULL");
  chain_keys(salt, tokens, n, chunk_tokens, keys_out);
  return BSR_OK;
}

static void free_session_res(SessionRes& r) {
  for (auto e : r.full_ev)
    if (e) (void)hipEventDestroy(e);
  for (auto e : r.free_ev)
    if (e) (void)hipEventDestroy(e);
  r.full_ev.clear();
  r.free_ev.clear();
  if (!r.static_scratch) {
    if (r.partials) (void)hipFree(r.partials);
    if (r.verify_aux) (void)hipFree(r.verify_aux);
    if (r.host_status) (void)hipHostFree(r.host_status);
  }
  r.partials = nullptr;
  r.verify_aux = nullptr;
  r.host_status = nullptr;
}

static int ctx_create(const bsr_layout* layout, const bsr_config* config, bsr_ctx** out, bool static_scratch) {
  if (!out) return fail_with(BSR_E_ARG, "out is NULL");
  *out = nullptr;
  if (int rc = check_layout(layout)) return rc;
  if (!config) return fail_with(BSR_E_ARG, "config is NULL");
  if (config->flags & ~(kTimingFlags | BSR_FLAG_TRUSTED_TABLES | BSR_FLAG_SDMA_COPIES | BSR_FLAG_TWO_STREAMS))
    return fail_with(BSR_E_ARG, "unknown config flags 0x%x", config->flags);
  // W = 0 is the legacy whole-plan mode (§4 "Restore-window configuration"):
  // each request's ring holds its whole plan and no slot is reused.
  const uint32_t W = config->window_chunks;
  uint32_t b = config->install_batch;
  // automatic: W - max(1, W/8) chunks per launch: large launches, and at
  // least one chunk-copy of slack before a slot's next copy needs its
  // install (W = 1 has no slack to give).  A whole-window launch makes the
  // first copy of every window wait for the previous window's install: at
  // W = 8 (512K 4-group workload, kernel staging copies) b = 8 restores
  // 55.4 GB/s, b = 4/6/7 56.3; at W = 16, b = 16 55.9, b = 8/12/14 56.7-56.8;
  // at W = 32, b = 32 56.0, b = 24/28 57.0.
  if (b == 0)
    b = W == 0 ? static_cast<uint32_t>(BSR_MAX_INSTALL_BATCH)
               : std::max(1u, std::min(W - std::max(1u, W / 8), static_cast<uint32_t>(BSR_MAX_INSTALL_BATCH)));
  if ((W && b > W) || b > BSR_MAX_INSTALL_BATCH)
    return fail_with(BSR_E_ARG, "install_batch %u must be <= min(W=%u, %d)", b, W, BSR_MAX_INSTALL_BATCH);
  // admission (§3 "Install locally": one bounded restore at a time; §7: a
  // global budget B over the rings of the bound requests)
  const uint64_t B = config->staging_budget_bytes;
  uint32_t M = config->max_bound_requests;
  if (M > BSR_MAX_BOUND_REQUESTS)
    return fail_with(BSR_E_ARG, "max_bound_requests %u exceeds %d", M, BSR_MAX_BOUND_REQUESTS);
  const uint64_t slot_bytes = bsr_slot_bytes(layout);
  const uint64_t min_ring = static_cast<uint64_t>(std::max(W, 1u)) * slot_bytes;
  if (static_scratch && (B != 0 || M > 1 || config->hip_device < 0))
    return fail_with(BSR_E_ARG, "a context without allocations has one session slot on a GPU: "
                                "staging_budget_bytes = 0, max_bound_requests <= 1, hip_device >= 0");
  if (B == 0) {
    if (M > 1) return fail_with(BSR_E_ARG, "max_bound_requests %u needs a staging budget (bounded-retrieve lock: 1)", M);
    M = 1;
  } else {
    if (B < min_ring)
      return fail_with(BSR_E_ARG, "staging budget %llu B holds no ring of %llu B", (unsigned long long)B,
                       (unsigned long long)min_ring);
    if (M == 0) M = static_cast<uint32_t>(std::min<uint64_t>(BSR_MAX_BOUND_REQUESTS, B / min_ring));
  }

  auto* c = new (std::nothrow) bsr_ctx();
  if (!c) return fail_with(BSR_E_NOMEM, "context allocation failed");
  build_geometry(layout, &c->geo);
  // one install launch of b chunks runs b x wg_per_chunk workgroups: HIP
  // takes at most 2^32 - 1 work-items in a grid dimension
  if (static_cast<uint64_t>(b) * c->geo.wg_per_chunk * bsr::kInstallThreads >= (1ull << 32)) {
    const uint32_t wpc = c->geo.wg_per_chunk;
    delete c;
    return fail_with(BSR_E_ARG, "an install launch of %u chunks x %u workgroups exceeds the grid limit; lower install_batch",
                     b, wpc);
  }
  c->cfg = *config;
  c->kernel_copies = (config->flags & BSR_FLAG_SDMA_COPIES) == 0;
  c->W = W;
  c->batch = b;
  // A request staged on one stream gains nothing from slack between its
  // copies and installs (stream order serialises them): its batches take the
  // whole window, which halves its launches at small W.  An install_batch
  // the caller sets holds for both.
  c->batch_one = config->install_batch ? b : std::min(W ? W : 32u, static_cast<uint32_t>(BSR_MAX_INSTALL_BATCH));
  while (c->batch_one > b && static_cast<uint64_t>(c->batch_one) * c->geo.wg_per_chunk * bsr::kInstallThreads >= (1ull << 32))
    --c->batch_one;
  c->device = config->hip_device;
  c->budget = B;
  c->store.index.resize(layout->n_groups);
  c->last.window_chunks = W;
  c->last.install_batch = b;
  c->last.slot_bytes = c->geo.slot_bytes;
  c->last.staging_required_bytes = c->geo.slot_bytes * W;
  c->last.first_failed_chunk = BSR_NO_CHUNK;
  c->res.resize(M);
  if (c->device >= 0) {
    int rc = BSR_OK;
    int n_dev = 0;
    if ((rc = hip_check(hipGetDeviceCount(&n_dev), "hipGetDeviceCount")) || c->device >= n_dev) {
      delete c;
      return rc ? rc : fail_with(BSR_E_DEVICE, "hip_device %d not present (%d devices)", config->hip_device, n_dev);
    }
    if ((rc = set_device(c))) {
      delete c;
      return rc;
    }
    // occupancy of the install kernel: each workgroup takes 1/kInstallWgPerCu
    // of the CU's LDS (at least what its planar pieces need)
    int lds_per_cu = 0, lds_per_block = 0;
    if ((rc = hip_check(hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, c->device),
                        "hipDeviceGetAttribute")) ||
        (rc = hip_check(hipDeviceGetAttribute(&lds_per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, c->device),
                        "hipDeviceGetAttribute"))) {
      delete c;
      return rc;
    }
    const uint32_t share = std::min<uint32_t>(static_cast<uint32_t>(lds_per_cu) / bsr::kInstallWgPerCu / 256 * 256,
                                              static_cast<uint32_t>(lds_per_block));
    if (c->geo.lds_bytes > static_cast<uint32_t>(lds_per_block)) {
      delete c;
      return fail_with(BSR_E_ARG, "planar pieces need %u B of LDS, the device has %d per workgroup", c->geo.lds_bytes,
                       lds_per_block);
    }
    c->geo.lds_bytes = std::max(c->geo.lds_bytes, share);
    // XCDs the dispatcher deals the install's workgroups to (eight on a
    // whole MI355X; fewer in a partitioned one); eight if the runtime cannot say
    int n_xcds = 0;
    if (hipDeviceGetAttribute(&n_xcds, hipDeviceAttributeNumberOfXccs, c->device) == hipSuccess && n_xcds >= 1)
      c->xcd_log2 = bsr::xcd_log2_of(n_xcds);
    else
      (void)hipGetLastError();
    auto aux_of = [&](uint32_t batch) {
      return align_up(static_cast<uint64_t>(batch) * c->geo.wg_per_chunk * bsr::kInstallWaves * sizeof(TagPair), kAlign) +
             sizeof(bsr::VerifyAux);
    };
    // the static array bounds one-stream batches too (never below b)
    if (static_scratch)
      while (c->batch_one > b && aux_of(c->batch_one) > bsr::kStaticScratchBytes) --c->batch_one;
    const uint32_t b_max = std::max(b, c->batch_one);
    c->partials_bytes = static_cast<uint64_t>(b_max) * c->geo.wg_per_chunk * bsr::kInstallWaves * sizeof(TagPair);
    c->aux_bytes = aux_of(b_max);
    uint8_t* scratch = nullptr;
    if (static_scratch) {
      if (c->aux_bytes > bsr::kStaticScratchBytes) {
        const uint64_t need = c->aux_bytes;
        delete c;
        return fail_with(BSR_E_ARG,
                         "install launches of %u chunks need %llu B of scratch; the static array holds %llu B "
                         "(lower install_batch)",
                         b, (unsigned long long)need, (unsigned long long)bsr::kStaticScratchBytes);
      }
      void* p = nullptr;
      bool busy = false;
      if ((rc = hip_check(bsr::static_scratch_claim(c->device, &p, &busy), "hipGetSymbolAddress(scratch)"))) {
        delete c;
        return rc;
      }
      if (busy) {
        delete c;
        return fail_with(BSR_E_BUSY, "another context of this process holds device %d's static scratch",
                         config->hip_device);
      }
      c->static_claimed = true;
      scratch = static_cast<uint8_t*>(p);
    }
    // event ring: the copy of chunk i waits for the release of chunk i - W,
    // recorded at most W batches earlier (W + 2 leaves a margin).  In
    // whole-plan mode no slot is reused, so no copy waits for a release and
    // two pairs serve any plan: a batch's copy event is waited for as soon
    // as it is recorded, and a later record does not move an enqueued wait.
    const uint32_t E = W ? W + 2 : 2;
    bool ok = true;
    for (SessionRes& r : c->res) {
      r.full_ev.assign(E, nullptr);
      r.free_ev.assign(E, nullptr);
      if (scratch) {  // the one session slot of a context without allocations
        r.static_scratch = true;
        r.partials = reinterpret_cast<TagPair*>(scratch);
        r.verify_aux = reinterpret_cast<bsr::VerifyAux*>(scratch + align_up(c->partials_bytes, kAlign));
        r.host_status = &r.status_buf;
      } else {
        ok = ok && hipMalloc(reinterpret_cast<void**>(&r.partials), c->partials_bytes) == hipSuccess &&
             hipMalloc(reinterpret_cast<void**>(&r.verify_aux), sizeof(bsr::VerifyAux)) == hipSuccess &&
             hipHostMalloc(reinterpret_cast<void**>(&r.host_status), sizeof(bsr_dev_status), hipHostMallocDefault) == hipSuccess;
      }
      for (uint32_t i = 0; ok && i < E; ++i)
        ok = hipEventCreateWithFlags(&r.full_ev[i], hipEventDisableTiming) == hipSuccess &&
             hipEventCreateWithFlags(&r.free_ev[i], hipEventDisableTiming) == hipSuccess;
    }
    if (!ok) {
      bsr_ctx_destroy(c);
      return fail_with(BSR_E_NOMEM, "device resources for W=%u x %u session slots could not be allocated", W, M);
    }
    c->last.aux_device_bytes = c->aux_bytes;
  }
  *out = c;
  return BSR_OK;
}

int bsr_ctx_create(const bsr_layout* layout, const bsr_config* config, bsr_ctx** out) {
  return ctx_create(layout, config, out, false);
}

int bsr_ctx_create_static(const bsr_layout* layout, const bsr_config* config, bsr_ctx** out) {
  return ctx_create(layout, config, out, true);
}


int bsr_ctx_destroy(bsr_ctx* c) {
  if (!c) return BSR_OK;
  c->ftier.close();
  if (c->device >= 0) {
    (void)hipSetDevice(c->device);
    for (auto& kv : c->bound) {
      Session& s = kv.second;
      if (s.copy) (void)hipStreamSynchronize(s.copy);
      if (s.compute) (void)hipStreamSynchronize(s.compute);
      for (auto* v : {&s.timing, &s.stage_timing})
        for (auto& pr : *v) {
          (void)hipEventDestroy(pr.first);
          (void)hipEventDestroy(pr.second);
        }
    }
    for (SessionRes& r : c->res) free_session_res(r);
    if (c->static_claimed) bsr::static_scratch_release(c->device);
    for (auto e : c->timing_pool) (void)hipEventDestroy(e);
    if (c->store.owned && c->store.arena) (void)hipHostFree(c->store.arena);
  }
  delete c;
  return BSR_OK;
}

// ---- store ------------------------------------------------------------------

static int store_init(bsr_ctx* c, uint8_t* arena, uint64_t bytes, bool owned) {
  Store& st = c->store;
  st.arena = arena;
  st.arena_bytes = bytes;
  st.owned = owned;
  st.block_stride = align_up(c->geo.slot_bytes, kArenaBlockAlign);
  const uint64_t nb = bytes / st.block_stride;
  st.n_blocks = static_cast<uint32_t>(std::min<uint64_t>(nb, 0xFFFFFFFEull));
  st.meta.assign(st.n_blocks, BlockMeta{});
  return BSR_OK;
}

int bsr_store_reserve(bsr_ctx* c, uint64_t bytes) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (c->store.arena) return fail_with(BSR_E_STATE, "store arena already set");
  if (int rc = set_device(c)) return rc;
  void* p = nullptr;
  if (hipHostMalloc(&p, bytes ? bytes : 1, hipHostMallocDefault) != hipSuccess || !p)
    return fail_with(BSR_E_NOMEM, "hipHostMalloc(%llu) failed", (unsigned long long)bytes);
  store_init(c, static_cast<uint8_t*>(p), bytes, true);
  void* dv = nullptr;
  if (hipHostGetDevicePointer(&dv, p, 0) == hipSuccess)
    c->store.arena_dev = static_cast<const uint8_t*>(dv);
  else
    (void)hipGetLastError();
  return BSR_OK;
}

// The device's view of a caller's arena, if HIP reports both its first and
// its last byte as pinned host memory mapped contiguously for the device;
// null otherwise (the copy engine then copies out of it).
static const uint8_t* pinned_device_view(const void* arena, uint64_t bytes) {
  if (!bytes) return nullptr;
  hipPointerAttribute_t a{}, b{};
  const uint8_t* last = static_cast<const uint8_t*>(arena) + (bytes - 1);
  if (hipPointerGetAttributes(&a, arena) != hipSuccess || hipPointerGetAttributes(&b, last) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  if (a.type != hipMemoryTypeHost || b.type != hipMemoryTypeHost || !a.devicePointer || !b.devicePointer)
    return nullptr;
  const uint8_t* d0 = static_cast<const uint8_t*>(a.devicePointer);
  if (static_cast<const uint8_t*>(b.devicePointer) != d0 + (bytes - 1)) return nullptr;
  return d0;
}

int bsr_store_adopt(bsr_ctx* c, void* host_arena, uint64_t bytes) {
  if (!c || !host_arena) return fail_with(BSR_E_ARG, "ctx or arena is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (c->store.arena) return fail_with(BSR_E_STATE, "store arena already set");
  store_init(c, static_cast<uint8_t*>(host_arena), bytes, false);
  if (c->device >= 0 && set_device(c) == BSR_OK) c->store.arena_dev = pinned_device_view(host_arena, bytes);
  return BSR_OK;
}

static void drop_entry(bsr_ctx* c, uint32_t g, uint64_t key) {
  auto& ix = c->store.index[g];
  auto it = ix.find(key);
  if (it == ix.end()) return;
  const uint32_t b = it->second.block;
  ix.erase(it);
  --c->store.n_entries;
  --c->store.meta[b].live_groups;
  c->store.maybe_free(b);
}

int bsr_store_put_chunk(bsr_ctx* c, uint64_t key, const void* const* payloads) {
  if (!c || !payloads) return fail_with(BSR_E_ARG, "ctx or payloads is NULL");
  const uint32_t G = c->geo.L.n_groups;
  for (uint32_t g = 0; g < G; ++g)
    if (!payloads[g]) return fail_with(BSR_E_ARG, "payload of group %u is NULL", g);
  uint32_t b;
  uint8_t* base;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    if (!c->store.arena) return fail_with(BSR_E_STATE, "no store arena (reserve or adopt first)");
    if (!c->store.alloc(&b)) return fail_with(BSR_E_NOMEM, "store arena full (%u chunks)", c->store.n_blocks);
    c->store.meta[b].refs = 1;  // keep the block private while it is filled
    base = c->store.block_ptr(b);
  }
  uint64_t tags[BSR_MAX_GROUPS];
  for (uint32_t g = 0; g < G; ++g) {
    uint8_t* dst = base + c->geo.offset[g];
    std::memcpy(dst, payloads[g], c->geo.payload[g]);
    const uint64_t pad = align_up(c->geo.payload[g], kAlign) - c->geo.payload[g];
    if (pad) std::memset(dst + c->geo.payload[g], 0, pad);
    tags[g] = tag_of(dst, c->geo.payload[g]);
  }
  std::lock_guard<std::mutex> lk(c->mu);
  for (uint32_t g = 0; g < G; ++g) {
    drop_entry(c, g, key);
    c->store.index[g][key] = Entry{b, tags[g]};
    ++c->store.meta[b].live_groups;
    ++c->store.n_entries;
  }
  c->store.meta[b].refs = 0;
  return BSR_OK;
}

int bsr_store_put_chunks(bsr_ctx* c, uint32_t n, const uint64_t* keys, const void* const* payloads) {
  if (!c || (n && (!keys || !payloads))) return fail_with(BSR_E_ARG, "ctx, keys or payloads is NULL");
  if (n == 0) return BSR_OK;
  const uint32_t G = c->geo.L.n_groups;
  for (uint64_t i = 0; i < static_cast<uint64_t>(n) * G; ++i)
    if (!payloads[i]) return fail_with(BSR_E_ARG, "payload of chunk %llu group %llu is NULL",
                                       (unsigned long long)(i / G), (unsigned long long)(i % G));
  std::vector<uint32_t> blocks(n);
  {
    std::lock_guard<std::mutex> lk(c->mu);
    Store& st = c->store;
    if (!st.arena) return fail_with(BSR_E_STATE, "no store arena (reserve or adopt first)");
    const uint64_t free_blocks = static_cast<uint64_t>(st.n_blocks - st.next_fresh) + st.free_list.size();
    if (free_blocks < n) return fail_with(BSR_E_NOMEM, "store arena has %llu free blocks, %u needed",
                                          (unsigned long long)free_blocks, n);
    const bool fresh_run = st.n_blocks - st.next_fresh >= n;
    for (uint32_t i = 0; i < n; ++i) {
      uint32_t b;
      if (fresh_run) {
        b = st.next_fresh++;
        st.meta[b] = BlockMeta{};
        ++st.blocks_in_use;
      } else {
        st.alloc(&b);  // cannot fail: enough blocks were counted above
      }
      st.meta[b].refs = 1;  // private while it is filled
      blocks[i] = b;
    }
  }
  std::vector<uint64_t> tags(static_cast<uint64_t>(n) * G);
  auto fill = [&](uint32_t lo, uint32_t hi) {
    for (uint32_t i = lo; i < hi; ++i) {
      uint8_t* base = c->store.block_ptr(blocks[i]);
      for (uint32_t g = 0; g < G; ++g) {
        uint8_t* dst = base + c->geo.offset[g];
        std::memcpy(dst, payloads[static_cast<uint64_t>(i) * G + g], c->geo.payload[g]);
        const uint64_t pad = align_up(c->geo.payload[g], kAlign) - c->geo.payload[g];
        if (pad) std::memset(dst + c->geo.payload[g], 0, pad);
        tags[static_cast<uint64_t>(i) * G + g] = tag_of(dst, c->geo.payload[g]);
      }
    }
  };
  unsigned nt = std::min(8u, std::max(1u, std::thread::hardware_concurrency()));
  if (n < 2 * nt) nt = 1;
  if (nt == 1) {
    fill(0, n);
  } else {
    std::vector<std::thread> th;
    const uint32_t per = (n + nt - 1) / nt;
    for (unsigned t = 0; t < nt; ++t) {
      const uint32_t lo = t * per, hi = std::min(n, lo + per);
      if (lo < hi) th.emplace_back(fill, lo, hi);
    }
    for (auto& x : th) x.join();
  }
  std::lock_guard<std::mutex> lk(c->mu);
  for (uint32_t i = 0; i < n; ++i) {
    for (uint32_t g = 0; g < G; ++g) {
      drop_entry(c, g, keys[i]);
      c->store.index[g][keys[i]] = Entry{blocks[i], tags[static_cast<uint64_t>(i) * G + g]};
      ++c->store.meta[blocks[i]].live_groups;
      ++c->store.n_entries;
    }
  }
  for (uint32_t i = 0; i < n; ++i) {
    c->store.meta[blocks[i]].refs = 0;
    c->store.maybe_free(blocks[i]);  // a key repeated within the call leaves its earlier block unused
  }
  return BSR_OK;
}

int bsr_store_remove(bsr_ctx* c, uint64_t key, int32_t group) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  const uint32_t G = c->geo.L.n_groups;
  if (group >= static_cast<int32_t>(G)) return fail_with(BSR_E_ARG, "group %d out of range", group);
  bool any = false;
  for (uint32_t g = 0; g < G; ++g) {
    if (group >= 0 && static_cast<uint32_t>(group) != g) continue;
    if (c->store.index[g].count(key)) {
      any = true;
      drop_entry(c, g, key);
    }
  }
  return any ? BSR_OK : fail_with(BSR_E_NOTFOUND, "no entry for key %016llx", (unsigned long long)key);
}

int bsr_store_payload(bsr_ctx* c, uint64_t key, uint32_t group, void** host_ptr, uint64_t* nbytes,
                      uint64_t* tag) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (group >= c->geo.L.n_groups) return fail_with(BSR_E_ARG, "group %u out of range", group);
  auto it = c->store.index[group].find(key);
  if (it == c->store.index[group].end())
    return fail_with(BSR_E_NOTFOUND, "no entry (%016llx, %u)", (unsigned long long)key, group);
  if (host_ptr) *host_ptr = c->store.block_ptr(it->second.block) + c->geo.offset[group];
  if (nbytes) *nbytes = c->geo.payload[group];
  if (tag) *tag = it->second.tag;
  return BSR_OK;
}

int bsr_store_count(bsr_ctx* c, uint64_t* n_entries, uint64_t* bytes_used) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (n_entries) *n_entries = c->store.n_entries;
  if (bytes_used) *bytes_used = static_cast<uint64_t>(c->store.blocks_in_use) * c->store.block_stride;
  return BSR_OK;
}

// ---- probe --------------------------------------------------------------------

int bsr_probe(bsr_ctx* c, uint64_t request_id, uint64_t salt, const int32_t* tokens, uint64_t n_tokens,
              uint32_t* n_hit_chunks, uint8_t* hit_bitmap, uint64_t* keys_out) {
  if (!c || !n_hit_chunks) return fail_with(BSR_E_ARG, "ctx or n_hit_chunks is NULL");
  if (!host_is_little_endian()) return fail_with(BSR_E_ARG, "big-endian host unsupported");
  const uint64_t t0 = now_ns();
  const uint32_t C = c->geo.L.chunk_tokens;
  const uint64_t N = n_tokens / C;
  if (N > 0xFFFFFFF0ull) return fail_with(BSR_E_ARG, "too many chunks");
  if (N && !tokens) return fail_with(BSR_E_ARG, "tokens is NULL");
  Request req;
  req.keys.resize(N);
  if (N) chain_keys(salt, tokens, N, C, req.keys.data());
  if (hit_bitmap) std::memset(hit_bitmap, 0, (N + 7) / 8);
  uint32_t n_hit = 0;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    if (c->bound.count(request_id))
      return fail_with(BSR_E_STATE, "request %llu is bound; end it before probing again", (unsigned long long)request_id);
    const bool local = c->force_local.count(request_id) != 0;
    bool prefix = true;
    const uint32_t G = c->geo.L.n_groups;
    req.tier.assign(N, kTierNone);
    const bool file_up = c->ftier.is_open() && c->ftier.available;
    for (uint64_t i = 0; i < N && !local; ++i) {
      // a chunk is a hit in the first available tier holding every group
      bool hit = c->tier0_available;
      for (uint32_t g = 0; g < G && hit; ++g) hit = c->store.index[g].count(req.keys[i]) != 0;
      if (hit) {
        req.tier[i] = kTierPinned;
      } else if (file_up) {
        hit = true;
        for (uint32_t g = 0; g < G && hit; ++g) hit = c->ftier.has(req.keys[i], g);
        if (hit) req.tier[i] = kTierFile;
      }
      if (hit && hit_bitmap) hit_bitmap[i >> 3] |= static_cast<uint8_t>(1u << (i & 7));
      if (!hit) prefix = false;
      if (prefix) ++n_hit;
    }
    req.n_probe = n_hit;
    req.probe_ns = now_ns() - t0;
    if (keys_out && N) std::memcpy(keys_out, req.keys.data(), N * 8);
    c->requests[request_id] = std::move(req);
  }
  *n_hit_chunks = n_hit;
  return BSR_OK;
}

// ---- bind ----------------------------------------------------------------------

int bsr_request_bind(bsr_ctx* c, uint64_t request_id, uint32_t n_hit, const bsr_group_dst* dst,
                     void* staging, uint64_t staging_bytes, bsr_dev_status* status, void* copy_stream,
                     void* compute_stream) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (int rc = set_device(c)) return rc;
  // Arguments and block tables first, without the context lock: the
  // readback waits for the caller's compute stream, and other requests'
  // calls must not wait for it.  The geometry read here never changes.
  // the install kernel's token arithmetic is 32-bit: the prefix plus two of
  // the largest blocks must stay below 2^32 tokens
  {
    uint64_t max_b = 0;
    for (uint32_t g = 0; g < c->geo.L.n_groups; ++g) max_b = std::max<uint64_t>(max_b, c->geo.L.groups[g].block_tokens);
    if (static_cast<uint64_t>(n_hit) * c->geo.L.chunk_tokens + 2 * max_b >= (1ull << 32))
      return fail_with(BSR_E_ARG, "a restored prefix must be shorter than 2^32 tokens less two blocks");
  }
  if (!dst || !staging || !status) return fail_with(BSR_E_ARG, "dst, staging or status is NULL");
  if (!copy_stream || !compute_stream || copy_stream == compute_stream)
    return fail_with(BSR_E_ARG, "copy and compute streams must be distinct non-null streams");
  const uint32_t window = c->W ? c->W : std::max(1u, n_hit);
  const uint64_t need = c->geo.slot_bytes * window;
  if (staging_bytes < need)
    return fail_with(BSR_E_STAGING, "staging %llu B < W x slot = %llu B", (unsigned long long)staging_bytes, (unsigned long long)need);
  if (reinterpret_cast<uintptr_t>(staging) % 256) return fail_with(BSR_E_ARG, "staging must be 256-byte aligned");

  const uint32_t G = c->geo.L.n_groups, C = c->geo.L.chunk_tokens;
  hipStream_t compute = static_cast<hipStream_t>(compute_stream);
  hipStream_t copy = static_cast<hipStream_t>(copy_stream);
  FinishParams fp{};
  fp.status = status;
  fp.n_groups = G;
  fp.chunk_tokens = C;
  fp.exposed_if_valid = static_cast<uint64_t>(n_hit) * C;
  const bool trusted = (c->cfg.flags & BSR_FLAG_TRUSTED_TABLES) != 0;
  InstallParams ip{};
  ip.h.ring = static_cast<const uint8_t*>(staging);
  ip.h.slot_bytes = c->geo.slot_bytes;
  ip.h.window = window;
  ip.h.chunk_tokens = C;
  ip.h.n_groups = G;
  ip.h.wg_per_chunk = c->geo.wg_per_chunk;
  ip.h.lds_bytes = c->geo.lds_bytes;
  ip.h.xcd_log2 = c->xcd_log2;
  ip.h.status = status;
  uint32_t total = 0;
  std::vector<int32_t> bt;
  for (uint32_t g = 0; g < G; ++g) {
    const bsr_group_dst& d = dst[g];
    const uint32_t B = c->geo.L.groups[g].block_tokens;
    const uint64_t nreq = (static_cast<uint64_t>(n_hit) * C + B - 1) / B;
    if (!d.block_table || !d.tensor_bases || !d.valid) return fail_with(BSR_E_ARG, "group %u: NULL destination pointer", g);
    if (d.n_blocks < nreq) return fail_with(BSR_E_ARG, "group %u: block table has %u blocks, prefix needs %llu", g, d.n_blocks, (unsigned long long)nreq);
    if (d.pool_blocks == 0) return fail_with(BSR_E_ARG, "group %u: pool_blocks is 0", g);
    if (!trusted) {
      // copy the advertised part of the block table back once and check it
      bt.resize(nreq);
      if (nreq) {
        int rc = hip_check(hipMemcpyAsync(bt.data(), d.block_table, nreq * 4, hipMemcpyDeviceToHost, compute), "block table readback");
        if (!rc) rc = hip_check(hipStreamSynchronize(compute), "hipStreamSynchronize");
        if (rc) return rc;
      }
      std::vector<uint8_t> seen(d.pool_blocks, 0);
      for (uint64_t k = 0; k < nreq; ++k) {
        const int32_t b = bt[k];
        if (b < 0 || static_cast<uint32_t>(b) >= d.pool_blocks)
          return fail_with(BSR_E_ARG, "group %u: block_table[%llu] = %d outside [0, %u)", g, (unsigned long long)k, b, d.pool_blocks);
        if (seen[b]++) return fail_with(BSR_E_ARG, "group %u: block %d appears twice in the prefix", g, b);
      }
    }
    // the group's record sits at its dispatch position
    uint32_t pos = 0;
    while (c->geo.order[pos] != g) ++pos;
    const GroupGeom& q = c->geo.gg[g];
    bsr::InstallGroup& ig = ip.g[pos];
    ig.per_chunk = c->geo.wg_start[g + 1] - c->geo.wg_start[g];
    ig.wg_start = c->geo.wg_start[g];
    ig.div_per_chunk = bsr::pack_fastdiv(q.div_per_chunk);
    ig.div_pieces = bsr::pack_fastdiv(q.div_pieces);
    ig.div_segs = bsr::pack_fastdiv(q.div_segs);
    ig.div_block = bsr::pack_fastdiv(q.div_block);
    ig.pieces_per_seg = q.pieces_per_seg;
    ig.segs_per_chunk = q.segs_per_chunk;
    ig.block_tokens = q.block_tokens;
    ig.record_bytes = q.record_bytes;
    ig.staged_off = q.staged_off;
    ig.piece = q.kind == BSR_KIND_CONTIG ? q.piece_bytes : q.piece_tokens;
    ig.kind = q.kind;
    ig.split_bytes = q.split_bytes;
    ig.n_blocks = d.n_blocks;
    ig.pool_blocks = d.pool_blocks;
    ig.block_table = d.block_table;
    ig.tensor_bases = reinterpret_cast<uint8_t* const*>(d.tensor_bases);
    ig.group = g;
    ig.prefix = c->geo.order_prefix[pos];
    ig.block_bytes = q.block_tokens * q.record_bytes;
    if (q.kind == BSR_KIND_PLANAR) {
      ig.div_p1 = bsr::pack_fastdiv(bsr::make_fastdiv(std::max(1u, q.split_bytes / 16)));
      ig.div_p2 = bsr::pack_fastdiv(bsr::make_fastdiv((q.record_bytes - q.split_bytes) / 4));
    }
    fp.g[g] = bsr::GroupValid{d.block_table, d.valid, static_cast<uint32_t>(nreq), d.pool_blocks, B, 0};
    total += static_cast<uint32_t>(nreq);
  }
  fp.total_blocks = total;

  std::lock_guard<std::mutex> lk(c->mu);
  if (c->bound.count(request_id)) return fail_with(BSR_E_STATE, "request %llu is already bound", (unsigned long long)request_id);
  auto it = c->requests.find(request_id);
  if (it == c->requests.end()) return fail_with(BSR_E_STATE, "request %llu was not probed", (unsigned long long)request_id);
  Request& rq = it->second;
  if (rq.phase != Phase::Probed) return fail_with(BSR_E_STATE, "request %llu already bound once; probe again", (unsigned long long)request_id);
  if (n_hit > rq.n_probe) return fail_with(BSR_E_ARG, "n_hit_chunks %u exceeds the probed prefix %u", n_hit, rq.n_probe);

  // admission: the bounded-retrieve lock, or the global budget B
  if (c->budget == 0) {
    if (!c->bound.empty()) {
      ++c->n_refused;
      return fail_with(BSR_E_BUSY, "request %llu holds the bounded-retrieve lock",
                       (unsigned long long)c->bound.begin()->first);
    }
  } else if (need > c->budget) {
    return fail_with(BSR_E_STAGING, "ring of %llu B exceeds the staging budget %llu B", (unsigned long long)need,
                     (unsigned long long)c->budget);
  } else if (c->bound_bytes + need > c->budget) {
    ++c->n_refused;
    return fail_with(BSR_E_BUSY, "staging budget: %llu B bound + %llu B > %llu B", (unsigned long long)c->bound_bytes,
                     (unsigned long long)need, (unsigned long long)c->budget);
  }
  uint32_t slot_res = 0;
  while (slot_res < c->res.size() && c->res[slot_res].in_use) ++slot_res;
  if (slot_res == c->res.size()) {
    ++c->n_refused;
    return fail_with(BSR_E_BUSY, "all %zu session slots are bound", c->res.size());
  }
  // concurrently bound requests must not share a ring or a status block
  {
    const uintptr_t r0 = reinterpret_cast<uintptr_t>(staging), r1 = r0 + need;
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(status), s1 = s0 + sizeof(bsr_dev_status);
    for (auto& kv : c->bound) {
      const Session& o = kv.second;
      const uintptr_t o0 = reinterpret_cast<uintptr_t>(o.staging), o1 = o0 + o.ring_bytes;
      const uintptr_t p0 = reinterpret_cast<uintptr_t>(o.status), p1 = p0 + sizeof(bsr_dev_status);
      if ((r0 < o1 && o0 < r1) || (s0 < p1 && p0 < s1) || (r0 < p1 && p0 < r1) || (s0 < o1 && o0 < s1))
        return fail_with(BSR_E_ARG, "staging or status overlaps that of bound request %llu", (unsigned long long)kv.first);
    }
  }
  SessionRes& res = c->res[slot_res];
  fp.verify_aux = res.verify_aux;
  ip.h.partials = res.partials;

  // begin: reset the status words and clear the advertised valid bytes
  FinishParams begin = fp;
  begin.mode = bsr::kFinishBegin;
  if (int rc = hip_check(bsr::launch_finish(begin, compute), "begin launch")) return rc;
  if (trusted) {
    FinishParams check = fp;
    check.mode = bsr::kFinishCheckTables;
    if (int rc = hip_check(bsr::launch_finish(check, compute), "block table check launch")) return rc;
  }
  // A request of at most kOneStreamBytes of chunks is staged on the compute
  // stream: its copies and installs are short, and the hand-over between two
  // streams (an event recorded on one, waited for on the other) costs about
  // as much as they do.
  const bool one_stream = !(c->cfg.flags & BSR_FLAG_TWO_STREAMS) &&
                          static_cast<uint64_t>(n_hit) * c->geo.slot_bytes <= kOneStreamBytes;
  // no copy of this request may overwrite the ring before earlier compute work is done
  if (!one_stream) {
    if (int rc = hip_check(hipEventRecord(res.free_ev[0], compute), "hipEventRecord")) return rc;
    if (int rc = hip_check(hipStreamWaitEvent(copy, res.free_ev[0], 0), "hipStreamWaitEvent")) return rc;
  }

  Session& s = c->bound[request_id];
  s = Session{};
  s.id = request_id;
  s.res = slot_res;
  s.ring_bytes = need;
  s.n_hit = n_hit;
  s.staging = static_cast<uint8_t*>(staging);
  s.status = status;
  s.one_stream = one_stream;
  s.time_flags = c->cfg.flags & kTimingFlags;
  s.batch = one_stream ? c->batch_one : c->batch;
  s.copy = one_stream ? compute : copy;
  s.compute = compute;
  s.ip = ip;
  s.fp = fp;
  s.window = window;
  s.slot_free_seq.assign(window, -1);
  s.slot_used.assign(window, 0);
  s.batch_seq = 1;  // event slot 0 is used by the bind fence above
  s.inject = c->inject;
  c->inject = Inject{};
  res.in_use = true;
  rq.phase = Phase::Bound;
  c->bound_bytes += need;
  c->peak_bound_bytes = std::max(c->peak_bound_bytes, c->bound_bytes);
  c->peak_bound = std::max(c->peak_bound, static_cast<uint32_t>(c->bound.size()));
  c->last_id = request_id;

  bsr_stats& st = s.st;
  st.request_id = request_id;
  st.n_hit_chunks = n_hit;
  st.window_chunks = c->W;  // 0: whole-plan mode
  st.install_batch = s.batch;
  st.slot_bytes = c->geo.slot_bytes;
  st.staging_required_bytes = need;
  st.aux_device_bytes = c->aux_bytes;
  st.first_failed_chunk = BSR_NO_CHUNK;
  st.probe_ns = rq.probe_ns;
  return BSR_OK;
}

// ---- restore window ------------------------------------------------------------

int bsr_restore_window(bsr_ctx* c, uint64_t request_id, uint32_t first_chunk, uint32_t n_chunks) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (int rc = set_device(c)) return rc;
  const uint64_t t_enter = now_ns();
  std::lock_guard<std::mutex> lk(c->mu);
  Session* sp = nullptr;
  if (int rc0 = find_active(c, request_id, &sp)) return rc0;
  Session& s = *sp;
  SessionRes& res = c->res[s.res];
  if (s.failed) return fail_with(BSR_E_STATE, "request %llu already failed", (unsigned long long)request_id);
  if (n_chunks == 0 || n_chunks > s.window) return fail_with(BSR_E_ARG, "n_chunks %u must be in 1..W=%u", n_chunks, s.window);
  if (first_chunk != s.next_chunk) return fail_with(BSR_E_STATE, "window starts at %u, expected %u", first_chunk, s.next_chunk);
  if (static_cast<uint64_t>(first_chunk) + n_chunks > s.n_hit)
    return fail_with(BSR_E_ARG, "window [%u, %u) beyond the bound prefix %u", first_chunk, first_chunk + n_chunks, s.n_hit);

  const Request& rq = c->requests[request_id];
  const uint32_t G = c->geo.L.n_groups;
  const uint32_t all_mask = (G >= 32) ? 0xFFFFFFFFu : ((1u << G) - 1);
  const uint32_t E = static_cast<uint32_t>(res.free_ev.size());
  // The install batch may span windows.  A copy into slot i mod W needs the
  // install of chunk i - W, which is never in the pending batch (it holds at
  // most install_batch - 1 <= W - 1 earlier chunks), so its release event has
  // been recorded already.
  std::vector<uint32_t>& batch = s.pend;
  const uint64_t t_window = now_ns();
  int rc = BSR_OK;

  // Chunks the probe found only in the file tier are read ahead by the
  // tier's readers into its bounce buffers (at most pool_size in flight) and
  // consumed in chunk order; each buffer is reused once the device copy out
  // of it has completed.
  std::vector<uint32_t> fchunks;
  for (uint32_t i = first_chunk; i < first_chunk + n_chunks; ++i)
    if (rq.tier[i] == kTierFile) fchunks.push_back(i);
  size_t f_sub = 0, f_used = 0;
  uint32_t P = 0;
  if (!fchunks.empty()) {
    std::string err;
    if (!c->ftier.is_open()) return fail_with(BSR_E_STATE, "the plan uses the file tier, which is closed");
    if (c->ftier.start(c->device, &err)) return fail_with(BSR_E_NOMEM, "%s", err.c_str());
    P = c->ftier.pool_size();
    for (; f_sub < fchunks.size() && f_sub < P; ++f_sub) c->ftier.submit(static_cast<uint32_t>(f_sub % P), rq.keys[fchunks[f_sub]]);
  }
  // Whatever path leaves this call, no read it queued may still be landing in
  // a bounce buffer: the next window (of this request or another) reuses them.
  struct DrainReads {
    bsr::FileTier& t;
    const bool any;
    ~DrainReads() {
      if (any) t.drain();
    }
  } drain_reads{c->ftier, !fchunks.empty()};
  const uint64_t deadline = c->cfg.window_timeout_ms ? t_window + static_cast<uint64_t>(c->cfg.window_timeout_ms) * 1000000ull : 0;

  // Consecutive chunks whose pinned sources are adjacent in the arena and
  // whose slots are adjacent in the ring are staged by one copy: every copy
  // pays a fixed start-up cost (a kernel launch, or the copy engine's own)
  // that a 16 MB chunk does not amortise.  A run waits once, for the release its first
  // chunk needs; a chunk needing a later release starts a new run, so no
  // copy waits longer than it would alone.  A run is always issued before
  // the batch holding its chunks is flushed, so the batch's copy event
  // covers it.
  struct Run {
    const uint8_t* src = nullptr;
    uint8_t* dst = nullptr;
    uint64_t bytes = 0;
    int64_t need = -1;
    uint32_t first = 0, count = 0;
  } run;
  auto issue_run = [&]() -> hipError_t {
    if (!run.count) return hipSuccess;
    hipError_t e = hipSuccess;
    if (!s.one_stream && run.need >= 0 && run.need > s.copy_waited_seq) {
      e = hipStreamWaitEvent(s.copy, res.free_ev[run.need % E], 0);
      if (e != hipSuccess) return e;
      s.copy_waited_seq = run.need;
    }
    e = stage_copy(c, s, run.dst, run.src, run.bytes, c->store.arena, c->store.arena_dev, c->store.arena_bytes);
    if (e == hipSuccess) run = Run{};
    return e;
  };
  // A run whose copy could not be enqueued leaves the batch again: its chunks
  // were never staged.
  auto fail_run = [&](hipError_t e) -> int {
    const std::string why = hipGetErrorString(e);
    const uint32_t first = run.first;
    for (uint32_t k = 0; k < run.count; ++k) {
      batch.pop_back();
      s.pend_tags.pop_back();
    }
    run = Run{};
    if (int r2 = flush_batch(c, s)) return launch_failed(c, s, r2);
    fail_with(BSR_E_TRANSFER, "chunk %u: staging copy failed: %s", first, why.c_str());
    return host_fail(c, s, BSR_FAIL_TRANSFER, first, all_mask, BSR_E_TRANSFER);
  };
  // install what is staged so far: the pending run's copy first
  auto flush_all = [&]() -> int {
    if (hipError_t e = issue_run()) return fail_run(e);
    if (int r2 = flush_batch(c, s)) return launch_failed(c, s, r2);
    return BSR_OK;
  };

  for (uint32_t i = first_chunk; i < first_chunk + n_chunks; ++i) {
    // injected host faults (forced from the host; kernels always exit normally)
    if (s.inject.kind == BSR_INJECT_DELAY_MS && s.inject.chunk == i)
      std::this_thread::sleep_for(std::chrono::milliseconds(s.inject.param));
    if (deadline && now_ns() > deadline) {
      if ((rc = flush_all())) return rc;
      fail_with(BSR_E_TIMEOUT, "window deadline %u ms exceeded at chunk %u", c->cfg.window_timeout_ms, i);
      return host_fail(c, s, BSR_FAIL_TIMEOUT, i, all_mask, BSR_E_TIMEOUT);
    }
    if (s.inject.kind == BSR_INJECT_TRANSFER_ERROR && s.inject.chunk == i) {
      if ((rc = flush_all())) return rc;
      fail_with(BSR_E_TRANSFER, "injected transfer error at chunk %u", i);
      return host_fail(c, s, BSR_FAIL_TRANSFER, i, all_mask, BSR_E_TRANSFER);
    }
    const uint64_t key = rq.keys[i];
    const bool from_file = rq.tier[i] == kTierFile;
    std::array<uint64_t, BSR_MAX_GROUPS> tg{};
    const uint8_t* src_block = nullptr;  // one contiguous slot-shaped source
    Entry ent[BSR_MAX_GROUPS];
    bool one_block = true;
    // fetch: every group's entry must still be present in the chunk's tier
    uint32_t missing = 0;
    if (!from_file) {
      for (uint32_t g = 0; g < G; ++g) {
        auto it = c->store.index[g].find(key);
        if (!c->tier0_available || it == c->store.index[g].end())
          missing |= 1u << g;
        else
          ent[g] = it->second;
      }
    } else {
      for (uint32_t g = 0; g < G; ++g)
        if (!c->ftier.available || !c->ftier.tag(key, g, &tg[g])) missing |= 1u << g;
    }
    if (missing) {
      if ((rc = flush_all())) return rc;
      fail_with(BSR_E_MISSING, "chunk %u: entries missing for group mask 0x%x", i, missing);
      return host_fail(c, s, BSR_FAIL_MISSING, i, missing, BSR_E_MISSING);
    }
    uint32_t bounce = 0;
    if (from_file) {
      // wait for the chunk's read (complete presence of the object)
      bounce = static_cast<uint32_t>(f_used % P);
      uint32_t present = 0;
      int os_err = 0;
      const int st = c->ftier.wait(bounce, deadline, &present, &os_err);
      if (st != bsr::FileTier::kReadOk || (present & all_mask) != all_mask) {
        if ((rc = flush_all())) return rc;
        if (st == bsr::FileTier::kReadPending) {
          fail_with(BSR_E_TIMEOUT, "window deadline %u ms exceeded reading chunk %u", c->cfg.window_timeout_ms, i);
          return host_fail(c, s, BSR_FAIL_TIMEOUT, i, all_mask, BSR_E_TIMEOUT);
        }
        if (st == bsr::FileTier::kReadIoError) {
          fail_with(BSR_E_TRANSFER, "chunk %u: file read failed: %s", i, std::strerror(os_err));
          return host_fail(c, s, BSR_FAIL_TRANSFER, i, all_mask, BSR_E_TRANSFER);
        }
        const uint32_t miss = st == bsr::FileTier::kReadOk ? (all_mask & ~present) : all_mask;
        fail_with(BSR_E_MISSING, "chunk %u: file entry missing for group mask 0x%x", i, miss);
        return host_fail(c, s, BSR_FAIL_MISSING, i, miss, BSR_E_MISSING);
      }
      src_block = c->ftier.bounce_data(bounce);
    } else {
      for (uint32_t g = 1; g < G; ++g) one_block = one_block && ent[g].block == ent[0].block;
      for (uint32_t g = 0; g < G; ++g) {
        tg[g] = ent[g].tag;
        if (g == 0 || !one_block) {
          ++c->store.meta[ent[g].block].refs;
          s.refs.push_back(ent[g].block);
        }
      }
      if (one_block) src_block = c->store.block_ptr(ent[0].block);
    }
    // the slot must have been released by the install of its previous chunk
    const uint32_t slot = i % s.window;
    // on one stream stream order releases the slot: nothing to wait for
    const int64_t need_seq = s.one_stream ? -1 : s.slot_free_seq[slot];
    uint8_t* dst = s.staging + static_cast<uint64_t>(slot) * c->geo.slot_bytes;
    hipError_t e = hipSuccess;
    if (!from_file && src_block) {
      // pinned, one block: extend the run or start a new one
      const int64_t need = need_seq > s.copy_waited_seq ? need_seq : -1;  // -1: nothing left to wait for
      const bool extends = run.count && run.src + run.bytes == src_block && run.dst + run.bytes == dst &&
                           need <= run.need;
      if (!extends) {
        if ((e = issue_run())) return fail_run(e);
        run.src = src_block;
        run.dst = dst;
        run.first = i;
        run.need = need_seq > s.copy_waited_seq ? need_seq : -1;  // issue_run may have waited
      }
      run.bytes += c->geo.slot_bytes;
      ++run.count;
    } else {
      if ((e = issue_run())) return fail_run(e);
      if (need_seq >= 0 && need_seq > s.copy_waited_seq) {
        if ((rc = hip_check(hipStreamWaitEvent(s.copy, res.free_ev[need_seq % E], 0), "hipStreamWaitEvent(free)")))
          return launch_failed(c, s, rc);
        s.copy_waited_seq = need_seq;
      }
      if (src_block && from_file) {
        e = stage_copy(c, s, dst, src_block, c->geo.slot_bytes, c->ftier.bounce_base(bounce),
                       c->ftier.bounce_device(bounce), c->ftier.file_bytes());
      } else if (src_block) {
        e = stage_copy(c, s, dst, src_block, c->geo.slot_bytes, c->store.arena, c->store.arena_dev,
                       c->store.arena_bytes);
      } else {
        for (uint32_t g = 0; g < G && e == hipSuccess; ++g)
          e = stage_copy(c, s, dst + c->geo.offset[g], c->store.block_ptr(ent[g].block) + c->geo.offset[g],
                         c->geo.payload[g], c->store.arena, c->store.arena_dev, c->store.arena_bytes);
      }
      if (e == hipSuccess && from_file) {
        // the bounce buffer is free again once this copy has run
        s.copy_dirty = true;
        e = hipEventRecord(c->ftier.bounce_event(bounce), s.copy);
        ++f_used;
        if (e == hipSuccess && f_sub < fchunks.size()) {
          c->ftier.submit(static_cast<uint32_t>(f_sub % P), rq.keys[fchunks[f_sub]]);
          ++f_sub;
        }
        ++s.st.file_tier_chunks;
      }
      if (e != hipSuccess) {
        const std::string why = hipGetErrorString(e);
        if ((rc = flush_batch(c, s))) return launch_failed(c, s, rc);
        fail_with(BSR_E_TRANSFER, "chunk %u: staging copy failed: %s", i, why.c_str());
        return host_fail(c, s, BSR_FAIL_TRANSFER, i, all_mask, BSR_E_TRANSFER);
      }
    }
    s.st.h2d_bytes += c->geo.slot_bytes;
    if (!s.slot_used[slot]) {
      s.slot_used[slot] = 1;
      ++s.slots_touched;
    }
    batch.push_back(i);
    s.pend_tags.push_back(tg);
    ++s.st.n_chunks_enqueued;
    if (batch.size() == s.batch)
      if ((rc = flush_all())) return rc;
  }
  if (hipError_t e = issue_run()) return fail_run(e);  // nothing of this call stays unstaged
  if (first_chunk + n_chunks == s.n_hit)
    if ((rc = flush_batch(c, s))) return launch_failed(c, s, rc);  // the prefix is complete
  s.next_chunk = first_chunk + n_chunks;
  ++s.st.n_windows;
  s.st.peak_live_staging_bytes = static_cast<uint64_t>(s.slots_touched) * c->geo.slot_bytes;
  if (!fchunks.empty()) s.st.host_bounce_bytes = c->ftier.bounce_bytes();
  s.st.enqueue_ns += now_ns() - t_enter;
  return BSR_OK;
}

int bsr_next_window(bsr_ctx* c, uint64_t request_id, uint32_t* first_chunk, uint32_t* n_chunks) {
  if (!c || !first_chunk || !n_chunks) return fail_with(BSR_E_ARG, "ctx or an out-parameter is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  Session* s = nullptr;
  if (int rc = find_active(c, request_id, &s)) return rc;
  *first_chunk = s->next_chunk;
  *n_chunks = s->failed ? 0 : std::min(s->window, s->n_hit - s->next_chunk);
  return BSR_OK;
}

int bsr_mark_group_invalid(bsr_ctx* c, uint64_t request_id, uint32_t group) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (int rc = set_device(c)) return rc;
  std::lock_guard<std::mutex> lk(c->mu);
  Session* s = nullptr;
  if (int rc = find_active(c, request_id, &s)) return rc;
  if (group >= c->geo.L.n_groups) return fail_with(BSR_E_ARG, "group %u out of range", group);
  if (int rc = enqueue_finish(c, *s, bsr::kFinishMarkGroup, 0, BSR_NO_CHUNK, group)) return launch_failed(c, *s, rc);
  return BSR_OK;
}

int bsr_invalidate(bsr_ctx* c, uint64_t request_id, int32_t reason) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (int rc = set_device(c)) return rc;
  std::lock_guard<std::mutex> lk(c->mu);
  Session* s = nullptr;
  if (int rc = find_active(c, request_id, &s)) return rc;
  if (reason <= BSR_FAIL_NONE || reason > BSR_FAIL_ABORT) return fail_with(BSR_E_ARG, "invalid reason %d", reason);
  c->force_local.insert(request_id);
  s->failed = true;
  if (s->host_fail == BSR_FAIL_NONE) s->host_fail = reason;
  return enqueue_finish(c, *s, bsr::kFinishInvalidate, static_cast<uint32_t>(reason), BSR_NO_CHUNK, 0);
}

// Wait for a bound request's device work, read its status, release its
// references and admission.  The context lock is dropped while the device
// work drains, so other requests keep going; the session is marked
// completing meanwhile, and no other call acts on it.  The session is gone
// when this returns.
static int complete_session(bsr_ctx* c, Session& s, std::unique_lock<std::mutex>& lk, bool run_commit,
                            uint64_t* exposed, int32_t* fallback) {
  SessionRes& res = c->res[s.res];
  bsr_stats& st = s.st;
  int rc = BSR_OK;
  if (run_commit) {
    if (s.failed || s.next_chunk < s.n_hit) {
      // a failure the host knows of, or an incomplete prefix, is never
      // exposed: invalidate right before the commit (on the device the first
      // recorded failure is kept, so repeating an earlier invalidate is harmless)
      const int reason = s.host_fail != BSR_FAIL_NONE ? s.host_fail : BSR_FAIL_ABORT;
      rc = enqueue_finish(c, s, bsr::kFinishInvalidate, static_cast<uint32_t>(reason), BSR_NO_CHUNK, 0);
      s.failed = true;
    }
    if (!rc) rc = enqueue_finish(c, s, bsr::kFinishCommit, 0, BSR_NO_CHUNK, 0);
  }
  if (!rc) rc = flush_batch(c, s);
  if (!rc) rc = hip_check(hipMemcpyAsync(res.host_status, s.status, sizeof(bsr_dev_status), hipMemcpyDeviceToHost, s.compute), "status readback");
  s.completing = true;
  const hipStream_t compute = s.compute, copy = s.copy;
  // Once the compute stream has waited for the last copy event, every copy
  // is behind its sync; the copy stream is synchronised only if it holds
  // work recorded after that (a run whose batch was never installed).
  const bool sync_copy = copy != compute && s.copy_dirty;
  const uint64_t t0 = now_ns();
  lk.unlock();
  int rc2 = hip_check(hipStreamSynchronize(compute), "hipStreamSynchronize(compute)");
  int rc3 = sync_copy ? hip_check(hipStreamSynchronize(copy), "hipStreamSynchronize(copy)") : BSR_OK;
  lk.lock();
  if (!rc) rc = rc2 ? rc2 : rc3;
  st.commit_wait_ns = now_ns() - t0;
  if (!rc) {
    const bsr_dev_status& h = *res.host_status;
    st.exposed_tokens = h.exposed_tokens;
    st.fallback = static_cast<int32_t>(h.fallback);
    st.fail_reason = static_cast<int32_t>(h.fail);
    st.first_failed_chunk = h.first_failed_chunk;
    uint32_t m = 0;
    for (uint32_t g = 0; g < c->geo.L.n_groups; ++g)
      if (h.q[g]) m |= 1u << g;
    st.q_mask = m;
    if (h.fallback) c->force_local.insert(s.id);
    if (exposed) *exposed = h.exposed_tokens;
    if (fallback) *fallback = static_cast<int32_t>(h.fallback);
  } else {
    c->force_local.insert(s.id);
    st.fallback = 1;
    if (exposed) *exposed = 0;
    if (fallback) *fallback = 1;
  }
  double tot = 0, mx = 0;
  for (auto& pr : s.timing) {
    float ms = 0;
    if (hipEventElapsedTime(&ms, pr.first, pr.second) == hipSuccess) {
      tot += ms;
      mx = std::max(mx, static_cast<double>(ms));
    }
    c->timing_pool.push_back(pr.first);
    c->timing_pool.push_back(pr.second);
  }
  s.timing.clear();
  st.install_ms_total = tot;
  st.install_ms_max = mx;
  double stot = 0;
  for (auto& pr : s.stage_timing) {
    float ms = 0;
    if (hipEventElapsedTime(&ms, pr.first, pr.second) == hipSuccess) stot += ms;
    c->timing_pool.push_back(pr.first);
    c->timing_pool.push_back(pr.second);
  }
  s.stage_timing.clear();
  st.stage_ms_total = stot;
  release_refs(c, s);
  const uint64_t id = s.id;
  auto it = c->requests.find(id);
  if (it != c->requests.end()) {
    it->second.phase = Phase::Done;
    it->second.has_stats = true;
    it->second.stats = st;
  }
  c->last = st;
  c->last_id = id;
  c->bound_bytes -= s.ring_bytes;
  res.in_use = false;
  c->bound.erase(id);  // s is gone from here on
  return rc;
}

int bsr_commit(bsr_ctx* c, uint64_t request_id, uint64_t* exposed_tokens, int32_t* fallback) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (int rc = set_device(c)) return rc;
  std::unique_lock<std::mutex> lk(c->mu);
  Session* s = nullptr;
  if (int rc = find_active(c, request_id, &s)) return rc;
  return complete_session(c, *s, lk, true, exposed_tokens, fallback);
}

int bsr_set_timing(bsr_ctx* c, uint32_t flags) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (flags & ~kTimingFlags) return fail_with(BSR_E_ARG, "flags 0x%x are not timing flags", flags);
  std::lock_guard<std::mutex> lk(c->mu);
  c->cfg.flags = (c->cfg.flags & ~kTimingFlags) | flags;
  return BSR_OK;
}

int bsr_request_running(bsr_ctx* c, uint64_t request_id) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  c->force_local.erase(request_id);
  return BSR_OK;
}

int bsr_request_end(bsr_ctx* c, uint64_t request_id) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::unique_lock<std::mutex> lk(c->mu);
  int rc = BSR_OK;
  if (Session* s = find_bound(c, request_id)) {
    if (s->completing) return fail_with(BSR_E_STATE, "request %llu is being completed", (unsigned long long)request_id);
    if ((rc = set_device(c))) return rc;
    rc = complete_session(c, *s, lk, false, nullptr, nullptr);
  }
  c->force_local.erase(request_id);
  c->requests.erase(request_id);
  return rc;
}

// ---- file-backed lower tier ----------------------------------------------------

int bsr_file_tier_open(bsr_ctx* c, const char* dir, uint32_t load_concurrency, uint32_t readahead_chunks,
                       uint32_t flags) {
  if (!c || !dir) return fail_with(BSR_E_ARG, "ctx or dir is NULL");
  if (load_concurrency == 0 || load_concurrency > 64) return fail_with(BSR_E_ARG, "load_concurrency must be 1..64");
  if (readahead_chunks && readahead_chunks < load_concurrency)
    return fail_with(BSR_E_ARG, "readahead_chunks must be 0 or >= load_concurrency");
  if (flags & ~BSR_FILE_DIRECT) return fail_with(BSR_E_ARG, "unknown flags 0x%x", flags);
  std::lock_guard<std::mutex> lk(c->mu);
  std::string err;
  if (c->ftier.open(dir, c->geo.L.n_groups, c->geo.slot_bytes, c->geo.offset, c->geo.payload, load_concurrency,
                    readahead_chunks, (flags & BSR_FILE_DIRECT) != 0, &err))
    return fail_with(BSR_E_ARG, "%s", err.c_str());
  return BSR_OK;
}

int bsr_file_tier_put_chunk(bsr_ctx* c, uint64_t key, const void* const* payloads) {
  if (!c || !payloads) return fail_with(BSR_E_ARG, "ctx or payloads is NULL");
  if (!c->ftier.is_open()) return fail_with(BSR_E_STATE, "file tier is not open");
  const uint32_t G = c->geo.L.n_groups;
  uint64_t tags[BSR_MAX_GROUPS] = {};
  for (uint32_t g = 0; g < G; ++g) {
    if (!payloads[g]) return fail_with(BSR_E_ARG, "payload of group %u is NULL", g);
    tags[g] = tag_of(static_cast<const uint8_t*>(payloads[g]), c->geo.payload[g]);
  }
  std::string err;
  if (c->ftier.put(key, payloads, tags, &err)) return fail_with(BSR_E_TRANSFER, "%s", err.c_str());
  return BSR_OK;
}

int bsr_file_tier_remove(bsr_ctx* c, uint64_t key, int32_t group) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (!c->ftier.is_open()) return fail_with(BSR_E_STATE, "file tier is not open");
  if (group >= static_cast<int32_t>(c->geo.L.n_groups)) return fail_with(BSR_E_ARG, "group %d out of range", group);
  std::string err;
  const int r = c->ftier.remove(key, group, &err);
  if (r > 0) return fail_with(BSR_E_NOTFOUND, "%s", err.c_str());
  if (r < 0) return fail_with(BSR_E_TRANSFER, "%s", err.c_str());
  return BSR_OK;
}

int bsr_file_tier_count(bsr_ctx* c, uint64_t* n_entries) {
  if (!c || !n_entries) return fail_with(BSR_E_ARG, "ctx or out is NULL");
  *n_entries = c->ftier.is_open() ? c->ftier.n_entries() : 0;
  return BSR_OK;
}

int bsr_tier_set_available(bsr_ctx* c, int32_t tier, int32_t available) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (tier == BSR_TIER_PINNED)
    c->tier0_available = available != 0;
  else if (tier == BSR_TIER_FILE)
    c->ftier.available = available != 0;
  else
    return fail_with(BSR_E_ARG, "unknown tier %d", tier);
  return BSR_OK;
}

int bsr_plan_tiers(bsr_ctx* c, uint64_t request_id, uint8_t* tier_of_chunk, uint32_t n_chunks) {
  if (!c || !tier_of_chunk) return fail_with(BSR_E_ARG, "ctx or out is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  auto it = c->requests.find(request_id);
  if (it == c->requests.end()) return fail_with(BSR_E_NOTFOUND, "request %llu was not probed", (unsigned long long)request_id);
  const auto& t = it->second.tier;
  for (uint32_t i = 0; i < n_chunks; ++i) tier_of_chunk[i] = i < t.size() ? t[i] : kTierNone;
  return BSR_OK;
}

int bsr_stats_get(bsr_ctx* c, bsr_stats* out) {
  if (!c || !out) return fail_with(BSR_E_ARG, "ctx or out is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  const Session* s = find_bound(c, c->last_id);
  *out = s ? s->st : c->last;
  return BSR_OK;
}

int bsr_request_stats(bsr_ctx* c, uint64_t request_id, bsr_stats* out) {
  if (!c || !out) return fail_with(BSR_E_ARG, "ctx or out is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  if (const Session* s = find_bound(c, request_id)) {
    *out = s->st;
    return BSR_OK;
  }
  auto it = c->requests.find(request_id);
  if (it == c->requests.end() || !it->second.has_stats)
    return fail_with(BSR_E_NOTFOUND, "no counters for request %llu", (unsigned long long)request_id);
  *out = it->second.stats;
  return BSR_OK;
}

int bsr_admission_get(bsr_ctx* c, bsr_admission* out) {
  if (!c || !out) return fail_with(BSR_E_ARG, "ctx or out is NULL");
  std::lock_guard<std::mutex> lk(c->mu);
  *out = bsr_admission{};
  out->staging_budget_bytes = c->budget;
  out->max_bound_requests = static_cast<uint32_t>(c->res.size());
  out->n_bound = static_cast<uint32_t>(c->bound.size());
  out->bound_staging_bytes = c->bound_bytes;
  out->peak_bound_staging_bytes = c->peak_bound_bytes;
  out->peak_n_bound = c->peak_bound;
  out->n_refused = c->n_refused;
  out->aux_device_bytes = c->device >= 0 ? c->aux_bytes * c->res.size() : 0;
  return BSR_OK;
}

int bsr_debug_inject(bsr_ctx* c, int32_t kind, uint32_t chunk, uint32_t param) {
  if (!c) return fail_with(BSR_E_ARG, "ctx is NULL");
  if (kind < BSR_INJECT_NONE || kind > BSR_INJECT_LAUNCH_ERROR) return fail_with(BSR_E_ARG, "unknown inject kind %d", kind);
  std::lock_guard<std::mutex> lk(c->mu);
  c->inject = Inject{kind, chunk, param};
  return BSR_OK;
}

int bsr_measure_scatter(bsr_ctx* c, uint32_t block_bytes, uint64_t data_bytes, uint32_t reps, uint64_t seed,
                        uint32_t flags, double* gbps) {
  if (flags & ~BSR_SCATTER_WARM_SOURCE) return fail_with(BSR_E_ARG, "unknown flags 0x%x", flags);
  if (!c || !gbps || reps == 0 || block_bytes == 0 || block_bytes % 16 || data_bytes < block_bytes)
    return fail_with(BSR_E_ARG, "bad arguments (block_bytes a positive multiple of 16, data_bytes >= block_bytes)");
  if (int rc = set_device(c)) return rc;
  const uint64_t nb = data_bytes / block_bytes;
  const uint64_t n_pieces = (block_bytes + bsr::kMaxPieceBytes - 1) / bsr::kMaxPieceBytes;
  const uint32_t piece = static_cast<uint32_t>(align_up((block_bytes + n_pieces - 1) / n_pieces, bsr::kPieceAlign));
  const uint32_t ppb = (block_bytes + piece - 1) / piece;
  if (nb * ppb >= (1ull << 31) || nb >= (1ull << 30)) return fail_with(BSR_E_ARG, "too many blocks for one launch");
  // destinations: nb distinct blocks of a pool twice the data, in a seeded random order
  std::vector<int32_t> perm(2 * nb);
  for (uint64_t i = 0; i < perm.size(); ++i) perm[i] = static_cast<int32_t>(i);
  uint64_t x = seed * 0x9E3779B97F4A7C15ull + 1;
  for (uint64_t i = perm.size() - 1; i > 0; --i) {  // Fisher-Yates with a splitmix64 stream
    x += 0x9E3779B97F4A7C15ull;
    uint64_t z = x;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    std::swap(perm[i], perm[z % (i + 1)]);
  }
  void* src = nullptr;
  void* pool = nullptr;
  void* dperm = nullptr;
  hipStream_t st = nullptr;
  hipEvent_t ev[2] = {};
  int rc = BSR_OK;
  if (hipMalloc(&src, nb * block_bytes) != hipSuccess || hipMalloc(&pool, 2 * nb * block_bytes) != hipSuccess ||
      hipMalloc(&dperm, nb * sizeof(int32_t)) != hipSuccess)
    rc = fail_with(BSR_E_NOMEM, "buffers for the scatter measurement");
  if (!rc) rc = hip_check(hipStreamCreate(&st), "hipStreamCreate");
  for (int i = 0; !rc && i < 2; ++i) rc = hip_check(hipEventCreate(&ev[i]), "hipEventCreate");
  if (!rc) rc = hip_check(hipMemcpy(dperm, perm.data(), nb * sizeof(int32_t), hipMemcpyHostToDevice), "hipMemcpy");
  if (!rc) rc = hip_check(hipMemset(src, 0x5a, nb * block_bytes), "hipMemset");
  bsr::ScatterParams p{static_cast<const uint8_t*>(src), static_cast<uint8_t*>(pool),
                       static_cast<const int32_t*>(dperm), block_bytes, piece, ppb, static_cast<uint32_t>(nb),
                       c->xcd_log2, bsr::xcd_remap_bound(static_cast<uint32_t>(nb * ppb), c->xcd_log2), c->geo.lds_bytes};
  if (!rc) {
    double best = 0;
    for (uint32_t r = 0; r < reps && !rc; ++r) {
      // the staging copy writes a slot right before the install reads it
      if (flags & BSR_SCATTER_WARM_SOURCE)
        rc = hip_check(hipMemsetAsync(src, 0x30 + r, nb * block_bytes, st), "hipMemsetAsync");
      if (!rc) rc = hip_check(hipEventRecord(ev[0], st), "hipEventRecord");
      if (!rc) rc = hip_check(bsr::launch_scatter(p, st), "scatter launch");
      if (!rc) rc = hip_check(hipEventRecord(ev[1], st), "hipEventRecord");
      if (!rc) rc = hip_check(hipEventSynchronize(ev[1]), "hipEventSynchronize");
      float ms = 0;
      if (!rc) rc = hip_check(hipEventElapsedTime(&ms, ev[0], ev[1]), "hipEventElapsedTime");
      if (!rc && ms > 0) best = std::max(best, 2.0 * nb * block_bytes / (ms * 1e-3) / 1e9);
    }
    *gbps = best;
  }
  if (st) (void)hipStreamSynchronize(st);
  for (auto e : ev)
    if (e) (void)hipEventDestroy(e);
  if (st) (void)hipStreamDestroy(st);
  if (dperm) (void)hipFree(dperm);
  if (pool) (void)hipFree(pool);
  if (src) (void)hipFree(src);
  return rc;
}

int bsr_measure_stage(bsr_ctx* c, uint64_t bytes, uint32_t reps, double* gbps) {
  if (!c || !gbps || bytes == 0 || reps == 0 || bytes % 16) return fail_with(BSR_E_ARG, "bad arguments");
  if (int rc = set_device(c)) return rc;
  void* h = nullptr;
  void* d = nullptr;
  void* hd = nullptr;
  hipStream_t st = nullptr;
  hipEvent_t ev[2] = {};
  int rc = BSR_OK;
  if (hipHostMalloc(&h, bytes, hipHostMallocDefault) != hipSuccess || hipMalloc(&d, bytes) != hipSuccess ||
      hipHostGetDevicePointer(&hd, h, 0) != hipSuccess)
    rc = fail_with(BSR_E_NOMEM, "buffers for the staging-copy measurement");
  if (!rc) rc = hip_check(hipStreamCreate(&st), "hipStreamCreate");
  for (int i = 0; !rc && i < 2; ++i) rc = hip_check(hipEventCreate(&ev[i]), "hipEventCreate");
  if (!rc) {
    std::memset(h, 0x5a, bytes);
    double best = 0;
    for (uint32_t r = 0; r < reps && !rc; ++r) {
      rc = hip_check(hipEventRecord(ev[0], st), "hipEventRecord");
      if (!rc) rc = hip_check(bsr::launch_stage(bsr::StageParams{static_cast<const uint8_t*>(hd), static_cast<uint8_t*>(d), bytes}, st), "staging copy");
      if (!rc) rc = hip_check(hipEventRecord(ev[1], st), "hipEventRecord");
      if (!rc) rc = hip_check(hipEventSynchronize(ev[1]), "hipEventSynchronize");
      float ms = 0;
      if (!rc) rc = hip_check(hipEventElapsedTime(&ms, ev[0], ev[1]), "hipEventElapsedTime");
      if (!rc && ms > 0) best = std::max(best, bytes / (ms * 1e-3) / 1e9);
    }
    *gbps = best;
  }
  if (st) (void)hipStreamSynchronize(st);
  for (auto e : ev)
    if (e) (void)hipEventDestroy(e);
  if (st) (void)hipStreamDestroy(st);
  if (d) (void)hipFree(d);
  if (h) (void)hipHostFree(h);
  return rc;
}

int bsr_measure_h2d(bsr_ctx* c, uint64_t bytes, uint32_t n_streams, uint32_t reps, double* gbps) {
  if (!c || !gbps || bytes == 0 || reps == 0) return fail_with(BSR_E_ARG, "bad arguments");
  if (n_streams < 1 || n_streams > 4) return fail_with(BSR_E_ARG, "n_streams must be 1..4");
  if (int rc = set_device(c)) return rc;
  void* h = nullptr;
  void* d = nullptr;
  hipStream_t st[4] = {};
  hipEvent_t ev[6] = {};
  int rc = BSR_OK;
  if (hipHostMalloc(&h, bytes, hipHostMallocDefault) != hipSuccess || hipMalloc(&d, bytes) != hipSuccess)
    rc = fail_with(BSR_E_NOMEM, "buffers for the H2D measurement");
  for (uint32_t i = 0; !rc && i < n_streams; ++i) rc = hip_check(hipStreamCreate(&st[i]), "hipStreamCreate");
  for (int i = 0; !rc && i < 6; ++i) rc = hip_check(hipEventCreate(&ev[i]), "hipEventCreate");
  if (!rc) {
    std::memset(h, 0x5a, bytes);
    double best = 0;
    const uint64_t part = (bytes / n_streams) & ~uint64_t(4095);
    for (uint32_t r = 0; r < reps && !rc; ++r) {
      rc = hip_check(hipEventRecord(ev[0], st[0]), "hipEventRecord");
      for (uint32_t i = 1; !rc && i < n_streams; ++i) rc = hip_check(hipStreamWaitEvent(st[i], ev[0], 0), "wait");
      for (uint32_t i = 0; !rc && i < n_streams; ++i) {
        const uint64_t off = part * i;
        const uint64_t len = (i + 1 == n_streams) ? bytes - off : part;
        rc = hip_check(hipMemcpyAsync(static_cast<uint8_t*>(d) + off, static_cast<uint8_t*>(h) + off, len, hipMemcpyHostToDevice, st[i]), "hipMemcpyAsync");
        if (!rc && i) rc = hip_check(hipEventRecord(ev[1 + i], st[i]), "hipEventRecord");
        if (!rc && i) rc = hip_check(hipStreamWaitEvent(st[0], ev[1 + i], 0), "wait");
      }
      if (!rc) rc = hip_check(hipEventRecord(ev[5], st[0]), "hipEventRecord");
      if (!rc) rc = hip_check(hipEventSynchronize(ev[5]), "hipEventSynchronize");
      float ms = 0;
      if (!rc) rc = hip_check(hipEventElapsedTime(&ms, ev[0], ev[5]), "hipEventElapsedTime");
      if (!rc && ms > 0) best = std::max(best, bytes / (ms * 1e-3) / 1e9);
    }
    *gbps = best;
  }
  for (uint32_t i = 0; i < n_streams; ++i)
    if (st[i]) (void)hipStreamSynchronize(st[i]);
  for (auto e : ev)
    if (e) (void)hipEventDestroy(e);
  for (auto s2 : st)
    if (s2) (void)hipStreamDestroy(s2);
  if (d) (void)hipFree(d);
  if (h) (void)hipHostFree(h);
  return rc;
}

}  // extern "C"
