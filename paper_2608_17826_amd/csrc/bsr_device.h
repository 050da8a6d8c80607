// Internal interface between the host runtime and the gfx950 kernels.
// Plain structs passed by value as kernel arguments; no HIP types leak into
// include/bsr.h.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "bsr.h"

namespace bsr {

#ifndef BSR_MAX_PIECE_BYTES
#define BSR_MAX_PIECE_BYTES 8192
#endif
#ifndef BSR_PLANAR_PIECE_BYTES
#define BSR_PLANAR_PIECE_BYTES 20480
#endif

#ifndef BSR_INSTALL_THREADS
#define BSR_INSTALL_THREADS 128
#endif
#ifndef BSR_INSTALL_WG_PER_CU
#define BSR_INSTALL_WG_PER_CU 4
#endif

constexpr int kInstallThreads = BSR_INSTALL_THREADS;  // wave64 multiples
constexpr int kInstallWaves = kInstallThreads / 64;
// contiguous segments are cut into equal pieces of at most this many bytes,
// each a multiple of kPieceAlign (one 16-byte vector per thread)
constexpr uint32_t kMaxPieceBytes = BSR_MAX_PIECE_BYTES;
constexpr uint32_t kPieceAlign = 16 * kInstallThreads;
// Install workgroups resident per CU.  Each holds one piece (8 KiB) of loads
// in flight, so four keep 32 KiB per CU in flight.  The install is a mixed
// read + write stream to scattered destinations; HBM moves it fastest with
// that much in flight, not with the most the CU can hold (a full CU keeps
// twice as much queued and runs about 4% slower).  The limit is applied by
// sizing each workgroup's dynamic LDS to 1/4 of the CU's.
constexpr uint32_t kInstallWgPerCu = BSR_INSTALL_WG_PER_CU;
// planar pieces (whole tokens) are staged through LDS up to this size
constexpr uint32_t kLdsCapBytes = BSR_PLANAR_PIECE_BYTES;

#ifndef BSR_XCD_RUN
#define BSR_XCD_RUN 36
#endif
// Work order across the XCDs.  The dispatcher hands workgroup b of a launch
// to XCD b mod X (X = 2^xcd_log2 XCDs in the device's partition: 8 on a
// whole MI355X), so consecutive work items (the pieces of one destination
// block) would run on X XCDs behind X L2s.  The install remaps b so that
// each XCD takes runs of kXcdRun consecutive work items instead: the
// pieces of a block then reach memory from one XCD.  Measured as a plain
// copy of the install's shape into random 73.7 KB blocks on eight XCDs:
// 69.5% of 8 TB/s round robin, 77.3% with runs of 9 (one block), 78.2% with
// 18, 77.9% with 36; into blocks in identity order 82% either way.  The
// remap is a permutation for any X; with one XCD it is the identity.
constexpr uint32_t kXcdRun = BSR_XCD_RUN;
static_assert(kXcdRun >= 1, "runs of at least one work item (1: round robin)");
// log2 of the XCD count the host reads from the device (a power of two;
// anything else is rounded down).
inline uint32_t xcd_log2_of(int n_xcds) {
  uint32_t l = 0;
  while (n_xcds > 1 && (2 << l) <= n_xcds) ++l;
  return l;
}
// Work items below the returned bound are remapped (whole spans of
// X * kXcdRun); the ragged rest keeps its order.
inline uint32_t xcd_remap_bound(uint32_t grid, uint32_t xcd_log2) {
  const uint32_t span = kXcdRun << xcd_log2;
  return kXcdRun > 1 && xcd_log2 > 0 ? grid / span * span : 0;
}

#if defined(__HIP__)
// Work item of hardware workgroup b (a permutation of [0, grid) whenever
// full = xcd_remap_bound(grid, xcd_log2)).
__device__ __forceinline__ uint32_t xcd_work_index(uint32_t b, uint32_t full, uint32_t xcd_log2) {
  if (b >= full) return b;
  const uint32_t xcd = b & ((1u << xcd_log2) - 1u), local = b >> xcd_log2;
  return ((local / kXcdRun * kXcdRun) << xcd_log2) + xcd * kXcdRun + local % kXcdRun;
}
#endif

// Tag partial of one install workgroup: sum and XOR of the little-endian u32
// words it read from the staged chunk.
struct TagPair {
  uint32_t sum;
  uint32_t x;
};

// Division of a 32-bit n by an invariant d as a multiply-high and two
// shifts (Granlund & Montgomery, "Division by invariant integers using
// multiplication", 1994, round-up multiplier): t = mulhi(m, n),
// n / d = (t + ((n - t) >> s1)) >> s2.  Built on the host (make_fastdiv).
struct FastDiv {
  uint32_t d, m, s1, s2;
#if defined(__HIP__)
  __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
    const uint32_t t = static_cast<uint32_t>((static_cast<uint64_t>(m) * n) >> 32);
    return (t + ((n - t) >> s1)) >> s2;
  }
#endif
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;  // l = ceil(log2 d)
  const uint64_t m = ((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d) + 1;
  return FastDiv{d, static_cast<uint32_t>(m), l < 1 ? l : 1u, l > 1 ? l - 1 : 0u};
}

// The same division packed for the install kernel: the multiplier and both
// shifts in two words (s = s1 | s2 << 8).
struct PackedDiv {
  uint32_t m, s;
};

inline PackedDiv pack_fastdiv(const FastDiv& f) { return PackedDiv{f.m, f.s1 | (f.s2 << 8)}; }

#if defined(__HIP__)
// (host-callable too, so that a CPU test checks the kernel's own division)
__host__ __device__ __forceinline__ uint32_t packed_div(uint32_t m, uint32_t s, uint32_t n) {
  const uint32_t t = static_cast<uint32_t>((static_cast<uint64_t>(m) * n) >> 32);
  return (t + ((n - t) >> (s & 0xffu))) >> (s >> 8);
}
#endif

// Per-group geometry of a layout, without request pointers (host side).
struct GroupGeom {
  uint32_t block_tokens;
  uint32_t n_tensors;
  uint32_t record_bytes;
  uint32_t kind;
  uint32_t split_bytes;
  uint32_t staged_off;      // byte offset of the group's entry inside a slot
  uint32_t segs_per_chunk;  // upper bound of destination blocks one chunk touches
  uint32_t pieces_per_seg;  // workgroups per (tensor, block) segment
  uint32_t piece_bytes;     // CONTIG: bytes per piece (multiple of 16)
  uint32_t piece_tokens;    // PLANAR: tokens per piece
  FastDiv div_pieces;       // by pieces_per_seg
  FastDiv div_segs;         // by segs_per_chunk
  FastDiv div_per_chunk;    // by the group's workgroups per chunk
  FastDiv div_block;        // by block_tokens
};

// Install kernel arguments.  A wave needs all of this before it can address
// its piece, so the kernel reads the head and then its group's record each
// as two 64-byte scalar loads issued together: two dependent rounds of
// argument reads in all.  Word positions are fixed by the static_asserts.
struct InstallHead {
  // words 0-15
  uint32_t n_chunks;        // chunks in this launch (<= BSR_MAX_INSTALL_BATCH, <= W)
  uint32_t first_chunk;     // global index of the launch's first chunk
  uint32_t chunk_tokens;
  uint32_t window;          // W (slots in the ring)
  uint32_t first_slot;      // first_chunk mod W
  uint32_t xcd_log2;        // log2 of the XCDs the dispatcher deals workgroups to
  uint32_t n_groups;
  uint32_t wg_per_chunk;    // workgroups per chunk, all groups
  // Workgroups are issued group by group (contiguous groups by descending
  // piece size, then block size, planar groups just before the last
  // contiguous group); within a group, chunk by chunk, first to last, or,
  // at odd dispatch positions when `serpentine` is 1, last to first.
  // start[o] is the first work item of dispatch position o in this launch
  // (n_chunks times the workgroups per chunk of the positions before it);
  // positions past the last group hold the grid size, which no work item
  // reaches.
  uint32_t start[BSR_MAX_GROUPS];
  // words 16-31
  const uint8_t* ring;
  uint64_t slot_bytes;
  const bsr_dev_status* status;
  TagPair* partials;        // [n_chunks * wg_per_chunk * kInstallWaves], one per wave, chunk-major
  uint32_t lds_bytes;       // dynamic LDS of this launch
  uint32_t xcd_full;        // hardware workgroups below it are remapped across the XCDs
  uint32_t serpentine;      // 1: odd dispatch positions take the launch's chunks last to first
  uint32_t pad[5];
};

struct InstallGroup {
  // words 0-15
  uint32_t per_chunk;       // workgroups per chunk of this group
  uint32_t wg_start;        // offset of the group's workgroups inside a chunk's tag partial slots
  PackedDiv div_per_chunk;
  PackedDiv div_pieces;
  PackedDiv div_segs;
  PackedDiv div_block;
  uint32_t pieces_per_seg;
  uint32_t segs_per_chunk;
  uint32_t block_tokens;
  uint32_t record_bytes;
  uint32_t staged_off;
  uint32_t piece;           // CONTIG: bytes per piece; PLANAR: tokens per piece
  // words 16-31
  uint32_t kind;
  uint32_t split_bytes;
  uint32_t n_blocks;        // entries of the block table
  uint32_t pool_blocks;
  const int32_t* block_table;
  uint8_t* const* tensor_bases;
  uint32_t group;           // index of the group in the layout
  PackedDiv div_p1;         // PLANAR: by plane-1 vectors per token (split_bytes / 16)
  PackedDiv div_p2;         // PLANAR: by plane-2 words per token ((record_bytes - split_bytes) / 4)
  uint32_t prefix;          // workgroups per chunk of the groups before this one in dispatch order
  uint32_t block_bytes;     // block_tokens * record_bytes (< 2^31)
  uint32_t pad[1];
};

static_assert(sizeof(InstallHead) == 128 && sizeof(InstallGroup) == 128, "two 64-byte scalar loads each");
static_assert(offsetof(InstallHead, ring) == 64 && offsetof(InstallGroup, kind) == 64, "second halves start at word 16");
static_assert(offsetof(InstallHead, start) == 32, "the group starts fill words 8-15");

struct InstallParams {
  InstallHead h;
  InstallGroup g[BSR_MAX_GROUPS];  // in dispatch order
};

// Device words the verify kernel uses across workgroups (library-owned,
// zeroed by the begin kernel and left zeroed by every verify launch).
struct VerifyAux {
  uint32_t bad[BSR_MAX_INSTALL_BATCH];  // per chunk of the launch: mask of mismatching groups
  uint32_t arrivals;                    // workgroups finished in the current launch
  uint32_t pad[15];
};

struct VerifyParams {
  const TagPair* partials;
  bsr_dev_status* status;
  VerifyAux* aux;
  uint32_t n_chunks;
  uint32_t first_chunk;
  uint32_t n_groups;
  uint32_t wg_per_chunk;
  uint32_t wg_start[BSR_MAX_GROUPS + 1];
  uint64_t expected[BSR_MAX_INSTALL_BATCH][BSR_MAX_GROUPS];  // stored tags
};

struct GroupValid {
  const int32_t* block_table;
  uint8_t* valid;
  uint32_t n_req_blocks;    // advertised blocks of this group
  uint32_t pool_blocks;
  uint32_t block_tokens;
  uint32_t pad;
};

// mode of the finishing kernel
enum FinishMode : uint32_t {
  kFinishBegin = 0,       // reset status, clear advertised valid bytes
  kFinishCommit = 1,      // Eq. 6: Q -> valid bytes, exposed, fallback
  kFinishInvalidate = 2,  // record failure, clear valid bytes, exposed = 0, fallback = 1
  kFinishMarkGroup = 3,   // q[group] = 0
  kFinishCheckTables = 4, // fail the request if an advertised block id is outside its pool
};

struct FinishParams {
  bsr_dev_status* status;
  VerifyAux* verify_aux;    // begin: zeroed
  uint32_t mode;
  uint32_t n_groups;
  uint32_t reason;          // invalidate: BSR_FAIL_*
  uint32_t chunk;           // invalidate: failing chunk or BSR_NO_CHUNK
  uint32_t group_mask;      // invalidate: groups whose q_g becomes 0; mark: the group
  uint32_t total_blocks;    // sum of n_req_blocks
  uint32_t chunk_tokens;
  uint64_t exposed_if_valid;
  GroupValid g[BSR_MAX_GROUPS];
};

// Staging copy (pinned host memory -> ring slot) done by a kernel on the
// copy stream instead of the copy engine.  src is the device's view of the
// pinned source, 16-byte aligned; dst is in the ring, 16-byte aligned; bytes
// is a multiple of 4.  The host checks both ranges before every launch.
struct StageParams {
  const uint8_t* src;
  uint8_t* dst;
  uint64_t bytes;
};
// Shape: the host link needs about its bandwidth-delay product in flight,
// and reads queued beyond it delay the install's HBM traffic when the two
// overlap.  24 workgroups x 256 threads x 2 vectors keep 192 KiB in flight.
// Measured on one box, 512K 4-group workload (grid x vectors, KiB in
// flight: restore GB/s at W = 32, install's share of 8 TB/s at W = 32 and
// W = 8): 24 x 2, 192: 56.84, 76.5%, 62.9%; 32 x 2, 256: 56.87, 74.3%,
// 55.8%; 48 x 1, 192: 56.61, 75.1% (W = 32 only); 16 x 2 and 32 x 1, 128:
// 56.44-56.59, 79.1%, 72.4%; 64 x 4, 1 MiB: installs three times slower.
// Staging that keeps less in flight moves less over the link (8 x 4, 128:
// 55.9 GB/s of link), so 192 KiB is the shape that keeps the link's rate.
#ifndef BSR_STAGE_GRID
#define BSR_STAGE_GRID 24
#endif
#ifndef BSR_STAGE_UNROLL
#define BSR_STAGE_UNROLL 2
#endif
constexpr int kStageThreads = 256;
constexpr int kStageUnroll = BSR_STAGE_UNROLL;  // 16-byte vectors in flight per thread
constexpr int kStageMaxGrid = BSR_STAGE_GRID;   // workgroups

// Scratch of a context that allocates nothing (bsr_ctx_create_static): one
// array per GPU in the library's code object, holding one session slot's
// install tag partials and verify words.  static_scratch_claim runs at the
// context's set-up with `device` current: the first claim on a device looks
// the array's device address up (hipGetSymbolAddress) and keeps it; a claim
// while another context of this process holds the device's array sets *busy.
constexpr uint64_t kStaticScratchBytes = BSR_STATIC_SCRATCH_BYTES;
constexpr int kMaxScratchDevices = 64;
hipError_t static_scratch_claim(int device, void** ptr, bool* busy);
void static_scratch_release(int device);

// Ceiling for the install (bsr_measure_scatter): a plain copy of whole
// blocks from a contiguous source into scattered destination blocks, with
// the install's workgroup shape, occupancy (lds_bytes) and XCD work order,
// and nothing else.
struct ScatterParams {
  const uint8_t* src;        // n_blocks x block_bytes, contiguous
  uint8_t* pool;             // destination pool of block_bytes blocks
  const int32_t* dst_block;  // destination block of each source block
  uint32_t block_bytes;      // a multiple of 16
  uint32_t piece_bytes;      // a multiple of kPieceAlign, at most kMaxPieceBytes
  uint32_t pieces_per_block;
  uint32_t n_blocks;
  uint32_t xcd_log2;
  uint32_t xcd_full;
  uint32_t lds_bytes;
};
hipError_t launch_scatter(const ScatterParams& p, hipStream_t s);

hipError_t launch_install(const InstallParams& p, uint32_t n_workgroups, hipStream_t s,
                          hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
hipError_t launch_verify(const VerifyParams& p, hipStream_t s);
hipError_t launch_stage(const StageParams& p, hipStream_t s, hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
hipError_t launch_finish(const FinishParams& p, hipStream_t s);

}  // namespace bsr
