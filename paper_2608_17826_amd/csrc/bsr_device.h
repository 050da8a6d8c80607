// Internal interface between the host runtime and the gfx950 kernels.
// Plain structs passed by value as kernel arguments; no HIP types leak into
// include/bsr.h.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "bsr.h"

namespace bsr {

constexpr int kInstallThreads = 256;     // 4 wave64 per workgroup
constexpr uint32_t kPieceBytes = 16384;  // contiguous-group bytes per workgroup
constexpr uint32_t kLdsCapBytes = 32768; // planar pieces staged through LDS up to this size

// Tag partial of one install workgroup: sum and XOR of the little-endian u32
// words it read from the staged chunk.
struct TagPair {
  uint32_t sum;
  uint32_t x;
};

// Per-group geometry of one install launch.
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
  uint32_t pool_blocks;
  uint32_t n_blocks;
  const int32_t* block_table;
  uint8_t* const* tensor_bases;
};

struct InstallParams {
  const uint8_t* ring;
  uint64_t slot_bytes;
  uint32_t window;          // W (slots in the ring)
  uint32_t chunk_tokens;
  uint32_t n_groups;
  uint32_t n_chunks;        // chunks in this launch (<= BSR_MAX_INSTALL_BATCH)
  uint32_t first_chunk;     // global index of the launch's first chunk
  uint32_t wg_per_chunk;    // workgroups per chunk, all groups
  uint32_t wg_start[BSR_MAX_GROUPS + 1];  // prefix of workgroups per group within a chunk
  uint32_t lds_bytes;       // dynamic LDS of this launch
  GroupGeom g[BSR_MAX_GROUPS];
  TagPair* partials;        // [n_chunks * wg_per_chunk], one per workgroup
  const bsr_dev_status* status;
};

struct VerifyParams {
  const TagPair* partials;
  bsr_dev_status* status;
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
};

// mode of the finishing kernel
enum FinishMode : uint32_t {
  kFinishBegin = 0,       // reset status, clear advertised valid bytes
  kFinishCommit = 1,      // Eq. 6: Q -> valid bytes, exposed, fallback
  kFinishInvalidate = 2,  // record failure, clear valid bytes, exposed = 0, fallback = 1
  kFinishMarkGroup = 3,   // q[group] = 0
};

struct FinishParams {
  bsr_dev_status* status;
  uint32_t mode;
  uint32_t n_groups;
  uint32_t reason;          // invalidate: BSR_FAIL_*
  uint32_t chunk;           // invalidate: failing chunk or BSR_NO_CHUNK
  uint32_t group_mask;      // invalidate: groups whose q_g becomes 0; mark: the group
  uint32_t total_blocks;    // sum of n_req_blocks
  uint64_t exposed_if_valid;
  GroupValid g[BSR_MAX_GROUPS];
};

hipError_t launch_install(const InstallParams& p, uint32_t n_workgroups, hipStream_t s);
hipError_t launch_verify(const VerifyParams& p, hipStream_t s);
hipError_t launch_finish(const FinishParams& p, hipStream_t s);

}  // namespace bsr
