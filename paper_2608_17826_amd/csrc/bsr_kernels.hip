// gfx950 kernels of the bounded-window restore.
//
// install : scatter staged chunks from the W-slot ring into every group's
//           paged blocks (§3 "Install locally"; §4 windowed retrieve, whose
//           per-window step moves the staged window into the engine's
//           blocks).  One
//           workgroup per piece of a (tensor, destination block) segment.
//           Contiguous groups move 16-byte vectors ring -> pool, all loads of
//           a piece issued before its destination is resolved; planar groups
//           (records split into a values plane and a scales plane inside a
//           block) stage the piece in LDS and write both planes with
//           coalesced stores.  Every wave also folds the words it read into
//           a (sum, xor) tag partial, and ballots the request's status words
//           first, so no workgroup installs past a failure.
// verify  : reduce the partials of each (chunk, group) and compare with the
//           tag recorded at store time; the first mismatching chunk, in
//           chunk order, fails the request (q_g = 0 for its mismatching
//           groups).
// finish  : begin (reset status, clear advertised valid bytes), commit
//           (Eq. 6), invalidate (§4 failed-block + HMA-aware invalidation),
//           mark one group invalid, check the block tables on the device.
//
// Nothing here is a dense contraction: the path is bound by HBM bandwidth
// (read the staged chunk once, write the paged blocks once).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "bsr_device.h"

#ifndef BSR_UNROLL
#define BSR_UNROLL 2    // 16-byte vectors per thread of a contiguous piece
#endif
#ifndef BSR_NT_LOAD
#define BSR_NT_LOAD 1   // staged chunks are read once: non-temporal loads
#endif
#ifndef BSR_NT_STORE
#define BSR_NT_STORE 1  // paged blocks are not re-read by this path: non-temporal stores
#endif


namespace bsr {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ T ld_stream(const T* p) {
#if BSR_NT_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void st_stream(T v, T* p) {
#if BSR_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

__device__ __forceinline__ void fold(const u32x4 v, uint32_t& s, uint32_t& x) {
  s += (v.x + v.y) + (v.z + v.w);
  x ^= (v.x ^ v.y) ^ (v.z ^ v.w);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ uint32_t wave_xor(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v ^= __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------------------
// contiguous piece that is not 16-byte aligned (records are multiples of 4
// bytes): 4-byte words
// ---------------------------------------------------------------------------
__device__ __forceinline__ void copy_words(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                           uint32_t len, uint32_t tid, uint32_t& s, uint32_t& x) {
  const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
  uint32_t* d1 = reinterpret_cast<uint32_t*>(dst);
  const uint32_t nw = len >> 2;
  for (uint32_t i = tid; i < nw; i += kInstallThreads) {
    const uint32_t w = s1[i];
    s += w;
    x ^= w;
    d1[i] = w;
  }
}

// ---------------------------------------------------------------------------
// planar segment piece: mu tokens of AoS records (r bytes each) starting at
// in-block position o.  Plane 1 gets the first sp bytes of each record at
// o*sp, plane 2 the remaining r-sp bytes at B*sp + o*(r-sp).
// ---------------------------------------------------------------------------
constexpr uint32_t kPlanarVecs = (kLdsCapBytes + kPieceAlign - 1) / kPieceAlign;  // vectors per thread

// Fast path, second half: the piece's words are in registers (v); stage them
// in LDS, then write plane 1 with 16-byte stores and plane 2 with 4-byte stores.
__device__ __forceinline__ void planar_from_regs(const u32x4 (&v)[kPlanarVecs], uint32_t nvec, uint8_t* dst1,
                                                 uint8_t* dst2, uint32_t mu, uint32_t r, uint32_t sp,
                                                 uint8_t* lds, uint32_t tid, uint32_t& s, uint32_t& x) {
  u32x4* l4 = reinterpret_cast<u32x4*>(lds);
#pragma unroll
  for (uint32_t u = 0; u < kPlanarVecs; ++u) {
    const uint32_t i = u * kInstallThreads + tid;
    if (i < nvec) {
      fold(v[u], s, x);
      l4[i] = v[u];
    }
  }
  __syncthreads();
  const uint32_t* l1 = reinterpret_cast<const uint32_t*>(lds);
  // plane 1: vector i covers token i / (sp/16), part i % (sp/16)
  const uint32_t vpt = sp >> 4;
  const uint32_t n1 = mu * vpt;
  u32x4* d4 = reinterpret_cast<u32x4*>(dst1);
  for (uint32_t i = tid; i < n1; i += kInstallThreads) {
    const uint32_t u = i / vpt;
    const uint32_t part = i - u * vpt;
    const uint32_t w0 = (u * r + part * 16) >> 2;
    u32x4 w;
    w.x = l1[w0];
    w.y = l1[w0 + 1];
    w.z = l1[w0 + 2];
    w.w = l1[w0 + 3];
    st_stream(w, d4 + i);
  }
  const uint32_t w2 = (r - sp) >> 2;
  const uint32_t n2 = mu * w2;
  uint32_t* d2 = reinterpret_cast<uint32_t*>(dst2);
  for (uint32_t i = tid; i < n2; i += kInstallThreads) {
    const uint32_t u = i / w2;
    const uint32_t wi = i - u * w2;
    d2[i] = l1[((u * r + sp) >> 2) + wi];
  }
}

// Any alignment: 4-byte words straight from the staged records.
__device__ __forceinline__ void planar_words(const uint8_t* __restrict__ src, uint8_t* dst1, uint8_t* dst2,
                                             uint32_t mu, uint32_t r, uint32_t sp, uint32_t tid, uint32_t& s,
                                             uint32_t& x) {
  const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
  uint32_t* d1 = reinterpret_cast<uint32_t*>(dst1);
  uint32_t* d2 = reinterpret_cast<uint32_t*>(dst2);
  const uint32_t rw = r >> 2, sw = sp >> 2, nw = (mu * r) >> 2;
  for (uint32_t i = tid; i < nw; i += kInstallThreads) {
    const uint32_t u = i / rw;
    const uint32_t wi = i - u * rw;
    const uint32_t w = s1[i];
    s += w;
    x ^= w;
    if (wi < sw)
      d1[u * sw + wi] = w;
    else
      d2[u * (rw - sw) + (wi - sw)] = w;
  }
}

__global__ __launch_bounds__(kInstallThreads) void k_install(const InstallParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  const uint32_t tid = threadIdx.x;
  const uint32_t lane = tid & 63;
  uint32_t rem = blockIdx.x;
  // work index -> (group, chunk, piece within the chunk's group range)
  uint32_t oi = 0, gi = p.order[0];
  for (;;) {
    const uint32_t n = (p.wg_start[gi + 1] - p.wg_start[gi]) * p.n_chunks;
    if (rem < n || oi + 1 == p.n_groups) break;
    rem -= n;
    gi = p.order[++oi];
  }
  const GroupGeom& G = p.g[gi];
  const uint32_t per_chunk = p.wg_start[gi + 1] - p.wg_start[gi];
  const uint32_t c = G.div_per_chunk.div(rem);
  rem -= c * per_chunk;
  const uint32_t wg = c * p.wg_per_chunk + p.wg_start[gi] + rem;  // chunk-major slot of the tag partials

  const uint32_t r1 = G.div_pieces.div(rem);
  const uint32_t piece = rem - r1 * G.pieces_per_seg;
  const uint32_t t = G.div_segs.div(r1);
  const uint32_t j = r1 - t * G.segs_per_chunk;

  const uint32_t chunk = p.first_chunk + c;
  const uint32_t slot = chunk - p.div_window.div(chunk) * p.window;
  const uint64_t C = p.chunk_tokens, B = G.block_tokens;
  const uint32_t tok0_32 = chunk * p.chunk_tokens;  // the bound prefix has < 2^32 tokens
  const uint64_t tok0 = tok0_32;
  const uint64_t k = G.div_block.div(tok0_32) + j;  // request block index
  const uint64_t blo = k * B;
  const uint64_t lo = tok0 > blo ? tok0 : blo;
  const uint64_t hi = (tok0 + C) < (blo + B) ? (tok0 + C) : (blo + B);

  uint32_t s = 0, x = 0;
  if (lo < hi && k < G.n_blocks) {
    // Metadata loads first (status words, destination block id, tensor base);
    // they resolve while the staged bytes are loaded: the source address
    // depends on none of them.
    bool bad = false;
    if (lane == 0)
      bad = p.status->fail != 0;
    else if (lane <= p.n_groups)
      bad = p.status->q[lane - 1] == 0;
    const int32_t b = G.block_table[k];
    uint8_t* const tbase = G.tensor_bases[t];

    const uint32_t r = G.record_bytes;
    const uint32_t m = static_cast<uint32_t>(hi - lo);
    const uint32_t q0 = static_cast<uint32_t>(lo - tok0);
    const uint32_t o0 = static_cast<uint32_t>(lo - blo);
    const uint8_t* src = p.ring + static_cast<uint64_t>(slot) * p.slot_bytes + G.staged_off +
                         (static_cast<uint64_t>(t) * C + q0) * r;
    if (G.kind == BSR_KIND_CONTIG) {
      const uint32_t seg = m * r;
      const uint32_t off = piece * G.piece_bytes;
      const uint32_t len = off < seg ? ((seg - off) < G.piece_bytes ? (seg - off) : G.piece_bytes) : 0;
      const uint8_t* sp = src + off;
      const uint32_t nvec = len >> 4;
      constexpr uint32_t U = BSR_UNROLL;
      static_assert(kMaxPieceBytes <= U * kPieceAlign, "a contiguous piece must fit one unrolled pass");
      const bool one_pass = ((reinterpret_cast<uintptr_t>(sp) | len) & 15u) == 0;
      u32x4 v[U];
      if (one_pass) {
#pragma unroll
        for (uint32_t u = 0; u < U; ++u) {
          const uint32_t i = u * kInstallThreads + tid;
          if (i < nvec) v[u] = ld_stream(reinterpret_cast<const u32x4*>(sp) + i);
        }
      }
      // Wave-level prefix check: a failure recorded by an earlier chunk (or an
      // invalid group) puts this chunk past the valid prefix; every wave
      // ballots the same words, so the whole workgroup agrees.
      const bool skip = __ballot(bad) != 0ull;
      if (!skip && b >= 0 && static_cast<uint32_t>(b) < G.pool_blocks && len) {
        uint8_t* dp = tbase + static_cast<uint64_t>(b) * B * r + static_cast<uint64_t>(o0) * r + off;
        if (one_pass && (reinterpret_cast<uintptr_t>(dp) & 15u) == 0) {
          u32x4* d4 = reinterpret_cast<u32x4*>(dp);
#pragma unroll
          for (uint32_t u = 0; u < U; ++u) {
            const uint32_t i = u * kInstallThreads + tid;
            if (i < nvec) {
              fold(v[u], s, x);
              st_stream(v[u], d4 + i);
            }
          }
        } else {
          copy_words(sp, dp, len, tid, s, x);
        }
      }
    } else {
      const uint32_t sp = G.split_bytes;
      const uint32_t u0 = piece * G.piece_tokens;
      const uint32_t mu = u0 < m ? ((m - u0) < G.piece_tokens ? (m - u0) : G.piece_tokens) : 0;
      const uint8_t* psrc = src + static_cast<uint64_t>(u0) * r;
      const uint32_t bytes = mu * r;
      const uint32_t nvec = bytes >> 4;
      const bool src_ok = ((reinterpret_cast<uintptr_t>(psrc) | bytes | sp) & 15u) == 0 && bytes <= p.lds_bytes;
      u32x4 v[kPlanarVecs];
      if (src_ok) {
#pragma unroll
        for (uint32_t u = 0; u < kPlanarVecs; ++u) {
          const uint32_t i = u * kInstallThreads + tid;
          if (i < nvec) v[u] = ld_stream(reinterpret_cast<const u32x4*>(psrc) + i);
        }
      }
      const bool skip = __ballot(bad) != 0ull;
      if (!skip && b >= 0 && static_cast<uint32_t>(b) < G.pool_blocks && mu) {
        uint8_t* blk = tbase + static_cast<uint64_t>(b) * B * r;
        uint8_t* dst1 = blk + static_cast<uint64_t>(o0 + u0) * sp;
        uint8_t* dst2 = blk + B * sp + static_cast<uint64_t>(o0 + u0) * (r - sp);
        if (src_ok && ((reinterpret_cast<uintptr_t>(dst1) & 15u) | (reinterpret_cast<uintptr_t>(dst2) & 3u)) == 0)
          planar_from_regs(v, nvec, dst1, dst2, mu, r, sp, lds, tid, s, x);
        else
          planar_words(psrc, dst1, dst2, mu, r, sp, tid, s, x);
      }
    }
  }

  // one tag partial per wave
  s = wave_sum(s);
  x = wave_xor(x);
  if (lane == 0) p.partials[wg * kInstallWaves + (tid >> 6)] = TagPair{s, x};
}

// One workgroup per (chunk, group) of the launch reduces that entry's wave
// partials and compares with the stored tag; the last workgroup to finish
// applies the first mismatching chunk, in chunk order, to the status words
// and leaves the shared words zeroed for the next launch.
__global__ __launch_bounds__(256) void k_verify(const VerifyParams p) {
  __shared__ uint32_t red_s[4], red_x[4];
  __shared__ uint32_t is_last;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t pair = blockIdx.x;
  const uint32_t c = pair / p.n_groups, g = pair - c * p.n_groups;
  const bool live = p.status->fail == 0;
  uint32_t s = 0, x = 0;
  if (live) {
    const uint32_t lo = (c * p.wg_per_chunk + p.wg_start[g]) * kInstallWaves;
    const uint32_t hi = (c * p.wg_per_chunk + p.wg_start[g + 1]) * kInstallWaves;
    for (uint32_t i = lo + tid; i < hi; i += 256) {
      const TagPair tp = p.partials[i];
      s += tp.sum;
      x ^= tp.x;
    }
  }
  s = wave_sum(s);
  x = wave_xor(x);
  if (lane == 0) {
    red_s[wave] = s;
    red_x[wave] = x;
  }
  __syncthreads();
  if (tid == 0) {
    if (live) {
      const uint32_t ts = (red_s[0] + red_s[1]) + (red_s[2] + red_s[3]);
      const uint32_t tx = (red_x[0] ^ red_x[1]) ^ (red_x[2] ^ red_x[3]);
      const uint64_t tag = (static_cast<uint64_t>(tx) << 32) | ts;
      if (tag != p.expected[c][g]) atomicOr(&p.aux->bad[c], 1u << g);
    }
    __threadfence();
    is_last = atomicAdd(&p.aux->arrivals, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (is_last && tid == 0) {
    __threadfence();
    bool applied = !live;
    for (uint32_t cc = 0; cc < p.n_chunks; ++cc) {
      const uint32_t m = atomicExch(&p.aux->bad[cc], 0u);
      if (m && !applied) {
        p.status->fail = BSR_FAIL_CORRUPT;
        p.status->first_failed_chunk = p.first_chunk + cc;
        for (uint32_t gg = 0; gg < p.n_groups; ++gg)
          if ((m >> gg) & 1u) p.status->q[gg] = 0;
        applied = true;
      }
    }
    atomicExch(&p.aux->arrivals, 0u);
  }
}

__global__ __launch_bounds__(256) void k_finish(const FinishParams p) {
  const uint32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
  bsr_dev_status* st = p.status;
  uint8_t value = 0;
  if (p.mode == kFinishMarkGroup) {
    if (gid == 0) st->q[p.group_mask] = 0;
    return;
  }
  if (p.mode == kFinishCheckTables) {
    // runs after begin, before any install: an advertised block id outside
    // its pool fails the request (the installs and commit never write it)
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t idx = gid; idx < p.total_blocks; idx += stride) {
      uint32_t g = 0, k = idx;
      while (g + 1 < p.n_groups && k >= p.g[g].n_req_blocks) {
        k -= p.g[g].n_req_blocks;
        ++g;
      }
      const int32_t b = p.g[g].block_table[k];
      if (b < 0 || static_cast<uint32_t>(b) >= p.g[g].pool_blocks) {
        atomicCAS(&st->fail, static_cast<uint32_t>(BSR_FAIL_NONE), static_cast<uint32_t>(BSR_FAIL_BLOCK_TABLE));
        atomicMin(&st->first_failed_chunk,
                  static_cast<uint32_t>(static_cast<uint64_t>(k) * p.g[g].block_tokens / p.chunk_tokens));
        st->q[g] = 0;
      }
    }
    return;
  }
  if (p.mode == kFinishBegin) {
    if (gid == 0) {
      st->fail = BSR_FAIL_NONE;
      st->first_failed_chunk = BSR_NO_CHUNK;
      for (int g = 0; g < BSR_MAX_GROUPS; ++g) st->q[g] = 1;
      st->exposed_tokens = 0;
      st->fallback = 0;
      st->phase = 1;
      st->reserved[0] = st->reserved[1] = 0;
      for (int i = 0; i < BSR_MAX_INSTALL_BATCH; ++i) p.verify_aux->bad[i] = 0;
      p.verify_aux->arrivals = 0;
    }
    value = 0;
  } else if (p.mode == kFinishCommit) {
    bool Q = st->fail == BSR_FAIL_NONE;
    for (uint32_t g = 0; g < p.n_groups; ++g) Q = Q && st->q[g] != 0;
    value = Q ? 1 : 0;
    if (gid == 0) {
      st->exposed_tokens = Q ? p.exposed_if_valid : 0;
      st->fallback = Q ? 0 : 1;
      st->phase = 2;
    }
  } else {  // invalidate
    if (gid == 0) {
      if (st->fail == BSR_FAIL_NONE) {
        st->fail = p.reason;
        st->first_failed_chunk = p.chunk;
        for (uint32_t g = 0; g < p.n_groups; ++g)
          if ((p.group_mask >> g) & 1u) st->q[g] = 0;
      }
      st->exposed_tokens = 0;
      st->fallback = 1;
      st->phase = 3;
    }
    value = 0;
  }
  const uint32_t stride = gridDim.x * blockDim.x;
  for (uint32_t idx = gid; idx < p.total_blocks; idx += stride) {
    uint32_t g = 0, k = idx;
    while (g + 1 < p.n_groups && k >= p.g[g].n_req_blocks) {
      k -= p.g[g].n_req_blocks;
      ++g;
    }
    const int32_t b = p.g[g].block_table[k];
    if (b >= 0 && static_cast<uint32_t>(b) < p.g[g].pool_blocks) p.g[g].valid[b] = value;
  }
}

hipError_t launch_install(const InstallParams& p, uint32_t n_workgroups, hipStream_t s, hipEvent_t start,
                          hipEvent_t stop) {
  if (start && stop) {
    // the events are stamped by the kernel's own dispatch (no marker packets)
    hipExtLaunchKernelGGL(k_install, dim3(n_workgroups), dim3(kInstallThreads), p.lds_bytes, s, start, stop, 0, p);
  } else {
    hipLaunchKernelGGL(k_install, dim3(n_workgroups), dim3(kInstallThreads), p.lds_bytes, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_verify(const VerifyParams& p, hipStream_t s) {
  hipLaunchKernelGGL(k_verify, dim3(p.n_chunks * p.n_groups), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_finish(const FinishParams& p, hipStream_t s) {
  uint32_t grid = (p.total_blocks + 255) / 256;
  if (grid == 0) grid = 1;
  if (grid > 1024) grid = 1024;
  hipLaunchKernelGGL(k_finish, dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace bsr
