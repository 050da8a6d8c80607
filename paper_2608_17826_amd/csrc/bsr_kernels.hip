// gfx950 kernels of the bounded-window restore.
//
// install : scatter staged chunks from the W-slot ring into every group's
//           paged blocks (§3 "Install locally"; §4 windowed retrieve,
//           "performs H2D installation" of the staged window).  One
//           workgroup per piece of a (tensor, destination block) segment.
//           Contiguous groups move 16-byte vectors ring -> pool; planar groups
//           (records split into a values plane and a scales plane inside a
//           block) stage the piece in LDS and write both planes with
//           coalesced stores.  Every workgroup also folds the words it read
//           into a (sum, xor) tag partial, and wave 0 ballots the request's
//           status words first, so no workgroup installs past a failure.
// verify  : reduce the partials of each (chunk, group) and compare with the
//           tag recorded at store time; the first mismatching chunk fails
//           the request (q_g = 0 for its mismatching groups).
// finish  : begin (reset status, clear advertised valid bytes), commit
//           (Eq. 6), invalidate (§4 failed-block + HMA-aware invalidation),
//           mark one group invalid.
//
// Nothing here is a dense contraction: the path is bound by HBM bandwidth
// (read the staged chunk once, write the paged blocks once).
#include <hip/hip_runtime.h>

#include "bsr_device.h"

namespace bsr {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
// contiguous segment piece: 16-byte vectors when everything is 16-aligned,
// else 4-byte words (records are multiples of 4 bytes)
// ---------------------------------------------------------------------------
__device__ __forceinline__ void copy_contig(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                            uint32_t len, uint32_t tid, uint32_t& s, uint32_t& x) {
  if (((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | len) & 15u) == 0) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* d4 = reinterpret_cast<u32x4*>(dst);
    const uint32_t nvec = len >> 4;
    constexpr uint32_t U = 4;
    for (uint32_t base = 0; base < nvec; base += U * kInstallThreads) {
      u32x4 v[U];
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const uint32_t i = base + u * kInstallThreads + tid;
        if (i < nvec) v[u] = __builtin_nontemporal_load(s4 + i);
      }
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const uint32_t i = base + u * kInstallThreads + tid;
        if (i < nvec) {
          fold(v[u], s, x);
          __builtin_nontemporal_store(v[u], d4 + i);
        }
      }
    }
  } else {
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
}

// ---------------------------------------------------------------------------
// planar segment piece: mu tokens of AoS records (r bytes each) starting at
// in-block position o.  Plane 1 gets the first sp bytes of each record at
// o*sp, plane 2 the remaining r-sp bytes at B*sp + o*(r-sp).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void copy_planar(const uint8_t* __restrict__ src, uint8_t* __restrict__ blk,
                                            uint32_t o, uint32_t mu, uint32_t r, uint32_t sp, uint32_t B,
                                            uint32_t lds_bytes, uint8_t* lds, uint32_t tid,
                                            uint32_t& s, uint32_t& x) {
  const uint32_t bytes = mu * r;
  uint8_t* dst1 = blk + static_cast<uint64_t>(o) * sp;
  uint8_t* dst2 = blk + static_cast<uint64_t>(B) * sp + static_cast<uint64_t>(o) * (r - sp);
  const bool fast = ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst1) | bytes | sp) & 15u) == 0 &&
                    (reinterpret_cast<uintptr_t>(dst2) & 3u) == 0 && bytes <= lds_bytes;
  if (fast) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* l4 = reinterpret_cast<u32x4*>(lds);
    const uint32_t nvec = bytes >> 4;
    for (uint32_t i = tid; i < nvec; i += kInstallThreads) {
      const u32x4 v = __builtin_nontemporal_load(s4 + i);
      fold(v, s, x);
      l4[i] = v;
    }
    __syncthreads();
    const uint32_t* l1 = reinterpret_cast<const uint32_t*>(lds);
    // plane 1: 16-byte stores; vector v covers token v / (sp/16), part v % (sp/16)
    const uint32_t vpt = sp >> 4;
    const uint32_t n1 = mu * vpt;
    u32x4* d4 = reinterpret_cast<u32x4*>(dst1);
    for (uint32_t i = tid; i < n1; i += kInstallThreads) {
      const uint32_t u = i / vpt;
      const uint32_t part = i - u * vpt;
      const uint32_t w0 = (u * r + part * 16) >> 2;
      u32x4 v;
      v.x = l1[w0];
      v.y = l1[w0 + 1];
      v.z = l1[w0 + 2];
      v.w = l1[w0 + 3];
      __builtin_nontemporal_store(v, d4 + i);
    }
    // plane 2: 4-byte stores
    const uint32_t w2 = (r - sp) >> 2;
    const uint32_t n2 = mu * w2;
    uint32_t* d2 = reinterpret_cast<uint32_t*>(dst2);
    for (uint32_t i = tid; i < n2; i += kInstallThreads) {
      const uint32_t u = i / w2;
      const uint32_t wi = i - u * w2;
      d2[i] = l1[((u * r + sp) >> 2) + wi];
    }
  } else {
    const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
    uint32_t* d1 = reinterpret_cast<uint32_t*>(dst1);
    uint32_t* d2 = reinterpret_cast<uint32_t*>(dst2);
    const uint32_t rw = r >> 2, sw = sp >> 2, nw = bytes >> 2;
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
}

__global__ __launch_bounds__(kInstallThreads) void k_install(const InstallParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ uint32_t red_s[kInstallThreads / 64], red_x[kInstallThreads / 64];
  __shared__ uint32_t skip_sh;

  const uint32_t tid = threadIdx.x;
  const uint32_t wg = blockIdx.x;
  const uint32_t c = wg / p.wg_per_chunk;
  uint32_t rem = wg - c * p.wg_per_chunk;
  uint32_t gi = 0;
  while (gi + 1 < p.n_groups && rem >= p.wg_start[gi + 1]) ++gi;
  rem -= p.wg_start[gi];
  const GroupGeom& G = p.g[gi];

  const uint32_t piece = rem % G.pieces_per_seg;
  rem /= G.pieces_per_seg;
  const uint32_t j = rem % G.segs_per_chunk;
  const uint32_t t = rem / G.segs_per_chunk;

  const uint32_t chunk = p.first_chunk + c;
  const uint32_t slot = chunk % p.window;
  const uint64_t C = p.chunk_tokens, B = G.block_tokens;
  const uint64_t tok0 = static_cast<uint64_t>(chunk) * C;
  const uint64_t k = tok0 / B + j;        // request block index
  const uint64_t blo = k * B;
  const uint64_t lo = tok0 > blo ? tok0 : blo;
  const uint64_t hi = (tok0 + C) < (blo + B) ? (tok0 + C) : (blo + B);

  // Wave-level prefix check: wave 0 ballots the request's status words
  // (fail, then q_g of every group); any failure recorded so far means this
  // chunk lies past the valid prefix, so the workgroup installs nothing.
  if (tid < 64) {
    bool bad = false;
    if (tid == 0)
      bad = p.status->fail != 0;
    else if (tid <= p.n_groups)
      bad = p.status->q[tid - 1] == 0;
    const uint64_t ballot = __ballot(bad);
    if (tid == 0) skip_sh = ballot != 0ull;
  }
  __syncthreads();

  uint32_t s = 0, x = 0;
  int32_t b = -1;
  if (lo < hi && k < G.n_blocks) b = G.block_table[k];
  const bool active = !skip_sh && b >= 0 && static_cast<uint32_t>(b) < G.pool_blocks;
  if (active) {
    const uint32_t r = G.record_bytes;
    const uint32_t m = static_cast<uint32_t>(hi - lo);
    const uint32_t q0 = static_cast<uint32_t>(lo - tok0);
    const uint32_t o0 = static_cast<uint32_t>(lo - blo);
    const uint8_t* src = p.ring + static_cast<uint64_t>(slot) * p.slot_bytes + G.staged_off +
                         (static_cast<uint64_t>(t) * C + q0) * r;
    uint8_t* blk = G.tensor_bases[t] + static_cast<uint64_t>(b) * B * r;
    if (G.kind == BSR_KIND_CONTIG) {
      const uint32_t seg = m * r;
      const uint32_t off = piece * G.piece_bytes;
      if (off < seg) {
        const uint32_t len = (seg - off) < G.piece_bytes ? (seg - off) : G.piece_bytes;
        copy_contig(src + off, blk + static_cast<uint64_t>(o0) * r + off, len, tid, s, x);
      }
    } else {
      const uint32_t u0 = piece * G.piece_tokens;
      if (u0 < m) {
        const uint32_t mu = (m - u0) < G.piece_tokens ? (m - u0) : G.piece_tokens;
        copy_planar(src + static_cast<uint64_t>(u0) * r, blk, o0 + u0, mu, r, G.split_bytes,
                    static_cast<uint32_t>(B), p.lds_bytes, lds, tid, s, x);
      }
    }
  }

  s = wave_sum(s);
  x = wave_xor(x);
  if ((tid & 63) == 0) {
    red_s[tid >> 6] = s;
    red_x[tid >> 6] = x;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t ts = 0, tx = 0;
#pragma unroll
    for (int w = 0; w < kInstallThreads / 64; ++w) {
      ts += red_s[w];
      tx ^= red_x[w];
    }
    p.partials[wg] = TagPair{ts, tx};
  }
}

__global__ __launch_bounds__(256) void k_verify(const VerifyParams p) {
  __shared__ uint32_t bad[BSR_MAX_INSTALL_BATCH];
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < BSR_MAX_INSTALL_BATCH) bad[tid] = 0;
  __syncthreads();
  const bool live = p.status->fail == 0;
  if (live) {
    const uint32_t n_pairs = p.n_chunks * p.n_groups;
    for (uint32_t pr = wave; pr < n_pairs; pr += 4) {
      const uint32_t c = pr / p.n_groups, g = pr - c * p.n_groups;
      const uint32_t lo = c * p.wg_per_chunk + p.wg_start[g];
      const uint32_t hi = c * p.wg_per_chunk + p.wg_start[g + 1];
      uint32_t s = 0, x = 0;
      for (uint32_t i = lo + lane; i < hi; i += 64) {
        const TagPair tp = p.partials[i];
        s += tp.sum;
        x ^= tp.x;
      }
      s = wave_sum(s);
      x = wave_xor(x);
      if (lane == 0) {
        const uint64_t tag = (static_cast<uint64_t>(x) << 32) | s;
        if (tag != p.expected[c][g]) atomicOr(&bad[c], 1u << g);
      }
    }
  }
  __syncthreads();
  if (tid == 0 && live) {
    for (uint32_t c = 0; c < p.n_chunks; ++c) {
      const uint32_t m = bad[c];
      if (m) {
        p.status->fail = BSR_FAIL_CORRUPT;
        p.status->first_failed_chunk = p.first_chunk + c;
        for (uint32_t g = 0; g < p.n_groups; ++g)
          if ((m >> g) & 1u) p.status->q[g] = 0;
        break;
      }
    }
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
  if (p.mode == kFinishBegin) {
    if (gid == 0) {
      st->fail = BSR_FAIL_NONE;
      st->first_failed_chunk = BSR_NO_CHUNK;
      for (int g = 0; g < BSR_MAX_GROUPS; ++g) st->q[g] = 1;
      st->exposed_tokens = 0;
      st->fallback = 0;
      st->phase = 1;
      st->reserved[0] = st->reserved[1] = 0;
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

hipError_t launch_install(const InstallParams& p, uint32_t n_workgroups, hipStream_t s) {
  hipLaunchKernelGGL(k_install, dim3(n_workgroups), dim3(kInstallThreads), p.lds_bytes, s, p);
  return hipGetLastError();
}

hipError_t launch_verify(const VerifyParams& p, hipStream_t s) {
  hipLaunchKernelGGL(k_verify, dim3(1), dim3(256), 0, s, p);
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
