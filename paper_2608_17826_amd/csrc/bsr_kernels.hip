// gfx950 kernels of the bounded-window restore.
//
// stage   : copy a run of staged chunks from pinned host memory into the
//           W-slot ring (§4 windowed retrieve: the window's objects are
//           brought into the local restore pool), read over the host link
//           by a small grid on the copy stream.
// install : scatter staged chunks from the W-slot ring into every group's
//           paged blocks (§3 "Install locally"; §4 windowed retrieve, whose
//           per-window step moves the staged window into the engine's
//           blocks).  One workgroup per piece of a (tensor, destination
//           block) segment; consecutive pieces are issued in runs to one
//           XCD, so a block's pieces share an L2.  A piece's 16-byte data
//           loads and one lane-parallel metadata load (block id, tensor
//           base, the request's status words) share one memory round trip;
//           a ballot over the status lanes is the prefix check, so no
//           workgroup installs past a failure.  Contiguous groups store the
//           vectors straight to the pool; planar groups (records split into
//           a values plane and a scales plane inside a block) stage the
//           piece in LDS and write both planes with coalesced stores.  Every
//           wave folds the words it read into a (sum, xor) tag partial.
// verify  : reduce the partials of each (chunk, group) and compare with the
//           tag recorded at store time; the first mismatching chunk, in
//           chunk order, fails the request (q_g = 0 for its mismatching
//           groups).
// finish  : begin (reset status, clear advertised valid bytes), commit
//           (Eq. 6), invalidate (§4 failed-block + HMA-aware invalidation),
//           mark one group invalid, check the block tables on the device.
//
// Nothing here is a dense contraction.  The staging copy is bound by the
// host link; the install by HBM bandwidth (read the staged chunk once,
// write the paged blocks once).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "bsr_device.h"

#ifndef BSR_UNROLL
#define BSR_UNROLL 4    // 16-byte vectors per thread of a contiguous piece
#endif
#ifndef BSR_NT_LOAD
#define BSR_NT_LOAD 1   // staged chunks are read once: non-temporal loads
#endif
#ifndef BSR_STAGE_NT_STORE
#define BSR_STAGE_NT_STORE 0  // staging-copy stores: 1 non-temporal, 0 ordinary
#endif


namespace bsr {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Ring and pool pointers are rebuilt from argument words and from tensor
// bases read out of device memory, so the compiler cannot tell that they
// point to global memory; every access goes through an explicit global
// pointer (global rather than flat instructions, which would also count
// against the LDS wait counter).
template <typename T>
__device__ __forceinline__ __attribute__((address_space(1))) T* global_ptr(T* p) {
  return (__attribute__((address_space(1))) T*)(p);
}

// Stores of a piece through a buffer resource whose base is the piece's
// (wave-uniform) destination and whose size is the piece's length: the
// hardware drops any store at or past that length.  kStoreAux is the cache
// policy (bit 0 sc0, bit 1 nt, bit 4 sc1): non-temporal at device scope
// (nt sc1).  Measured on the install: nt alone 68.6%, nt sc0 68.5%, nt sc1
// 69.6%, nt sc0 sc1 69.6% of 8 TB/s; the paged blocks are not read again
// by this path, and device scope is all that the later kernels and the
// host's synchronised reads need.
#ifndef BSR_STORE_AUX
#define BSR_STORE_AUX 18
#endif
constexpr int kStoreAux = BSR_STORE_AUX;
constexpr int kRsrcWord3 = 0x00020000;  // raw 32-bit elements, gfx9-family resource format
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t piece_rsrc(uint8_t* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, static_cast<int>(bytes), kRsrcWord3);
}

__device__ __forceinline__ void st_piece16(u32x4 v, __amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), r, static_cast<int>(byte_off), 0, kStoreAux);
}

__device__ __forceinline__ void st_piece4(uint32_t v, __amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  __builtin_amdgcn_raw_buffer_store_b32(static_cast<int>(v), r, static_cast<int>(byte_off), 0, kStoreAux);
}

// The install's loads are issued explicitly: a piece's data loads, then its
// metadata load, then one wait for all of them, in a single asm statement.
// Left to itself the compiler sinks the data loads below the metadata check
// (into the branch that stores them), which turns one memory round trip into
// two.  Inside one statement the loaded registers are only defined once the
// wait has passed, so no instruction can read them early, and early-clobber
// outputs keep every destination apart from the addresses of later loads.
// One burst shape per per-thread load count the kernel is built with.
#if BSR_NT_LOAD
#define BSR_LDX4(d, a) "global_load_dwordx4 %" #d ", %" #a ", off nt\n\t"
#else
#define BSR_LDX4(d, a) "global_load_dwordx4 %" #d ", %" #a ", off\n\t"
#endif
#define BSR_LD1(d, a) "global_load_dword %" #d ", %" #a ", off\n\t"
#define BSR_WAIT "s_waitcnt vmcnt(0)"

template <int N>
struct LoadBurst;  // N 16-byte stream loads + one metadata word, waited for together

template <>
struct LoadBurst<2> {
  static __device__ __forceinline__ void run(u32x4 (&v)[2], uint32_t& w, const u32x4* const (&a)[2],
                                             const uint32_t* am) {
    asm volatile(BSR_LDX4(0, 3) BSR_LDX4(1, 4) BSR_LD1(2, 5) BSR_WAIT
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(w)
                 : "v"(a[0]), "v"(a[1]), "v"(am)
                 : "memory");
  }
};

template <>
struct LoadBurst<4> {
  static __device__ __forceinline__ void run(u32x4 (&v)[4], uint32_t& w, const u32x4* const (&a)[4],
                                             const uint32_t* am) {
    asm volatile(BSR_LDX4(0, 5) BSR_LDX4(1, 6) BSR_LDX4(2, 7) BSR_LDX4(3, 8) BSR_LD1(4, 9) BSR_WAIT
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(w)
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(am)
                 : "memory");
  }
};

template <>
struct LoadBurst<5> {
  static __device__ __forceinline__ void run(u32x4 (&v)[5], uint32_t& w, const u32x4* const (&a)[5],
                                             const uint32_t* am) {
    asm volatile(BSR_LDX4(0, 6) BSR_LDX4(1, 7) BSR_LDX4(2, 8) BSR_LDX4(3, 9) BSR_LDX4(4, 10) BSR_LD1(5, 11) BSR_WAIT
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(w)
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(am)
                 : "memory");
  }
};

template <>
struct LoadBurst<10> {
  static __device__ __forceinline__ void run(u32x4 (&v)[10], uint32_t& w, const u32x4* const (&a)[10],
                                             const uint32_t* am) {
    asm volatile(BSR_LDX4(0, 11) BSR_LDX4(1, 12) BSR_LDX4(2, 13) BSR_LDX4(3, 14) BSR_LDX4(4, 15)
                 BSR_LDX4(5, 16) BSR_LDX4(6, 17) BSR_LDX4(7, 18) BSR_LDX4(8, 19) BSR_LDX4(9, 20)
                 BSR_LD1(10, 21) BSR_WAIT
                 : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]),
                   "=&v"(v[7]), "=&v"(v[8]), "=&v"(v[9]), "=&v"(w)
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7]),
                   "v"(a[8]), "v"(a[9]), "v"(am)
                 : "memory");
  }
};

__device__ __forceinline__ void fold(const u32x4 v, uint32_t& s, uint32_t& x) {
  s += (v.x + v.y) + (v.z + v.w);
  x ^= (v.x ^ v.y) ^ (v.z ^ v.w);
}

// Wave-wide sum and XOR of a per-lane word, returned as a wave-uniform value.
// Within each 16-lane row, lanes exchange with DPP moves (quad swaps 1 and 2,
// then the mirrored half-row and row), so every lane of a row holds the row's
// total; the four row totals are then read out of lanes 0, 16, 32 and 48.
// No LDS traffic: the tag costs a few VALU cycles per wave.
template <int kCtrl>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), kCtrl, 0xF, 0xF, false));
}
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppRowMirror = 0x140;  // lane i of a row reads lane 15 - i
constexpr int kDppHalfMirror = 0x141; // lane i of a half-row reads lane 7 - i

__device__ __forceinline__ uint32_t row_lane(uint32_t v, int lane) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), lane));
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  v += dpp<kDppQuadSwap1>(v);
  v += dpp<kDppQuadSwap2>(v);
  v += dpp<kDppHalfMirror>(v);
  v += dpp<kDppRowMirror>(v);
  return (row_lane(v, 0) + row_lane(v, 16)) + (row_lane(v, 32) + row_lane(v, 48));
}

__device__ __forceinline__ uint32_t wave_xor(uint32_t v) {
  v ^= dpp<kDppQuadSwap1>(v);
  v ^= dpp<kDppQuadSwap2>(v);
  v ^= dpp<kDppHalfMirror>(v);
  v ^= dpp<kDppRowMirror>(v);
  return (row_lane(v, 0) ^ row_lane(v, 16)) ^ (row_lane(v, 32) ^ row_lane(v, 48));
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
    const uint32_t w = *global_ptr(s1 + i);
    s += w;
    x ^= w;
    *global_ptr(d1 + i) = w;
  }
}

// ---------------------------------------------------------------------------
// planar segment piece: mu tokens of AoS records (r bytes each) starting at
// in-block position o.  Plane 1 gets the first sp bytes of each record at
// o*sp, plane 2 the remaining r-sp bytes at B*sp + o*(r-sp).
// ---------------------------------------------------------------------------
constexpr uint32_t kPlanarVecs = (kLdsCapBytes + kPieceAlign - 1) / kPieceAlign;  // vectors per thread
static_assert(kPlanarVecs * kPieceAlign >= kLdsCapBytes, "a planar piece of kLdsCapBytes fits the registers");

// Fast path, second half: the piece's words are in registers (v); stage them
// in LDS, then write plane 1 with 16-byte stores and plane 2 with 4-byte
// stores.  Plane 1 has fewer vectors than the piece (split < record), so it
// fits the same per-thread count: every thread reads all its plane-1 vectors
// out of LDS at once (indices clamped to the last, no per-lane branch) and
// waits once, instead of once per vector.  d1/d2 are the divisions by the
// plane-1 vectors and plane-2 words per token.
__device__ __forceinline__ void planar_from_regs(const u32x4 (&v)[kPlanarVecs], uint32_t nvec, uint8_t* dst1,
                                                 uint8_t* dst2, uint32_t mu, uint32_t r, uint32_t sp,
                                                 const PackedDiv d1, const PackedDiv d2, uint8_t* lds,
                                                 uint32_t tid, uint32_t& s, uint32_t& x) {
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
  // plane 1: vector i covers token i / vpt, part i % vpt
  const uint32_t vpt = sp >> 4;
  const uint32_t n1 = mu * vpt;  // n1 * 16 < mu * r <= kLdsCapBytes: at most kPlanarVecs per thread
  u32x4 w[kPlanarVecs];
#pragma unroll
  for (uint32_t u = 0; u < kPlanarVecs; ++u) {
    const uint32_t i0 = u * kInstallThreads + tid;
    const uint32_t i = i0 < n1 ? i0 : n1 - 1;
    const uint32_t tk = packed_div(d1.m, d1.s, i);
    const uint32_t w0 = (tk * r + (i - tk * vpt) * 16) >> 2;
    w[u].x = l1[w0];
    w[u].y = l1[w0 + 1];
    w[u].z = l1[w0 + 2];
    w[u].w = l1[w0 + 3];
  }
  const __amdgpu_buffer_rsrc_t r1 = piece_rsrc(dst1, n1 * 16u);
#pragma unroll
  for (uint32_t u = 0; u < kPlanarVecs; ++u) {
    const uint32_t i = u * kInstallThreads + tid;
    if (i < n1) st_piece16(w[u], r1, i * 16u);
  }
  const uint32_t w2 = (r - sp) >> 2;
  const uint32_t n2 = mu * w2;
  const __amdgpu_buffer_rsrc_t r2 = piece_rsrc(dst2, n2 * 4u);
  for (uint32_t i = tid; i < n2; i += kInstallThreads) {
    const uint32_t tk = packed_div(d2.m, d2.s, i);
    st_piece4(l1[((tk * r + sp) >> 2) + (i - tk * w2)], r2, i * 4u);
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
    const uint32_t w = *global_ptr(s1 + i);
    s += w;
    x ^= w;
    if (wi < sw)
      *global_ptr(d1 + u * sw + wi) = w;
    else
      *global_ptr(d2 + u * (rw - sw) + (wi - sw)) = w;
  }
}

// Destination metadata of one segment and the request's status words,
// fetched by one vector load per wave issued right after the piece's data
// loads: lane 0 reads the destination block id, lanes 1-2 the two halves of
// the tensor base, lane 3 the fail word and lanes 4.. the per-group q_g.  The
// data and the metadata then arrive in one memory round trip, and the values
// are broadcast from their lanes.
struct SegMeta {
  int32_t block;
  uint8_t* tensor_base;
  bool past_prefix;  // a failure is recorded, or some group is invalid
};

__device__ __forceinline__ const uint32_t* meta_addr(const bsr_dev_status* status, const int32_t* block_table,
                                                     uint8_t* const* tensor_bases, uint32_t k, uint32_t t,
                                                     uint32_t lane) {
  const uint32_t* st = reinterpret_cast<const uint32_t*>(status);
  const uint32_t* a = st;  // lane 3 and every lane past the q words: the fail word
  if (lane == 0) a = reinterpret_cast<const uint32_t*>(block_table + k);
  if (lane == 1 || lane == 2) a = reinterpret_cast<const uint32_t*>(tensor_bases + t) + (lane - 1);
  if (lane >= 4 && lane < 4 + BSR_MAX_GROUPS) a = st + 2 + (lane - 4);  // q[lane - 4]
  return a;
}

__device__ __forceinline__ SegMeta broadcast_meta(uint32_t w, uint32_t lane, uint32_t n_groups) {
  SegMeta m;
  m.block = static_cast<int32_t>(row_lane(w, 0));
  // both halves widened from uint32_t: the builtin returns int, and a
  // widened int would sign-extend a low half whose bit 31 is set
  const uint64_t lo = row_lane(w, 1), hi = row_lane(w, 2);
  m.tensor_base = reinterpret_cast<uint8_t*>(lo | (hi << 32));
  // Prefix check: a failure recorded by an earlier chunk, or an invalid
  // group, puts this chunk past the valid prefix.  Nothing writes the status
  // words while installs run, so every wave sees the same values and the
  // whole workgroup agrees.
  const bool bad = (lane == 3 && w != 0) || (lane >= 4 && lane < 4 + n_groups && w == 0);
  m.past_prefix = __ballot(bad) != 0ull;
  return m;
}

// 128 bytes of kernel arguments as two 64-byte vectors: each becomes one
// scalar load, and both are issued before either is waited for.
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
template <typename T>
union ArgWords {
  u32x16 v[2];
  T s;
};

template <typename T>
__device__ __forceinline__ T load_args(const T* src) {
  static_assert(sizeof(T) == sizeof(u32x16) * 2, "argument blocks are 128 bytes");
  ArgWords<T> w;
  const u32x16* v = reinterpret_cast<const u32x16*>(src);
  w.v[0] = v[0];
  w.v[1] = v[1];
  return w.s;
}

// acc + (a >= b) for wave-uniform a, b: a scalar compare and an add of its
// carry.  (Written as C, the comparison becomes a lane mask that is turned
// back into an integer through a vector register, several instructions and
// a vector-to-scalar transfer per comparison.)
__device__ __forceinline__ uint32_t add_if_ge(uint32_t acc, uint32_t a, uint32_t b) {
  asm("s_cmp_ge_u32 %1, %2\n\ts_addc_u32 %0, %0, 0" : "+s"(acc) : "s"(a), "s"(b) : "scc");
  return acc;
}

__global__ __launch_bounds__(kInstallThreads) void k_install(const InstallParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  const uint32_t tid = threadIdx.x;
  const uint32_t lane = tid & 63;
  const InstallHead H = load_args(&p.h);
  // work index -> dispatch position (the group), then (chunk, piece within
  // the chunk's group range)
  const uint32_t bid = xcd_work_index(blockIdx.x, H.xcd_full, H.xcd_log2);
  // Every wave runs this decode before its first data load, and that delay
  // costs bandwidth, so it is kept short: about 120 scalar instructions
  // (256 extra ones per wave cost a plain copy of this shape about 3 points
  // of HBM bandwidth, 128 about 0.3).  The dispatch position is the count
  // of group starts at or below bid (the starts increase with the
  // position).
  uint32_t oi = 0;
#pragma unroll
  for (uint32_t q = 1; q < BSR_MAX_GROUPS; ++q) oi = add_if_ge(oi, bid, H.start[q]);
  const InstallGroup G = load_args(&p.g[oi]);
  uint32_t rem = bid - H.n_chunks * G.prefix;
  const uint32_t cf = packed_div(G.div_per_chunk.m, G.div_per_chunk.s, rem);
  rem -= cf * G.per_chunk;
  const uint32_t c = (oi & H.serpentine) ? H.n_chunks - 1 - cf : cf;  // launch-relative chunk
  const uint32_t wg = c * H.wg_per_chunk + G.wg_start + rem;  // chunk-major slot of the tag partials

  const uint32_t r1 = packed_div(G.div_pieces.m, G.div_pieces.s, rem);
  const uint32_t piece = rem - r1 * G.pieces_per_seg;
  const uint32_t t = packed_div(G.div_segs.m, G.div_segs.s, r1);
  const uint32_t j = r1 - t * G.segs_per_chunk;

  const uint32_t chunk = H.first_chunk + c;
  const uint32_t slot0 = H.first_slot + c;  // c < n_chunks <= W
  const uint32_t slot = slot0 >= H.window ? slot0 - H.window : slot0;
  // Token positions in 32 bits: the bound prefix plus two blocks stays
  // below 2^32 tokens (checked when the request is bound).
  const uint32_t C = H.chunk_tokens, B = G.block_tokens;
  const uint32_t tok0 = chunk * C;
  const uint32_t k = packed_div(G.div_block.m, G.div_block.s, tok0) + j;  // request block index
  const uint32_t blo = k * B;
  const uint32_t lo = tok0 > blo ? tok0 : blo;
  const uint32_t hi = (tok0 + C) < (blo + B) ? (tok0 + C) : (blo + B);

  uint32_t s = 0, x = 0;
  if (lo < hi && k < G.n_blocks) {
    const uint32_t r = G.record_bytes;
    const uint32_t m = hi - lo;
    const uint32_t q0 = lo - tok0;
    const uint32_t o0 = lo - blo;
    // offsets inside a slot and inside a block fit 32 bits (slot < 4 GiB,
    // block < 2 GiB)
    const uint8_t* src = H.ring + static_cast<uint64_t>(slot) * H.slot_bytes + (G.staged_off + (t * C + q0) * r);
    if (G.kind == BSR_KIND_CONTIG) {
      const uint32_t seg = m * r;
      const uint32_t off = piece * G.piece;
      const uint32_t len = off < seg ? ((seg - off) < G.piece ? (seg - off) : G.piece) : 0;
      const uint8_t* sp = src + off;
      const uint32_t nvec = len >> 4;
      constexpr uint32_t U = BSR_UNROLL;
      static_assert(kMaxPieceBytes <= U * kPieceAlign, "a contiguous piece must fit one unrolled pass");
      const bool one_pass = ((reinterpret_cast<uintptr_t>(sp) | len) & 15u) == 0 && nvec != 0;
      // Every lane loads, with no branch around the loads (a branch would
      // make the compiler wait for them where its paths join, before the
      // metadata load is issued): lanes past the piece's end reload its last
      // vector, and a piece that takes the word path loads the ring's first
      // vector instead, a valid aligned address whose value is not used.
      const u32x4* s4 = reinterpret_cast<const u32x4*>(one_pass ? sp : H.ring);
      const uint32_t last = one_pass ? nvec - 1 : 0;
      const u32x4* at[U];
#pragma unroll
      for (uint32_t u = 0; u < U; ++u) {
        const uint32_t i = u * kInstallThreads + tid;
        at[u] = s4 + (i < last ? i : last);
      }
      u32x4 v[U];
      uint32_t mw;
      LoadBurst<U>::run(v, mw, at, meta_addr(H.status, G.block_table, G.tensor_bases, k, t, lane));
      const SegMeta md = broadcast_meta(mw, lane, H.n_groups);
      if (!md.past_prefix && md.block >= 0 && static_cast<uint32_t>(md.block) < G.pool_blocks && len) {
        uint8_t* dp = md.tensor_base + static_cast<uint64_t>(md.block) * G.block_bytes + (o0 * r + off);
        if (one_pass && (reinterpret_cast<uintptr_t>(dp) & 15u) == 0) {
          const __amdgpu_buffer_rsrc_t rs = piece_rsrc(dp, len);
#pragma unroll
          for (uint32_t u = 0; u < U; ++u) {
            const uint32_t i = u * kInstallThreads + tid;
            if (i < nvec) {
              fold(v[u], s, x);
              st_piece16(v[u], rs, i * 16u);
            }
          }
        } else {
          copy_words(sp, dp, len, tid, s, x);
        }
      }
    } else {
      const uint32_t sp = G.split_bytes;
      const uint32_t u0 = piece * G.piece;
      const uint32_t mu = u0 < m ? ((m - u0) < G.piece ? (m - u0) : G.piece) : 0;
      const uint8_t* psrc = src + u0 * r;
      const uint32_t bytes = mu * r;
      const uint32_t nvec = bytes >> 4;
      const bool src_ok =
          ((reinterpret_cast<uintptr_t>(psrc) | bytes | sp) & 15u) == 0 && bytes <= kLdsCapBytes &&
          bytes <= H.lds_bytes && nvec != 0;  // the piece fits the registers (v) and the LDS
      // unconditional loads, as for contiguous pieces
      const u32x4* s4 = reinterpret_cast<const u32x4*>(src_ok ? psrc : H.ring);
      const uint32_t last = src_ok ? nvec - 1 : 0;
      const u32x4* at[kPlanarVecs];
#pragma unroll
      for (uint32_t u = 0; u < kPlanarVecs; ++u) {
        const uint32_t i = u * kInstallThreads + tid;
        at[u] = s4 + (i < last ? i : last);
      }
      u32x4 v[kPlanarVecs];
      uint32_t mw;
      LoadBurst<kPlanarVecs>::run(v, mw, at, meta_addr(H.status, G.block_table, G.tensor_bases, k, t, lane));
      const SegMeta md = broadcast_meta(mw, lane, H.n_groups);
      if (!md.past_prefix && md.block >= 0 && static_cast<uint32_t>(md.block) < G.pool_blocks && mu) {
        uint8_t* blk = md.tensor_base + static_cast<uint64_t>(md.block) * G.block_bytes;
        uint8_t* dst1 = blk + (o0 + u0) * sp;
        uint8_t* dst2 = blk + (B * sp + (o0 + u0) * (r - sp));
        if (src_ok && ((reinterpret_cast<uintptr_t>(dst1) & 15u) | (reinterpret_cast<uintptr_t>(dst2) & 3u)) == 0)
          planar_from_regs(v, nvec, dst1, dst2, mu, r, sp, G.div_p1, G.div_p2, lds, tid, s, x);
        else
          planar_words(psrc, dst1, dst2, mu, r, sp, tid, s, x);
      }
    }
  }

  // one tag partial per wave
  s = wave_sum(s);
  x = wave_xor(x);
  // TagPair {sum, xor} as one little-endian 8-byte word
  static_assert(sizeof(TagPair) == 8 && offsetof(TagPair, x) == 4, "sum in the low word");
  if (lane == 0)
    *global_ptr(reinterpret_cast<uint64_t*>(H.partials) + wg * kInstallWaves + (tid >> 6)) =
        static_cast<uint64_t>(s) | (static_cast<uint64_t>(x) << 32);
}

// One workgroup per (chunk, group) of the launch reduces that entry's wave
// partials and compares with the stored tag; the last workgroup to finish
// applies the first mismatching chunk, in chunk order, to the status words
// and leaves the shared words zeroed for the next launch.  Both halves are
// latency-bound, so each keeps its memory accesses in flight together: a
// thread loads up to kVerifyUnroll partials before adding any, and the last
// workgroup takes every chunk's mismatch word in one exchange per lane.
constexpr uint32_t kVerifyThreads = 256;
constexpr uint32_t kVerifyUnroll = 8;
static_assert(BSR_MAX_INSTALL_BATCH <= 64, "one lane of the first wave per chunk of a launch");

__global__ __launch_bounds__(kVerifyThreads) void k_verify(const VerifyParams p) {
  __shared__ uint32_t red_s[4], red_x[4];
  __shared__ uint32_t is_last;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t pair = blockIdx.x;
  const uint32_t c = pair / p.n_groups, g = pair - c * p.n_groups;
  // The install's own prefix test: with a failure recorded or some group
  // already invalid (q_g = 0, e.g. reported by the engine between windows),
  // the launch's chunks are past the valid prefix and installed nothing, so
  // their partials are not compared (an empty partial is no corruption).
  // Nothing writes the status words between an install and its verify.
  bool live = p.status->fail == 0;
  for (uint32_t gg = 0; gg < p.n_groups; ++gg) live = live && p.status->q[gg] != 0;
  uint32_t s = 0, x = 0;
  if (live) {
    const uint32_t lo = (c * p.wg_per_chunk + p.wg_start[g]) * kInstallWaves;
    const uint32_t hi = (c * p.wg_per_chunk + p.wg_start[g + 1]) * kInstallWaves;
    for (uint32_t i0 = lo + tid; i0 < hi; i0 += kVerifyThreads * kVerifyUnroll) {
      TagPair tp[kVerifyUnroll];
#pragma unroll
      for (uint32_t u = 0; u < kVerifyUnroll; ++u) {
        const uint32_t i = i0 + u * kVerifyThreads;
        tp[u] = i < hi ? p.partials[i] : TagPair{0u, 0u};
      }
#pragma unroll
      for (uint32_t u = 0; u < kVerifyUnroll; ++u) {
        s += tp[u].sum;
        x ^= tp[u].x;
      }
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
  if (is_last && wave == 0) {
    __threadfence();
    // lane cc takes chunk cc's mismatch mask and leaves the word zeroed
    const uint32_t m = lane < p.n_chunks ? atomicExch(&p.aux->bad[lane], 0u) : 0u;
    const uint64_t any = __ballot(m != 0u);
    // the first mismatching chunk in chunk order fails the request, unless a
    // failure was recorded before this launch
    if (live && any != 0ull && lane == static_cast<uint32_t>(__builtin_ctzll(any))) {
      p.status->fail = BSR_FAIL_CORRUPT;
      p.status->first_failed_chunk = p.first_chunk + lane;
      for (uint32_t gg = 0; gg < p.n_groups; ++gg)
        if ((m >> gg) & 1u) p.status->q[gg] = 0;
    }
    if (lane == 0) atomicExch(&p.aux->arrivals, 0u);
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

// Staging copy: pinned host memory (the device's view of it) into a ring
// slot, read over the host link by a small grid (kStageMaxGrid workgroups,
// kStageUnroll 16-byte loads in flight per thread before its stores).  The
// stores are ordinary: the install reads the slot next, and non-temporal
// stores made overlapping installs slower (16 x 4 at W = 32: 167 against
// 155 us per launch).  Compared with the copy engine (hipMemcpyAsync), a
// kernel's completion hands over to the install on the compute stream
// sooner, which is most of what a small window lost per window.
__global__ __launch_bounds__(kStageThreads) void k_stage(const StageParams p) {
  const u32x4* __restrict__ s4 = reinterpret_cast<const u32x4*>(p.src);
  u32x4* __restrict__ d4 = reinterpret_cast<u32x4*>(p.dst);
  const uint64_t nvec = p.bytes >> 4;
  const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kStageThreads;
  for (uint64_t base = static_cast<uint64_t>(blockIdx.x) * kStageThreads + threadIdx.x; base < nvec;
       base += stride * kStageUnroll) {
    u32x4 v[kStageUnroll];
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const uint64_t i = base + u * stride;
      if (i < nvec) v[u] = *global_ptr(s4 + i);
    }
#pragma unroll
    for (int u = 0; u < kStageUnroll; ++u) {
      const uint64_t i = base + u * stride;
#if BSR_STAGE_NT_STORE
      if (i < nvec) __builtin_nontemporal_store(v[u], global_ptr(d4 + i));
#else
      if (i < nvec) *global_ptr(d4 + i) = v[u];
#endif
    }
  }
  // a tail of up to three words
  const uint64_t w0 = nvec * 4, nw = p.bytes >> 2;
  if (blockIdx.x == 0 && w0 + threadIdx.x < nw)
    *global_ptr(reinterpret_cast<uint32_t*>(p.dst) + w0 + threadIdx.x) =
        *global_ptr(reinterpret_cast<const uint32_t*>(p.src) + w0 + threadIdx.x);
}

// Plain scattered block copy (the install's ceiling, see ScatterParams):
// one workgroup per piece of a block, every thread four 16-byte vectors.
// The piece's data loads and the destination block id share one memory
// round trip (the install's load burst), and the stores are the install's
// (non-temporal, device scope, through a buffer resource).
__global__ __launch_bounds__(kInstallThreads) void k_scatter(const ScatterParams p) {
  const uint32_t tid = threadIdx.x;
  const uint32_t w = xcd_work_index(blockIdx.x, p.xcd_full, p.xcd_log2);
  const uint32_t blk = w / p.pieces_per_block, piece = w - blk * p.pieces_per_block;
  if (blk >= p.n_blocks) return;
  const uint32_t off = piece * p.piece_bytes;
  const uint32_t len = (p.block_bytes - off) < p.piece_bytes ? (p.block_bytes - off) : p.piece_bytes;
  const u32x4* s4 = reinterpret_cast<const u32x4*>(p.src + static_cast<uint64_t>(blk) * p.block_bytes + off);
  const uint32_t nvec = len >> 4;  // >= 1: len is a positive multiple of 16
  constexpr uint32_t U = BSR_UNROLL;
  const u32x4* at[U];
#pragma unroll
  for (uint32_t u = 0; u < U; ++u) {
    const uint32_t i = u * kInstallThreads + tid;
    at[u] = s4 + (i < nvec - 1 ? i : nvec - 1);
  }
  u32x4 v[U];
  uint32_t mw;
  LoadBurst<U>::run(v, mw, at, reinterpret_cast<const uint32_t*>(p.dst_block + blk));
  const int32_t b = static_cast<int32_t>(row_lane(mw, 0));
  uint8_t* dst = p.pool + static_cast<uint64_t>(b) * p.block_bytes + off;
  const __amdgpu_buffer_rsrc_t rs = piece_rsrc(dst, len);
#pragma unroll
  for (uint32_t u = 0; u < U; ++u) {
    const uint32_t i = u * kInstallThreads + tid;
    if (i < nvec) st_piece16(v[u], rs, i * 16u);
  }
}

hipError_t launch_scatter(const ScatterParams& p, hipStream_t s) {
  if (p.xcd_log2 > 5 || p.pieces_per_block == 0 || p.piece_bytes > kMaxPieceBytes || p.piece_bytes % kPieceAlign ||
      p.block_bytes % 16 || static_cast<uint64_t>(p.pieces_per_block) * p.piece_bytes < p.block_bytes)
    return hipErrorInvalidValue;
  const uint64_t grid = static_cast<uint64_t>(p.n_blocks) * p.pieces_per_block;
  if (grid == 0 || grid >= (1ull << 31) || p.xcd_full != xcd_remap_bound(static_cast<uint32_t>(grid), p.xcd_log2))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_scatter, dim3(static_cast<uint32_t>(grid)), dim3(kInstallThreads), p.lds_bytes, s, p);
  return hipGetLastError();
}

// The static scratch.  In host code `scratch` names a host-side stand-in,
// not device memory: only the address from hipGetSymbolAddress, taken per
// device with that device current, is ever passed to a kernel or a copy.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
bool g_scratch_claimed[kMaxScratchDevices] = {};
}  // namespace

hipError_t static_scratch_claim(int device, void** ptr, bool* busy) {
  *ptr = nullptr;
  *busy = false;
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_claimed[device]) {
    *busy = true;
    return hipSuccess;
  }
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
  }
  g_scratch_claimed[device] = true;
  *ptr = g_scratch_ptr[device];
  return hipSuccess;
}

void static_scratch_release(int device) {
  if (device < 0 || device >= kMaxScratchDevices) return;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  g_scratch_claimed[device] = false;
}

hipError_t launch_install(const InstallParams& p, uint32_t n_workgroups, hipStream_t s, hipEvent_t start,
                          hipEvent_t stop) {
  // the XCD remap is a permutation of the grid only for whole spans inside it
  if (p.h.xcd_log2 > 5 || p.h.xcd_full != xcd_remap_bound(n_workgroups, p.h.xcd_log2)) return hipErrorInvalidValue;
  if (start && stop) {
    // the events are stamped by the kernel's own dispatch (no marker packets)
    hipExtLaunchKernelGGL(k_install, dim3(n_workgroups), dim3(kInstallThreads), p.h.lds_bytes, s, start, stop, 0, p);
  } else {
    hipLaunchKernelGGL(k_install, dim3(n_workgroups), dim3(kInstallThreads), p.h.lds_bytes, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_stage(const StageParams& p, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  if (((reinterpret_cast<uintptr_t>(p.src) | reinterpret_cast<uintptr_t>(p.dst)) & 15u) || (p.bytes & 3u))
    return hipErrorInvalidValue;
  if (p.bytes == 0) return hipSuccess;
  const uint64_t per_wg = static_cast<uint64_t>(kStageThreads) * kStageUnroll * 16;
  const uint32_t grid = static_cast<uint32_t>(std::min<uint64_t>(kStageMaxGrid, (p.bytes + per_wg - 1) / per_wg));
  if (start && stop)
    hipExtLaunchKernelGGL(k_stage, dim3(grid), dim3(kStageThreads), 0, s, start, stop, 0, p);
  else
    hipLaunchKernelGGL(k_stage, dim3(grid), dim3(kStageThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_verify(const VerifyParams& p, hipStream_t s) {
  hipLaunchKernelGGL(k_verify, dim3(p.n_chunks * p.n_groups), dim3(kVerifyThreads), 0, s, p);
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
