// A torch-free restore through the C ABI: HIP runtime calls for memory and
// streams, include/bsr.h for everything else.  Two groups with one block per
// chunk (a contiguous group of two 1,152-byte-record tensors and a planar
// group of 132-byte records split 128 + 4), 43 chunks stored in bulk,
// W = 8 (five whole windows and a ragged one of 3, as bsr_next_window plans
// them), a reversed block table.  With block = chunk the expected pool image
// is plain concatenation, checked byte for byte here, together with the
// exposure, the valid bytes, the staging peak and the untouched blocks.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "bsr.h"

#define CHECK(cond)                                                                          \
  do {                                                                                       \
    if (!(cond)) {                                                                           \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, bsr_last_error()); \
      return 1;                                                                              \
    }                                                                                        \
  } while (0)
#define HIP(x) CHECK((x) == hipSuccess)

namespace {

constexpr uint32_t C = 64, N = 43, W = 8, POOL = N + 3;
constexpr uint32_t T0 = 2, R0 = 1152, T1 = 1, R1 = 132, S1 = 128;

uint8_t byte_of(uint32_t chunk, uint32_t group, uint64_t i) {
  uint64_t x = (static_cast<uint64_t>(chunk) << 40) ^ (static_cast<uint64_t>(group) << 32) ^ i;
  x = (x ^ (x >> 31)) * 0x7fb5d329728ea185ull;  // an integer mix; any bijection-like scramble will do
  x = (x ^ (x >> 27)) * 0x81dadef4bc2dd44dull;
  return static_cast<uint8_t>(x ^ (x >> 33));
}

}  // namespace

int main() {
  int n_dev = 0;
  HIP(hipGetDeviceCount(&n_dev));
  CHECK(n_dev > 0);
  HIP(hipSetDevice(0));

  bsr_layout L{};
  L.chunk_tokens = C;
  L.n_groups = 2;
  L.groups[0] = bsr_group_desc{C, T0, R0, BSR_KIND_CONTIG, 0};
  L.groups[1] = bsr_group_desc{C, T1, R1, BSR_KIND_PLANAR, S1};
  const uint64_t pay0 = uint64_t(T0) * C * R0, pay1 = uint64_t(T1) * C * R1;
  const uint64_t slot = bsr_slot_bytes(&L);
  CHECK(slot > 0);

  bsr_config cfg{};
  cfg.window_chunks = W;
  cfg.hip_device = 0;
  bsr_ctx* ctx = nullptr;
  CHECK(bsr_ctx_create(&L, &cfg, &ctx) == BSR_OK);
  CHECK(bsr_store_reserve(ctx, (slot + 4095) / 4096 * 4096 * (N + 1)) == BSR_OK);

  std::vector<int32_t> tokens(N * C);
  for (uint32_t i = 0; i < tokens.size(); ++i) tokens[i] = static_cast<int32_t>((i * 2654435761u) % 129280u);
  const uint64_t salt = 12345;
  std::vector<uint64_t> keys(N);
  CHECK(bsr_chunk_keys(salt, tokens.data(), tokens.size(), C, keys.data()) == BSR_OK);
  std::vector<std::vector<uint8_t>> payload(2 * N);
  std::vector<const void*> ptrs(2 * N);
  for (uint32_t i = 0; i < N; ++i)
    for (uint32_t g = 0; g < 2; ++g) {
      auto& p = payload[2 * i + g];
      p.resize(g ? pay1 : pay0);
      for (uint64_t b = 0; b < p.size(); ++b) p[b] = byte_of(i, g, b);
      ptrs[2 * i + g] = p.data();
    }
  CHECK(bsr_store_put_chunks(ctx, N, keys.data(), ptrs.data()) == BSR_OK);

  uint32_t n_hit = 0;
  CHECK(bsr_probe(ctx, 1, salt, tokens.data(), tokens.size(), &n_hit, nullptr, nullptr) == BSR_OK);
  CHECK(n_hit == N);

  // destination: pools of POOL blocks per tensor, chunk k -> block N-1-k
  const uint64_t blk0 = uint64_t(C) * R0, blk1 = uint64_t(C) * R1;
  void* pools[T0 + T1];
  for (uint32_t t = 0; t < T0; ++t) {
    HIP(hipMalloc(&pools[t], POOL * blk0));
    HIP(hipMemset(pools[t], 0xA5, POOL * blk0));
  }
  HIP(hipMalloc(&pools[T0], POOL * blk1));
  HIP(hipMemset(pools[T0], 0xA5, POOL * blk1));
  std::vector<int32_t> table(N);
  for (uint32_t k = 0; k < N; ++k) table[k] = static_cast<int32_t>(N - 1 - k);
  int32_t* d_table = nullptr;
  void** d_bases0 = nullptr;
  void** d_bases1 = nullptr;
  uint8_t *d_valid0 = nullptr, *d_valid1 = nullptr;
  HIP(hipMalloc(&d_table, N * 4));
  HIP(hipMemcpy(d_table, table.data(), N * 4, hipMemcpyHostToDevice));
  HIP(hipMalloc(reinterpret_cast<void**>(&d_bases0), T0 * sizeof(void*)));
  HIP(hipMemcpy(d_bases0, pools, T0 * sizeof(void*), hipMemcpyHostToDevice));
  HIP(hipMalloc(reinterpret_cast<void**>(&d_bases1), sizeof(void*)));
  HIP(hipMemcpy(d_bases1, &pools[T0], sizeof(void*), hipMemcpyHostToDevice));
  HIP(hipMalloc(reinterpret_cast<void**>(&d_valid0), POOL));
  HIP(hipMalloc(reinterpret_cast<void**>(&d_valid1), POOL));
  HIP(hipMemset(d_valid0, 0, POOL));
  HIP(hipMemset(d_valid1, 0, POOL));
  bsr_group_dst dst[2];
  dst[0] = bsr_group_dst{d_table, d_bases0, d_valid0, N, POOL};
  dst[1] = bsr_group_dst{d_table, d_bases1, d_valid1, N, POOL};

  const uint64_t ring_bytes = bsr_plan_staging_bytes(ctx, N);
  CHECK(ring_bytes == W * slot);
  void* ring = nullptr;
  bsr_dev_status* status = nullptr;
  HIP(hipMalloc(&ring, ring_bytes));
  HIP(hipMalloc(reinterpret_cast<void**>(&status), sizeof(bsr_dev_status)));
  hipStream_t copy, compute;
  HIP(hipStreamCreate(&copy));
  HIP(hipStreamCreate(&compute));
  HIP(hipDeviceSynchronize());

  CHECK(bsr_request_bind(ctx, 1, N, dst, ring, ring_bytes, status, copy, compute) == BSR_OK);
  // the windows as the library plans them: [0, W), [W, 2W), ..., a ragged last one
  uint32_t first = 0, n = 0, n_windows = 0;
  for (;;) {
    CHECK(bsr_next_window(ctx, 1, &first, &n) == BSR_OK);
    if (n == 0) break;
    CHECK(first == n_windows * W && n == (first + W <= N ? W : N - first));
    CHECK(bsr_restore_window(ctx, 1, first, n) == BSR_OK);
    ++n_windows;
  }
  CHECK(first == N && n_windows == (N + W - 1) / W);
  uint64_t exposed = 0;
  int32_t fallback = -1;
  CHECK(bsr_commit(ctx, 1, &exposed, &fallback) == BSR_OK);
  CHECK(exposed == uint64_t(N) * C && fallback == 0);
  bsr_stats st{};
  CHECK(bsr_request_stats(ctx, 1, &st) == BSR_OK);
  CHECK(st.peak_live_staging_bytes == W * slot && st.h2d_bytes == N * slot);

  // the image: block N-1-k of tensor t holds chunk k's records of tensor t
  std::vector<uint8_t> host(POOL * blk0);
  for (uint32_t t = 0; t < T0; ++t) {
    HIP(hipMemcpy(host.data(), pools[t], POOL * blk0, hipMemcpyDeviceToHost));
    for (uint32_t k = 0; k < N; ++k)
      CHECK(std::memcmp(host.data() + (N - 1 - k) * blk0, payload[2 * k].data() + t * blk0, blk0) == 0);
    for (uint64_t b = N * blk0; b < POOL * blk0; ++b) CHECK(host[b] == 0xA5);
  }
  HIP(hipMemcpy(host.data(), pools[T0], POOL * blk1, hipMemcpyDeviceToHost));
  for (uint32_t k = 0; k < N; ++k) {
    const uint8_t* blk = host.data() + (N - 1 - k) * blk1;
    const uint8_t* rec = payload[2 * k + 1].data();
    for (uint32_t o = 0; o < C; ++o) {
      CHECK(std::memcmp(blk + o * S1, rec + o * R1, S1) == 0);                          // values plane
      CHECK(std::memcmp(blk + C * S1 + o * (R1 - S1), rec + o * R1 + S1, R1 - S1) == 0);  // scales plane
    }
  }
  uint8_t v0[POOL], v1[POOL];
  HIP(hipMemcpy(v0, d_valid0, POOL, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(v1, d_valid1, POOL, hipMemcpyDeviceToHost));
  for (uint32_t b = 0; b < POOL; ++b) CHECK(v0[b] == (b < N) && v1[b] == (b < N));

  CHECK(bsr_request_end(ctx, 1) == BSR_OK);
  CHECK(bsr_ctx_destroy(ctx) == BSR_OK);
  HIP(hipStreamDestroy(copy));
  HIP(hipStreamDestroy(compute));
  for (void* p : pools) HIP(hipFree(p));
  HIP(hipFree(ring));
  HIP(hipFree(status));
  HIP(hipFree(d_table));
  HIP(hipFree(d_bases0));
  HIP(hipFree(d_bases1));
  HIP(hipFree(d_valid0));
  HIP(hipFree(d_valid1));
  std::printf("ok %u chunks, %llu bytes\n", N, static_cast<unsigned long long>(N * (pay0 + pay1)));
  return 0;
}
