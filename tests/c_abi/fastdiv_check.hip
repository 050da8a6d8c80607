// CPU check of the install kernel's division by invariant integers: the
// host builds (m, s1, s2) for a divisor d (make_fastdiv) and packs it
// (pack_fastdiv); the kernel divides with packed_div.  For every d in
// [1, 65536] and a set of larger divisors up to 2^32 - 1, the quotient must
// equal n / d for numerators at and around multiples of d, at the ends of
// the 32-bit range, and at pseudo-random points.  Host code only: no GPU.
#include <cstdint>
#include <cstdio>

#include "bsr_device.h"

static uint32_t xs = 0x9E3779B9u;
static uint32_t next_rand() {  // xorshift32
  xs ^= xs << 13;
  xs ^= xs >> 17;
  xs ^= xs << 5;
  return xs;
}

static bool check_divisor(uint32_t d, uint64_t* checks) {
  const bsr::FastDiv f = bsr::make_fastdiv(d);
  const bsr::PackedDiv p = bsr::pack_fastdiv(f);
  auto one = [&](uint32_t n) -> bool {
    ++*checks;
    const uint32_t want = n / d;
    const uint32_t a = f.div(n), b = bsr::packed_div(p.m, p.s, n);
    if (a != want || b != want) {
      printf("MISMATCH d=%u n=%u want=%u div=%u packed=%u\n", d, n, want, a, b);
      return false;
    }
    return true;
  };
  const uint32_t ends[] = {0u, 1u, 2u, 0x7FFFFFFFu, 0x80000000u, 0xFFFFFFFEu, 0xFFFFFFFFu};
  for (uint32_t n : ends)
    if (!one(n)) return false;
  // around the first multiples and the last multiples below 2^32
  const uint64_t top = 0xFFFFFFFFull / d;
  for (uint64_t k = 1; k <= 64 && k <= top; ++k) {
    for (uint64_t v : {k * d - 1, k * d, k * d + 1})
      if (v <= 0xFFFFFFFFull && !one(static_cast<uint32_t>(v))) return false;
    const uint64_t kk = top - (k - 1);
    for (uint64_t v : {kk * d - 1, kk * d, kk * d + 1})
      if (kk >= 1 && v <= 0xFFFFFFFFull && !one(static_cast<uint32_t>(v))) return false;
  }
  for (int i = 0; i < 256; ++i)
    if (!one(next_rand())) return false;
  return true;
}

int main() {
  uint64_t checks = 0;
  for (uint32_t d = 1; d <= 65536; ++d)
    if (!check_divisor(d, &checks)) return 1;
  for (int e = 17; e < 32; ++e) {
    const uint32_t p2 = 1u << e;
    for (uint32_t d : {p2 - 1, p2, p2 + 1, p2 + 12345u})
      if (!check_divisor(d, &checks)) return 1;
  }
  for (uint32_t d : {0x7FFFFFFFu, 0x80000001u, 0xFFFFFFFEu, 0xFFFFFFFFu, 147456u, 9707520u, 16404480u})
    if (!check_divisor(d, &checks)) return 1;
  for (int i = 0; i < 4096; ++i)
    if (!check_divisor(next_rand() | 1u, &checks)) return 1;
  printf("checks %llu\nok\n", static_cast<unsigned long long>(checks));
  return 0;
}
