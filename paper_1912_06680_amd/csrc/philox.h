// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC'11): a counter-based generator, so every value is a
// pure function of (counter, key) and needs no generator state on the
// device.  Each round takes two 64 x 64 -> 128-bit products; the key is
// bumped by the Weyl increments between rounds.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace o5 {

constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;  // golden ratio
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;  // sqrt(3) - 1

__device__ __forceinline__ void philox4x64_10(uint64_t& c0, uint64_t& c1, uint64_t& c2, uint64_t& c3, uint64_t k0,
                                              uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const uint64_t hi0 = __umul64hi(kPhiloxM0, c0), lo0 = kPhiloxM0 * c0;
    const uint64_t hi1 = __umul64hi(kPhiloxM1, c2), lo1 = kPhiloxM1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
}

// U in (0, 1) from the top 24 bits of a word: ((word >> 40) + 1/2) / 2^24,
// exact in fp32.
__device__ __forceinline__ float philox_uniform24(uint64_t word) {
  return (static_cast<float>(word >> 40) + 0.5f) * 5.9604644775390625e-08f;  // 2^-24
}

}  // namespace o5
