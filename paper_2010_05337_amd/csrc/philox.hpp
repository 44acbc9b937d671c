// Counter-based random draws for the sampler (device side).
//
// Philox4x32-10 as defined by Salmon, Moraes, Dror & Shaw ("Parallel random
// numbers: as easy as 1, 2, 3", SC'11): ten rounds of two 32x32->64-bit
// multiplications on lanes 0 and 2, with the key advanced by the Weyl
// constants between rounds.  A draw in [0, m) follows Lemire ("Fast random
// integer generation in an interval", ACM TOMACS 2019): the high word of
// x*m, rejecting x when the low word falls below (2^32 - m) mod m.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmb {

struct Philox4 {
  uint32_t w[4];
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                 uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // one 32x32->64-bit product per lane pair (a single v_mad_u64_u32
    // instead of a low and a high multiply)
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c0;
    const uint64_t p2 = static_cast<uint64_t>(0xCD9E8D57u) * c2;
    const uint32_t a0 = static_cast<uint32_t>(p0), h0 = static_cast<uint32_t>(p0 >> 32);
    const uint32_t a2 = static_cast<uint32_t>(p2), h2 = static_cast<uint32_t>(p2 >> 32);
    const uint32_t n0 = h2 ^ c1 ^ k0;
    const uint32_t n2 = h0 ^ c3 ^ k1;
    c0 = n0;
    c1 = a2;
    c2 = n2;
    c3 = a0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return Philox4{{c0, c1, c2, c3}};
}

// i-th draw of vertex v at layer l, uniform in [0, m), m >= 1.  Each word
// is rejected with probability below m / 2^32 <= 1/2, so the bound on the
// number of Philox blocks (2^20 blocks, 2^22 words) is never reached; it
// only guarantees that the loop ends.
__device__ __forceinline__ uint32_t draw_below(uint32_t k0, uint32_t k1, uint32_t v, uint32_t l,
                                               uint32_t i, uint32_t m) {
  for (uint32_t block = 0; block < (1u << 20); ++block) {
    const Philox4 x = philox4x32_10(v, l, i, block, k0, k1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t prod = static_cast<uint64_t>(x.w[q]) * m;
      const uint32_t low = static_cast<uint32_t>(prod);
      // low >= m can never be below the threshold (which is < m), so the
      // division is only paid on the rare path.
      if (low >= m || low >= (0u - m) % m) return static_cast<uint32_t>(prod >> 32);
    }
  }
  return m - 1;
}

}  // namespace gmb
