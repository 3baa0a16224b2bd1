// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy
// as 1, 2, 3", SC'11): 4x32-bit counter, 2x32-bit key, ten rounds; each round
// multiplies counter words 0 and 2 by fixed constants and mixes the 64-bit
// product halves with words 1, 3 and the key, which is advanced by two Weyl
// increments between rounds.  Device implementation.
#pragma once
#include "common.hpp"

namespace rgd {

RGD_DEV uint32_t philox4x32_10_w0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                  uint32_t k0, uint32_t k1) {
  const uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  const uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += kW0; k1 += kW1; }
    const uint32_t hi0 = __umulhi(kM0, c0), lo0 = kM0 * c0;
    const uint32_t hi1 = __umulhi(kM1, c2), lo1 = kM1 * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
  return c0;
}

// Uniform in [0,1) with 24 random bits: word 0 of Philox(key = seed split
// low/high, counter = (ctr, stream, 0, 0)), top 24 bits scaled by 2^-24.
RGD_DEV float philox_uniform(uint64_t seed, uint32_t ctr, uint32_t stream) {
  const uint32_t w = philox4x32_10_w0(ctr, stream, 0u, 0u, uint32_t(seed), uint32_t(seed >> 32));
  return float(w >> 8) * (1.0f / 16777216.0f);
}

}  // namespace rgd
