// Philox4x64-10 counter-based generator (Salmon, Moraes, Dror, Shaw, "Parallel
// Random Numbers: As Easy as 1, 2, 3", SC'11) and the uniforms SpS draws.
//
// Counter (c0..c3) = (j, b, loop, purpose), key = (seed, 0). The uniform is
// the top 24 bits of output word 0 scaled by 2^-24: a value on the 2^-24
// grid in [0, 1), exact in fp32.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sps {

__device__ __forceinline__ uint64_t philox_word0(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                 uint64_t k0, uint64_t k1) {
  // Round multipliers and Weyl increments of the 4x64 variant (SC'11, Sec. 5).
  const uint64_t kMul0 = 0xD2E7470EE14C6C93ull, kMul1 = 0xCA5A826395121157ull;
  const uint64_t kInc0 = 0x9E3779B97F4A7C15ull, kInc1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hi0 = __umul64hi(kMul0, c0), lo0 = kMul0 * c0;
    const uint64_t hi1 = __umul64hi(kMul1, c2), lo1 = kMul1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += kInc0; k1 += kInc1;
  }
  return c0;
}

__device__ __forceinline__ float philox_uniform(uint64_t seed, uint64_t loop, uint32_t purpose,
                                                uint32_t b, uint32_t j) {
  const uint64_t x0 = philox_word0(j, b, loop, purpose, seed, 0);
  return static_cast<float>(static_cast<uint32_t>(x0 >> 40)) * 0x1p-24f;
}

}  // namespace sps
