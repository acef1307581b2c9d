// Philox4x64-10 counter-based generator shared by the sampling kernels
// (drafting, accept / residual draws, AR steps, Poisson drafting). Every draw
// of the sampler is keyed by a 4-word counter (sequence, round or event
// index, slot, purpose tag) under the run's seed.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tppsd {

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon et al., SC'11) and uniforms on the 2^-24 odd grid
// ---------------------------------------------------------------------------

enum { TAG_AR = 1, TAG_DRAFT = 2, TAG_ACCEPT = 3, TAG_RES_T = 4, TAG_RES_K = 5, TAG_BONUS = 6 };

__device__ __forceinline__ void philox_uniforms(uint64_t seed, uint64_t c0, uint64_t c1, uint64_t c2,
                                                uint64_t c3, float u[4]) {
  uint64_t x0 = c0, x1 = c1, x2 = c2, x3 = c3;
  uint64_t k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
    uint64_t lo0 = m0 * x0, hi0 = __umul64hi(m0, x0);
    uint64_t lo1 = m1 * x2, hi1 = __umul64hi(m1, x2);
    uint64_t y0 = hi1 ^ x1 ^ k0, y2 = hi0 ^ x3 ^ k1;
    x0 = y0;
    x1 = lo1;
    x2 = y2;
    x3 = lo0;
  }
  // top 23 bits -> (2 m + 1) 2^-24, exact in float32
  u[0] = (float)(2ull * (x0 >> 41) + 1ull) * 0x1p-24f;
  u[1] = (float)(2ull * (x1 >> 41) + 1ull) * 0x1p-24f;
  u[2] = (float)(2ull * (x2 >> 41) + 1ull) * 0x1p-24f;
  u[3] = (float)(2ull * (x3 >> 41) + 1ull) * 0x1p-24f;
}

}  // namespace tppsd
