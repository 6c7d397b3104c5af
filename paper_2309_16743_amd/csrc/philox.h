// Philox4x64-10 counter-based generator (Salmon, Moraes, Dror, Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC'11), device side, and the
// multiply-high range map floor(w * n / 2^64) (Lemire, 2019, without the
// rejection step).  Used for every random draw of the reservoir and for the
// surrogate's initialisation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ot {

enum : uint64_t { kKindSample = 1, kKindEvict = 2, kKindInit = 3 };

struct u64x4 {
  uint64_t x, y, z, w;
};

__device__ __forceinline__ u64x4 philox4x64_10(u64x4 c, uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t hi0 = __umul64hi(M0, c.x), lo0 = M0 * c.x;
    const uint64_t hi1 = __umul64hi(M1, c.z), lo1 = M1 * c.z;
    c = u64x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
    k0 += W0;
    k1 += W1;
  }
  return c;
}

// Word 0 of the block at counter (j, ticket, kind, 0), key (seed, 0).
__device__ __forceinline__ uint64_t draw_word(uint64_t seed, uint64_t j, uint64_t ticket,
                                              uint64_t kind) {
  return philox4x64_10(u64x4{j, ticket, kind, 0}, seed, 0).x;
}

// floor(w * n / 2^64): an index in [0, n).
__device__ __forceinline__ uint64_t range_map(uint64_t w, uint64_t n) { return __umul64hi(w, n); }

}  // namespace ot
