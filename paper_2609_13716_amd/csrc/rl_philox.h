// Device-side counter-based random draws: Philox4x64-10 and what is derived
// from it (32-bit draws, range maps, Gumbel noise).
//
// Philox4x64-10 follows Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers:
// As Easy as 1, 2, 3" (SC'11): 4 x 64-bit counter, 2 x 64-bit key, 10 rounds
// of two 64x64->128 multiplies whose high halves are xored into the other
// counter words together with the round key; the key advances by two Weyl
// increments between rounds.  Key = (seed, 0), counter = (env, t, sub, tag).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rl {

enum : uint64_t { TAG_RESET = 1, TAG_ACTION = 2, TAG_LAYOUT = 3 };

struct Block4 {
  uint64_t w0, w1, w2, w3;
};

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                uint64_t k0, uint64_t k1) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    const uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Block4{c0, c1, c2, c3};
}

__device__ __forceinline__ Block4 draw_block(uint64_t seed, uint64_t env, uint64_t t, uint64_t sub,
                                             uint64_t tag) {
  return philox4x64_10(env, t, sub, tag, seed, 0);
}

__device__ __forceinline__ uint64_t block_word(const Block4& b, int i) {
  return i == 0 ? b.w0 : i == 1 ? b.w1 : i == 2 ? b.w2 : b.w3;
}

// 32-bit draw j (0..7) of a block: word j / 2, high half for even j.
__device__ __forceinline__ uint32_t block_u32(const Block4& b, int j) {
  const uint64_t w = block_word(b, j >> 1);
  return (j & 1) ? (uint32_t)w : (uint32_t)(w >> 32);
}

// floor(u * n / 2^32): maps a 32-bit draw onto 0..n-1.
__device__ __forceinline__ uint32_t range_map(uint32_t u, uint32_t n) {
  return (uint32_t)(((uint64_t)u * (uint64_t)n) >> 32);
}

// Standard Gumbel noise of a 24-bit uniform integer: -ln(-ln((u + 1/2) 2^-24))
// evaluated in double precision, rounded once to float.
__device__ __forceinline__ float gumbel24(uint32_t u24) {
  const double x = ((double)u24 + 0.5) * (1.0 / 16777216.0);
  return (float)(-log(-log(x)));
}

}  // namespace rl
