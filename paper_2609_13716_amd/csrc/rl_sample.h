// Gumbel-max action sampling on the device.
//
// Action a of agent i of global env `env` at step t draws its noise from
// Philox block (seed; env, t, i * 256 + a / 8, TAG_ACTION), 32-bit draw a % 8
// of that block (word (a % 8) / 2, high half for even a), keeping its top 24
// bits.  The score float32(logit + g) of an illegal action or a NaN score is
// -inf; the action is the first index of the largest score, 0 if all are -inf.
#pragma once
#include <math.h>

#include "rl_philox.h"

namespace rl {

__device__ __forceinline__ float action_noise(uint64_t seed, uint64_t env, uint64_t t, int agent, int a) {
  const Block4 b = draw_block(seed, env, t, (uint64_t)agent * 256u + (uint64_t)(a >> 3), TAG_ACTION);
  return gumbel24(block_u32(b, a & 7) >> 8);
}

__device__ __forceinline__ float action_score(float logit, float noise, bool legal) {
#pragma clang fp contract(off)
  const float s = logit + noise;
  return (legal & (s == s)) ? s : -INFINITY;
}

// log pi(a) of a softmax over the n logits l[0..n-1] (all legal), in float32:
// l[a] - (m + log(sum exp(l - m))) with m the largest logit.
__device__ __forceinline__ float log_softmax_at(const float* l, int n, int a) {
  float m = l[0];
  for (int i = 1; i < n; ++i) m = fmaxf(m, l[i]);
  float s = 0.f;
  for (int i = 0; i < n; ++i) s += expf(l[i] - m);
  return l[a] - (m + logf(s));
}

}  // namespace rl
