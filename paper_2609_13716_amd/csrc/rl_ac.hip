// Generalised advantage estimation over a stored trajectory: one thread per
// (env, agent), a backward scan over the steps.  Memory-bound: each step reads
// the env's reward and done (shared by its agents) and the agent's value, and
// writes its advantage and return; consecutive threads touch consecutive
// (env, agent) entries of every [T, E, A] array.
#include "rl_internal.h"

namespace rl {

__global__ __launch_bounds__(NTHREADS) void gae_kernel(const float* __restrict__ reward,
                                                       const uint8_t* __restrict__ done,
                                                       const float* __restrict__ value,
                                                       const float* __restrict__ value_last, int T, int E, int A,
                                                       float gamma, float gl, float* __restrict__ adv,
                                                       float* __restrict__ ret) {
  const int64_t i = (int64_t)blockIdx.x * NTHREADS + threadIdx.x;  // env * A + agent
  const int64_t n = (int64_t)E * A;
  if (i >= n) return;
  const int64_t e = i / A;
  float nv = value_last[i], na = 0.f;
  for (int t = T - 1; t >= 0; --t) {
    const size_t ti = (size_t)t * n + i;
    const float keep = done[(size_t)t * E + e] == 0 ? 1.f : 0.f;
    const float v = value[ti];
    const float delta = reward[(size_t)t * E + e] + gamma * keep * nv - v;
    na = delta + gl * keep * na;
    adv[ti] = na;
    if (ret) ret[ti] = na + v;
    nv = v;
  }
}

hipError_t launch_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last, int T,
                      int E, int A, float gamma, float lambda, float* adv, float* ret, hipStream_t s) {
  const int64_t n = (int64_t)E * A;
  gae_kernel<<<dim3((unsigned)((n + NTHREADS - 1) / NTHREADS)), NTHREADS, 0, s>>>(
      reward, done, value, value_last, T, E, A, gamma, gamma * lambda, adv, ret);
  return hipGetLastError();
}

}  // namespace rl
