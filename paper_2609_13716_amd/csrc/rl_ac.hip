// Generalised advantage estimation over a stored trajectory: one thread per
// (env, agent), a backward scan over the steps (inputs of 16 steps loaded
// ahead of the dependent recurrence).  Memory-bound: each step reads
// the env's reward and done (shared by its agents) and the agent's value, and
// writes its advantage and return; consecutive threads touch consecutive
// (env, agent) entries of every [T, E, A] array.
#include "rl_internal.h"

namespace rl {

constexpr int GAE_NT = 64;  // one wave per workgroup: E * A chains spread over as many CUs as possible
constexpr int GAE_U = 16;   // steps whose inputs are loaded ahead of the dependent recurrence

__global__ __launch_bounds__(GAE_NT) void gae_kernel(const float* __restrict__ reward,
                                                     const uint8_t* __restrict__ done,
                                                     const float* __restrict__ value,
                                                     const float* __restrict__ value_last, int T, int E, int A,
                                                     float gamma, float gl, float* __restrict__ adv,
                                                     float* __restrict__ ret) {
  const int64_t i = (int64_t)blockIdx.x * GAE_NT + threadIdx.x;  // env * A + agent
  const int64_t n = (int64_t)E * A;
  if (i >= n) return;
  const int64_t e = i / A;
  float nv = value_last[i], na = 0.f;
  for (int t1 = T; t1 > 0; t1 -= GAE_U) {  // steps t1-1 down to max(t1-GAE_U, 0)
    float r[GAE_U], v[GAE_U], keep[GAE_U];
#pragma unroll
    for (int u = 0; u < GAE_U; ++u) {
      const int t = t1 - 1 - u;
      if (t >= 0) {
        r[u] = reward[(size_t)t * E + e];
        keep[u] = done[(size_t)t * E + e] == 0 ? 1.f : 0.f;
        v[u] = value[(size_t)t * n + i];
      }
    }
#pragma unroll
    for (int u = 0; u < GAE_U; ++u) {
      const int t = t1 - 1 - u;
      if (t >= 0) {
        const float delta = r[u] + gamma * keep[u] * nv - v[u];
        na = delta + gl * keep[u] * na;
        const size_t ti = (size_t)t * n + i;
        adv[ti] = na;
        if (ret) ret[ti] = na + v[u];
        nv = v[u];
      }
    }
  }
}

hipError_t launch_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last, int T,
                      int E, int A, float gamma, float lambda, float* adv, float* ret, hipStream_t s) {
  const int64_t n = (int64_t)E * A;
  gae_kernel<<<dim3((unsigned)((n + GAE_NT - 1) / GAE_NT)), GAE_NT, 0, s>>>(reward, done, value, value_last, T, E,
                                                                           A, gamma, gamma * lambda, adv, ret);
  return hipGetLastError();
}

}  // namespace rl
