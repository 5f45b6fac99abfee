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

// The same recurrence cut into GAE_CH chunks of steps per chain, the chunks
// run side by side: A_t = delta_t + c_t A_{t+1} (c_t = gamma lambda (1 - d_t))
// is affine in A_{t+1}, so each chunk first folds its steps into
// A_start = a + p A_after (a: the chunk's advantage at its first step with
// A_after = 0, p: the product of its c_t); one wave then runs the short
// recurrence over the chunks' (a, p) pairs for every chain, and each chunk
// replays its steps from its true A_after, writing the outputs.  Inputs are
// read twice; a workgroup holds 64 chains (one per lane) x GAE_CH chunks (one
// per wave), so chains of 128 steps spread over 16 times more waves.
constexpr int GAE_CH = 16;

__global__ __launch_bounds__(64 * GAE_CH) void gae_chunk_kernel(const float* __restrict__ reward,
                                                               const uint8_t* __restrict__ done,
                                                               const float* __restrict__ value,
                                                               const float* __restrict__ value_last, int T, int E,
                                                               int A, float gamma, float gl, float* __restrict__ adv,
                                                               float* __restrict__ ret) {
  __shared__ float s_a[GAE_CH][64], s_p[GAE_CH][64], s_in[GAE_CH][64];
  const int lane = threadIdx.x & 63, ch = threadIdx.x >> 6;
  const int64_t n = (int64_t)E * A;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;  // env * A + agent
  const bool ok = i < n;
  const int64_t e = ok ? i / A : 0;
  const int L = (T + GAE_CH - 1) / GAE_CH;
  const int t_lo = min(T, ch * L), t_hi = min(T, t_lo + L);
  // pass 1: fold the chunk's steps
  float a = 0.f, pr = 1.f;
  if (ok) {
    float nv = t_hi < T ? value[(size_t)t_hi * n + i] : value_last[i];
    for (int t = t_hi - 1; t >= t_lo; --t) {
      const float keep = done[(size_t)t * E + e] == 0 ? 1.f : 0.f;
      const float v = value[(size_t)t * n + i];
      const float delta = reward[(size_t)t * E + e] + gamma * keep * nv - v;
      a = delta + gl * keep * a;
      pr *= gl * keep;
      nv = v;
    }
  }
  s_a[ch][lane] = a;
  s_p[ch][lane] = pr;
  __syncthreads();
  if (ch == 0) {  // advantage after each chunk, from the last chunk backwards
    float after = 0.f;
    for (int j = GAE_CH - 1; j >= 0; --j) {
      s_in[j][lane] = after;
      after = s_a[j][lane] + s_p[j][lane] * after;
    }
  }
  __syncthreads();
  if (!ok) return;
  // pass 2: the chunk's steps from its true advantage after it
  a = s_in[ch][lane];
  float nv = t_hi < T ? value[(size_t)t_hi * n + i] : value_last[i];
  for (int t = t_hi - 1; t >= t_lo; --t) {
    const float keep = done[(size_t)t * E + e] == 0 ? 1.f : 0.f;
    const float v = value[(size_t)t * n + i];
    const float delta = reward[(size_t)t * E + e] + gamma * keep * nv - v;
    a = delta + gl * keep * a;
    const size_t ti = (size_t)t * n + i;
    adv[ti] = a;
    if (ret) ret[ti] = a + v;
    nv = v;
  }
}

hipError_t launch_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last, int T,
                      int E, int A, float gamma, float lambda, float* adv, float* ret, hipStream_t s) {
  const int64_t n = (int64_t)E * A;
  if (T >= 2 * GAE_CH) {  // long chains: chunked
    gae_chunk_kernel<<<dim3((unsigned)((n + 63) / 64)), 64 * GAE_CH, 0, s>>>(reward, done, value, value_last, T, E, A,
                                                                             gamma, gamma * lambda, adv, ret);
  } else {
    gae_kernel<<<dim3((unsigned)((n + GAE_NT - 1) / GAE_NT)), GAE_NT, 0, s>>>(reward, done, value, value_last, T, E,
                                                                             A, gamma, gamma * lambda, adv, ret);
  }
  return hipGetLastError();
}

}  // namespace rl
