// Standalone policy forward (obs -> logits on the MFMA MLP), standalone
// Gumbel-max sampling from given logits, and the sampler's noise function.
#include "rl_internal.h"
#include "rl_sample.h"

namespace rl {

struct PolicyLayout {
  int BM;              // rows per workgroup
  int ldx, ld1, ld2;
  size_t off_x, off_h1, off_h2, off_logit, total;
};

static PolicyLayout make_policy_layout(const PolicyArgs& pol, int BM) {
  PolicyLayout L;
  const size_t es = pol.dt == DT_F32 ? 4 : 2;
  L.BM = BM;
  L.ldx = pol.dt == DT_F32 ? lds_ld<DT_F32>(pol.D) : lds_ld<DT_BF16>(pol.D);
  L.ld1 = pol.dt == DT_F32 ? lds_ld<DT_F32>(pol.H1) : lds_ld<DT_BF16>(pol.H1);
  L.ld2 = pol.dt == DT_F32 ? lds_ld<DT_F32>(pol.H2) : lds_ld<DT_BF16>(pol.H2);
  size_t o = 0;
  L.off_x = o;     o += (size_t)BM * L.ldx * es;  o = (o + 15) & ~(size_t)15;
  L.off_h1 = o;    o += (size_t)BM * L.ld1 * es;  o = (o + 15) & ~(size_t)15;
  L.off_h2 = o;    o += (size_t)BM * L.ld2 * es;  o = (o + 15) & ~(size_t)15;
  L.off_logit = o; o += (size_t)BM * MAX_NA * 4;
  L.total = o;
  return L;
}

static PolicyLayout pick_policy_layout(const PolicyArgs& pol) {
  for (int bm = 64; bm >= 16; bm >>= 1) {
    const PolicyLayout L = make_policy_layout(pol, bm);
    if (L.total <= MAX_LDS_BYTES) return L;
  }
  return make_policy_layout(pol, 16);
}

size_t policy_lds_bytes(const PolicyArgs& pol) { return pick_policy_layout(pol).total; }

template <int DT>
__global__ __launch_bounds__(NTHREADS) void policy_forward_kernel(PolicyArgs pol, PolicyLayout PL,
                                                                  const void* __restrict__ obs_v,
                                                                  const uint8_t* __restrict__ legal, int64_t rows,
                                                                  float* __restrict__ logits) {
  using T = typename DType<DT>::T;
  extern __shared__ __align__(16) uint8_t smem[];
  T* xs = reinterpret_cast<T*>(smem + PL.off_x);
  T* h1 = reinterpret_cast<T*>(smem + PL.off_h1);
  T* h2 = reinterpret_cast<T*>(smem + PL.off_h2);
  float* lg = reinterpret_cast<float*>(smem + PL.off_logit);
  const T* obs = static_cast<const T*>(obs_v);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int BM = PL.BM, D = pol.D, NA = pol.NA;
  const int64_t row0 = (int64_t)blockIdx.x * BM;
  const int nrow = (int)min((int64_t)BM, rows - row0);

  // stage the observation tile, zero-padded to ldx columns and BM rows
  for (int idx = tid; idx < BM * PL.ldx; idx += NTHREADS) {
    const int r = idx / PL.ldx, k = idx - r * PL.ldx;
    xs[idx] = (r < nrow && k < D) ? obs[(size_t)(row0 + r) * D + k] : (T)0;
  }
  // zero the K padding of the hidden tiles
  for (int idx = tid; idx < BM * PL.ld1; idx += NTHREADS) h1[idx] = (T)0;
  for (int idx = tid; idx < BM * PL.ld2; idx += NTHREADS) h2[idx] = (T)0;
  __syncthreads();
  mlp_hidden<DT>(xs, PL.ldx, BM, D, static_cast<const T*>(pol.W[0]), static_cast<const T*>(pol.b[0]), pol.H1, h1,
                 PL.ld1, wave, NTHREADS / 64, lane);
  __syncthreads();
  mlp_hidden<DT>(h1, PL.ld1, BM, pol.H1, static_cast<const T*>(pol.W[1]), static_cast<const T*>(pol.b[1]), pol.H2,
                 h2, PL.ld2, wave, NTHREADS / 64, lane);
  __syncthreads();
  mlp_logits<DT>(h2, PL.ld2, BM, pol.H2, static_cast<const T*>(pol.W[2]), static_cast<const T*>(pol.b[2]), NA, lg,
                 MAX_NA, wave, NTHREADS / 64, lane);
  __syncthreads();
  for (int idx = tid; idx < nrow * NA; idx += NTHREADS) {
    const int r = idx / NA, a = idx - r * NA;
    const size_t gi = (size_t)row0 * NA + idx;
    const bool ok = legal == nullptr || legal[gi] != 0;
    logits[gi] = ok ? lg[r * MAX_NA + a] : -INFINITY;
  }
}

hipError_t launch_policy_forward(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                 float* logits, hipStream_t s) {
  const PolicyLayout PL = pick_policy_layout(pol);
  const dim3 grid((unsigned)((rows + PL.BM - 1) / PL.BM));
  if (pol.dt == DT_F32) {
    static bool attr = false;
    if (!attr) {
      hipError_t e = hipFuncSetAttribute((const void*)policy_forward_kernel<DT_F32>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)MAX_LDS_BYTES);
      if (e != hipSuccess) return e;
      attr = true;
    }
    policy_forward_kernel<DT_F32><<<grid, NTHREADS, PL.total, s>>>(pol, PL, obs, legal, rows, logits);
  } else {
    static bool attr = false;
    if (!attr) {
      hipError_t e = hipFuncSetAttribute((const void*)policy_forward_kernel<DT_BF16>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)MAX_LDS_BYTES);
      if (e != hipSuccess) return e;
      attr = true;
    }
    policy_forward_kernel<DT_BF16><<<grid, NTHREADS, PL.total, s>>>(pol, PL, obs, legal, rows, logits);
  }
  return hipGetLastError();
}

// One thread per (env, agent) row: noise, scores, first argmax.
__global__ __launch_bounds__(NTHREADS) void sample_kernel(uint64_t seed, int64_t env_base, int E, int A, int NA,
                                                          uint64_t t, const float* __restrict__ logits,
                                                          const uint8_t* __restrict__ legal,
                                                          int32_t* __restrict__ actions) {
  const int64_t row = (int64_t)blockIdx.x * NTHREADS + threadIdx.x;
  if (row >= (int64_t)E * A) return;
  const int e = (int)(row / A), ag = (int)(row - (int64_t)e * A);
  int best = 0;
  float bs = -INFINITY;
  for (int a = 0; a < NA; ++a) {
    const size_t i = (size_t)row * NA + a;
    const float g = action_noise(seed, (uint64_t)(env_base + e), t, ag, a);
    const float v = action_score(logits[i], g, legal == nullptr || legal[i] != 0);
    if (v > bs) {
      bs = v;
      best = a;
    }
  }
  actions[row] = best;
}

hipError_t launch_sample(uint64_t seed, int64_t env_base, int E, int A, int NA, uint64_t t, const float* logits,
                         const uint8_t* legal, int32_t* actions, hipStream_t s) {
  const int64_t rows = (int64_t)E * A;
  sample_kernel<<<dim3((unsigned)((rows + NTHREADS - 1) / NTHREADS)), NTHREADS, 0, s>>>(seed, env_base, E, A, NA, t,
                                                                                       logits, legal, actions);
  return hipGetLastError();
}

__global__ __launch_bounds__(NTHREADS) void gumbel_kernel(const uint32_t* __restrict__ u, int64_t n,
                                                          float* __restrict__ g) {
  const int64_t i = (int64_t)blockIdx.x * NTHREADS + threadIdx.x;
  if (i < n) g[i] = gumbel24(u[i] & 0xffffffu);
}

hipError_t launch_gumbel(const uint32_t* u, int64_t n, float* g, hipStream_t s) {
  gumbel_kernel<<<dim3((unsigned)((n + NTHREADS - 1) / NTHREADS)), NTHREADS, 0, s>>>(u, n, g);
  return hipGetLastError();
}

}  // namespace rl
