// Standalone policy forward (obs -> logits on the MFMA MLP), standalone
// Gumbel-max sampling from given logits, and the sampler's noise function.
#include "rl_internal.h"
#include "rl_regmlp.h"
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
  mlp_input_layer<DT>(xs, PL.ldx, nullptr, BM, D, static_cast<const T*>(pol.W[0]), static_cast<const T*>(pol.b[0]), pol.H1, h1,
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

// Persistent policy forward for compile-time sizes: each workgroup keeps the
// layer-1/2 weights in registers and layer 3 in LDS, and loops over tiles of
// MT * 16 rows (stage the observation tile with 16-byte loads, three MFMA
// layers computed transposed, masked logits out).  MINB workgroups share a
// CU so that one's loads overlap another's matrix work.
template <int DT, int D, int H1, int H2, int NA, int NW, int MT, int MINB>
__global__ __launch_bounds__(NW * 64, MINB) void policy_fwd_reg_kernel(PolicyArgs pol, const void* __restrict__ obs_v,
                                                                       const uint8_t* __restrict__ legal,
                                                                       int64_t rows, float* __restrict__ logits) {
  using T = typename DType<DT>::T;
  using B = typename BOperand<DT>::type;
  constexpr int NT = NW * 64, BM = MT * 16;
  constexpr int LDX = lds_ld<DT>(D), LD1 = lds_ld<DT>(H1), LD2 = lds_ld<DT>(H2);
  constexpr int K3 = round_up(H2, DType<DT>::KS) / DType<DT>::KS;
  constexpr int VE = 16 / sizeof(T);
  static_assert(D % VE == 0, "observation rows are whole 16-byte vectors");
  static_assert(NA <= 16, "one transposed M tile of actions");
  static_assert(MT <= NW, "one layer-3 M tile per wave");
  __shared__ __align__(16) T xs[BM * LDX];
  __shared__ __align__(16) T h1s[BM * LD1];
  __shared__ __align__(16) T h2s[BM * LD2];
  __shared__ __align__(16) B w3s[K3 * 64];
  const T* obs = static_cast<const T*>(obs_v);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  RegLayer<DT, D, H1, NW> L1;
  RegLayer<DT, H1, H2, NW> L2;
  L1.load(static_cast<const T*>(pol.W[0]), static_cast<const T*>(pol.b[0]), wave, lane);
  L2.load(static_cast<const T*>(pol.W[1]), static_cast<const T*>(pol.b[1]), wave, lane);
  if (tid < 64) {
    const int n = lane & 15;
    const T* row = static_cast<const T*>(pol.W[2]) + (size_t)(n < NA ? n : 0) * H2;
#pragma unroll
    for (int ks = 0; ks < K3; ++ks) w3s[ks * 64 + lane] = load_operand_global<DT, H2>(row, H2, ks, lane, n < NA);
  }
  float b3r[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int a = 4 * (lane >> 4) + r;
    b3r[r] = a < NA ? DType<DT>::to_f32(static_cast<const T*>(pol.b[2])[a]) : 0.f;
  }
  for (int i = tid; i < BM * LDX; i += NT) xs[i] = (T)0;
  for (int i = tid; i < BM * LD1; i += NT) h1s[i] = (T)0;
  for (int i = tid; i < BM * LD2; i += NT) h2s[i] = (T)0;
  __syncthreads();

  // Software pipeline over this workgroup's tiles: the observation tile of
  // the next iteration is loaded into registers while the current one is
  // computed, and a tile's logits are stored at the start of the next
  // iteration, after that prefetch is issued, so that waiting for the
  // prefetch never waits for just-issued stores.
  const int64_t ntiles = (rows + BM - 1) / BM;
  constexpr int VPR = D / VE, NV = BM * VPR, IT = (NV + NT - 1) / NT;
  u32x4 v[IT];
  auto prefetch = [&](int64_t tile) {
    const int64_t row0 = tile * BM;
    const int nrow = tile < ntiles ? (int)min((int64_t)BM, rows - row0) : 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = tid + it * NT;
      const int r = i / VPR, c = (i - r * VPR) * VE;
      v[it] = (i < NV && r < nrow) ? *reinterpret_cast<const u32x4*>(obs + (size_t)(row0 + r) * D + c)
                                    : u32x4{0u, 0u, 0u, 0u};
    }
  };
  float lg[4] = {0.f, 0.f, 0.f, 0.f};
  int64_t lg_row = -1;  // global row of the pending logits (-1: none)
  auto store_logits = [&]() {
    if (lg_row >= 0) {
      const size_t gr = (size_t)lg_row * NA;
      const int g = lane >> 4;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = 4 * g + r;
        if (a < NA) {
          const bool ok = legal == nullptr || legal[gr + a] != 0;
          logits[gr + a] = ok ? lg[r] : -INFINITY;
        }
      }
    }
  };
  prefetch(blockIdx.x);
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t row0 = tile * BM;
    const int nrow = (int)min((int64_t)BM, rows - row0);
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = tid + it * NT;
      const int r = i / VPR, c = (i - r * VPR) * VE;
      if (i < NV) *reinterpret_cast<u32x4*>(xs + r * LDX + c) = v[it];
    }
    __syncthreads();
    if (tile + gridDim.x < ntiles) prefetch(tile + gridDim.x);
    store_logits();
    lg_row = -1;
    {
      f32x4 acc[MT][RegLayer<DT, D, H1, NW>::OWN];
      L1.template run<MT>(xs, LDX, acc, wave, lane);
      L1.template store_tanh<MT>(acc, h1s, LD1, wave, lane);
    }
    __syncthreads();
    {
      f32x4 acc[MT][RegLayer<DT, H1, H2, NW>::OWN];
      L2.template run<MT>(h1s, LD1, acc, wave, lane);
      L2.template store_tanh<MT>(acc, h2s, LD2, wave, lane);
    }
    __syncthreads();
    if (wave < MT) {
      const int row = wave * 16 + (lane & 15);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < K3; ++ks)
        acc = mfma16<DT>(w3s[ks * 64 + lane], load_operand_lds<DT>(h2s, LD2, row, ks, lane), acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) lg[r] = acc[r] + b3r[r];
      lg_row = row < nrow ? row0 + row : -1;
    }
  }
  store_logits();
}

template <int DT, int D, int H1, int H2, int NA, int NW, int MT, int MINB>
static hipError_t launch_policy_reg(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                    float* logits, hipStream_t s) {
  constexpr int BM = MT * 16;
  const int64_t ntiles = (rows + BM - 1) / BM;
  const unsigned grid = (unsigned)(ntiles < (int64_t)256 * MINB ? ntiles : (int64_t)256 * MINB);
  policy_fwd_reg_kernel<DT, D, H1, H2, NA, NW, MT, MINB><<<dim3(grid), NW * 64, 0, s>>>(pol, obs, legal, rows, logits);
  return hipGetLastError();
}

static bool try_launch_policy_reg(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                  float* logits, hipStream_t s, hipError_t* err) {
#define RL_PF_CASE(DTV, DV, H1V, H2V, NAV, NWV, MTV, MINBV)                                              \
  if (pol.dt == DTV && pol.D == DV && pol.H1 == H1V && pol.H2 == H2V && pol.NA == NAV) {                   \
    *err = launch_policy_reg<DTV, DV, H1V, H2V, NAV, NWV, MTV, MINBV>(pol, obs, legal, rows, logits, s); \
    return true;                                                                                         \
  }
  // (dtype, D, H1, H2, nA, waves, 16-row M tiles per workgroup tile, workgroups per CU)
  RL_PF_CASE(DT_BF16, 192, 128, 128, 6, 4, 4, 2)
  RL_PF_CASE(DT_F32, 192, 128, 128, 6, 4, 4, 1)
  RL_PF_CASE(DT_BF16, 192, 64, 64, 6, 4, 4, 2)
  RL_PF_CASE(DT_F32, 192, 64, 64, 6, 4, 4, 2)
#undef RL_PF_CASE
  return false;
}

hipError_t launch_policy_forward(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                 float* logits, hipStream_t s) {
  hipError_t err;
  if (try_launch_policy_reg(pol, obs, legal, rows, logits, s, &err)) return err;
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
