// Level-Based Foraging kernels: episode init, env-only stepping with injected
// actions, and the fused persistent rollout (observe -> MLP -> sample -> step
// -> auto-reset) for one tile of TILE_E envs per workgroup.
//
// Work split inside a workgroup (256 threads, 4 waves):
//   * env logic: lane e of wave 0 owns env e of the tile and keeps its whole
//     state in registers for the duration of the kernel (read from HBM once,
//     written back once);
//   * observations: every thread encodes 8 consecutive features at a time
//     from two per-env byte grids in LDS (agent level and food level at each
//     cell) that the env lanes repaint after each transition, and writes them
//     with 16-byte stores, so the observation rows of the tile (contiguous in
//     [E, A, D]) are written fully coalesced;
//   * policy: the tile's R = TILE_E * A rows go through the MFMA MLP
//     (rl_mlp.h) with operand tiles in LDS;
//   * sampling: one thread per (row, action) draws the Gumbel noise.
#include "rl_internal.h"
#include "rl_sample.h"

namespace rl {

struct LbfMagic {
  uint32_t d, a, hw, na;
};

static LbfMagic make_magic(const LbfParams& p, int na) {
  return LbfMagic{div_magic((uint32_t)p.D), div_magic((uint32_t)p.A), div_magic((uint32_t)p.HW),
                  div_magic((uint32_t)na)};
}

struct LbfLds {
  uint8_t* agrid;  // [TILE_E][256]: level of the agent on each cell, 0 = none
  uint8_t* fgrid;  // [TILE_E][256]: level of the uneaten food on each cell, 0 = none
  int* acell;      // [TILE_E][LBF_MAXA]: agent cells
};

// Write (on) or erase (!on) env `el`'s agents and uneaten foods in the LDS
// grids.  Cell ids are masked to the grid buffer so that a malformed state
// supplied by the caller cannot address LDS outside its own env's grid.
__device__ __forceinline__ void lbf_paint(const LbfParams& p, const LbfEnv& s, int el, const LbfLds& L, bool on) {
  constexpr int CM = LBF_MAXCELLS - 1;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < p.A) {
      L.agrid[el * LBF_MAXCELLS + (s.acell[i] & CM)] = on ? (uint8_t)s.alevel[i] : 0;
      if (on) L.acell[el * LBF_MAXA + i] = s.acell[i];
    }
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < p.F && !((s.eaten >> j) & 1u))
      L.fgrid[el * LBF_MAXCELLS + (s.fcell[j] & CM)] = on ? (uint8_t)s.flevel[j] : 0;
}

template <typename OT>
__device__ __forceinline__ OT small_int_to(uint32_t v);
template <>
__device__ __forceinline__ float small_int_to<float>(uint32_t v) {
  return (float)v;
}
template <>
__device__ __forceinline__ uint16_t small_int_to<uint16_t>(uint32_t v) {
  return (uint16_t)(__float_as_uint((float)v) >> 16);  // exact: small integers are bf16 values
}

// Observation rows of the tile: element (r, k) with r = el * A + a.
// gdst: the tile's first element in global [.., A, D] (or null); ldst: LDS
// operand tile with leading dimension ldl (or null).  Rows of envs beyond
// te_valid are zero in LDS and not written to global memory.
template <typename OT>
__device__ __forceinline__ void lbf_encode(const LbfParams& p, const LbfMagic& m, int te_valid, const LbfLds& L,
                                           OT* __restrict__ gdst, OT* __restrict__ ldst, int ldl, int tid) {
  const int A = p.A, D = p.D, HW = p.HW;
  if ((D & 7) == 0 && (HW & 7) == 0) {
    const int nvec = TILE_E * A * (D >> 3);
    for (int v = tid; v < nvec; v += NTHREADS) {
      const int idx = v << 3;
      const int r = fdiv(idx, m.d), k = idx - r * D;
      const int el = fdiv(r, m.a), a = r - el * A;
      const int plane = fdiv(k, m.hw), cell0 = k - plane * HW;
      uint64_t bytes = 0;
      if (el < te_valid) {
        if (plane == 0) {
          bytes = *reinterpret_cast<const uint64_t*>(L.agrid + el * LBF_MAXCELLS + cell0);
        } else if (plane == 1) {
          bytes = *reinterpret_cast<const uint64_t*>(L.fgrid + el * LBF_MAXCELLS + cell0);
        } else {
          const int c = L.acell[el * LBF_MAXA + a] - cell0;
          if (c >= 0 && c < 8) bytes = 1ull << (8 * c);
        }
      }
      OT vals[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) vals[q] = small_int_to<OT>((uint32_t)(bytes >> (8 * q)) & 0xffu);
      if constexpr (sizeof(OT) == 2) {
        u32x4 w;
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = (uint32_t)vals[2 * q] | ((uint32_t)vals[2 * q + 1] << 16);
        if (ldst) *reinterpret_cast<u32x4*>(ldst + (size_t)r * ldl + k) = w;
        if (gdst && el < te_valid) *reinterpret_cast<u32x4*>(gdst + idx) = w;
      } else {
        const f32x4 w0 = {vals[0], vals[1], vals[2], vals[3]};
        const f32x4 w1 = {vals[4], vals[5], vals[6], vals[7]};
        if (ldst) {
          *reinterpret_cast<f32x4*>(ldst + (size_t)r * ldl + k) = w0;
          *reinterpret_cast<f32x4*>(ldst + (size_t)r * ldl + k + 4) = w1;
        }
        if (gdst && el < te_valid) {
          *reinterpret_cast<f32x4*>(gdst + idx) = w0;
          *reinterpret_cast<f32x4*>(gdst + idx + 4) = w1;
        }
      }
    }
  } else {
    const int total = TILE_E * A * D;
    for (int idx = tid; idx < total; idx += NTHREADS) {
      const int r = fdiv(idx, m.d), k = idx - r * D;
      const int el = fdiv(r, m.a), a = r - el * A;
      const int plane = fdiv(k, m.hw), cell = k - plane * HW;
      uint32_t v = 0;
      if (el < te_valid) {
        if (plane == 0)
          v = L.agrid[el * LBF_MAXCELLS + cell];
        else if (plane == 1)
          v = L.fgrid[el * LBF_MAXCELLS + cell];
        else
          v = L.acell[el * LBF_MAXA + a] == cell ? 1u : 0u;
      }
      const OT ov = small_int_to<OT>(v);
      if (ldst) ldst[(size_t)r * ldl + k] = ov;
      if (gdst && el < te_valid) gdst[idx] = ov;
    }
  }
}

__device__ __forceinline__ void lbf_write_legal(const LbfParams& p, int te_valid, uint8_t* __restrict__ g, int tid) {
  const int n = te_valid * p.A * LBF_NACT;
  for (int i = tid; i < n; i += NTHREADS) g[i] = 1;
}

__device__ __forceinline__ void zero_lds(void* base, size_t bytes, int tid) {
  uint32_t* w = reinterpret_cast<uint32_t*>(base);
  for (size_t i = tid; i < bytes / 4; i += NTHREADS) w[i] = 0u;
}

// ---------------------------------------------------------------- init ----

template <typename OT>
__global__ __launch_bounds__(NTHREADS) void lbf_init_kernel(LbfParams p, LbfMagic m, int32_t* __restrict__ state,
                                                            OT* __restrict__ obs, uint8_t* __restrict__ legal) {
  __shared__ __align__(16) uint8_t agrid[TILE_E * LBF_MAXCELLS];
  __shared__ __align__(16) uint8_t fgrid[TILE_E * LBF_MAXCELLS];
  __shared__ int acell[TILE_E * LBF_MAXA];
  const LbfLds L{agrid, fgrid, acell};
  const int tid = threadIdx.x;
  const int e0 = blockIdx.x * TILE_E;
  const int te_valid = min(TILE_E, p.E - e0);
  zero_lds(agrid, sizeof(agrid), tid);
  zero_lds(fgrid, sizeof(fgrid), tid);
  __syncthreads();
  if (tid < te_valid) {
    LbfEnv s{};
    lbf_reset(p, (uint64_t)(p.env_base + e0 + tid), 0, s);
    lbf_store(state, p, e0 + tid, s);
    lbf_paint(p, s, tid, L, true);
  }
  __syncthreads();
  if (obs) lbf_encode<OT>(p, m, te_valid, L, obs + (size_t)e0 * p.A * p.D, nullptr, 0, tid);
  if (legal) lbf_write_legal(p, te_valid, legal + (size_t)e0 * p.A * LBF_NACT, tid);
}

// ------------------------------------------------------------ env-only ----

template <typename OT>
__global__ __launch_bounds__(NTHREADS) void lbf_step_kernel(LbfParams p, LbfMagic m, int32_t* __restrict__ state,
                                                            uint64_t t0, int n_steps,
                                                            const int32_t* __restrict__ actions,
                                                            OT* __restrict__ obs, float* __restrict__ reward,
                                                            uint8_t* __restrict__ done, uint8_t* __restrict__ legal) {
  __shared__ __align__(16) uint8_t agrid[TILE_E * LBF_MAXCELLS];
  __shared__ __align__(16) uint8_t fgrid[TILE_E * LBF_MAXCELLS];
  __shared__ int acell[TILE_E * LBF_MAXA];
  const LbfLds L{agrid, fgrid, acell};
  const int tid = threadIdx.x;
  const int e0 = blockIdx.x * TILE_E;
  const int te_valid = min(TILE_E, p.E - e0);
  const int A = p.A;
  zero_lds(agrid, sizeof(agrid), tid);
  zero_lds(fgrid, sizeof(fgrid), tid);
  __syncthreads();
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  LbfEnv s{};
  if (envlane) {
    lbf_load(state, p, e, s);
    lbf_paint(p, s, tid, L, true);
  }
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    __syncthreads();  // the encoders of the previous step are done with the grids
    if (envlane) {
      int act[LBF_MAXA];
#pragma unroll
      for (int i = 0; i < LBF_MAXA; ++i)
        act[i] = i < A ? actions[((size_t)k * p.E + e) * A + i] : 0;
      lbf_paint(p, s, tid, L, false);
      float r;
      uint32_t d;
      lbf_transition(p, s, act, r, d);
      if (d) lbf_reset(p, (uint64_t)(p.env_base + e), t + 1, s);
      lbf_paint(p, s, tid, L, true);
      if (reward) reward[(size_t)k * p.E + e] = r;
      if (done) done[(size_t)k * p.E + e] = (uint8_t)d;
    }
    __syncthreads();
    if (obs) lbf_encode<OT>(p, m, te_valid, L, obs + ((size_t)k * p.E + e0) * A * p.D, nullptr, 0, tid);
    if (legal) lbf_write_legal(p, te_valid, legal + ((size_t)k * p.E + e0) * A * LBF_NACT, tid);
  }
  if (envlane) lbf_store(state, p, e, s);
}

// ------------------------------------------------------ fused rollout ----

template <int DT>
__global__ __launch_bounds__(NTHREADS) void lbf_run_kernel(LbfParams p, LbfMagic m, PolicyArgs pol,
                                                           int32_t* __restrict__ state, uint64_t t0, int n_steps,
                                                           TrajArgs out) {
  using T = typename DType<DT>::T;
  extern __shared__ __align__(16) uint8_t smem[];
  const RunLayout RL = make_run_layout(p.A, p.D, pol.H1, pol.H2, DT);
  const LbfLds L{smem + RL.off_agrid, smem + RL.off_fgrid, reinterpret_cast<int*>(smem + RL.off_acell)};
  int* act_lds = reinterpret_cast<int*>(smem + RL.off_act);
  T* xs = reinterpret_cast<T*>(smem + RL.off_x);
  T* h1 = reinterpret_cast<T*>(smem + RL.off_h1);
  T* h2 = reinterpret_cast<T*>(smem + RL.off_h2);
  float* lg = reinterpret_cast<float*>(smem + RL.off_logit);
  float* sc = reinterpret_cast<float*>(smem + RL.off_score);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TILE_E;
  const int te_valid = min(TILE_E, p.E - e0);
  const int A = p.A, D = p.D, NA = pol.NA, R = RL.R;
  const T* W1 = static_cast<const T*>(pol.W[0]);
  const T* W2 = static_cast<const T*>(pol.W[1]);
  const T* W3 = static_cast<const T*>(pol.W[2]);
  const T* b1 = static_cast<const T*>(pol.b[0]);
  const T* b2 = static_cast<const T*>(pol.b[1]);
  const T* b3 = static_cast<const T*>(pol.b[2]);
  T* gobs = static_cast<T*>(out.obs);

  zero_lds(smem, RL.total, tid);  // zero grids and the K padding of every operand tile
  __syncthreads();
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  const uint64_t genv = (uint64_t)(p.env_base + e);
  LbfEnv s{};
  if (envlane) {
    lbf_load(state, p, e, s);
    lbf_paint(p, s, tid, L, true);
  }
  __syncthreads();

  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    // o_t -> LDS operand tile (+ trajectory)
    lbf_encode<T>(p, m, te_valid, L, gobs ? gobs + ((size_t)k * p.E + e0) * A * D : nullptr, xs, RL.ldx, tid);
    __syncthreads();
    mlp_hidden<DT>(xs, RL.ldx, R, D, W1, b1, pol.H1, h1, RL.ld1, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_hidden<DT>(h1, RL.ld1, R, pol.H1, W2, b2, pol.H2, h2, RL.ld2, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_logits<DT>(h2, RL.ld2, R, pol.H2, W3, b3, NA, lg, MAX_NA, wave, NTHREADS / 64, lane);
    __syncthreads();
    // Gumbel scores per (row, action); every LBF action is legal
    for (int idx = tid; idx < R * NA; idx += NTHREADS) {
      const int r = fdiv(idx, m.na), a = idx - r * NA;
      const int el = fdiv(r, m.a), ag = r - el * A;
      if (el < te_valid) {
        const float g = action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t, ag, a);
        sc[r * MAX_NA + a] = action_score(lg[r * MAX_NA + a], g, true);
        if (out.logits) out.logits[((size_t)k * p.E + e0) * A * NA + idx] = lg[r * MAX_NA + a];
      }
    }
    __syncthreads();
    for (int r = tid; r < R; r += NTHREADS) {
      const int el = fdiv(r, m.a);
      if (el < te_valid) {
        int best = 0;
        float bs = -INFINITY;
        for (int a = 0; a < NA; ++a) {
          const float v = sc[r * MAX_NA + a];
          if (v > bs) {
            bs = v;
            best = a;
          }
        }
        act_lds[r] = best;
        if (out.actions) out.actions[((size_t)k * p.E + e0) * A + r] = best;
      }
    }
    __syncthreads();
    if (envlane) {
      int act[LBF_MAXA];
#pragma unroll
      for (int i = 0; i < LBF_MAXA; ++i) act[i] = i < A ? act_lds[tid * A + i] : 0;
      lbf_paint(p, s, tid, L, false);
      float r;
      uint32_t d;
      lbf_transition(p, s, act, r, d);
      if (d) lbf_reset(p, genv, t + 1, s);
      lbf_paint(p, s, tid, L, true);
      if (out.reward) out.reward[(size_t)k * p.E + e] = r;
      if (out.done) out.done[(size_t)k * p.E + e] = (uint8_t)d;
    }
    __syncthreads();
  }
  if (out.obs_last)
    lbf_encode<T>(p, m, te_valid, L, static_cast<T*>(out.obs_last) + (size_t)e0 * A * D, nullptr, 0, tid);
  if (envlane) lbf_store(state, p, e, s);
}

// ------------------------------------------------------------ launchers ----

static dim3 tiles(int E) { return dim3((unsigned)((E + TILE_E - 1) / TILE_E)); }

hipError_t launch_lbf_init(const LbfParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal,
                           hipStream_t s) {
  const LbfMagic m = make_magic(p, LBF_NACT);
  if (obs_dt == DT_F32)
    lbf_init_kernel<float><<<tiles(p.E), NTHREADS, 0, s>>>(p, m, state, static_cast<float*>(obs), legal);
  else
    lbf_init_kernel<uint16_t><<<tiles(p.E), NTHREADS, 0, s>>>(p, m, state, static_cast<uint16_t*>(obs), legal);
  return hipGetLastError();
}

hipError_t launch_lbf_step(const LbfParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                           void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s) {
  const LbfMagic m = make_magic(p, LBF_NACT);
  if (obs_dt == DT_F32)
    lbf_step_kernel<float><<<tiles(p.E), NTHREADS, 0, s>>>(p, m, state, t0, n_steps, actions,
                                                           static_cast<float*>(obs), reward, done, legal);
  else
    lbf_step_kernel<uint16_t><<<tiles(p.E), NTHREADS, 0, s>>>(p, m, state, t0, n_steps, actions,
                                                              static_cast<uint16_t*>(obs), reward, done, legal);
  return hipGetLastError();
}

hipError_t launch_lbf_run(const LbfParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                          const TrajArgs& out, hipStream_t s) {
  const LbfMagic m = make_magic(p, pol.NA);
  const RunLayout RL = make_run_layout(p.A, p.D, pol.H1, pol.H2, pol.dt);
  if (pol.dt == DT_F32) {
    static bool attr_f32 = false;
    if (!attr_f32) {
      hipError_t e = hipFuncSetAttribute((const void*)lbf_run_kernel<DT_F32>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)MAX_LDS_BYTES);
      if (e != hipSuccess) return e;
      attr_f32 = true;
    }
    lbf_run_kernel<DT_F32><<<tiles(p.E), NTHREADS, RL.total, s>>>(p, m, pol, state, t0, n_steps, out);
  } else {
    static bool attr_bf16 = false;
    if (!attr_bf16) {
      hipError_t e = hipFuncSetAttribute((const void*)lbf_run_kernel<DT_BF16>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)MAX_LDS_BYTES);
      if (e != hipSuccess) return e;
      attr_bf16 = true;
    }
    lbf_run_kernel<DT_BF16><<<tiles(p.E), NTHREADS, RL.total, s>>>(p, m, pol, state, t0, n_steps, out);
  }
  return hipGetLastError();
}

}  // namespace rl
