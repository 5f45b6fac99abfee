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
#include "rl_regmlp.h"
#include "rl_sample.h"

namespace rl {

RL_STAMP_TABLE


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
template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_paint(const LbfParams& p, const LbfEnv& s, int el, const LbfLds& L, bool on) {
  constexpr int CM = LBF_MAXCELLS - 1;
  const int A = AC ? AC : p.A, F = FC ? FC : p.F;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A) {
      L.agrid[el * LBF_MAXCELLS + (s.acell[i] & CM)] = on ? (uint8_t)s.alevel[i] : 0;
      if (on) L.acell[el * LBF_MAXA + i] = s.acell[i];
    }
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F && !((s.eaten >> j) & 1u))
      L.fgrid[el * LBF_MAXCELLS + (s.fcell[j] & CM)] = on ? (uint8_t)s.flevel[j] : 0;
}

// Observation rows of the tile: element (r, k) with r = el * A + a.
// gdst: the tile's first element in global [.., A, D] (or null); ldst: LDS
// operand tile with leading dimension ldl (or null).  Rows of envs beyond
// te_valid are zero in LDS and not written to global memory.
template <typename OT, int TE = TILE_E, int NT = NTHREADS>
__device__ __forceinline__ void lbf_encode(const LbfParams& p, const LbfMagic& m, int te_valid, const LbfLds& L,
                                           OT* __restrict__ gdst, OT* __restrict__ ldst, int ldl, int tid) {
  const int A = p.A, D = p.D, HW = p.HW;
  if ((D & 7) == 0 && (HW & 7) == 0) {
    const int nvec = TE * A * (D >> 3);
    for (int v = tid; v < nvec; v += NT) {
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
    const int total = TE * A * D;
    for (int idx = tid; idx < total; idx += NT) {
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

// lbf_encode with the tile shape known at compile time (D and the grid size
// multiples of 8): every 16-byte vector of the tile is handled by one thread
// in a fully unrolled loop, so the LDS grid reads of all iterations are in
// flight together.
template <typename OT, int TE, int A, int D, int NT>
__device__ __forceinline__ void lbf_encode_ct(int te_valid, const LbfLds& L, OT* __restrict__ gdst,
                                              OT* __restrict__ ldst, int ldl, int tid) {
  constexpr int HW = D / 3;
  static_assert(D % 8 == 0 && HW % 8 == 0, "vectorised encoder needs 8-aligned planes");
  constexpr int NV = TE * A * D / 8;
  constexpr int ITERS = (NV + NT - 1) / NT;
  uint64_t bytes[ITERS];
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int v = tid + it * NT;
    bytes[it] = 0;
    if (v < NV) {
      const int idx = v * 8;
      const int r = idx / D, k = idx - r * D;
      const int el = r / A, a = r - el * A;
      const int plane = k / HW, cell0 = k - plane * HW;
      if (el < te_valid) {
        if (plane == 0) {
          bytes[it] = *reinterpret_cast<const uint64_t*>(L.agrid + el * LBF_MAXCELLS + cell0);
        } else if (plane == 1) {
          bytes[it] = *reinterpret_cast<const uint64_t*>(L.fgrid + el * LBF_MAXCELLS + cell0);
        } else {
          const int c = L.acell[el * LBF_MAXA + a] - cell0;
          if (c >= 0 && c < 8) bytes[it] = 1ull << (8 * c);
        }
      }
    }
  }
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int v = tid + it * NT;
    if (v >= NV) continue;
    const int idx = v * 8;
    const int r = idx / D, k = idx - r * D;
    const int el = r / A;
    OT vals[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) vals[q] = small_int_to<OT>((uint32_t)(bytes[it] >> (8 * q)) & 0xffu);
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
}

template <int NT = NTHREADS>
__device__ __forceinline__ void lbf_write_legal(const LbfParams& p, int te_valid, uint8_t* __restrict__ g, int tid) {
  const int n = te_valid * p.A * LBF_NACT;
  for (int i = tid; i < n; i += NT) g[i] = 1;
}

// ---------------------------------------------------------------- init ----

// RESET: draw every env's first episode (step 0) and store it; otherwise
// only observe the stored states.
template <typename OT, bool RESET = true>
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
    if constexpr (RESET) {
      lbf_reset(p, (uint64_t)(p.env_base + e0 + tid), 0, s);
      lbf_store(state, p, e0 + tid, s);
    } else {
      lbf_load(state, p, e0 + tid, s);
    }
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
  __shared__ int32_t act_lds[ACT_CHUNK * TILE_E * LBF_MAXA];
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
  for (int k0 = 0; k0 < n_steps; k0 += ACT_CHUNK) {
    const int nk = min(ACT_CHUNK, n_steps - k0);
    __syncthreads();  // the previous chunk's actions are consumed
    // no global loads inside the step loop: a load there would wait for every earlier trajectory store
    stage_actions<TILE_E * LBF_MAXA, NTHREADS>(actions, p.E, e0, te_valid * A, A, k0, nk, act_lds, tid);
    for (int kk = 0; kk < nk; ++kk) {
      const int k = k0 + kk;
      const uint64_t t = t0 + (uint64_t)k;
      __syncthreads();  // the encoders of the previous step are done with the grids (and the actions are staged)
      if (envlane) {
        int act[LBF_MAXA];
#pragma unroll
        for (int i = 0; i < LBF_MAXA; ++i) act[i] = i < A ? act_lds[kk * TILE_E * LBF_MAXA + tid * A + i] : 0;
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
  const int A = p.A, D = p.D, NOUT = pol.NA, NA = NOUT - pol.VH, R = RL.R;
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
  int tkind[LBF_MAXA] = {-1, -1, -1, -1};  // heuristic teammates of this env's agents (-1: the policy)
  int start[LBF_MAXA] = {0, 0, 0, 0};       // the agents' cells at the start of the current episode
  if (envlane) {
    lbf_load(state, p, e, s);
    lbf_paint(p, s, tid, L, true);
    if (out.teammates) {
#pragma unroll
      for (int i = 0; i < LBF_MAXA; ++i) {
        const int kd = i < A ? out.teammates[(size_t)e * A + i] : -1;
        tkind[i] = (kd >= 0 && kd < LBF_NHEUR) ? kd : -1;
      }
      lbf_start_cells(p, genv, t0, s, start);
    }
  }
  __syncthreads();

  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    // o_t -> LDS operand tile (+ trajectory)
    lbf_encode<T>(p, m, te_valid, L, gobs ? gobs + ((size_t)k * p.E + e0) * A * D : nullptr, xs, RL.ldx, tid);
    __syncthreads();
    mlp_input_layer<DT>(xs, RL.ldx, nullptr, R, D, W1, b1, pol.H1, h1, RL.ld1, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_hidden<DT>(h1, RL.ld1, R, pol.H1, W2, b2, pol.H2, h2, RL.ld2, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_logits<DT>(h2, RL.ld2, R, pol.H2, W3, b3, NOUT, lg, MAX_NA, wave, NTHREADS / 64, lane);
    __syncthreads();
    if (out.teammates) {  // heuristic agents: logits 0 for their action, -inf for the others
      if (envlane) {
#pragma unroll
        for (int i = 0; i < LBF_MAXA; ++i)
          if (tkind[i] >= 0) {
            const int act = lbf_heuristic_action(p, s, i, tkind[i], start[i]);
            float* l = lg + (tid * A + i) * MAX_NA;
            for (int a = 0; a < NA; ++a) l[a] = a == act ? 0.f : -INFINITY;
          }
      }
      __syncthreads();
    }
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
        const size_t gr = ((size_t)k * p.E + e0) * A + r;
        if (out.actions) out.actions[gr] = best;
        if (out.logp) out.logp[gr] = log_softmax_at(lg + r * MAX_NA, NA, best);
        if (out.value) out.value[gr] = lg[r * MAX_NA + NA];
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
      if (d) {
        lbf_reset(p, genv, t + 1, s);
#pragma unroll
        for (int i = 0; i < LBF_MAXA; ++i) start[i] = s.acell[i];
      }
      lbf_paint(p, s, tid, L, true);
      if (out.reward) out.reward[(size_t)k * p.E + e] = r;
      if (out.done) out.done[(size_t)k * p.E + e] = (uint8_t)d;
    }
    __syncthreads();
  }
  if (out.obs_last || out.value_last)
    lbf_encode<T>(p, m, te_valid, L, out.obs_last ? static_cast<T*>(out.obs_last) + (size_t)e0 * A * D : nullptr,
                  out.value_last ? xs : nullptr, RL.ldx, tid);
  if (out.value_last) {  // V(o_{t0+T}): one more pass of the network over the final observation
    __syncthreads();
    mlp_input_layer<DT>(xs, RL.ldx, nullptr, R, D, W1, b1, pol.H1, h1, RL.ld1, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_hidden<DT>(h1, RL.ld1, R, pol.H1, W2, b2, pol.H2, h2, RL.ld2, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_logits<DT>(h2, RL.ld2, R, pol.H2, W3, b3, NOUT, lg, MAX_NA, wave, NTHREADS / 64, lane);
    __syncthreads();
    for (int r = tid; r < te_valid * A; r += NTHREADS) out.value_last[(size_t)e0 * A + r] = lg[r * MAX_NA + NA];
  }
  if (envlane) lbf_store(state, p, e, s);
}

// ------------------------------------------- population rollout ----
//
// rollout_run_pop: the rollout of lbf_run_kernel where agent a of env e acts
// with policy pidx[e * A + a] of a population of n_pol networks of one shape,
// stacked in memory (the ego agent and its teammates of the ad hoc teamwork
// objective, Section 3).  At the start each workgroup sorts its rows by policy
// (the assignment is fixed for the rollout); every step it runs the three MFMA
// layers once per policy present, on that policy's rows only (rows gathered
// by index into the operand), and scatters the logits back to their rows.
// Cost per step grows with the number of distinct policies in a tile.  An
// index outside 0..n_pol-1 selects policy 0.
size_t lbf_pop_lds_bytes(const LbfParams& p, const PolicyArgs& pol) {
  const RunLayout RL = make_run_layout(p.A, p.D, pol.H1, pol.H2, pol.dt);
  const size_t off = (RL.total + 15) & ~(size_t)15;
  return off + (size_t)(3 * RL.R + 17) * 4 + (size_t)RL.R * MAX_NA * 4;
}

__device__ __forceinline__ bool pop_two_slots(const int32_t* __restrict__ pidx, int e0, int te_valid, int A,
                                              int n_pol, int& q0, int& q1);

// skip_two: tiles whose agents use at most two policies are left alone (the
// two-policy kernel has run them).
template <int DT, bool PK>
__global__ __launch_bounds__(NTHREADS) void lbf_run_pop_kernel(LbfParams p, LbfMagic m, PolicyArgs pol, int n_pol,
                                                               const int32_t* __restrict__ pidx,
                                                               int32_t* __restrict__ state, uint64_t t0,
                                                               int n_steps, TrajArgs out, int skip_two) {
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
  const int R = RL.R;
  int* order = reinterpret_cast<int*>(smem + ((RL.total + 15) & ~(size_t)15));  // R + 16 row indices, by policy
  int* gstart = order + R + 16;                                                  // group g: order[gstart[g] .. gstart[g+1])
  int* gpid = gstart + R + 1;                                                    // policy of group g
  float* lgc = reinterpret_cast<float*>(gpid + R);                               // a group's logits, compact rows
  __shared__ int ngroups;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TILE_E;
  const int te_valid = min(TILE_E, p.E - e0);
  const int A = p.A, D = p.D, NA = pol.NA, H1 = pol.H1, H2 = pol.H2;
  const int dims4[4] = {D, H1, H2, NA};
  T* gobs = static_cast<T*>(out.obs);
  if (skip_two) {
    __shared__ int two;
    if (tid == 0) {
      int q0, q1;
      two = pop_two_slots(pidx, e0, te_valid, A, n_pol, q0, q1) ? 1 : 0;
    }
    __syncthreads();
    if (two) return;
  }

  zero_lds(smem, RL.total, tid);  // zero grids and the K padding of every operand tile
  if (tid == 0) {
    // group the live rows (te_valid * A <= 64) by policy, in order of first appearance
    const int nr = te_valid * A;
    uint64_t left = nr >= 64 ? ~0ull : ((1ull << nr) - 1ull);
    int ng = 0, pos = 0;
    while (left) {
      const int r0 = __builtin_ctzll(left);
      const int raw0 = pidx[(size_t)e0 * A + r0];
      const int id0 = (unsigned)raw0 < (unsigned)n_pol ? raw0 : 0;
      gpid[ng] = id0;
      gstart[ng] = pos;
      for (int r = r0; r < nr; ++r) {
        if (!((left >> r) & 1ull)) continue;
        const int raw = pidx[(size_t)e0 * A + r];
        if (((unsigned)raw < (unsigned)n_pol ? raw : 0) == id0) {
          order[pos++] = r;
          left &= ~(1ull << r);
        }
      }
      ++ng;
    }
    gstart[ng] = pos;
    for (int i = pos; i < R + 16; ++i) order[i] = 0;  // padding rows of the last MFMA row tile
    ngroups = ng;
  }
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
  const int ng = ngroups;

  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    lbf_encode<T>(p, m, te_valid, L, gobs ? gobs + ((size_t)k * p.E + e0) * A * D : nullptr, xs, RL.ldx, tid);
    __syncthreads();
    for (int g = 0; g < ng; ++g) {
      const int g0 = gstart[g], cnt = gstart[g + 1] - g0;
      const int R16 = (cnt + 15) & ~15;
      const size_t q = (size_t)gpid[g];
      const T* W1 = static_cast<const T*>(pol.W[0]) + q * H1 * D;
      const T* W2 = static_cast<const T*>(pol.W[1]) + q * H2 * H1;
      const T* W3 = static_cast<const T*>(pol.W[2]) + q * NA * H2;
      const T* b1 = static_cast<const T*>(pol.b[0]) + q * H1;
      const T* b2 = static_cast<const T*>(pol.b[1]) + q * H2;
      const T* b3 = static_cast<const T*>(pol.b[2]) + q * NA;
      // PK: policy q's fragment-major copy starts q whole packed policies in
      const size_t pq = PK ? q * (packed_layer_offset(dims4, 2) + packed_layer_bytes(NA, H2)) : 0;
      const T* Wp1 = PK ? reinterpret_cast<const T*>(static_cast<const uint8_t*>(pol.Wp[0]) + pq) : nullptr;
      const T* Wp2 = PK ? reinterpret_cast<const T*>(static_cast<const uint8_t*>(pol.Wp[1]) + pq) : nullptr;
      const T* Wp3 = PK ? reinterpret_cast<const T*>(static_cast<const uint8_t*>(pol.Wp[2]) + pq) : nullptr;
      mlp_input_layer<DT, PK>(xs, RL.ldx, order + g0, R16, D, W1, b1, H1, h1, RL.ld1, wave, NTHREADS / 64, lane, Wp1);
      __syncthreads();
      mlp_hidden<DT, PK>(h1, RL.ld1, R16, H1, W2, b2, H2, h2, RL.ld2, wave, NTHREADS / 64, lane, Wp2);
      __syncthreads();
      mlp_logits<DT, PK>(h2, RL.ld2, R16, H2, W3, b3, NA, lgc, MAX_NA, wave, NTHREADS / 64, lane, Wp3);
      __syncthreads();
      for (int idx = tid; idx < cnt * NA; idx += NTHREADS) {
        const int r = idx / NA, a = idx - r * NA;
        lg[order[g0 + r] * MAX_NA + a] = lgc[r * MAX_NA + a];
      }
      __syncthreads();
    }
    // Gumbel scores per (row, action); every LBF action is legal
    for (int idx = tid; idx < R * NA; idx += NTHREADS) {
      const int r = fdiv(idx, m.na), a = idx - r * NA;
      const int el = fdiv(r, m.a), ag = r - el * A;
      if (el < te_valid) {
        const float gn = action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t, ag, a);
        sc[r * MAX_NA + a] = action_score(lg[r * MAX_NA + a], gn, true);
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

// ------------------------------------ fused rollout, weights in registers ----

// Field-wise copy of the A agents and F foods of an env state (a whole-struct
// copy to or from LDS would turn the register copy into private memory).
template <int A, int F>
__device__ __forceinline__ void lbf_copy(LbfEnv& d, const LbfEnv& s) {
#pragma unroll
  for (int i = 0; i < A; ++i) {
    d.acell[i] = s.acell[i];
    d.alevel[i] = s.alevel[i];
  }
#pragma unroll
  for (int j = 0; j < F; ++j) {
    d.fcell[j] = s.fcell[j];
    d.flevel[j] = s.flevel[j];
  }
  d.eaten = s.eaten;
  d.steps = s.steps;
  d.den = s.den;
}

constexpr int NOISE_STEPS = 16;

// Write (on) or erase (!on) env el's non-zero observation features directly
// in the MFMA operand tile: for each of its A rows, plane 0 holds every
// agent's level at its cell, plane 1 every uneaten food's level, plane 2 a 1
// at the row's own agent.  Cell ids are clamped into the grid so that a
// malformed caller-supplied state cannot address outside the row.
// AMT > 0: the tile's rows are agent-major, row i * AMT + el (AMT envs per
// tile); otherwise env-major, row el * A + i.
template <typename T, int A, int F, int AMT = 0>
__device__ __forceinline__ void lbf_paint_tile(const LbfEnv& s, int el, T* xs, int ldx, int HW, bool on) {
  const uint32_t cmax = (uint32_t)HW - 1u;
  const T one = on ? small_int_to<T>(1u) : (T)0;
#pragma unroll
  for (int i = 0; i < A; ++i) {
    T* xr = xs + (AMT ? i * AMT + el : el * A + i) * ldx;
#pragma unroll
    for (int q = 0; q < A; ++q) xr[min((uint32_t)s.acell[q], cmax)] = on ? small_int_to<T>((uint32_t)s.alevel[q]) : (T)0;
#pragma unroll
    for (int j = 0; j < F; ++j)  // an eaten food writes 0 at its own (distinct) cell: no branch
      xr[HW + min((uint32_t)s.fcell[j], cmax)] =
          (on && !((s.eaten >> j) & 1u)) ? small_int_to<T>((uint32_t)s.flevel[j]) : (T)0;
    xr[2 * HW + min((uint32_t)s.acell[i], cmax)] = one;
  }
}

// Copy the tile's live observation rows from LDS to global [.., A, D] rows
// with 16-byte vectors (g == nullptr: no copy).  CLEAR: each vector is
// zeroed in LDS after it is read, which leaves the tile blank for the next
// paint.  The vectors of a thread go in groups of G: all reads of a group
// are issued before its first store, so a group waits for LDS once.
// AMT > 0: the LDS rows are agent-major (row a * AMT + el, AMT envs of A
// agents) and go to global rows el * A + a.
template <typename T, int R, int D, int LDX, int NT, bool CLEAR = false, int G = 4, int AMT = 0, int A = 1>
__device__ __forceinline__ void copy_obs_rows(T* xs, T* __restrict__ g, int rows_live, int tid) {
  constexpr int VE = 16 / sizeof(T);
  static_assert(AMT == 0 || D % VE == 0, "agent-major tiles need whole-vector rows");
  if constexpr (D % VE != 0 && LDX == D) {
    // Rows that are not whole vectors, unpadded in LDS as in global memory:
    // the tile is one contiguous block of R * D elements, copied as 16-byte
    // vectors; the vector that ends the live rows goes element by element.
    static_assert((R * D) % VE == 0, "the tile must be whole 16-byte vectors");
    constexpr int NV = R * D / VE;
    constexpr int IT = (NV + NT - 1) / NT;
    const int nlive = rows_live * D;
#pragma unroll
    for (int i0 = 0; i0 < IT; i0 += G) {
      u32x4 val[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int v = tid + (i0 + j) * NT;
        if (i0 + j < IT && (NV % NT == 0 || v < NV)) val[j] = *reinterpret_cast<const u32x4*>(xs + v * VE);
      }
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int v = tid + (i0 + j) * NT, e0 = v * VE;
        if (i0 + j < IT && (NV % NT == 0 || v < NV) && e0 < nlive) {
          if (g) {
            if (e0 + VE <= nlive) {
              *reinterpret_cast<u32x4*>(g + e0) = val[j];
            } else {
#pragma unroll
              for (int q = 0; q < VE; ++q)
                if (e0 + q < nlive) g[e0 + q] = xs[e0 + q];
            }
          }
          if constexpr (CLEAR) *reinterpret_cast<u32x4*>(xs + e0) = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
    return;
  } else if constexpr (D % VE != 0) {
    // Rows that are not whole vectors (e.g. the 7x7 grid's 147 features): the
    // tile's rows are contiguous in global memory, so the tile goes out as
    // R * D elements in 16-byte vectors, each gathered element by element
    // from the (padded) LDS rows; the vector that ends the live rows is
    // stored element by element.
    static_assert((R * D) % VE == 0, "the tile must be whole 16-byte vectors");
    constexpr int NV = R * D / VE;
    constexpr int IT = (NV + NT - 1) / NT;
    const int nlive = rows_live * D;
#pragma unroll
    for (int i0 = 0; i0 < IT; i0 += G) {
      uint32_t w[G][4];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int v = tid + (i0 + j) * NT;
#pragma unroll
        for (int q = 0; q < 4; ++q) w[j][q] = 0u;
        if (i0 + j < IT && (NV % NT == 0 || v < NV)) {
#pragma unroll
          for (int q = 0; q < VE; ++q) {
            const int el = v * VE + q, r = el / D, c = el - r * D;
            const T x = xs[r * LDX + c];
            if constexpr (sizeof(T) == 2)
              w[j][q >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, x) << (16 * (q & 1));
            else
              w[j][q] = __builtin_bit_cast(uint32_t, x);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int v = tid + (i0 + j) * NT;
        const int e0 = v * VE;
        if (i0 + j < IT && (NV % NT == 0 || v < NV) && e0 < nlive) {
          if (g) {
            if (e0 + VE <= nlive) {
              *reinterpret_cast<u32x4*>(g + e0) = u32x4{w[j][0], w[j][1], w[j][2], w[j][3]};
            } else {
#pragma unroll
              for (int q = 0; q < VE; ++q)
                if (e0 + q < nlive) {
                  const uint32_t bits = sizeof(T) == 2 ? (w[j][q >> 1] >> (16 * (q & 1))) & 0xffffu : w[j][q];
                  if constexpr (sizeof(T) == 2)
                    g[e0 + q] = __builtin_bit_cast(T, (uint16_t)bits);
                  else
                    g[e0 + q] = __builtin_bit_cast(T, bits);
                }
            }
          }
          if constexpr (CLEAR) {
#pragma unroll
            for (int q = 0; q < VE; ++q) {
              const int el = e0 + q, r = el / D, c = el - r * D;
              if (el < nlive) xs[r * LDX + c] = (T)0;
            }
          }
        }
      }
    }
    return;
  }
  constexpr int VPR = D / VE > 0 ? D / VE : 1;
  constexpr int NV = R * VPR;
  constexpr int IT = (NV + NT - 1) / NT;
#pragma unroll
  for (int i0 = 0; i0 < IT; i0 += G) {
    u32x4 val[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int v = tid + (i0 + j) * NT;
      const int r = v / VPR, c = (v - r * VPR) * VE;
      // rows past rows_live are inside the tile: reading them is harmless
      if (i0 + j < IT && (NV % NT == 0 || v < NV)) val[j] = *reinterpret_cast<const u32x4*>(xs + r * LDX + c);
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int v = tid + (i0 + j) * NT;
      const int r = v / VPR, c = (v - r * VPR) * VE;
      const int gr = AMT ? (r % AMT) * A + r / AMT : r;  // global row of LDS row r
      const bool live = AMT ? (r % AMT) * A < rows_live : r < rows_live;
      if (i0 + j < IT && (NV % NT == 0 || v < NV) && live) {
        if (g) *reinterpret_cast<u32x4*>(g + (size_t)gr * D + c) = val[j];
        if constexpr (CLEAR) *reinterpret_cast<u32x4*>(xs + r * LDX + c) = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
}

// The value of lane l in the partner group of 16 lanes (groups 0 <-> 1, 2 <-> 3).
__device__ __forceinline__ float partner16(float x) {
  const auto pr = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(((threadIdx.x >> 4) & 1) ? pr[0] : pr[1]);
}

// log pi(a) of a row of the transposed layer 3, whose NA <= 8 action logits
// sit in two partner lane groups (actions 4 g + r in logit[r] of group g):
// a float32 log-softmax with the max and the exp-sum combined over the pair.
// Both lanes of a pair return the same value (a sum of two floats commutes).
template <int NA>
__device__ __forceinline__ float row_log_pi(const float (&logit)[4], int g, int a) {
  float m = -INFINITY;
#pragma unroll
  for (int r = 0; r < 4; ++r)
    if (4 * g + r < NA) m = fmaxf(m, logit[r]);
  m = fmaxf(m, partner16(m));
  float sum = 0.f, c = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (4 * g + r < NA) sum += expf(logit[r] - m);
    if (4 * g + r == a) c = logit[r];
  }
  sum += partner16(sum);
  const float oc = partner16(c);
  return ((a >> 2) == g ? c : oc) - (m + logf(sum));
}

// Same step as lbf_run_kernel for compile-time policy sizes, restructured for
// latency:
//   * layer-1/2 weights live in registers (S1: layer 1 streamed from the
//     packed copy) and layer 3 in LDS for the whole rollout; layers are
//     computed transposed so each lane ends with four consecutive outputs of
//     one row, with all of a layer's LDS operands read ahead of its MFMAs;
//   * observations are painted by the env lanes straight into the layer-1
//     operand tile (only the non-zero features are written); with two tiles
//     (one M tile) the other waves copy o_t to the trajectory while the env
//     wave steps, otherwise all waves copy it while the layer-2 MFMAs run;
//     either way the copy clears the tile behind it;
//   * the Philox action draws of NOISE_STEPS steps are made in one batch by
//     all lanes; the Gumbel noise of step k+1 is evaluated from them by the
//     other waves while the env wave steps the envs at step k;
//   * one "env wave" (wave 0, at raised issue priority: its serial section is
//     the longest stage) computes layer 3, the Gumbel argmax (in registers
//     plus one v_permlane16_swap) and steps the TE envs, drawing the reset
//     blocks of ended episodes on idle lanes in parallel; with several M
//     tiles, wave m computes layer 3 and the argmax of tile m and the env
//     wave steps the envs after a barrier.
// TE envs per workgroup; the launch bounds let MINB workgroups share a CU.
// VH: layer 3 has one more output, the value head V(o) of an actor-critic
// network, written with log pi of each sampled action and, after the last
// step, V of the final observation.
// TM: agents whose teammates entry is a heuristic kind act with that
// heuristic (evaluated by the env lanes) instead of the network.
template <int DT, int GH, int GW, int H1, int H2, int NA, int A, int F, int TE, int NW, int MINB, bool VH = false,
          bool TM = false, bool S1 = false>
__global__ __launch_bounds__(NW * 64, MINB) void lbf_rollout_kernel(LbfParams p, PolicyArgs pol,
                                                                    int32_t* __restrict__ state, uint64_t t0,
                                                                    int n_steps, TrajArgs out) {
  using T = typename DType<DT>::T;
  using B = typename BOperand<DT>::type;
  constexpr int HW = GH * GW, D = 3 * HW;
  constexpr int NT = NW * 64;
  constexpr int R = TE * A;
  constexpr int MT = (R + 15) / 16;
  constexpr int RP = MT * 16;
  // With one M tile and A dividing 16, env e lives in lane e * A of wave 0,
  // which after the argmax already holds its first agent's action; the
  // others come from the next lanes by DPP row shifts (no LDS round trip).
  constexpr bool DIRECT = MT == 1 && 16 % A == 0;
  constexpr int ESTRIDE = DIRECT ? A : 1;  // lane of env e = e * ESTRIDE
  constexpr bool SPLIT3 = MT > 1 && MT <= NW;
  constexpr int LDX = lds_ld<DT>(D), LD1 = lds_ld<DT>(H1), LD2 = lds_ld<DT>(H2);
  constexpr int K3 = round_up(H2, DType<DT>::KS) / DType<DT>::KS;
  // LEAN: the resident weights leave too few registers for the env step, so
  // the biases and the env state wait in LDS between uses.
  constexpr int REG_BUDGET = 512 / ((NW * MINB + 3) / 4);
  // S1: layer 1 streams its weights from L2 (StreamLayer) instead of holding them
  constexpr int L1REGS = S1 ? StreamLayer<DT_BF16, D, H1, NW>::WREGS : RegLayer<DT, D, H1, NW>::WREGS;
  constexpr bool LEAN = S1 || L1REGS + RegLayer<DT, H1, H2, NW>::WREGS + 160 > REG_BUDGET;
  using L1T = std::conditional_t<S1, StreamLayer<DT_BF16, D, H1, NW, LEAN>, RegLayer<DT, D, H1, NW, LEAN>>;
  static_assert(!S1 || DT == DT_BF16, "streamed layer 1: bf16");
  constexpr int NOUT = NA + (VH ? 1 : 0);  // layer-3 outputs: the actions, then the value
  static_assert(NA <= 8 && NOUT <= 8, "one Philox block of action noise per row; outputs in two lane groups");
  static_assert(!(VH && LEAN), "the value head runs on shapes whose env state stays in registers");
  static_assert(!(VH && TM), "heuristic teammates run without the value head");
  static_assert(TE <= 64, "env lanes live in wave 0");
  static_assert(TE * ((2 * A + 2 * F + 7) / 8) <= 64, "one lane per reset block");

  // DB (one M tile): two observation tiles; o_t is read by layer 1 from tile
  // t % 2 while the env wave paints o_{t+1} onto the other one, and the other
  // waves copy o_t to the trajectory (clearing it) while the env wave steps.
  // Otherwise one tile, copied under the layer-2 MFMAs.
  constexpr bool DB = MT == 1;
  __shared__ __align__(16) T xs[DB ? 2 : 1][RP * LDX];
  __shared__ __align__(16) T h1s[RP * LD1];
  __shared__ __align__(16) T h2s[RP * LD2];
  __shared__ __align__(16) B w3s[K3 * 64];
  __shared__ int act_s[RP];
  __shared__ uint32_t words[NOISE_STEPS * RP * 8];  // action Philox draws per (step, row)
  __shared__ __align__(16) float nz[2][RP * 8];     // Gumbel noise per (row, action), by step parity
  __shared__ uint32_t rdraw[TE * LBF_MAX_DRAWS];    // reset draws of envs being reset
  __shared__ __align__(16) float bias_s[LEAN ? H1 + H2 : 4];
  __shared__ LbfEnv env_s[LEAN ? TE : 1];
  __shared__ int tk_s[TM ? RP : 1];  // TM: heuristic kind of each row (-1: the network)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE;
  const int te_valid = min(TE, p.E - e0);
  const int E = p.E;
  constexpr int ew = 0;  // the env wave
  constexpr int nd = 2 * A + 2 * F;
  constexpr int nblk = (nd + 7) >> 3;
  // Gumbel noise of (row, action) items i0, i0 + stride, ... from the Philox
  // draws of batch slot sn
  auto draw_noise = [&](int sn, float* noise, int i0, int stride) {
    for (int i = i0; i < R * NA; i += stride) {
      const int row = i / NA, a = i - row * NA;
      noise[row * 8 + a] = gumbel24(words[(sn * RP + row) * 8 + a] >> 8);
    }
  };

  L1T L1;
  RegLayer<DT, H1, H2, NW, LEAN> L2;
  if constexpr (LEAN) {
    for (int i = tid; i < H1 + H2; i += NT)
      bias_s[i] = DType<DT>::to_f32(i < H1 ? static_cast<const T*>(pol.b[0])[i] : static_cast<const T*>(pol.b[1])[i - H1]);
  }
  if constexpr (S1)
    L1.load(static_cast<const T*>(pol.b[0]), wave, lane, static_cast<const T*>(pol.Wp[0]));
  else
    L1.load(static_cast<const T*>(pol.W[0]), static_cast<const T*>(pol.b[0]), wave, lane);
  L2.load(static_cast<const T*>(pol.W[1]), static_cast<const T*>(pol.b[1]), wave, lane);
  if (tid < 64) {
    const int n = lane & 15;
    const T* row = static_cast<const T*>(pol.W[2]) + (size_t)(n < NOUT ? n : 0) * H2;
#pragma unroll
    for (int ks = 0; ks < K3; ++ks) w3s[ks * 64 + lane] = load_operand_global<DT, H2>(row, H2, ks, lane, n < NOUT);
  }
  float b3r[4];  // bias of outputs 4 * (lane / 16) + r, for the transposed layer 3
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int act = 4 * (lane >> 4) + r;
    b3r[r] = act < NOUT ? DType<DT>::to_f32(static_cast<const T*>(pol.b[2])[act]) : 0.f;
  }

  if constexpr (TM) {
    for (int row = tid; row < RP; row += NT) {
      const int kd = row < te_valid * A ? out.teammates[(size_t)e0 * A + row] : -1;
      tk_s[row] = (kd >= 0 && kd < LBF_NHEUR) ? kd : -1;
    }
  }
  // zero the operand tiles (their K padding and unused rows stay zero)
  for (int i = tid; i < (DB ? 2 : 1) * RP * LDX; i += NT) (&xs[0][0])[i] = (T)0;
  for (int i = tid; i < RP * LD1; i += NT) h1s[i] = (T)0;
  for (int i = tid; i < RP * LD2; i += NT) h2s[i] = (T)0;
  __syncthreads();
  const int el = lane / ESTRIDE;  // env of this lane (when it is an env lane)
  const bool envlane = wave == ew && lane % ESTRIDE == 0 && el < te_valid;
  const int e = e0 + el;
  // The env state; when LEAN it is kept in LDS between steps and reloaded by
  // the whole env wave, so it is dead (not holding registers) during the MLP.
  LbfEnv s{};
  int start[TM ? LBF_MAXA : 1] = {};  // TM: the agents' cells at the start of the current episode
  if (envlane) {
    lbf_load<A, F>(state, p, e, s);
    lbf_paint_tile<T, A, F>(s, el, xs[0], LDX, HW, true);
    if constexpr (LEAN) lbf_copy<A, F>(env_s[el], s);
    if constexpr (TM) lbf_start_cells<A, F>(p, (uint64_t)(p.env_base + e), t0, s, start);
  }
  // Let the prologue loads land here, once (see lbf_env_kernel).
  __builtin_amdgcn_s_waitcnt(0);
  // the env wave's serial section sets the pace: it goes first when the waves
  // sharing its SIMD are ready to issue too
  if (wave == ew) __builtin_amdgcn_s_setprio(3);

  RL_STAMP_BEGIN
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    const int sn = k % NOISE_STEPS;
    T* xcur = xs[DB ? (k & 1) : 0];       // o_t
    T* xnext = xs[DB ? ((k + 1) & 1) : 0];  // o_{t+1}, painted by the env wave
    __syncthreads();  // the env wave is done with the previous step (tile, noise, actions)
    RL_STAMP(0)
    if (sn == 0) {
      // Philox action draws of the next NOISE_STEPS steps, one block (8 draws)
      // per (step, row), in one pass over all lanes
      const int nb = min(NOISE_STEPS, n_steps - k);
      for (int i = tid; i < nb * R; i += NT) {
        const int st = i / R, row = i - st * R;
        const int el = row / A, ag = row - el * A;
        if (el < te_valid) {
          const Block4 b = draw_block(p.seed, (uint64_t)(p.env_base + e0 + el), t + st, (uint64_t)ag * 256u,
                                      TAG_ACTION);
          uint32_t* d = words + (st * RP + row) * 8;
#pragma unroll
          for (int q = 0; q < 8; ++q) d[q] = block_u32(b, q);
        }
      }
      __syncthreads();
      draw_noise(0, nz[k & 1], tid, NT);  // noise of the batch's first step
      __syncthreads();
    }
    RL_STAMP(1)
    {
      f32x4 acc[MT][L1T::OWN];
      L1.template run<MT>(xcur, LDX, acc, wave, lane);
      L1.template store_tanh<MT>(acc, h1s, LD1, wave, lane, bias_s);
    }
    __syncthreads();
    RL_STAMP(2)
    {
      f32x4 acc[MT][RegLayer<DT, H1, H2, NW, LEAN>::OWN];
      L2.template run<MT>(h1s, LD1, acc, wave, lane);
      // (one tile) o_t to the trajectory while the layer-2 MFMAs run, clearing
      // the tile behind the copy (the env wave paints o_{t+1} onto it after layer 3)
      if constexpr (!DB) {
        int ct = tid;
        if constexpr (S1) asm volatile("" : "+v"(ct));  // (its addresses formed here, not held across the loop)
        copy_obs_rows<T, R, D, LDX, NT, true>(
            xcur, out.obs ? static_cast<T*>(out.obs) + ((size_t)k * E + e0) * A * D : nullptr, te_valid * A, ct);
      }
      L2.template store_tanh<MT>(acc, h2s, LD2, wave, lane, bias_s + H1);
    }
    __syncthreads();
    RL_STAMP(3)
    // Layer 3 transposed, logits^T = W3 h2^T: lane holds row (lane % 16) of
    // an M tile and actions 4 * (lane / 16) + r in accumulator element r.
    // Each lane takes the Gumbel argmax of its four actions; one lane swap
    // with the partner group (actions 0-3 <-> 4-7) finishes the row.
    const int g = lane >> 4;
    // Layer 3 of NTL M tiles from m0: the K steps run in order over the tiles
    // at once (one W3 operand serves every tile), their LDS operands read PF3
    // K steps ahead of the MFMAs that use them, each into its own registers,
    // so the chains do not wait out an LDS latency per K step.  (The lane
    // index is made opaque here so that the W3 reads are not hoisted out of
    // the step loop into registers held through the whole step.)
    auto l3_tiles = [&](auto ntl_c, int m0, auto& acc3) {
      constexpr int NTL = decltype(ntl_c)::value;
      constexpr int PF3 = K3 < 4 ? K3 : NTL > 2 ? 2 : 4;  // (fewer where three M tiles crowd the registers)
      int ln = lane;
      asm volatile("" : "+v"(ln));
      B wq[PF3], hq[PF3][NTL];
      auto fetch3 = [&](int ks, int q) {
        wq[q] = w3s[ks * 64 + ln];
#pragma unroll
        for (int m = 0; m < NTL; ++m) hq[q][m] = load_operand_lds<DT>(h2s, LD2, (m0 + m) * 16 + (ln & 15), ks, ln);
      };
#pragma unroll
      for (int m = 0; m < NTL; ++m) acc3[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < PF3; ++q) fetch3(q, q);
#pragma unroll
      for (int ks = 0; ks < K3; ++ks) {
#pragma unroll
        for (int m = 0; m < NTL; ++m) acc3[m] = mfma16<DT>(wq[ks % PF3], hq[ks % PF3][m], acc3[m]);
        if (ks + PF3 < K3) fetch3(ks + PF3, ks % PF3);
      }
    };
    // The Gumbel argmax of M tile mt and its outputs; returns this lane's
    // row's action (valid in lane groups 0 and 1).
    auto l3_argmax = [&](int mt, const f32x4 acc) -> int {
      const int row = mt * 16 + (lane & 15);
      const f32x4 nz4 = *reinterpret_cast<const f32x4*>(&nz[k & 1][row * 8 + 4 * (g & 1)]);
      float best_s = -INFINITY;
      int best_a = 0;
      float logit[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int act = 4 * g + r;
        logit[r] = acc[r] + b3r[r];
        const float sc = action_score(logit[r], nz4[r], (act < NA) & (row < R));
        const bool take = (r == 0) | (sc > best_s);
        best_s = take ? sc : best_s;
        best_a = take ? act : best_a;
      }
      {
        const auto ps = __builtin_amdgcn_permlane16_swap(__float_as_uint(best_s), __float_as_uint(best_s), false,
                                                         false);
        const auto pa = __builtin_amdgcn_permlane16_swap((uint32_t)best_a, (uint32_t)best_a, false, false);
        const float os = __uint_as_float((g & 1) ? ps[0] : ps[1]);
        const int oa = (int)((g & 1) ? pa[0] : pa[1]);
        const bool take = (os > best_s) | ((os == best_s) & (oa < best_a));
        best_s = take ? os : best_s;
        best_a = take ? oa : best_a;
      }
      const bool live = row < te_valid * A;
      const bool heur = TM && live && tk_s[TM ? row : 0] >= 0;  // (kinds set in the prologue)
      if (live && g == 0) {
        if constexpr (!DIRECT) act_s[row] = best_a;
        if (out.actions && !heur) out.actions[((size_t)k * E + e0) * A + row] = best_a;
      }
      if constexpr (VH) {
        const size_t gr = ((size_t)k * E + e0) * A + row;
        if (live && g == NA / 4 && out.value) out.value[gr] = logit[NA % 4];
        if (out.logp) {
          const float lp = row_log_pi<NA>(logit, g, best_a);
          if (live && g == 0) out.logp[gr] = lp;
        }
      }
      if (out.logits && live && g < 2 && !heur) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * g + r < NA) out.logits[(((size_t)k * E + e0) * A + row) * NA + 4 * g + r] = logit[r];
      }
      return best_a;
    };
    // SPLIT3: with several M tiles, wave m runs layer 3 and the argmax of
    // tile m before a barrier, instead of the env wave running them all.
    if constexpr (SPLIT3) {
      if (wave < MT) {
        f32x4 acc3[1];
        l3_tiles(std::integral_constant<int, 1>{}, wave, acc3);
        l3_argmax(wave, acc3[0]);
      }
      __syncthreads();
      RL_STAMP(4)
    }
    if (wave == ew) {
      if constexpr (LEAN) lbf_copy<A, F>(s, env_s[min(el, TE - 1)]);
      int act_d[LBF_MAXA] = {0, 0, 0, 0};  // DIRECT: this lane's env's actions
      if constexpr (!SPLIT3) {
        f32x4 acc3[MT];
        l3_tiles(std::integral_constant<int, MT>{}, 0, acc3);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int best_a = l3_argmax(mt, acc3[mt]);
          if constexpr (DIRECT) {
            act_d[0] = best_a;
            if constexpr (A > 1) act_d[1] = __builtin_amdgcn_update_dpp(0, best_a, 0x101, 0xf, 0xf, false);  // row_shl:1
            if constexpr (A > 2) act_d[2] = __builtin_amdgcn_update_dpp(0, best_a, 0x102, 0xf, 0xf, false);
            if constexpr (A > 3) act_d[3] = __builtin_amdgcn_update_dpp(0, best_a, 0x103, 0xf, 0xf, false);
          }
        }
      }
      if constexpr (!DIRECT && !SPLIT3) wave_lds_sync();
      uint32_t d = 0;
      RL_STAMP(4)
      float r = 0.f;
      if (envlane) {
        int act[LBF_MAXA];
#pragma unroll
        for (int i = 0; i < LBF_MAXA; ++i) {
          if constexpr (DIRECT)
            act[i] = act_d[i];
          else
            act[i] = i < A ? act_s[lane * A + i] : 0;
        }
        if constexpr (TM) {  // heuristic agents: their action, and logits 0 for it / -inf for the others
#pragma unroll
          for (int i = 0; i < A; ++i) {
            const int kd = tk_s[el * A + i];
            if (kd >= 0) {
              act[i] = lbf_heuristic_action(p, s, i, kd, start[TM ? i : 0]);
              const size_t gr = ((size_t)k * E + e) * A + i;
              if (out.actions) out.actions[gr] = act[i];
              if (out.logits)
#pragma unroll
                for (int a = 0; a < NA; ++a) out.logits[gr * NA + a] = a == act[i] ? 0.f : -INFINITY;
            }
          }
        }
        lbf_transition<A, F, GH, GW>(p, s, act, r, d);
      }
      // reset blocks of every env that ended, one Philox block per lane
      RL_STAMP(5)
      const uint64_t done_mask = __ballot(envlane && d != 0);
      if (done_mask) {
        const int j = lane / nblk, blk = lane - j * nblk;
        if (j < TE && ((done_mask >> (j * ESTRIDE)) & 1ull)) {
          const Block4 b = draw_block(p.seed, (uint64_t)(p.env_base + e0 + j), t + 1, (uint64_t)blk, TAG_RESET);
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (blk * 8 + q < LBF_MAX_DRAWS) rdraw[j * LBF_MAX_DRAWS + blk * 8 + q] = block_u32(b, q);
        }
        wave_lds_sync();
        if (envlane && d) {
          uint32_t dw[LBF_MAX_DRAWS];
#pragma unroll
          for (int q = 0; q < LBF_MAX_DRAWS; ++q) dw[q] = q < nd ? rdraw[el * LBF_MAX_DRAWS + q] : 0u;
          lbf_reset_from_draws<A, F>(p, dw, s);
          if constexpr (TM) {
#pragma unroll
            for (int i = 0; i < A; ++i) start[i] = s.acell[i];
          }
        }
      }
      RL_STAMP(6)
      if (envlane) {
        lbf_paint_tile<T, A, F>(s, el, xnext, LDX, HW, true);
        if (out.reward) out.reward[(size_t)k * E + e] = r;
        if (out.done) out.done[(size_t)k * E + e] = (uint8_t)d;
        if constexpr (LEAN) lbf_copy<A, F>(env_s[el], s);
      }
      RL_STAMP(7)
    } else {
      // the other waves, while the env wave steps: (two tiles) o_t to the
      // trajectory, clearing its tile; the Gumbel noise of the next step (a new
      // batch's first step is drawn with the batch)
      if constexpr (DB)
        copy_obs_rows<T, R, D, LDX, NT - 64, true>(
            xcur, out.obs ? static_cast<T*>(out.obs) + ((size_t)k * E + e0) * A * D : nullptr, te_valid * A,
            tid - 64);
      RL_STAMP(8)
      if (k + 1 < n_steps && (k + 1) % NOISE_STEPS != 0)
        draw_noise((k + 1) % NOISE_STEPS, nz[(k + 1) & 1], (wave - 1) * 64 + lane, (NW - 1) * 64);
      RL_STAMP(9)
    }
  }
  RL_STAMP_END(wave)
  __syncthreads();
  T* xlast = xs[DB ? (n_steps & 1) : 0];  // o_{t0+T}
  if (out.obs_last)
    copy_obs_rows<T, R, D, LDX, NT>(xlast, static_cast<T*>(out.obs_last) + (size_t)e0 * A * D, te_valid * A, tid);
  if constexpr (VH) {
    if (out.value_last) {  // V(o_{t0+T}): one more pass of the network over the final tile
      {
        f32x4 acc[MT][L1T::OWN];
        L1.template run<MT>(xlast, LDX, acc, wave, lane);
        L1.template store_tanh<MT>(acc, h1s, LD1, wave, lane, bias_s);
      }
      __syncthreads();
      {
        f32x4 acc[MT][RegLayer<DT, H1, H2, NW, LEAN>::OWN];
        L2.template run<MT>(h1s, LD1, acc, wave, lane);
        L2.template store_tanh<MT>(acc, h2s, LD2, wave, lane, bias_s + H1);
      }
      __syncthreads();
      if (wave == ew) {  // (the whole wave takes part in the MFMAs)
        for (int mt = 0; mt < MT; ++mt) {
          const int row = mt * 16 + (lane & 15);
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < K3; ++ks)
            acc = mfma16<DT>(w3s[ks * 64 + lane], load_operand_lds<DT>(h2s, LD2, row, ks, lane), acc);
          if ((lane >> 4) == NA / 4 && row < te_valid * A)
            out.value_last[(size_t)e0 * A + row] = acc[NA % 4] + b3r[NA % 4];
        }
      }
    }
  }
  if constexpr (LEAN) lbf_copy<A, F>(s, env_s[min(el, TE - 1)]);
  if (envlane) lbf_store<A, F>(state, p, e, s);
}

// Compile-time shapes that run on lbf_rollout_kernel (everything else uses
// lbf_run_kernel): LBF 8x8 with 2 agents and 3 foods (obs 192) under 64- and
// 128-wide layers.
template <int DT, int GH, int GW, int H1, int H2, int A, int F, int TE, int NW, int MINB, bool VH, bool TM,
          bool S1 = false>
static hipError_t launch_rollout_reg(const LbfParams& p, const LbfMagic&, const PolicyArgs& pol, int32_t* state,
                                     uint64_t t0, int n_steps, const TrajArgs& out, hipStream_t s) {
  auto kern = lbf_rollout_kernel<DT, GH, GW, H1, H2, LBF_NACT, A, F, TE, NW, MINB, VH, TM, S1>;
  const dim3 grid((unsigned)((p.E + TE - 1) / TE));
  kern<<<grid, NW * 64, 0, s>>>(p, pol, state, t0, n_steps, out);
  return hipGetLastError();
}

static bool try_launch_rollout_reg(const LbfParams& p, const LbfMagic& m, const PolicyArgs& pol, int32_t* state,
                                   uint64_t t0, int n_steps, const TrajArgs& out, hipStream_t s, hipError_t* err) {
  if (pol.NA != LBF_NACT + pol.VH) return false;
  const bool tm = out.teammates != nullptr;
#define RL_REG_CASE_T(DTV, GHV, GWV, H1V, H2V, AV, FV, TEV, NWV, MINBV, VHV, TMV)                              \
  if (pol.dt == DTV && p.H == GHV && p.W == GWV && pol.H1 == H1V && pol.H2 == H2V && p.A == AV &&            \
      p.F == FV && pol.VH == VHV && tm == TMV) {                                                             \
    *err = launch_rollout_reg<DTV, GHV, GWV, H1V, H2V, AV, FV, TEV, NWV, MINBV, VHV, TMV>(p, m, pol, state,   \
                                                                                          t0, n_steps, out, s); \
    return true;                                                                                             \
  }
#define RL_REG_CASE(DTV, GHV, GWV, H1V, H2V, AV, FV, TEV, NWV, MINBV, VHV) \
  RL_REG_CASE_T(DTV, GHV, GWV, H1V, H2V, AV, FV, TEV, NWV, MINBV, VHV, false)
  // (dtype, grid rows, grid cols, hidden, hidden, agents, foods, envs per workgroup, waves, workgroups per CU,
  //  value head)
  RL_REG_CASE(DT_F32, 8, 8, 64, 64, 2, 3, 8, 4, 2, 0)
  RL_REG_CASE(DT_BF16, 8, 8, 64, 64, 2, 3, 8, 4, 2, 0)
  RL_REG_CASE(DT_F32, 8, 8, 128, 128, 2, 3, 16, 8, 1, 0)
  RL_REG_CASE(DT_BF16, 8, 8, 128, 128, 2, 3, 8, 4, 2, 0)
  if (pol.dt == DT_BF16 && p.H == 12 && p.W == 12 && pol.H1 == 256 && pol.H2 == 256 && p.A == 3 && p.F == 6 &&
      !pol.VH && !tm) {
    // layer 1 (432 x 256) streamed from the packed copy: both layers resident
    // spill; without a packed copy they stay resident all the same
    if (pol.Wp[0] != nullptr)
      *err = launch_rollout_reg<DT_BF16, 12, 12, 256, 256, 3, 6, 16, 8, 1, false, false, true>(p, m, pol, state, t0,
                                                                                            n_steps, out, s);
    else
      *err = launch_rollout_reg<DT_BF16, 12, 12, 256, 256, 3, 6, 16, 8, 1, false, false, false>(p, m, pol, state, t0,
                                                                                             n_steps, out, s);
    return true;
  }
  RL_REG_CASE(DT_BF16, 7, 7, 128, 128, 2, 3, 8, 4, 2, 0)
  RL_REG_CASE(DT_F32, 8, 8, 64, 64, 2, 3, 8, 4, 2, 1)
  RL_REG_CASE(DT_BF16, 8, 8, 64, 64, 2, 3, 8, 4, 2, 1)
  RL_REG_CASE(DT_F32, 8, 8, 128, 128, 2, 3, 16, 4, 1, 1)
  RL_REG_CASE(DT_BF16, 8, 8, 128, 128, 2, 3, 8, 4, 2, 1)
  // (heuristic teammates)
  RL_REG_CASE_T(DT_BF16, 7, 7, 128, 128, 2, 3, 8, 4, 2, 0, true)
  RL_REG_CASE_T(DT_BF16, 7, 7, 64, 64, 2, 3, 8, 4, 2, 0, true)
  RL_REG_CASE_T(DT_BF16, 8, 8, 128, 128, 2, 3, 8, 4, 2, 0, true)
  RL_REG_CASE_T(DT_F32, 8, 8, 64, 64, 2, 3, 8, 4, 2, 0, true)
#undef RL_REG_CASE
#undef RL_REG_CASE_T
  return false;
}

// ------------------------- population rollout, two resident policies ----
//
// rollout_run_pop for the common case of at most two distinct policies among
// a tile's agents (the ego and one teammate per block of envs): both
// policies' layer-1/2 weights stay in registers for the whole rollout, as in
// lbf_rollout_kernel.  The tile's rows are agent-major (row a * TE + el), so
// with the ego on agent 0 and a teammate on agent 1 each 16-row MFMA tile
// holds a single policy and runs its own weights only; a tile whose rows mix
// the two policies runs both and each lane keeps its row's result.  Tiles
// with three or more policies are left to lbf_run_pop_kernel (launched after
// this kernel with skip_two set), which skips the tiles handled here.

// Policies of a tile's agents (an index outside the population selects policy
// 0): slot 0 is the policy of env e0's agent 0, slot 1 the first other policy
// in row order (slot 0 again when there is none).  True iff every agent of the
// tile uses one of the two.
__device__ __forceinline__ bool pop_two_slots(const int32_t* __restrict__ pidx, int e0, int te_valid, int A,
                                              int n_pol, int& q0, int& q1) {
  const int nr = te_valid * A;
  q0 = -1;
  q1 = -1;
  bool ok = true;
  for (int r = 0; r < nr; ++r) {
    const int raw = pidx[(size_t)e0 * A + r];
    const int id = (unsigned)raw < (unsigned)n_pol ? raw : 0;
    if (q0 < 0) {
      q0 = id;
    } else if (id != q0) {
      if (q1 < 0) q1 = id;
      else if (id != q1) ok = false;
    }
  }
  if (q1 < 0) q1 = q0;
  return ok;
}

template <int GH, int GW, int H1, int H2, int A, int F, int TE, int NW>
__global__ __launch_bounds__(NW * 64, 1) void lbf_pop2_kernel(LbfParams p, PolicyArgs pol, int n_pol,
                                                             const int32_t* __restrict__ pidx,
                                                             int32_t* __restrict__ state, uint64_t t0, int n_steps,
                                                             TrajArgs out) {
  constexpr int DT = DT_BF16;
  using T = uint16_t;
  using B = u32x4;
  constexpr int HW = GH * GW, D = 3 * HW;
  constexpr int NT = NW * 64;
  constexpr int R = TE * A;
  constexpr int MT = (R + 15) / 16;
  constexpr int RP = MT * 16;
  constexpr int NA = LBF_NACT;
  constexpr int LDX = lds_ld<DT>(D), LD1 = lds_ld<DT>(H1), LD2 = lds_ld<DT>(H2);
  constexpr int K3 = round_up(H2, 32) / 32;
  using L1T = RegLayer<DT, D, H1, NW, true>;
  using L2T = RegLayer<DT, H1, H2, NW, true>;
  static_assert(TE == 16, "agent-major rows: M tile m holds agent m of the tile's 16 envs");
  static_assert(L1T::NT % NW == 0 && L2T::NT % NW == 0, "every wave owns whole output tiles");

  __shared__ __align__(16) T xs[RP * LDX];
  __shared__ __align__(16) T h1s[RP * LD1];
  __shared__ __align__(16) T h2s[RP * LD2];
  __shared__ __align__(16) B w3s[2][K3 * 64];
  __shared__ __align__(16) float bias_s[2][H1 + H2];
  __shared__ float b3s[2][8];
  __shared__ int act_s[RP];
  __shared__ int slot_s[RP];  // 0 or 1: the resident policy of each row
  __shared__ int ctl_s[2 + MT];  // the two policies' indices (-1: the tile is not handled here), slot masks per M tile
  __shared__ uint32_t words[NOISE_STEPS * RP * 8];
  __shared__ __align__(16) float nz[2][RP * 8];
  __shared__ uint32_t rdraw[TE * LBF_MAX_DRAWS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE;
  const int te_valid = min(TE, p.E - e0);
  const int E = p.E;
  constexpr int nd = 2 * A + 2 * F;
  constexpr int nblk = (nd + 7) >> 3;
  static_assert(TE * nblk <= 64, "one lane per reset block");

  if (tid == 0) {
    int q0, q1;
    const bool ok = pop_two_slots(pidx, e0, te_valid, A, n_pol, q0, q1);
    ctl_s[0] = ok ? q0 : -1;
    ctl_s[1] = q1;
  }
  __syncthreads();
  if (ctl_s[0] < 0) return;  // three or more policies: lbf_run_pop_kernel runs this tile
  const int q0 = ctl_s[0], q1 = ctl_s[1];
  for (int row = tid; row < RP; row += NT) {
    const int el = row % TE, ag = row / TE;
    int sl = 0;
    if (el < te_valid && ag < A) {
      const int raw = pidx[(size_t)(e0 + el) * A + ag];
      sl = ((unsigned)raw < (unsigned)n_pol ? raw : 0) == q0 ? 0 : 1;
    }
    slot_s[row] = sl;
  }
  __syncthreads();
  if (tid < MT) {  // which slots the live rows of M tile tid use
    int msk = 0;
    for (int r = 0; r < 16; ++r) {
      const int row = tid * 16 + r;
      if (row < R && row % TE < te_valid) msk |= 1 << slot_s[row];
    }
    ctl_s[2 + tid] = msk;
  }

  // weights: layers 1 and 2 of both policies in registers, layer 3 and the biases in LDS
  const T* W1 = static_cast<const T*>(pol.W[0]);
  const T* W2 = static_cast<const T*>(pol.W[1]);
  const T* W3 = static_cast<const T*>(pol.W[2]);
  const T* b1 = static_cast<const T*>(pol.b[0]);
  const T* b2 = static_cast<const T*>(pol.b[1]);
  const T* b3 = static_cast<const T*>(pol.b[2]);
  L1T L1a, L1b;
  L2T L2a, L2b;
  L1a.load(W1 + (size_t)q0 * H1 * D, b1, wave, lane);
  L2a.load(W2 + (size_t)q0 * H2 * H1, b2, wave, lane);
  if (q1 != q0) {
    L1b.load(W1 + (size_t)q1 * H1 * D, b1, wave, lane);
    L2b.load(W2 + (size_t)q1 * H2 * H1, b2, wave, lane);
  }
  for (int i = tid; i < 2 * (H1 + H2); i += NT) {
    const int sl = i / (H1 + H2), j = i - sl * (H1 + H2);
    const size_t q = sl ? q1 : q0;
    bias_s[sl][j] = bf16_to_f32(j < H1 ? b1[q * H1 + j] : b2[q * H2 + j - H1]);
  }
  if (tid < 128) {
    const int sl = tid >> 6, n = lane & 15;
    const size_t q = sl ? q1 : q0;
    const T* row = W3 + (q * NA + (n < NA ? n : 0)) * H2;
#pragma unroll
    for (int ks = 0; ks < K3; ++ks) w3s[sl][ks * 64 + lane] = load_operand_global<DT, H2>(row, H2, ks, lane, n < NA);
    if (lane < 8) b3s[sl][lane] = lane < NA ? bf16_to_f32(b3[q * NA + lane]) : 0.f;
  }
  for (int i = tid; i < RP * LDX; i += NT) xs[i] = (T)0;
  for (int i = tid; i < RP * LD1; i += NT) h1s[i] = (T)0;
  for (int i = tid; i < RP * LD2; i += NT) h2s[i] = (T)0;
  __syncthreads();
  int tmask[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) tmask[m] = __builtin_amdgcn_readfirstlane(ctl_s[2 + m]);
  const bool envlane = wave == 0 && lane < te_valid;
  const int el = lane, e = e0 + el;
  LbfEnv s{};
  if (envlane) {
    lbf_load<A, F>(state, p, e, s);
    lbf_paint_tile<T, A, F, TE>(s, el, xs, LDX, HW, true);
  }
  __builtin_amdgcn_s_waitcnt(0);

  auto draw_noise = [&](int sn, float* noise, int i0, int stride) {
    for (int i = i0; i < R * NA; i += stride) {
      const int row = i / NA, a = i - row * NA;
      noise[row * 8 + a] = gumbel24(words[(sn * RP + row) * 8 + a] >> 8);
    }
  };
  // one layer over every M tile: each tile runs the weights of the slots its
  // rows use, each lane keeps its own row's result, then bias + tanh in bf16
  auto layer = [&](const auto& La, const auto& Lb, const T* in, int ldi, T* outp, int ldo, const float* bias0,
                   const float* bias1) {
    using LT = std::decay_t<decltype(La)>;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      f32x4 a0[1][LT::OWN], a1[1][LT::OWN];
#pragma unroll
      for (int o = 0; o < LT::OWN; ++o) a0[0][o] = a1[0][o] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (tmask[m] & 1) La.template run<1>(in + m * 16 * ldi, ldi, a0, wave, lane);
      if (tmask[m] & 2) Lb.template run<1>(in + m * 16 * ldi, ldi, a1, wave, lane);
      const int sl = slot_s[m * 16 + (lane & 15)];
#pragma unroll
      for (int o = 0; o < LT::OWN; ++o)
        La.store_block(sl ? a1[0][o] : a0[0][o], outp + m * 16 * ldo, ldo, 0, o, wave, lane, sl ? bias1 : bias0);
    }
  };

  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    const int sn = k % NOISE_STEPS;
    __syncthreads();
    if (sn == 0) {
      const int nb = min(NOISE_STEPS, n_steps - k);
      for (int i = tid; i < nb * R; i += NT) {
        const int st = i / R, row = i - st * R;
        const int rel = row % TE, ag = row / TE;
        if (rel < te_valid) {
          const Block4 b = draw_block(p.seed, (uint64_t)(p.env_base + e0 + rel), t + st, (uint64_t)ag * 256u,
                                      TAG_ACTION);
          uint32_t* d = words + (st * RP + row) * 8;
#pragma unroll
          for (int q = 0; q < 8; ++q) d[q] = block_u32(b, q);
        }
      }
      __syncthreads();
      draw_noise(0, nz[k & 1], tid, NT);
      __syncthreads();
    }
    layer(L1a, L1b, xs, LDX, h1s, LD1, bias_s[0], bias_s[1]);
    __syncthreads();
    copy_obs_rows<T, R, D, LDX, NT, true, 4, TE, A>(
        xs, out.obs ? static_cast<T*>(out.obs) + ((size_t)k * E + e0) * A * D : nullptr, te_valid * A, tid);
    layer(L2a, L2b, h1s, LD1, h2s, LD2, bias_s[0] + H1, bias_s[1] + H1);
    __syncthreads();
    // wave m: layer 3 and the Gumbel argmax of M tile m; then the env wave steps
    static_assert(MT <= NW, "one wave per M tile of layer 3");
    if (wave < MT) {
      const int g = lane >> 4;
      {
        const int m = wave;
        int tm = 0;  // tmask[m] (without indexing the register array at run time)
#pragma unroll
        for (int q = 0; q < MT; ++q) tm = q == m ? tmask[q] : tm;
        const int row = m * 16 + (lane & 15);
        const int rel = row % TE, ag = row / TE;
        const int sl = slot_s[row];
        const f32x4 nz4 = *reinterpret_cast<const f32x4*>(&nz[k & 1][row * 8 + 4 * (g & 1)]);
        f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
        // the row operands (shared by both policies' chains), then each
        // policy's W3 operands, all read before the MFMAs that use them
        B hq[K3];
#pragma unroll
        for (int ks = 0; ks < K3; ++ks) hq[ks] = load_operand_lds<DT>(h2s, LD2, row, ks, lane);
        if (tm & 1) {
          B wq[K3];
#pragma unroll
          for (int ks = 0; ks < K3; ++ks) wq[ks] = w3s[0][ks * 64 + lane];
#pragma unroll
          for (int ks = 0; ks < K3; ++ks) a0 = mfma16<DT>(wq[ks], hq[ks], a0);
        }
        if (tm & 2) {
          B wq[K3];
#pragma unroll
          for (int ks = 0; ks < K3; ++ks) wq[ks] = w3s[1][ks * 64 + lane];
#pragma unroll
          for (int ks = 0; ks < K3; ++ks) a1 = mfma16<DT>(wq[ks], hq[ks], a1);
        }
        float best_s = -INFINITY;
        int best_a = 0;
        float logit[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int act = 4 * g + r;
          logit[r] = (sl ? a1[r] : a0[r]) + b3s[sl][act & 7];
          const float sc = action_score(logit[r], nz4[r], (act < NA) & (row < R));
          const bool take = (r == 0) | (sc > best_s);
          best_s = take ? sc : best_s;
          best_a = take ? act : best_a;
        }
        {
          const auto ps = __builtin_amdgcn_permlane16_swap(__float_as_uint(best_s), __float_as_uint(best_s), false,
                                                           false);
          const auto pa = __builtin_amdgcn_permlane16_swap((uint32_t)best_a, (uint32_t)best_a, false, false);
          const float os = __uint_as_float((g & 1) ? ps[0] : ps[1]);
          const int oa = (int)((g & 1) ? pa[0] : pa[1]);
          const bool take = (os > best_s) | ((os == best_s) & (oa < best_a));
          best_s = take ? os : best_s;
          best_a = take ? oa : best_a;
        }
        const bool live = row < R && rel < te_valid;
        const size_t gr = ((size_t)k * E + e0 + rel) * A + ag;
        if (live && g == 0) {
          act_s[row] = best_a;
          if (out.actions) out.actions[gr] = best_a;
        }
        if (out.logits && live && g < 2) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (4 * g + r < NA) out.logits[gr * NA + 4 * g + r] = logit[r];
        }
      }
    }
    __syncthreads();
    if (wave == 0) {
      uint32_t d = 0;
      float r = 0.f;
      if (envlane) {
        int act[LBF_MAXA];
#pragma unroll
        for (int i = 0; i < LBF_MAXA; ++i) act[i] = i < A ? act_s[i * TE + el] : 0;
        lbf_transition<A, F, GH, GW>(p, s, act, r, d);
      }
      const uint64_t done_mask = __ballot(envlane && d != 0);
      if (done_mask) {
        const int j = lane / nblk, blk = lane - j * nblk;
        if (j < TE && ((done_mask >> j) & 1ull)) {
          const Block4 b = draw_block(p.seed, (uint64_t)(p.env_base + e0 + j), t + 1, (uint64_t)blk, TAG_RESET);
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (blk * 8 + q < LBF_MAX_DRAWS) rdraw[j * LBF_MAX_DRAWS + blk * 8 + q] = block_u32(b, q);
        }
        wave_lds_sync();
        if (envlane && d) {
          uint32_t dw[LBF_MAX_DRAWS];
#pragma unroll
          for (int q = 0; q < LBF_MAX_DRAWS; ++q) dw[q] = q < nd ? rdraw[el * LBF_MAX_DRAWS + q] : 0u;
          lbf_reset_from_draws<A, F>(p, dw, s);
        }
      }
      if (envlane) {
        lbf_paint_tile<T, A, F, TE>(s, el, xs, LDX, HW, true);
        if (out.reward) out.reward[(size_t)k * E + e] = r;
        if (out.done) out.done[(size_t)k * E + e] = (uint8_t)d;
      }
    } else if (k + 1 < n_steps && (k + 1) % NOISE_STEPS != 0) {
      draw_noise((k + 1) % NOISE_STEPS, nz[(k + 1) & 1], (wave - 1) * 64 + lane, (NW - 1) * 64);
    }
  }
  __syncthreads();
  if (out.obs_last)
    copy_obs_rows<T, R, D, LDX, NT, false, 4, TE, A>(xs, static_cast<T*>(out.obs_last) + (size_t)e0 * A * D,
                                                     te_valid * A, tid);
  if (envlane) lbf_store<A, F>(state, p, e, s);
}

hipError_t launch_lbf_run_pop(const LbfParams& p, const PolicyArgs& pol, int n_pol, const int32_t* pidx,
                              int32_t* state, uint64_t t0, int n_steps, const TrajArgs& out, hipStream_t s) {
  const LbfMagic m = make_magic(p, pol.NA);
  // the register-resident two-policy kernel for its compiled shape; the
  // generic kernel then runs only the tiles with three or more policies
  int skip_two = 0;
  if (pol.dt == DT_BF16 && p.H == 8 && p.W == 8 && p.A == 2 && p.F == 3 && pol.H1 == 128 && pol.H2 == 128 &&
      pol.NA == LBF_NACT && TILE_E == 16) {
    lbf_pop2_kernel<8, 8, 128, 128, 2, 3, 16, 8><<<dim3((unsigned)((p.E + 15) / 16)), 512, 0, s>>>(
        p, pol, n_pol, pidx, state, t0, n_steps, out);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    skip_two = 1;
  }
  const size_t lds = lbf_pop_lds_bytes(p, pol);
  const dim3 grid((unsigned)((p.E + TILE_E - 1) / TILE_E));
  // the dynamic limit leaves room for the kernel's few bytes of static LDS
  const int max_dyn = (int)(MAX_LDS_BYTES - LBF_POP_STATIC_LDS);
  if (pol.dt == DT_F32) {
    static bool attr = false;
    if (!attr) {
      const hipError_t e = hipFuncSetAttribute((const void*)lbf_run_pop_kernel<DT_F32, false>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, max_dyn);
      if (e != hipSuccess) return e;
      attr = true;
    }
    lbf_run_pop_kernel<DT_F32, false><<<grid, NTHREADS, lds, s>>>(p, m, pol, n_pol, pidx, state, t0, n_steps, out, skip_two);
  } else if (pol.Wp[0] != nullptr) {  // fragment-major weights
    static bool attr = false;
    if (!attr) {
      const hipError_t e = hipFuncSetAttribute((const void*)lbf_run_pop_kernel<DT_BF16, true>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, max_dyn);
      if (e != hipSuccess) return e;
      attr = true;
    }
    lbf_run_pop_kernel<DT_BF16, true><<<grid, NTHREADS, lds, s>>>(p, m, pol, n_pol, pidx, state, t0, n_steps, out, skip_two);
  } else {
    static bool attr = false;
    if (!attr) {
      const hipError_t e = hipFuncSetAttribute((const void*)lbf_run_pop_kernel<DT_BF16, false>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, max_dyn);
      if (e != hipSuccess) return e;
      attr = true;
    }
    lbf_run_pop_kernel<DT_BF16, false><<<grid, NTHREADS, lds, s>>>(p, m, pol, n_pol, pidx, state, t0, n_steps, out, skip_two);
  }
  return hipGetLastError();
}

// ------------------------------------- env-only steps ----
//
// rollout_step for compile-time LBF shapes.  The env wave runs S steps
// between workgroup barriers: per step the transition and the resets of the
// episodes that ended.  Everything else, and everything that touches global
// memory inside the step loop, is left to the other ("copy") waves:
//   * wave 0 (env), at raised issue priority (its chain sets the pace): the
//     env state lives in registers; on grids of at most 64 cells the 8 lanes
//     of a group hold one env and resolve its transition together
//     (lbf_transition_group), otherwise lane e holds env e.  The actions come
//     from LDS one step ahead.  The reset draws of the envs that ended are
//     made in parallel, one Philox block per lane.  The env's first lane
//     publishes the post-step state, reward and done of each step to LDS
//     (double-buffered by barrier interval);
//   * waves 1..NCW (copy): after a barrier, each for its own share of the
//     rows and for each of the S steps just run, paint o_{t+1} from the
//     published states onto the step's observation tile (one non-zero
//     feature per lane), copy the rows to the trajectory with 16-byte stores,
//     clearing them behind the copy, and write the rewards, dones and legal
//     masks, while wave 0 runs the next S steps; at the start of each chunk
//     of ACT_CHUNK steps they stage the next chunk's actions into the other
//     half of a double buffer (a global load waits for its wave's earlier
//     stores, so wave 0 issues none inside the loop).
template <typename OT, int GH, int GW, int A, int F, int TE, int NCW, int S>
__global__ __launch_bounds__(64 * (NCW + 1)) void lbf_env_kernel(LbfParams p, int32_t* __restrict__ state,
                                                                 uint64_t t0, int n_steps,
                                                                 const int32_t* __restrict__ actions,
                                                                 OT* __restrict__ obs, float* __restrict__ reward,
                                                                 uint8_t* __restrict__ done,
                                                                 uint8_t* __restrict__ legal) {
  constexpr int HW = GH * GW, D = 3 * HW, R = TE * A;
  constexpr int NT = 64 * (NCW + 1), NC = 64 * NCW;
  constexpr bool GRP = HW <= 64 && A <= 4 && F <= 8 && TE == 8;  // lane groups of 8 per env
  constexpr int G = GRP ? 8 : 1;
  constexpr int nd = 2 * A + 2 * F;
  constexpr int nblk = (nd + 7) >> 3;
  static_assert(TE * G <= 64 && TE * nblk <= 64, "env lanes in wave 0, and one lane per reset block");
  constexpr int CH = ACT_CHUNK;
  static_assert(CH % S == 0, "barrier groups of S steps do not straddle action chunks");
  static_assert(R % NCW == 0, "whole rows per copy wave");
  constexpr int RW = R / NCW, NSLOT = A + F + 1;    // rows per copy wave; non-zero features per row
  __shared__ __align__(16) OT xs[S][R * D];         // o_{t+1} of a step, painted and copied by the copy waves
  __shared__ LbfEnv pub[2][S][TE];                  // post-step state of step k in pub[(k / S) % 2][k % S]
  __shared__ int32_t act_lds[2][CH * TE * A];      // actions of chunk c in act_lds[c % 2]
  __shared__ uint32_t rdraw[TE * LBF_MAX_DRAWS];   // reset draws of the envs that ended
  __shared__ float rw_s[2][S][TE];                 // reward and done of step k, as its tile
  __shared__ uint32_t dn_s[2][S][TE];
  constexpr int GC = (R * D * sizeof(OT) / 16 + NC - 1) / NC < 4 ? (R * D * sizeof(OT) / 16 + NC - 1) / NC : 4;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE;
  const int te_valid = min(TE, p.E - e0);
  const int E = p.E;
  const int el = lane / G;                          // wave 0: env of this lane
  const bool grplane = wave == 0 && el < te_valid;  // lanes holding env el's state
  const bool envlane = grplane && lane % G == 0;    // the lane that writes env el's outputs
  const int e = e0 + el;
  const int ea = min(el, TE - 1) * A;  // this lane's env's first action in a step's staged actions

  zero_lds<NT>(xs, sizeof(xs), tid);
  stage_actions<TE * A, NT>(actions, E, e0, te_valid * A, A, 0, min(CH, n_steps), act_lds[0], tid);
  LbfEnv s{};
  if (grplane) lbf_load<A, F>(state, p, e, s);
  if (wave == 0) __builtin_amdgcn_s_setprio(3);  // (the env wave's chain sets the pace)
  for (int k0 = 0; k0 < n_steps; k0 += CH) {
    const int nk = min(CH, n_steps - k0);
    const int32_t* acts = act_lds[(k0 / CH) & 1];
    __syncthreads();  // this chunk's actions are staged
    int act[LBF_MAXA] = {0, 0, 0, 0};
    if (wave == 0) {
#pragma unroll
      for (int i = 0; i < A; ++i) act[i] = acts[ea + i];
    }
    for (int kb = 0; kb < nk; kb += S) {
      const int ns = min(S, nk - kb);
      const int pr = ((k0 + kb) / S) & 1;  // the tiles of these steps
      if (wave == 0) {
#pragma unroll 1
        for (int u = 0; u < ns; ++u) {
          const int kk = kb + u, k = k0 + kk;
          const uint64_t t = t0 + (uint64_t)k;
          uint32_t d = 0;
          float r = 0.f;
          if constexpr (GRP) {
            lbf_transition_group<A, F, GH, GW>(p, s, act, r, d);  // every lane of the wave
          } else {
            if (grplane) lbf_transition<A, F, GH, GW>(p, s, act, r, d);
          }
          if (kk + 1 < nk) {  // the next step's actions, ahead of need
#pragma unroll
            for (int i = 0; i < A; ++i) act[i] = acts[(kk + 1) * TE * A + ea + i];
          }
          // resets of the envs that ended, drawn at t + 1: one Philox block per lane
          const uint64_t done_mask = __ballot(envlane && d != 0);
          if (done_mask) {
            const int j = lane / nblk, blk = lane - j * nblk;
            if (j < TE && ((done_mask >> (j * G)) & 1ull)) {
              const Block4 b = draw_block(p.seed, (uint64_t)(p.env_base + e0 + j), t + 1, (uint64_t)blk, TAG_RESET);
#pragma unroll
              for (int q = 0; q < 8; ++q)
                if (blk * 8 + q < LBF_MAX_DRAWS) rdraw[j * LBF_MAX_DRAWS + blk * 8 + q] = block_u32(b, q);
            }
            wave_lds_sync();
            if (grplane && d) {
              uint32_t dw[LBF_MAX_DRAWS];
#pragma unroll
              for (int q = 0; q < LBF_MAX_DRAWS; ++q) dw[q] = q < nd ? rdraw[el * LBF_MAX_DRAWS + q] : 0u;
              lbf_reset_from_draws<A, F>(p, dw, s);
            }
          }
          if (envlane) {
            if (obs) lbf_copy<A, F>(pub[pr][u][el], s);
            rw_s[pr][u][el] = r;
            dn_s[pr][u][el] = d;
          }
        }
      }
      __syncthreads();  // these steps published (and the previous ones copied out)
      if (wave != 0) {
        const int ct = tid - 64;  // 0 .. NC-1
        const int r0 = (wave - 1) * RW, live = max(0, min(RW, te_valid * A - r0));  // this wave's rows
        for (int u = 0; u < ns; ++u) {
          const int k = k0 + kb + u;
          if (obs && live > 0) {
            // paint the wave's rows of o_{t+1} from the published states, one
            // non-zero feature per lane (the tile is blank: the copy clears it)
            OT* tile = xs[u] + r0 * D;
            for (int it = lane; it < live * NSLOT; it += 64) {
              const int rl = it / NSLOT, c = it - rl * NSLOT, row = r0 + rl, en = row / A, i = row - en * A;
              const LbfEnv& st = pub[pr][u][en];
              int cell, plane;
              uint32_t v;
              if (c < A) {
                cell = st.acell[c], plane = 0, v = (uint32_t)st.alevel[c];
              } else if (c < A + F) {
                const int j = c - A;
                cell = st.fcell[j], plane = 1, v = ((st.eaten >> j) & 1u) ? 0u : (uint32_t)st.flevel[j];
              } else {
                cell = st.acell[i], plane = 2, v = 1u;
              }
              // (cells clamped into the grid: a malformed state cannot address outside the row)
              if (v) tile[rl * D + plane * HW + min((uint32_t)cell, (uint32_t)HW - 1u)] = small_int_to<OT>(v);
            }
            wave_lds_sync();
            copy_obs_rows<OT, RW, D, D, 64, true, GC>(tile, obs + ((size_t)k * E + e0) * A * D + (size_t)r0 * D,
                                                      live, lane);
            wave_lds_sync();
          }
          if (ct < te_valid) {
            if (reward) reward[(size_t)k * E + e0 + ct] = rw_s[pr][u][ct];
            if (done) done[(size_t)k * E + e0 + ct] = (uint8_t)dn_s[pr][u][ct];
          }
          if (legal && wave == 1)
            lbf_write_legal<64>(p, te_valid, legal + ((size_t)k * E + e0) * A * LBF_NACT, lane);
        }
        if (kb == 0 && k0 + CH < n_steps)  // the next chunk's actions, into the other buffer
          stage_actions<TE * A, NC>(actions, E, e0, te_valid * A, A, k0 + CH, min(CH, n_steps - k0 - CH),
                                    act_lds[(k0 / CH + 1) & 1], ct);
      }
    }
  }
  if (envlane) lbf_store<A, F>(state, p, e, s);
}

// The float32 env-only path, in three waves.  With float32 observations a
// step's tile is twice as large, and the copy-wave kernel above loses to this
// design (measured on the 8x8 workload: 0.150 against 0.177 ms), which keeps
// the resets off the env lanes by building them ahead of need:
//   * wave 0 (env): lanes 0..TE-1 keep the env state in registers, read their
//     actions from LDS one step ahead, run the transition, take the next
//     episode's state from the reset ring when an episode ends, and publish
//     the post-step state to an LDS snapshot;
//   * wave 1 (observe): after the step's barrier, paints the snapshot into
//     the observation tile (one lane per observation row), copies the tile to
//     the trajectory with 16-byte stores, clearing it behind the copy, and
//     writes the legal masks, while wave 0 runs step k+1;
//   * wave 2 (reset): a reset state depends only on (seed, env, step), so it
//     is built ahead of need: every LBF_RB steps, the states that would start
//     an episode at each of the steps LBF_RB..2 LBF_RB-1 ahead, one
//     (env, step) per lane, into a ring of 2 LBF_RB slots.
constexpr int LBF_RB = 4;  // steps of reset states built per batch

template <typename T, int A, int F>
__device__ __forceinline__ void lbf_paint_row(const LbfEnv& s, int i, T* xr, int HW) {
  const uint32_t cmax = (uint32_t)HW - 1u;
#pragma unroll
  for (int q = 0; q < A; ++q) xr[min((uint32_t)s.acell[q], cmax)] = small_int_to<T>((uint32_t)s.alevel[q]);
#pragma unroll
  for (int j = 0; j < F; ++j)  // an eaten food writes 0 at its own (distinct) cell: no branch
    xr[HW + min((uint32_t)s.fcell[j], cmax)] = !((s.eaten >> j) & 1u) ? small_int_to<T>((uint32_t)s.flevel[j]) : (T)0;
  xr[2 * HW + min((uint32_t)s.acell[i], cmax)] = small_int_to<T>(1u);
}

template <typename OT, int GH, int GW, int A, int F, int TE>
__global__ __launch_bounds__(192) void lbf_env3_kernel(LbfParams p, int32_t* __restrict__ state, uint64_t t0,
                                                       int n_steps, const int32_t* __restrict__ actions,
                                                       OT* __restrict__ obs, float* __restrict__ reward,
                                                       uint8_t* __restrict__ done, uint8_t* __restrict__ legal) {
  constexpr int HW = GH * GW, D = 3 * HW, R = TE * A;
  constexpr int RS = 2 * LBF_RB;  // reset ring slots: slot k % RS holds the state an episode ending at step k restarts from
  static_assert(TE <= 64 && TE * RS <= 64, "one lane per env, and per (env, step) of the first reset batch");
  static_assert(ACT_CHUNK % LBF_RB == 0, "batches do not straddle action chunks");
  __shared__ __align__(16) OT xs[R * D];
  __shared__ int32_t act_lds[ACT_CHUNK * TE * A];
  __shared__ LbfEnv snap[2][TE];   // post-step state of step k, in slot k % 2
  __shared__ LbfEnv ring[RS][TE];  // reset states
  constexpr int GC = (R * D * sizeof(OT) / 16 + 63) / 64 < 8 ? (R * D * sizeof(OT) / 16 + 63) / 64 : 8;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE;
  const int te_valid = min(TE, p.E - e0);
  const int E = p.E;
  const bool envlane = wave == 0 && lane < te_valid;
  const int e = e0 + lane;
  // wave 2: reset states of steps k0 .. k0+n-1 (drawn at t0 + step + 1), one (env, step) per lane
  auto build_resets = [&](int k0, int n) {
    const int j = lane % TE, u = lane / TE;
    if (u < n && j < te_valid) {
      LbfEnv r{};
      lbf_reset<A, F>(p, (uint64_t)(p.env_base + e0 + j), t0 + (uint64_t)(k0 + u) + 1, r);
      lbf_copy<A, F>(ring[(k0 + u) % RS][j], r);
    }
  };

  zero_lds<192>(xs, sizeof(xs), tid);
  if (wave == 2) build_resets(0, RS);
  LbfEnv s{};
  if (envlane) lbf_load<A, F>(state, p, e, s);
  if (wave == 0) __builtin_amdgcn_s_setprio(3);  // (the transition wave's chain sets the pace)
  for (int k0 = 0; k0 < n_steps; k0 += ACT_CHUNK) {
    const int nk = min(ACT_CHUNK, n_steps - k0);
    stage_actions<TE * A, 192>(actions, E, e0, te_valid * A, A, k0, nk, act_lds, tid);
    __syncthreads();
    int act[LBF_MAXA] = {0, 0, 0, 0};
    if (envlane) {
#pragma unroll
      for (int i = 0; i < A; ++i) act[i] = act_lds[lane * A + i];
    }
    for (int kk = 0; kk < nk; ++kk) {
      const int k = k0 + kk;
      if (wave == 0) {
        if (envlane) {
          uint32_t d = 0;
          float r = 0.f;
          lbf_transition<A, F, GH, GW>(p, s, act, r, d);
          if (d) lbf_copy<A, F>(s, ring[k % RS][lane]);
          lbf_copy<A, F>(snap[k & 1][lane], s);
          if (reward) reward[(size_t)k * E + e] = r;
          if (done) done[(size_t)k * E + e] = (uint8_t)d;
          if (kk + 1 < nk) {
#pragma unroll
            for (int i = 0; i < A; ++i) act[i] = act_lds[(kk + 1) * TE * A + lane * A + i];
          }
        }
      } else if (wave == 2) {
        // slots of steps k+RB .. k+2RB-1: last read at steps k-RB .. k-1
        if (k % LBF_RB == 0) build_resets(k + LBF_RB, LBF_RB);
      }
      __syncthreads();  // snapshot k published (and snapshot k-1 observed)
      if (wave == 1) {
        if (obs) {
          if (lane < te_valid * A) {
            const int el = lane / A, i = lane - el * A;
            lbf_paint_row<OT, A, F>(snap[k & 1][el], i, xs + lane * D, HW);
          }
          copy_obs_rows<OT, R, D, D, 64, true, GC>(xs, obs + ((size_t)k * E + e0) * A * D, te_valid * A, lane);
        }
        if (legal) lbf_write_legal<64>(p, te_valid, legal + ((size_t)k * E + e0) * A * LBF_NACT, lane);
      }
    }
    __syncthreads();  // the chunk's actions are read (and its last tile copied) before the next chunk
  }
  if (envlane) lbf_store<A, F>(state, p, e, s);
}

template <typename OT, int GH, int GW, int A, int F, int TE>
static hipError_t launch_env_ct(const LbfParams& p, int32_t* state, uint64_t t0, int n_steps,
                                const int32_t* actions, void* obs, float* reward, uint8_t* done, uint8_t* legal,
                                hipStream_t s) {
  // bf16: two copy waves keep up with the env wave; steps per barrier: as
  // many as two pairs of tiles fit in a quarter of the LDS
  // (float32 observations: the three-wave kernel)
  if constexpr (sizeof(OT) == 4) {
    lbf_env3_kernel<OT, GH, GW, A, F, TE><<<dim3((unsigned)((p.E + TE - 1) / TE)), 192, 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<OT*>(obs), reward, done, legal);
  } else {
    constexpr int NCW = 2;
    constexpr size_t TILE = (size_t)TE * A * 3 * GH * GW * sizeof(OT);
    constexpr int S = 4 * TILE <= MAX_LDS_BYTES / 4 ? 4 : 2 * TILE <= MAX_LDS_BYTES / 4 ? 2 : 1;
    lbf_env_kernel<OT, GH, GW, A, F, TE, NCW, S><<<dim3((unsigned)((p.E + TE - 1) / TE)), 64 * (NCW + 1), 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<OT*>(obs), reward, done, legal);
  }
  return hipGetLastError();
}

static bool try_launch_env_ct(const LbfParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                              void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s,
                              hipError_t* err) {
  if (p.H == 8 && p.W == 8 && p.A == 2 && p.F == 3) {
    *err = obs_dt == DT_F32 ? launch_env_ct<float, 8, 8, 2, 3, 8>(p, state, t0, n_steps, actions, obs, reward, done,
                                                                   legal, s)
                            : launch_env_ct<uint16_t, 8, 8, 2, 3, 8>(p, state, t0, n_steps, actions, obs, reward,
                                                                      done, legal, s);
    return true;
  }
  if (p.H == 7 && p.W == 7 && p.A == 2 && p.F == 3) {
    *err = obs_dt == DT_F32 ? launch_env_ct<float, 7, 7, 2, 3, 8>(p, state, t0, n_steps, actions, obs, reward, done,
                                                                   legal, s)
                            : launch_env_ct<uint16_t, 7, 7, 2, 3, 8>(p, state, t0, n_steps, actions, obs, reward,
                                                                      done, legal, s);
    return true;
  }
  if (p.H == 12 && p.W == 12 && p.A == 3 && p.F == 6) {
    *err = obs_dt == DT_F32 ? launch_env_ct<float, 12, 12, 3, 6, 8>(p, state, t0, n_steps, actions, obs, reward,
                                                                     done, legal, s)
                            : launch_env_ct<uint16_t, 12, 12, 3, 6, 8>(p, state, t0, n_steps, actions, obs, reward,
                                                                        done, legal, s);
    return true;
  }
  return false;
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

hipError_t launch_lbf_observe(const LbfParams& p, const int32_t* state, uint16_t* obs, hipStream_t s) {
  const LbfMagic m = make_magic(p, LBF_NACT);
  lbf_init_kernel<uint16_t, false><<<tiles(p.E), NTHREADS, 0, s>>>(p, m, const_cast<int32_t*>(state), obs, nullptr);
  return hipGetLastError();
}

hipError_t launch_lbf_step(const LbfParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                           void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s) {
  hipError_t err;
  if (try_launch_env_ct(p, state, t0, n_steps, actions, obs, obs_dt, reward, done, legal, s, &err)) return err;
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
  const LbfMagic m = make_magic(p, pol.NA - pol.VH);
  hipError_t err;
  if (try_launch_rollout_reg(p, m, pol, state, t0, n_steps, out, s, &err)) return err;
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

RL_STAMP_EXPORT(lbf)
