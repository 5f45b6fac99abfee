// Overcooked-style kitchen kernels: init (layout + first episode), env-only
// steps with injected actions, and the fused rollout.
//
// Each workgroup owns a tile of envs; env lane e keeps its kitchen in registers
// (cell sets as 45-bit masks).  Observations live in an LDS tile of
// 2 rows per env x 1170 features: the layout planes are painted once (the
// kitchen never changes), and each step the env lanes erase and repaint only
// the features that can change (agents, facings, held items, pots, and the
// counters whose item changed); the tile is then copied to the trajectory.
// The fused rollout runs the policy with the streaming MFMA MLP of rl_mlp.h
// (weights read from L2 every step) and samples one action per (row, action)
// lane.
#include "rl_internal.h"
#include "rl_overcooked.h"
#include "rl_sample.h"

namespace rl {

RL_STAMP_TABLE


constexpr int OC_TE = 8;  // envs per workgroup of the init kernel (one wave)
// env-only kernel: envs per workgroup and threads (one env wave, the rest copy)
constexpr int OC_ENV_TE_BF16 = 16, OC_ENV_NT_BF16 = 256;
constexpr int OC_ENV_TE_F32 = 8, OC_ENV_NT_F32 = 256;

template <typename T>
__device__ __forceinline__ void oc_put(T* xr, int plane, int cell, uint32_t v) {
  xr[plane * OC_NCELL + cell] = small_int_to<T>(v);
}

// Layout planes 10-14 of both rows of env el (never change during a launch).
template <typename T>
__device__ __forceinline__ void oc_paint_static(const OcEnv& s, T* tile, int ld, int el) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    T* xr = tile + (size_t)(el * 2 + i) * ld;
    const uint64_t kinds[5] = {s.counter, s.onion, s.plate, s.pot, s.serve};
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      uint64_t m = kinds[k];
      while (m) {
        oc_put(xr, 10 + k, __builtin_ctzll(m), 1u);
        m &= m - 1;
      }
    }
  }
}

// Agent, facing, held and pot features of both rows (on: write, else erase).
template <typename T>
__device__ __forceinline__ void oc_paint_agents(const OcEnv& s, T* tile, int ld, int el, bool on) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    T* xr = tile + (size_t)(el * 2 + i) * ld;
    const int me = i, ot = 1 - i;
    const uint32_t one = on ? 1u : 0u;
    oc_put(xr, 0, s.acell[me], one);
    oc_put(xr, 1, s.acell[ot], one);
    oc_put(xr, 2 + (s.face[me] & 3), s.acell[me], one);
    oc_put(xr, 6 + (s.face[ot] & 3), s.acell[ot], one);
    if (s.held[me]) oc_put(xr, 17 + (s.held[me] & 3), s.acell[me], one);
    if (s.held[ot]) oc_put(xr, 20 + (s.held[ot] & 3), s.acell[ot], one);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      if (s.pcell[j] >= 0) {
        oc_put(xr, 24, s.pcell[j], on ? (uint32_t)s.pon[j] : 0u);
        oc_put(xr, 25, s.pcell[j], on ? (uint32_t)s.ptm[j] : 0u);
      }
  }
}

// Item features (planes 15-17) at the counters in `cells`: erase all three,
// then write the item currently there.
template <typename T>
__device__ __forceinline__ void oc_paint_items(const OcEnv& s, T* tile, int ld, int el, uint64_t cells) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    T* xr = tile + (size_t)(el * 2 + i) * ld;
    uint64_t m = cells;
    while (m) {
      const int c = __builtin_ctzll(m);
      m &= m - 1;
      oc_put(xr, 15, c, 0u);
      oc_put(xr, 16, c, 0u);
      oc_put(xr, 17, c, 0u);
      const int it = oc_item_at(s, c);
      if (it) oc_put(xr, 14 + it, c, 1u);
    }
  }
}

template <typename T>
__device__ __forceinline__ void oc_paint_all(const OcEnv& s, T* tile, int ld, int el) {
  oc_paint_static(s, tile, ld, el);
  oc_paint_agents(s, tile, ld, el, true);
  oc_paint_items(s, tile, ld, el, s.it_onion | s.it_plate | s.it_soup);
}

// One env step of env lane el (tile rows el*2, el*2+1 kept in sync).
template <typename T>
__device__ __forceinline__ void oc_step_lane(const OcParams& p, OcEnv& s, int el, uint64_t genv, uint64_t t,
                                             const int (&act)[2], T* tile, int ld, float& r, uint32_t& d) {
  oc_paint_agents(s, tile, ld, el, false);
  uint64_t changed;
  oc_transition(p, s, act, r, d, changed);
  if (d) {
    const uint64_t had = s.it_onion | s.it_plate | s.it_soup;
    oc_reset(p, genv, t + 1, s);
    oc_paint_items(s, tile, ld, el, had | changed);
  } else {
    oc_paint_items(s, tile, ld, el, changed);
  }
  oc_paint_agents(s, tile, ld, el, true);
}

// -------------------------------------------------------------- init ----

template <typename OT>
__global__ __launch_bounds__(64) void oc_init_kernel(OcParams p, int32_t* __restrict__ state, OT* __restrict__ obs,
                                                     uint8_t* __restrict__ legal) {
  __shared__ __align__(16) OT tile[OC_TE * 2 * OC_D];
  const int lane = threadIdx.x, e0 = blockIdx.x * OC_TE, te_valid = min(OC_TE, p.E - e0);
  zero_lds<64>(tile, sizeof(tile), lane);
  wave_lds_sync();
  if (lane < te_valid) {
    OcEnv s;
    const uint64_t genv = (uint64_t)(p.env_base + e0 + lane);
    oc_layout(p, genv, s);
    oc_reset(p, genv, 0, s);
    oc_store(state, p.E, e0 + lane, s);
    oc_paint_all(s, tile, OC_D, lane);
  }
  wave_lds_sync();
  if (obs) copy_tile(tile, obs + (size_t)e0 * 2 * OC_D, te_valid * 2 * OC_D, lane, 64);
  if (legal)
    for (int i = lane; i < te_valid * 2 * OC_NACT; i += 64) legal[(size_t)e0 * 2 * OC_NACT + i] = 1;
}

// ---------------------------------------------------------- env-only ----

// One workgroup steps TE kitchens with two observation tiles: step k's tile
// is tile[k & 1]. The env lanes (wave 0) run step k's transition and bring
// tile[k & 1] from o_{k-2} up to o_k while the other waves copy tile
// [(k-1) & 1] (o_{k-1}) to the trajectory; one barrier per step. Going from
// o_{k-2} to o_k erases the agents of s_{k-2}, repaints the counters whose
// item changed in either step and paints the agents of s_k (the agent,
// facing, held and pot planes never overlap the item planes). Before the
// first step both tiles hold the launch's observation, whose agents are
// those of the launch state.
template <typename OT, int TE, int NT>
__global__ __launch_bounds__(NT) void oc_env_kernel(OcParams p, int32_t* __restrict__ state, uint64_t t0, int n_steps,
                                                    const int32_t* __restrict__ actions, OT* __restrict__ obs,
                                                    float* __restrict__ reward, uint8_t* __restrict__ done,
                                                    uint8_t* __restrict__ legal) {
  static_assert(TE <= 64 && NT % 64 == 0 && NT >= 128, "env lanes in wave 0, copy waves after it");
  constexpr int TS = TE * 2 * OC_D;
  __shared__ __align__(16) OT tile[2 * TS];
  __shared__ int32_t act_lds[ACT_CHUNK * TE * 2];
  const int tid = threadIdx.x, e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0);
  const int E = p.E;
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  zero_lds<NT>(tile, sizeof(tile), tid);
  __syncthreads();
  OcEnv s, s_pp;  // s_pp: the state whose agents tile[k & 1] shows when step k starts
  uint64_t mask_prev = 0;  // counters whose item changed in the previous step
  if (envlane) {
    oc_load(state, E, e, s);
    oc_paint_all(s, tile, OC_D, tid);
    oc_paint_all(s, tile + TS, OC_D, tid);
    s_pp = s;
  }
  if (tid < 64) __builtin_amdgcn_s_setprio(3);
  auto emit = [&](int k, int i0, int stride) {
    if (obs) copy_tile(tile + (k & 1) * TS, obs + ((size_t)k * E + e0) * 2 * OC_D, te_valid * 2 * OC_D, i0, stride);
    if (legal)
      for (int i = i0; i < te_valid * 2 * OC_NACT; i += stride) legal[((size_t)k * E + e0) * 2 * OC_NACT + i] = 1;
  };
  for (int k0 = 0; k0 < n_steps; k0 += ACT_CHUNK) {
    const int nk = min(ACT_CHUNK, n_steps - k0);
    // no global loads inside the step loop: a load there would wait for every earlier trajectory store
    stage_actions<TE * 2, NT>(actions, E, e0, te_valid * 2, 2, k0, nk, act_lds, tid);
    __syncthreads();
    for (int kk = 0; kk < nk; ++kk) {
      const int k = k0 + kk;
      const uint64_t t = t0 + (uint64_t)k;
      if (envlane) {
        const int act[2] = {act_lds[kk * TE * 2 + tid * 2], act_lds[kk * TE * 2 + tid * 2 + 1]};
        const OcEnv s_prev = s;
        float r;
        uint32_t d;
        uint64_t changed;
        oc_transition(p, s, act, r, d, changed);
        if (d) {
          changed |= s.it_onion | s.it_plate | s.it_soup;
          oc_reset(p, (uint64_t)(p.env_base + e), t + 1, s);
        }
        if (reward) reward[(size_t)k * E + e] = r;
        if (done) done[(size_t)k * E + e] = (uint8_t)d;
        OT* tk = tile + (k & 1) * TS;
        oc_paint_agents(s_pp, tk, OC_D, tid, false);
        oc_paint_items(s, tk, OC_D, tid, mask_prev | changed);
        oc_paint_agents(s, tk, OC_D, tid, true);
        s_pp = s_prev;
        mask_prev = changed;
      } else if (tid >= 64 && k > 0) {
        emit(k - 1, tid - 64, NT - 64);
      }
      __syncthreads();
    }
  }
  if (n_steps > 0) emit(n_steps - 1, tid, NT);
  if (envlane) oc_store(state, E, e, s);
}

// ----------------------------------------------------- fused rollout ----

constexpr int OC_RUN_NT = 512;  // 8 waves: the streamed MLP's chains of a workgroup spread over twice the waves

template <int DT, int TE, bool PK>
__global__ __launch_bounds__(OC_RUN_NT) void oc_run_kernel(OcParams p, PolicyArgs pol, int32_t* __restrict__ state,
                                                          uint64_t t0, int n_steps, TrajArgs out) {
  using T = typename DType<DT>::T;
  constexpr int R = TE * 2, NA = OC_NACT;
  constexpr int LDX = lds_ld<DT>(OC_D);
  extern __shared__ __align__(16) uint8_t smem[];
  const int ld1 = lds_ld<DT>(pol.H1), ld2 = lds_ld<DT>(pol.H2);
  T* xs = reinterpret_cast<T*>(smem);
  T* h1 = xs + R * LDX;
  T* h2 = h1 + R * ld1;
  float* lg = reinterpret_cast<float*>(h2 + R * ld2);
  float* sc = lg + R * MAX_NA;
  int* act_s = reinterpret_cast<int*>(sc + R * MAX_NA);
  float* nz = reinterpret_cast<float*>(act_s + R);  // Gumbel noise of the next step's (row, action)
  const size_t total = (size_t)((uint8_t*)(nz + R * MAX_NA) - smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0), E = p.E;
  const T* W1 = static_cast<const T*>(pol.W[0]);
  const T* W2 = static_cast<const T*>(pol.W[1]);
  const T* W3 = static_cast<const T*>(pol.W[2]);
  const T* b1 = static_cast<const T*>(pol.b[0]);
  const T* b2 = static_cast<const T*>(pol.b[1]);
  const T* b3 = static_cast<const T*>(pol.b[2]);
  zero_lds<OC_RUN_NT>(smem, total, tid);
  __syncthreads();
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  // the noise of step kn's (row, action) items, threads i0, i0 + stride, ...
  auto draw_noise = [&](int kn, int i0, int stride) {
    for (int idx = i0; idx < R * NA; idx += stride) {
      const int r = idx / NA, a = idx - r * NA, el = r >> 1, ag = r & 1;
      nz[r * MAX_NA + a] =
          el < te_valid ? action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t0 + (uint64_t)kn, ag, a) : 0.f;
    }
  };
  OcEnv s;
  if (envlane) {
    oc_load(state, E, e, s);
    oc_paint_all(s, xs, LDX, tid);
  }
  if (n_steps > 0) draw_noise(0, tid, OC_RUN_NT);
  __builtin_amdgcn_s_waitcnt(0);
  RL_STAMP_BEGIN
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    __syncthreads();  // the env lanes' repaint of the previous step is visible
    RL_STAMP(0)
    mlp_input_layer_const<DT, OC_D, PK>(xs, LDX, nullptr, R, W1, b1, pol.H1, h1, ld1, wave, OC_RUN_NT / 64, lane,
                                        static_cast<const T*>(pol.Wp[0]));
    __syncthreads();
    RL_STAMP(1)
    mlp_hidden<DT, PK>(h1, ld1, R, pol.H1, W2, b2, pol.H2, h2, ld2, wave, OC_RUN_NT / 64, lane,
                       static_cast<const T*>(pol.Wp[1]));
    __syncthreads();
    RL_STAMP(2)
    mlp_logits<DT, PK>(h2, ld2, R, pol.H2, W3, b3, NA, lg, MAX_NA, wave, OC_RUN_NT / 64, lane,
                       static_cast<const T*>(pol.Wp[2]));
    __syncthreads();
    RL_STAMP(3)
    for (int idx = tid; idx < R * NA; idx += OC_RUN_NT) {
      const int r = idx / NA, a = idx - r * NA, el = r >> 1, ag = r & 1;
      if (el < te_valid) {
        sc[r * MAX_NA + a] = action_score(lg[r * MAX_NA + a], nz[r * MAX_NA + a], true);
        if (out.logits) out.logits[((size_t)k * E + e0) * 2 * NA + idx] = lg[r * MAX_NA + a];
      }
    }
    RL_STAMP(4)
    __syncthreads();
    RL_STAMP(6)
    if (tid < R && (tid >> 1) < te_valid) {
      int best = 0;
      float bs = -INFINITY;
      for (int a = 0; a < NA; ++a) {
        const float v = sc[tid * MAX_NA + a];
        if (v > bs) {
          bs = v;
          best = a;
        }
      }
      act_s[tid] = best;
      if (out.actions) out.actions[((size_t)k * E + e0) * 2 + tid] = best;
    }
    __syncthreads();
    RL_STAMP(7)
    // The env lanes step the kitchens (oc_step_lane, with the tile's repaint
    // deferred) while the other waves copy o_t to the trajectory (after the
    // step's weight loads: a wave's loads wait for its earlier stores, one
    // in-order counter); after a barrier the env lanes repaint.  The other
    // waves draw the next step's noise (it depends on nothing the step
    // computes) during the repaint, or, with no trajectory copy, during the
    // transition.
    OcEnv s_old;
    uint64_t changed = 0, had = 0;
    uint32_t d = 0;
    if (envlane) {
      const int act[2] = {act_s[tid * 2], act_s[tid * 2 + 1]};
      float r;
      s_old = s;
      oc_transition(p, s, act, r, d, changed);
      if (d) {
        had = s.it_onion | s.it_plate | s.it_soup;
        oc_reset(p, (uint64_t)(p.env_base + e), t + 1, s);
      }
      if (out.reward) out.reward[(size_t)k * E + e] = r;
      if (out.done) out.done[(size_t)k * E + e] = (uint8_t)d;
    } else if (tid >= 64) {
      if (out.obs)
        copy_rows_global16(xs, LDX, static_cast<T*>(out.obs) + ((size_t)k * E + e0) * 2 * OC_D, OC_D,
                           te_valid * 2, tid - 64, OC_RUN_NT - 64);
      RL_STAMP(5)
      if (!out.obs && k + 1 < n_steps) draw_noise(k + 1, tid - 64, OC_RUN_NT - 64);
    }
    RL_STAMP(8)
    __syncthreads();  // o_t is copied out
    RL_STAMP(9)
    if (envlane) {  // the tile becomes o_{t+1}: oc_step_lane's paints, in its order
      oc_paint_agents(s_old, xs, LDX, tid, false);
      oc_paint_items(s, xs, LDX, tid, d ? (had | changed) : changed);
      oc_paint_agents(s, xs, LDX, tid, true);
    } else if (tid >= 64 && out.obs && k + 1 < n_steps) {
      draw_noise(k + 1, tid - 64, OC_RUN_NT - 64);
    }
    RL_STAMP(10)
  }
  RL_STAMP_END(wave == 0 ? 0 : 1)
  __syncthreads();
  if (out.obs_last)
    copy_rows_global16(xs, LDX, static_cast<T*>(out.obs_last) + (size_t)e0 * 2 * OC_D, OC_D, te_valid * 2, tid,
                       OC_RUN_NT);
  if (envlane) oc_store(state, E, e, s);
}

// ---------------------------------------------------------- launchers ----

static dim3 oc_tiles(int E, int te) { return dim3((unsigned)((E + te - 1) / te)); }

// LDS of the fused kitchen rollout with te envs (2 * te policy rows) per workgroup.
static size_t oc_run_lds_bytes_te(const PolicyArgs& pol, int te) {
  const int R = te * 2;
  const size_t es = pol.dt == DT_F32 ? 4 : 2;
  const int ldx = pol.dt == DT_F32 ? lds_ld<DT_F32>(OC_D) : lds_ld<DT_BF16>(OC_D);
  const int ld1 = pol.dt == DT_F32 ? lds_ld<DT_F32>(pol.H1) : lds_ld<DT_BF16>(pol.H1);
  const int ld2 = pol.dt == DT_F32 ? lds_ld<DT_F32>(pol.H2) : lds_ld<DT_BF16>(pol.H2);
  return (size_t)R * (ldx + ld1 + ld2) * es + (size_t)R * MAX_NA * 4 * 3 + (size_t)R * 4;
}

// 16 envs per workgroup (two row tiles share every weight fragment) when their tiles fit in LDS, else 8.
static int oc_run_te(const PolicyArgs& pol) { return oc_run_lds_bytes_te(pol, 16) <= MAX_LDS_BYTES ? 16 : 8; }

size_t oc_run_lds_bytes(const PolicyArgs& pol) { return oc_run_lds_bytes_te(pol, oc_run_te(pol)); }

hipError_t launch_oc_init(const OcParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal, hipStream_t s) {
  if (obs_dt == DT_F32)
    oc_init_kernel<float><<<oc_tiles(p.E, OC_TE), 64, 0, s>>>(p, state, static_cast<float*>(obs), legal);
  else
    oc_init_kernel<uint16_t><<<oc_tiles(p.E, OC_TE), 64, 0, s>>>(p, state, static_cast<uint16_t*>(obs), legal);
  return hipGetLastError();
}

hipError_t launch_oc_step(const OcParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                          void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s) {
  if (obs_dt == DT_F32)
    oc_env_kernel<float, OC_ENV_TE_F32, OC_ENV_NT_F32><<<oc_tiles(p.E, OC_ENV_TE_F32), OC_ENV_NT_F32, 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<float*>(obs), reward, done, legal);
  else
    oc_env_kernel<uint16_t, OC_ENV_TE_BF16, OC_ENV_NT_BF16><<<oc_tiles(p.E, OC_ENV_TE_BF16), OC_ENV_NT_BF16, 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<uint16_t*>(obs), reward, done, legal);
  return hipGetLastError();
}

template <int DT, int TE, bool PK>
static hipError_t launch_oc_run_te(const OcParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0,
                                   int n_steps, const TrajArgs& out, size_t lds, hipStream_t s) {
  hipError_t e = hipFuncSetAttribute((const void*)oc_run_kernel<DT, TE, PK>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  oc_run_kernel<DT, TE, PK><<<oc_tiles(p.E, TE), OC_RUN_NT, lds, s>>>(p, pol, state, t0, n_steps, out);
  return hipGetLastError();
}

hipError_t launch_oc_run(const OcParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                         const TrajArgs& out, hipStream_t s) {
  const int te = oc_run_te(pol);
  const size_t lds = oc_run_lds_bytes_te(pol, te);
  if (pol.dt == DT_F32)
    return te == 16 ? launch_oc_run_te<DT_F32, 16, false>(p, pol, state, t0, n_steps, out, lds, s)
                    : launch_oc_run_te<DT_F32, 8, false>(p, pol, state, t0, n_steps, out, lds, s);
  if (pol.Wp[0] != nullptr)  // fragment-major weights
    return te == 16 ? launch_oc_run_te<DT_BF16, 16, true>(p, pol, state, t0, n_steps, out, lds, s)
                    : launch_oc_run_te<DT_BF16, 8, true>(p, pol, state, t0, n_steps, out, lds, s);
  return te == 16 ? launch_oc_run_te<DT_BF16, 16, false>(p, pol, state, t0, n_steps, out, lds, s)
                  : launch_oc_run_te<DT_BF16, 8, false>(p, pol, state, t0, n_steps, out, lds, s);
}

}  // namespace rl

RL_STAMP_EXPORT(oc)
