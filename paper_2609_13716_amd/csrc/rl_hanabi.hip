// Two-player Hanabi kernels: init (deal), env-only steps with injected
// actions, and the fused rollout.
//
// Env lane e of wave 0 holds its game in registers (rl_hanabi.h).  After
// every move it publishes what the observation reads (HnView) and the
// mover's legal-action mask to LDS; then all threads of the workgroup paint
// the two 658-feature observations of every env of the tile, feature-parallel
// (consecutive lanes take consecutive features of one row), into an LDS tile
// that is copied to the trajectory.  In the fused rollout only the mover's
// row goes through the policy (the other player has no legal action): its
// rows are gathered from the tile by index, and the MLP is the streaming
// MFMA MLP of rl_mlp.h.
#include "rl_hanabi.h"
#include "rl_internal.h"
#include "rl_sample.h"

namespace rl {

constexpr int HN_DECK_SLOT = 52;  // LDS bytes of one lane's Fisher-Yates deck

struct HnTile {
  HnView view;
  uint32_t legal;  // mover's 20-bit legal mask
};

// Paint rows 2*el + me (el < te_valid) of the observation tile.
template <typename T, int TE, int NT>
__device__ __forceinline__ void hn_paint(const HnTile* __restrict__ envs, int te_valid, T* tile, int ld, int tid) {
  const int n = 2 * te_valid * HN_OBS;
  for (int idx = tid; idx < n; idx += NT) {
    const int r = idx / HN_OBS, f = idx - r * HN_OBS;
    tile[(size_t)r * ld + f] = small_int_to<T>(hn_feature(envs[r >> 1].view, r & 1, f));
  }
}

// Copy `rows` rows of `len` elements from an LDS tile (leading dimension ld)
// to consecutive global rows; rows of 4-byte multiples, 4-byte words.
template <typename T, int NT>
__device__ __forceinline__ void hn_copy_rows(const T* src, int ld, T* __restrict__ dst, int len, int rows, int tid) {
  constexpr int PER = 4 / (int)sizeof(T);
  const int wpr = len / PER, ldw = ld / PER;
  const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
  uint32_t* g = reinterpret_cast<uint32_t*>(dst);
  for (int i = tid; i < rows * wpr; i += NT) {
    const int r = i / wpr, w = i - r * wpr;
    g[i] = s[r * ldw + w];
  }
}

// Legal masks of both players of envs 0..te_valid-1 ([env][agent][20] bytes).
template <int NT>
__device__ __forceinline__ void hn_write_legal(const HnTile* __restrict__ envs, int te_valid, uint8_t* __restrict__ g,
                                               int tid) {
  for (int i = tid; i < te_valid * 2 * HN_NACT; i += NT) {
    const int el = i / (2 * HN_NACT), rem = i - el * 2 * HN_NACT, ag = rem / HN_NACT, a = rem - ag * HN_NACT;
    g[i] = (ag == envs[el].view.cur) ? (uint8_t)((envs[el].legal >> a) & 1u) : (uint8_t)0;
  }
}

__device__ __forceinline__ void hn_publish(const HnEnv& s, HnTile& t) {
  hn_view(s, t.view);
  t.legal = hn_legal(s);
}

// -------------------------------------------------------------- init ----

template <typename OT, int TE>
__global__ __launch_bounds__(NTHREADS) void hn_init_kernel(HnParams p, int32_t* __restrict__ state,
                                                           OT* __restrict__ obs, uint8_t* __restrict__ legal) {
  __shared__ HnTile envs[TE];
  __shared__ __align__(16) uint8_t decks[TE][HN_DECK_SLOT];
  __shared__ __align__(16) OT tile[2 * TE * HN_OBS];
  const int tid = threadIdx.x, e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0);
  if (tid < te_valid) {
    HnEnv s;
    hn_reset(p, (uint64_t)(p.env_base + e0 + tid), 0, s, decks[tid]);
    hn_store(state, p.E, e0 + tid, s);
    hn_publish(s, envs[tid]);
  }
  __syncthreads();
  if (obs) {
    hn_paint<OT, TE, NTHREADS>(envs, te_valid, tile, HN_OBS, tid);
    __syncthreads();
    hn_copy_rows<OT, NTHREADS>(tile, HN_OBS, obs + (size_t)e0 * 2 * HN_OBS, HN_OBS, 2 * te_valid, tid);
  }
  if (legal) hn_write_legal<NTHREADS>(envs, te_valid, legal + (size_t)e0 * 2 * HN_NACT, tid);
}

// ---------------------------------------------------------- env-only ----

template <typename OT, int TE>
__global__ __launch_bounds__(NTHREADS) void hn_env_kernel(HnParams p, int32_t* __restrict__ state, uint64_t t0,
                                                          int n_steps, const int32_t* __restrict__ actions,
                                                          OT* __restrict__ obs, float* __restrict__ reward,
                                                          uint8_t* __restrict__ done, uint8_t* __restrict__ legal) {
  __shared__ HnTile envs[TE];
  __shared__ __align__(16) uint8_t decks[TE][HN_DECK_SLOT];
  __shared__ __align__(16) OT tile[2 * TE * HN_OBS];
  const int tid = threadIdx.x, e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0), E = p.E;
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  HnEnv s;
  if (envlane) hn_load(state, E, e, s);
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    if (envlane) {
      float r;
      uint32_t d;
      hn_transition(p, s, actions[((size_t)k * E + e) * 2 + s.cur], r, d);
      if (d) hn_reset(p, (uint64_t)(p.env_base + e), t + 1, s, decks[tid]);
      hn_publish(s, envs[tid]);
      if (reward) reward[(size_t)k * E + e] = r;
      if (done) done[(size_t)k * E + e] = (uint8_t)d;
    }
    __syncthreads();
    if (obs) {
      hn_paint<OT, TE, NTHREADS>(envs, te_valid, tile, HN_OBS, tid);
      __syncthreads();
      hn_copy_rows<OT, NTHREADS>(tile, HN_OBS, obs + ((size_t)k * E + e0) * 2 * HN_OBS, HN_OBS, 2 * te_valid, tid);
    }
    if (legal) hn_write_legal<NTHREADS>(envs, te_valid, legal + ((size_t)k * E + e0) * 2 * HN_NACT, tid);
    __syncthreads();  // the tile and masks are read before the next move rewrites them
  }
  if (envlane) hn_store(state, E, e, s);
}

// ----------------------------------------------------- fused rollout ----

constexpr int HN_RUN_TE = 16;  // envs (and mover rows) per workgroup

struct HnRunLayout {
  int ldx, ld1, ld2;
  size_t off_x, off_h1, off_h2, off_lg, off_sc, off_env, off_deck, off_rows, total;
};

__host__ __device__ inline HnRunLayout hn_run_layout(int H1, int H2, int dt) {
  HnRunLayout L;
  const size_t es = dt == DT_F32 ? 4 : 2;
  L.ldx = dt == DT_F32 ? lds_ld<DT_F32>(HN_OBS) : lds_ld<DT_BF16>(HN_OBS);
  L.ld1 = dt == DT_F32 ? lds_ld<DT_F32>(H1) : lds_ld<DT_BF16>(H1);
  L.ld2 = dt == DT_F32 ? lds_ld<DT_F32>(H2) : lds_ld<DT_BF16>(H2);
  size_t o = 0;
  L.off_x = o;    o += (size_t)2 * HN_RUN_TE * L.ldx * es;
  L.off_h1 = o;   o += (size_t)HN_RUN_TE * L.ld1 * es;
  L.off_h2 = o;   o += (size_t)HN_RUN_TE * L.ld2 * es;
  L.off_lg = o;   o += (size_t)HN_RUN_TE * MAX_NA * 4;
  L.off_sc = o;   o += (size_t)HN_RUN_TE * MAX_NA * 4;
  L.off_env = o;  o += (size_t)HN_RUN_TE * sizeof(HnTile);
  o = (o + 15) & ~(size_t)15;
  L.off_deck = o; o += (size_t)HN_RUN_TE * HN_DECK_SLOT;
  L.off_rows = o; o += (size_t)HN_RUN_TE * 4;
  L.total = o;
  return L;
}

size_t hn_run_lds_bytes(const PolicyArgs& pol) { return hn_run_layout(pol.H1, pol.H2, pol.dt).total; }

template <int DT>
__global__ __launch_bounds__(NTHREADS) void hn_run_kernel(HnParams p, PolicyArgs pol, int32_t* __restrict__ state,
                                                          uint64_t t0, int n_steps, TrajArgs out) {
  using T = typename DType<DT>::T;
  constexpr int TE = HN_RUN_TE, NA = HN_NACT;
  extern __shared__ __align__(16) uint8_t smem[];
  const HnRunLayout L = hn_run_layout(pol.H1, pol.H2, DT);
  T* xs = reinterpret_cast<T*>(smem + L.off_x);
  T* h1 = reinterpret_cast<T*>(smem + L.off_h1);
  T* h2 = reinterpret_cast<T*>(smem + L.off_h2);
  float* lg = reinterpret_cast<float*>(smem + L.off_lg);
  float* sc = reinterpret_cast<float*>(smem + L.off_sc);
  HnTile* envs = reinterpret_cast<HnTile*>(smem + L.off_env);
  uint8_t* decks = smem + L.off_deck;
  int* rows = reinterpret_cast<int*>(smem + L.off_rows);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0), E = p.E;
  const T* W1 = static_cast<const T*>(pol.W[0]);
  const T* W2 = static_cast<const T*>(pol.W[1]);
  const T* W3 = static_cast<const T*>(pol.W[2]);
  const T* b1 = static_cast<const T*>(pol.b[0]);
  const T* b2 = static_cast<const T*>(pol.b[1]);
  const T* b3 = static_cast<const T*>(pol.b[2]);
  zero_lds(smem, L.total, tid);
  __syncthreads();
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  HnEnv s;
  if (envlane) {
    hn_load(state, E, e, s);
    hn_publish(s, envs[tid]);
  }
  if (tid < TE) rows[tid] = 2 * tid + (envlane ? s.cur : 0);  // the mover's row (a zero row for padding)
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    __syncthreads();  // the previous move's views are published
    hn_paint<T, TE, NTHREADS>(envs, te_valid, xs, L.ldx, tid);
    __syncthreads();
    if (out.obs)
      hn_copy_rows<T, NTHREADS>(xs, L.ldx, static_cast<T*>(out.obs) + ((size_t)k * E + e0) * 2 * HN_OBS, HN_OBS,
                                2 * te_valid, tid);
    mlp_hidden_rows<DT>(xs, L.ldx, rows, TE, HN_OBS, W1, b1, pol.H1, h1, L.ld1, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_hidden<DT>(h1, L.ld1, TE, pol.H1, W2, b2, pol.H2, h2, L.ld2, wave, NTHREADS / 64, lane);
    __syncthreads();
    mlp_logits<DT>(h2, L.ld2, TE, pol.H2, W3, b3, NA, lg, MAX_NA, wave, NTHREADS / 64, lane);
    __syncthreads();
    for (int idx = tid; idx < te_valid * NA; idx += NTHREADS) {
      const int el = idx / NA, a = idx - el * NA;
      const int cur = envs[el].view.cur;
      const bool ok = (envs[el].legal >> a) & 1u;
      const float g = action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t, cur, a);
      sc[el * MAX_NA + a] = action_score(lg[el * MAX_NA + a], g, ok);
      if (out.logits) {
        float* lo = out.logits + ((size_t)k * E + e0 + el) * 2 * NA;
        lo[cur * NA + a] = ok ? lg[el * MAX_NA + a] : -INFINITY;
        lo[(1 - cur) * NA + a] = -INFINITY;
      }
    }
    __syncthreads();
    if (envlane) {
      int best = 0;
      float bs = -INFINITY;
      for (int a = 0; a < NA; ++a) {
        const float v = sc[tid * MAX_NA + a];
        if (v > bs) {
          bs = v;
          best = a;
        }
      }
      if (out.actions) {
        out.actions[((size_t)k * E + e) * 2 + s.cur] = best;
        out.actions[((size_t)k * E + e) * 2 + 1 - s.cur] = 0;
      }
      float r;
      uint32_t d;
      hn_transition(p, s, best, r, d);
      if (d) hn_reset(p, (uint64_t)(p.env_base + e), t + 1, s, decks + tid * HN_DECK_SLOT);
      hn_publish(s, envs[tid]);
      rows[tid] = 2 * tid + s.cur;
      if (out.reward) out.reward[(size_t)k * E + e] = r;
      if (out.done) out.done[(size_t)k * E + e] = (uint8_t)d;
    }
  }
  __syncthreads();
  if (out.obs_last) {
    hn_paint<T, TE, NTHREADS>(envs, te_valid, xs, L.ldx, tid);
    __syncthreads();
    hn_copy_rows<T, NTHREADS>(xs, L.ldx, static_cast<T*>(out.obs_last) + (size_t)e0 * 2 * HN_OBS, HN_OBS,
                              2 * te_valid, tid);
  }
  if (envlane) hn_store(state, E, e, s);
}

// ---------------------------------------------------------- launchers ----

constexpr int HN_ENV_TE = 8;  // envs per workgroup of the init and env-only kernels

static dim3 hn_tiles(int E, int te) { return dim3((unsigned)((E + te - 1) / te)); }

hipError_t launch_hn_init(const HnParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal, hipStream_t s) {
  if (obs_dt == DT_F32)
    hn_init_kernel<float, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(p, state, static_cast<float*>(obs),
                                                                                  legal);
  else
    hn_init_kernel<uint16_t, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(
        p, state, static_cast<uint16_t*>(obs), legal);
  return hipGetLastError();
}

hipError_t launch_hn_step(const HnParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                          void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s) {
  if (obs_dt == DT_F32)
    hn_env_kernel<float, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<float*>(obs), reward, done, legal);
  else
    hn_env_kernel<uint16_t, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<uint16_t*>(obs), reward, done, legal);
  return hipGetLastError();
}

hipError_t launch_hn_run(const HnParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                         const TrajArgs& out, hipStream_t s) {
  const size_t lds = hn_run_lds_bytes(pol);
  const void* fn = pol.dt == DT_F32 ? (const void*)hn_run_kernel<DT_F32> : (const void*)hn_run_kernel<DT_BF16>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)MAX_LDS_BYTES);
  if (e != hipSuccess) return e;
  if (pol.dt == DT_F32)
    hn_run_kernel<DT_F32><<<hn_tiles(p.E, HN_RUN_TE), NTHREADS, lds, s>>>(p, pol, state, t0, n_steps, out);
  else
    hn_run_kernel<DT_BF16><<<hn_tiles(p.E, HN_RUN_TE), NTHREADS, lds, s>>>(p, pol, state, t0, n_steps, out);
  return hipGetLastError();
}

}  // namespace rl
