// Internal interface between the C-ABI layer and the kernel translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rl_lbf.h"
#include "rl_mlp.h"
#include "rl_hanabi.h"
#include "rl_overcooked.h"

namespace rl {

constexpr int TILE_E = 16;     // envs per workgroup in the env and rollout kernels
constexpr int NTHREADS = 256;  // threads per workgroup (4 waves of 64)
constexpr int MAX_NA = 32;     // largest action count of a policy head

// Exact division by small divisors: x / d == umulhi(x, ceil(2^32 / d)) for
// d >= 2 and x < 2^32 / d; d == 1 is flagged by magic == 0.
__host__ __device__ inline uint32_t div_magic(uint32_t d) {
  return d <= 1 ? 0u : (uint32_t)((((uint64_t)1 << 32) + d - 1) / d);
}
__device__ __forceinline__ int fdiv(int x, uint32_t magic) {
  return magic ? (int)__umulhi((uint32_t)x, magic) : x;
}

// Phase stamps, compiled in only by the instrumented build (RL_PHASE_STAMPS;
// every macro is empty otherwise).  Each wave adds the shader-clock cycles
// (s_memtime) between consecutive marks of a kernel's step loop to
// per-phase counters and, when the kernel ends, into a device table
// [role][phase] summed over the grid (the role is the wave's part in its
// workgroup, chosen by the kernel; the last phase counter of a role counts
// its waves).  A translation unit that stamps declares
// its table with RL_STAMP_TABLE and exports a reader with
// RL_STAMP_EXPORT(unit): rl_phase_stamps_<unit>(out, reset) copies the
// table to `out` (RL_STAMP_ROLES x RL_STAMP_PHASES counters) and clears it
// when `reset` is non-zero.
constexpr int RL_STAMP_PHASES = 12, RL_STAMP_ROLES = 8;
#ifdef RL_PHASE_STAMPS
#define RL_STAMP_TABLE static __device__ unsigned long long rl_stamp_table[RL_STAMP_ROLES * RL_STAMP_PHASES];
#define RL_STAMP_BEGIN                                   \
  uint64_t rl_st_last = __builtin_amdgcn_s_memtime(); \
  uint64_t rl_st[RL_STAMP_PHASES] = {};
#define RL_STAMP(i)                                            \
  {                                                            \
    const uint64_t rl_now = __builtin_amdgcn_s_memtime();     \
    rl_st[i] += rl_now - rl_st_last;                           \
    rl_st_last = rl_now;                                       \
  }
#define RL_STAMP_END(role)                                                                   \
  rl_st[RL_STAMP_PHASES - 1] = 1; /* the last counter counts the waves of the role */       \
  if ((threadIdx.x & 63) == 0)                                                               \
    for (int rl_i = 0; rl_i < RL_STAMP_PHASES; ++rl_i)                                       \
      atomicAdd(&rl_stamp_table[((role) % RL_STAMP_ROLES) * RL_STAMP_PHASES + rl_i], rl_st[rl_i]);
#define RL_STAMP_EXPORT(unit)                                                                          \
  extern "C" int rl_phase_stamps_##unit(unsigned long long* out, int reset) {                          \
    hipError_t e = hipMemcpyFromSymbol(out, HIP_SYMBOL(rl::rl_stamp_table), sizeof(rl::rl_stamp_table)); \
    if (e == hipSuccess && reset) {                                                                    \
      static unsigned long long zero[rl::RL_STAMP_ROLES * rl::RL_STAMP_PHASES] = {};                   \
      e = hipMemcpyToSymbol(HIP_SYMBOL(rl::rl_stamp_table), zero, sizeof(zero));                       \
    }                                                                                                  \
    return (int)e;                                                                                     \
  }
#else
#define RL_STAMP_TABLE
#define RL_STAMP_BEGIN
#define RL_STAMP(i)
#define RL_STAMP_END(role)
#define RL_STAMP_EXPORT(unit)
#endif

// Make this wave's earlier LDS writes visible to its later LDS reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int NT = NTHREADS>
__device__ __forceinline__ void zero_lds(void* base, size_t bytes, int tid) {
  uint32_t* w = reinterpret_cast<uint32_t*>(base);
  for (size_t i = tid; i < bytes / 4; i += NT) w[i] = 0u;
}

// Copy n elements from LDS (16-byte aligned) to global (4-byte aligned):
// 16-byte stores when the destination allows, 4-byte words otherwise.
template <typename T>
__device__ __forceinline__ void copy_tile(const T* src, T* __restrict__ dst, int n, int tid, int nt) {
  const int nbytes = n * (int)sizeof(T);
  int done_words = 0;
  if ((reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* g4 = reinterpret_cast<u32x4*>(dst);
    const int nq = nbytes >> 4;
    for (int i = tid; i < nq; i += nt) g4[i] = s4[i];
    done_words = nq * 4;
  }
  const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
  uint32_t* g = reinterpret_cast<uint32_t*>(dst);
  for (int i = done_words + tid; i < (nbytes >> 2); i += nt) g[i] = s[i];
}

// Copy `rows` rows of `len` elements (len * sizeof(T) a multiple of 4) from
// an LDS tile whose rows start 16-byte aligned (leading dimension ld) to
// consecutive global rows that are 4-byte aligned: per row, the words before
// the first 16-byte boundary and after the last one go as 4-byte stores, the
// rest as 16-byte stores (their LDS source is read as four words).
template <typename T>
__device__ __forceinline__ void copy_rows_global16(const T* src, int ld, T* __restrict__ dst, int len, int rows,
                                                   int tid, int nt) {
  const int lb = len * (int)sizeof(T), ldb = ld * (int)sizeof(T);
  const int maxch = lb / 16;
  const uint8_t* s8 = reinterpret_cast<const uint8_t*>(src);
  uint8_t* d8 = reinterpret_cast<uint8_t*>(dst);
  // 16-byte body
  for (int i = tid; i < rows * maxch; i += nt) {
    const int r = i / maxch, c = i - r * maxch;
    uint8_t* drow = d8 + (size_t)r * lb;
    const int head = (int)((16 - (reinterpret_cast<uintptr_t>(drow) & 15)) & 15);
    if (c < (lb - head) / 16) {
      const uint32_t* sp = reinterpret_cast<const uint32_t*>(s8 + (size_t)r * ldb + head + 16 * c);
      const u32x4 v = {sp[0], sp[1], sp[2], sp[3]};
      *reinterpret_cast<u32x4*>(drow + head + 16 * c) = v;
    }
  }
  // head and tail words (at most 3 + 3 per row)
  for (int i = tid; i < rows * 8; i += nt) {
    const int r = i >> 3, q = i & 7;
    uint8_t* drow = d8 + (size_t)r * lb;
    const int head = (int)((16 - (reinterpret_cast<uintptr_t>(drow) & 15)) & 15);
    const int h = head < lb ? head : lb;
    const int tail0 = h + (lb - h) / 16 * 16;
    const int off = q < 4 ? 4 * q : tail0 + 4 * (q - 4);
    if ((q < 4 && off < h) || (q >= 4 && off < lb))
      *reinterpret_cast<uint32_t*>(drow + off) = *reinterpret_cast<const uint32_t*>(s8 + (size_t)r * ldb + off);
  }
}

// Injected actions are staged through LDS in chunks of this many steps.
constexpr int ACT_CHUNK = 64;

// Stage the actions of steps k0 .. k0+nk-1 of one env tile into LDS: the
// tile's `live` contiguous int32 per step (its envs x A agents) go to
// lds[kk * PER + j]; PER is the full tile's count.
template <int PER, int NT>
__device__ __forceinline__ void stage_actions(const int32_t* __restrict__ actions, int E, int e0, int live, int A,
                                              int k0, int nk, int32_t* lds, int tid) {
  for (int i = tid; i < nk * PER; i += NT) {
    const int kk = i / PER, j = i - kk * PER;
    lds[i] = j < live ? actions[((size_t)(k0 + kk) * E + e0) * A + j] : 0;
  }
}

struct PolicyArgs {
  int dt;  // DT_F32 / DT_BF16
  int D, H1, H2, NA;  // NA: outputs of layer 3 (actions, plus the value when VH)
  const void* W[3];
  const void* b[3];
  int VH = 0;  // 1: the last of the NA outputs is the critic's value V(o), the others are action logits
  // bf16 only: the layers' fragment-major copies (nullptr: read W; see
  // packed_layer_offset), used by the streamed-weight rollout kernels
  const void* Wp[3] = {nullptr, nullptr, nullptr};
};

// Fragment-major copy of a bf16 layer W [N x K] (the nn.Linear layout): for
// 16-row tile t and 32-wide K step s, the MFMA B operands of the 64 lanes
// (lane l: row 16t + l % 16, k = 32s + 8(l / 16) .. +7, zero outside W) are
// 1 KB at element ((t * S + s) * 64 + l) * 8, S = ceil(K / 32).  The three
// layers of a policy follow one another, each at a 256-byte boundary.
__host__ __device__ inline size_t packed_layer_bytes(int N, int K) {
  return (size_t)((N + 15) / 16) * (size_t)((K + 31) / 32) * 1024;
}
__host__ __device__ inline size_t packed_layer_offset(const int (&dims)[4], int layer) {
  size_t o = 0;
  for (int l = 0; l < layer; ++l) o += (packed_layer_bytes(dims[l + 1], dims[l]) + 255) & ~(size_t)255;
  return o;
}

struct TrajArgs {
  void* obs;
  int32_t* actions;
  float* logits;
  float* reward;
  uint8_t* done;
  void* obs_last;
  float* value = nullptr;       // [T, E, A] V(o_t) (value head only)
  float* logp = nullptr;        // [T, E, A] log pi(a_t | o_t) of the sampled action
  float* value_last = nullptr;  // [E, A] V(o_{t0+T})
  const int32_t* teammates = nullptr;  // [E, A] heuristic kind per agent (LBF_NHEUR kinds), else the policy
};

// LDS layout of the fused rollout kernel for one env tile of TILE_E envs.
struct RunLayout {
  int R;               // policy rows per tile = TILE_E * A (a multiple of 16)
  int ldx, ld1, ld2;   // leading dimensions of the obs, h1 and h2 tiles (elements)
  size_t off_agrid, off_fgrid, off_acell, off_act, off_x, off_h1, off_h2, off_logit, off_score;
  size_t total;        // bytes
};

__host__ __device__ inline RunLayout make_run_layout(int A, int D, int H1, int H2, int dt) {
  RunLayout L;
  const size_t es = dt == DT_F32 ? 4 : 2;
  L.R = TILE_E * A;
  L.ldx = dt == DT_F32 ? lds_ld<DT_F32>(D) : lds_ld<DT_BF16>(D);
  L.ld1 = dt == DT_F32 ? lds_ld<DT_F32>(H1) : lds_ld<DT_BF16>(H1);
  L.ld2 = dt == DT_F32 ? lds_ld<DT_F32>(H2) : lds_ld<DT_BF16>(H2);
  size_t o = 0;
  L.off_agrid = o; o += (size_t)TILE_E * LBF_MAXCELLS;
  L.off_fgrid = o; o += (size_t)TILE_E * LBF_MAXCELLS;
  L.off_acell = o; o += (size_t)TILE_E * LBF_MAXA * 4;
  L.off_act = o;   o += (size_t)L.R * 4;
  L.off_x = o;     o += (size_t)L.R * L.ldx * es;
  o = (o + 15) & ~(size_t)15;
  L.off_h1 = o;    o += (size_t)L.R * L.ld1 * es;
  o = (o + 15) & ~(size_t)15;
  L.off_h2 = o;    o += (size_t)L.R * L.ld2 * es;
  o = (o + 15) & ~(size_t)15;
  L.off_logit = o; o += (size_t)L.R * MAX_NA * 4;
  L.off_score = o; o += (size_t)L.R * MAX_NA * 4;
  L.total = o;
  return L;
}

constexpr size_t MAX_LDS_BYTES = 160 * 1024;

hipError_t launch_lbf_init(const LbfParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal,
                           hipStream_t s);
hipError_t launch_lbf_step(const LbfParams& p, int32_t* state, uint64_t t0, int n_steps,
                           const int32_t* actions, void* obs, int obs_dt, float* reward, uint8_t* done,
                           uint8_t* legal, hipStream_t s);
hipError_t launch_lbf_run(const LbfParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                          const TrajArgs& out, hipStream_t s);
// Observe the stored LBF states into obs [E, A, D] bf16 (no reset).
hipError_t launch_lbf_observe(const LbfParams& p, const int32_t* state, uint16_t* obs, hipStream_t s);

// Recurrent S5 actor-critic (rl_s5.hip): bf16 dense layers, float32 S5.
struct S5Net {
  int D, H, P, F, NA;
  const void* w_enc;  // [H, D]
  const void* b_enc;
  const float* lbar;  // [2, P] discretised diagonal (real, imaginary)
  const float* bbar;  // [2, P, H]
  const float* c;     // [2, H, P]
  const float* d;     // [H]
  const void* actor_w[4];
  const void* actor_b[4];
  const void* critic_w[4];
  const void* critic_b[4];
};
struct S5Workspace {
  size_t off_obs, off_y, off_h, off_act, off_wcat, bytes;
};
S5Workspace s5_workspace(const LbfParams& p, const S5Net& net);
size_t s5_front_lds_bytes(int D, int H, int P);
hipError_t launch_s5_discretize(int P, int H, const float* lam, const float* log_dt, const float* b, float* lbar,
                                float* bbar, hipStream_t s);
hipError_t launch_s5_rollout(const LbfParams& p, const S5Net& net, int32_t* state, float* carry, uint64_t t0,
                             int n_steps, const TrajArgs& out, void* workspace, hipStream_t s);
// The allocation-free S5 rollout's workspace: a file-scope device array of
// S5_SCRATCH_BYTES per GPU; s5_scratch_ptr resolves the current GPU's copy
// (hipGetSymbolAddress, once per device) and returns its device address.
constexpr size_t S5_SCRATCH_BYTES = (size_t)80 << 20;
hipError_t s5_scratch_ptr(void** out);

// Generalised advantage estimation over [T, E, A] values (rl_ac.hip).
hipError_t launch_gae(const float* reward, const uint8_t* done, const float* value, const float* value_last, int T,
                      int E, int A, float gamma, float lambda, float* adv, float* ret, hipStream_t s);

// Population rollout (LBF): agent a of env e acts with policy pidx[e * A + a]
// of n_pol networks stacked in pol's weight arrays.
constexpr size_t LBF_POP_STATIC_LDS = 64;  // bytes of static LDS the population kernel may declare
size_t lbf_pop_lds_bytes(const LbfParams& p, const PolicyArgs& pol);
hipError_t launch_lbf_run_pop(const LbfParams& p, const PolicyArgs& pol, int n_pol, const int32_t* pidx,
                              int32_t* state, uint64_t t0, int n_steps, const TrajArgs& out, hipStream_t s);

hipError_t launch_oc_init(const OcParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal, hipStream_t s);
hipError_t launch_oc_step(const OcParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                          void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s);
size_t oc_run_lds_bytes(const PolicyArgs& pol);
hipError_t launch_oc_run(const OcParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                         const TrajArgs& out, hipStream_t s);

hipError_t launch_hn_init(const HnParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal, hipStream_t s);
hipError_t launch_hn_step(const HnParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                          void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s);
size_t hn_run_lds_bytes(const PolicyArgs& pol);
hipError_t launch_hn_run(const HnParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                         const TrajArgs& out, hipStream_t s);

size_t policy_lds_bytes(const PolicyArgs& pol);
hipError_t launch_policy_pack(const PolicyArgs& pol, void* packed, hipStream_t s);
hipError_t launch_policy_forward(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                 float* logits, hipStream_t s);
hipError_t launch_sample(uint64_t seed, int64_t env_base, int E, int A, int NA, uint64_t t, const float* logits,
                         const uint8_t* legal, int32_t* actions, hipStream_t s);
hipError_t launch_gumbel(const uint32_t* u, int64_t n, float* g, hipStream_t s);

}  // namespace rl
