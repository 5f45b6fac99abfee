// Standalone policy forward (obs -> logits on the MFMA MLP), standalone
// Gumbel-max sampling from given logits, and the sampler's noise function.
#include <type_traits>

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

// Software-pipelined variant for the narrow bf16 policies (one workgroup of
// 4 waves per CU).  In a 128-wide layer the tanh epilogue (two
// transcendental instructions per value) takes longer than the layer's
// MFMAs, so each wave overlaps one tile's epilogue with the next tile's
// matrix products: iteration j of a workgroup runs
//   phase A: layer 3 of tile j-2 (logits out), layer-1 MFMAs of tile j+1
//            interleaved with the layer-1 epilogue of tile j;
//   phase B: the observation tile of j+2 staged from registers, the load of
//            tile j+3 issued, layer-2 MFMAs of tile j interleaved with the
//            layer-2 epilogue of tile j-1;
// with one barrier after each phase.  The observation tile is double
// buffered; h1 and h2 have one buffer each (every write of one is separated
// from the reads of its previous contents by a barrier).  Tiles past this
// workgroup's last are computed from zeros and never stored.  Every output
// is the same MFMA chain and epilogue as policy_fwd_reg_kernel and the
// rollout kernels, so the logits are bit-identical to theirs.
template <int D, int H1, int H2, int NA, int MT, int MINB>
__global__ __launch_bounds__(256, MINB) void policy_fwd_pipe_kernel(PolicyArgs pol, const void* __restrict__ obs_v,
                                                                  const uint8_t* __restrict__ legal, int64_t rows,
                                                                  float* __restrict__ logits) {
  constexpr int DT = DT_BF16, NW = 4, NT = NW * 64, BM = MT * 16;
  using T = typename DType<DT>::T;
  using B = typename BOperand<DT>::type;
  constexpr int LDX = lds_ld<DT>(D), LD1 = lds_ld<DT>(H1), LD2 = lds_ld<DT>(H2);
  constexpr int K3 = round_up(H2, DType<DT>::KS) / DType<DT>::KS;
  constexpr int VE = 16 / sizeof(T);
  // rows of D elements: whole 16-byte vectors, or (FLAT) a tile read as one
  // flat block of BM * D elements (16-byte aligned when BM * D is a multiple
  // of 8) and scattered into the LDS rows element by element
  constexpr bool FLAT = D % VE != 0;
  static_assert(!FLAT || (BM * D) % VE == 0, "flat observation tiles start on 16-byte boundaries");
  static_assert(NA <= 16, "one transposed M tile of actions");
  static_assert(MT <= NW, "one layer-3 M tile per wave");
  __shared__ __align__(16) T xs[2][BM * LDX];
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
  for (int i = tid; i < 2 * BM * LDX; i += NT) (&xs[0][0])[i] = (T)0;
  for (int i = tid; i < BM * LD1; i += NT) h1s[i] = (T)0;
  for (int i = tid; i < BM * LD2; i += NT) h2s[i] = (T)0;

  const int64_t ntiles = (rows + BM - 1) / BM;
  const int nt = (int64_t)blockIdx.x < ntiles ? (int)((ntiles - 1 - blockIdx.x) / gridDim.x) + 1 : 0;
  auto tile_of = [&](int j) { return (int64_t)blockIdx.x + (int64_t)j * gridDim.x; };
  constexpr int VPR = D / VE, NV = FLAT ? BM * D / VE : BM * VPR, IT = (NV + NT - 1) / NT;
  u32x4 v[IT];
  auto prefetch = [&](int j) {  // tile j of this workgroup into registers (zeros past the last)
    const int64_t row0 = tile_of(j) * BM;
    const int nrow = j < nt ? (int)min((int64_t)BM, rows - row0) : 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = tid + it * NT;
      if constexpr (FLAT) {
        // flat element i * VE of the tile; the vector that holds the tile's
        // last element is read element by element (nothing past the batch)
        const int nel = nrow * D, e0 = i * VE;
        const T* src = obs + (size_t)row0 * D + e0;
        if (i < NV && e0 + VE <= nel) {
          v[it] = *reinterpret_cast<const u32x4*>(src);
        } else {
          uint32_t h[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t lo = (i < NV && e0 + 2 * q < nel) ? (uint32_t)src[2 * q] : 0u;
            const uint32_t hi = (i < NV && e0 + 2 * q + 1 < nel) ? (uint32_t)src[2 * q + 1] : 0u;
            h[q] = lo | (hi << 16);
          }
          v[it] = u32x4{h[0], h[1], h[2], h[3]};
        }
      } else {
        const int r = i / VPR, c = (i - r * VPR) * VE;
        v[it] = (i < NV && r < nrow) ? *reinterpret_cast<const u32x4*>(obs + (size_t)(row0 + r) * D + c)
                                      : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto stage = [&](T* dst) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = tid + it * NT;
      if (i >= NV) continue;
      if constexpr (FLAT) {
#pragma unroll
        for (int q = 0; q < VE; ++q) {
          const int el = i * VE + q, r = el / D, c = el - r * D;
          dst[r * LDX + c] = (T)((v[it][q >> 1] >> (16 * (q & 1))) & 0xffffu);
        }
      } else {
        const int r = i / VPR, c = (i - r * VPR) * VE;
        *reinterpret_cast<u32x4*>(dst + r * LDX + c) = v[it];
      }
    }
  };

  __syncthreads();  // zero fill done before the staging writes
  prefetch(0);
  stage(xs[0]);
  prefetch(1);
  stage(xs[1]);
  prefetch(2);
  __syncthreads();
  f32x4 acc1[MT][RegLayer<DT, D, H1, NW>::OWN];
  f32x4 acc2[MT][RegLayer<DT, H1, H2, NW>::OWN];
  L1.template run<MT>(xs[0], LDX, acc1, wave, lane);
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int o = 0; o < RegLayer<DT, H1, H2, NW>::OWN; ++o) acc2[m][o] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int j = 0;; ++j) {
    // phase A
    if (j >= 2 && wave < MT) {
      const int row = wave * 16 + (lane & 15);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < K3; ++ks)
        acc = mfma16<DT>(w3s[ks * 64 + lane], load_operand_lds<DT>(h2s, LD2, row, ks, lane), acc);
      const int64_t row0 = tile_of(j - 2) * BM;
      if (row0 + row < rows) {
        const size_t gr = (size_t)(row0 + row) * NA;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int a = 4 * (lane >> 4) + r;
          if (a < NA) {
            const bool ok = legal == nullptr || legal[gr + a] != 0;
            logits[gr + a] = ok ? acc[r] + b3r[r] : -INFINITY;
          }
        }
      }
    }
    if (j == nt + 1) break;
    L1.template run_overlapped<MT>(xs[(j + 1) & 1], LDX, acc1, h1s, LD1, wave, lane);
    __syncthreads();
    // phase B
    stage(xs[j & 1]);
    prefetch(j + 3);
    L2.template run_overlapped<MT>(h1s, LD1, acc2, h2s, LD2, wave, lane);
    __syncthreads();
  }
}

template <int D, int H1, int H2, int NA, int MT, int MINB>
static hipError_t launch_policy_pipe(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                     float* logits, hipStream_t s) {
  constexpr int BM = MT * 16;
  const int64_t ntiles = (rows + BM - 1) / BM;
  const unsigned grid = (unsigned)(ntiles < (int64_t)256 * MINB ? ntiles : (int64_t)256 * MINB);
  policy_fwd_pipe_kernel<D, H1, H2, NA, MT, MINB><<<dim3(grid), 256, 0, s>>>(pol, obs, legal, rows, logits);
  return hipGetLastError();
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
  if (pol.dt == DT_BF16 && pol.D == 192 && pol.H1 == 128 && pol.H2 == 128 && pol.NA == 6) {
    *err = launch_policy_pipe<192, 128, 128, 6, 2, 2>(pol, obs, legal, rows, logits, s);
    return true;
  }
  if (pol.dt == DT_BF16 && pol.D == 147 && pol.H1 == 128 && pol.H2 == 128 && pol.NA == 6) {  // 7 x 7 LBF
    *err = launch_policy_pipe<147, 128, 128, 6, 2, 2>(pol, obs, legal, rows, logits, s);
    return true;
  }
  RL_PF_CASE(DT_F32, 192, 128, 128, 6, 4, 4, 1)
  RL_PF_CASE(DT_BF16, 192, 64, 64, 6, 4, 4, 2)
  RL_PF_CASE(DT_F32, 192, 64, 64, 6, 4, 4, 2)
#undef RL_PF_CASE
  return false;
}

// ------------------------------------------------ tiled policy forward ----
//
// bf16 policy forward for wide layers (the 12x12 LBF, kitchen and Hanabi
// policies), structured as three chained GEMMs per tile of BM rows:
//   * 4 waves in a 2 x 2 grid over (output units, rows); each wave holds the
//     fp32 accumulators of HMAX/2 units x BM/2 rows for a whole layer;
//   * layer-1 weights and observations, and layer-2 weights, are staged
//     through a ring of NB LDS buffers, one K slice of 32 at a time; every
//     weight byte staged serves all BM rows of the tile.  With NB = 3 the
//     global loads of slice s+3 are issued a full step before they are
//     stored to LDS, and the MFMA operands of slice s+1 are read from LDS
//     while the MFMAs of slice s run;
//   * h1 stays in LDS; h2 overwrites it once layer 2 has read it;
//   * layer 3 is computed transposed (actions x rows) from h2.
// As in the register-resident kernels, every output is one MFMA chain over K
// in increasing order, bias added after, so the logits are bit-identical to
// the other policy paths.
constexpr int PT_KC = 32;  // K slice per step: one bf16 MFMA K step
constexpr int PT_NT = 256;

template <int HMAX, int BM, int NB>
struct PtLayout {
  static constexpr int LDH = HMAX + 8;  // pitch of the resident activation tile
  static constexpr size_t H_BYTES = (size_t)BM * LDH * 2;
  static constexpr size_t W_BYTES = (size_t)HMAX * PT_KC * 2;  // one staged weight slice
  static constexpr size_t X_BYTES = (size_t)BM * PT_KC * 2;    // one staged observation slice
  static constexpr size_t OFF_W = H_BYTES;
  static constexpr size_t OFF_X = OFF_W + NB * W_BYTES;
  static constexpr size_t OFF_B = OFF_X + NB * X_BYTES;  // fp32 biases of layers 1 and 2
  static constexpr size_t TOTAL = OFF_B + 2 * HMAX * 4;
};

// Element offset of 16-byte vector q (k = 8q..8q+7) of row n in a staged
// slice: rows of 64 bytes, vectors XOR-swizzled by (n / 2) % 4 so that any 8
// consecutive rows of an MFMA operand read fill the 32 LDS banks without
// conflict.  The swizzle does not change when n moves by 16 (an operand tile).
__device__ __forceinline__ int pt_slot(int n, int q) { return n * PT_KC + 8 * (q ^ ((n >> 1) & 3)); }

// Buffer resource over `bytes` bytes at p (raw: loads past the end read 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pt_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Zero the elements of an 8-element bf16 vector at or beyond `left` (the
// number of the vector's elements that lie inside the row).
__device__ __forceinline__ u32x4 pt_mask8(u32x4 v, int left) {
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t m = 2 * d + 1 < left ? 0xffffffffu : 2 * d < left ? 0x0000ffffu : 0u;
    v[d] &= m;
  }
  return v;
}

template <int HMAX, int BM, int NB, int MINB, bool PK>
__global__ __launch_bounds__(PT_NT, MINB) void policy_fwd_tiled_kernel(PolicyArgs pol, const uint16_t* __restrict__ obs,
                                                                 const uint8_t* __restrict__ legal, int64_t rows,
                                                                 float* __restrict__ logits) {
  using L = PtLayout<HMAX, BM, NB>;
  constexpr int UT = HMAX / 32;  // unit tiles of a wave (half the units)
  constexpr int RT = BM / 32;    // row tiles of a wave (half the rows)
  constexpr int HH = HMAX / 2;   // units of a wave
  constexpr int WV = HMAX * 4 / PT_NT, XV = (BM * 4 + PT_NT - 1) / PT_NT;  // staged vectors per thread
  static_assert(NB == 2 || NB == 3, "two or three slice buffers");
  static_assert(HMAX * 4 % PT_NT == 0, "whole weight vectors per thread");
  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem);
  uint16_t* wst = reinterpret_cast<uint16_t*>(smem + L::OFF_W);
  uint16_t* xst = reinterpret_cast<uint16_t*>(smem + L::OFF_X);
  float* bias_s = reinterpret_cast<float*>(smem + L::OFF_B);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wu = wave & 1, wr = wave >> 1;
  const int D = pol.D, NA = pol.NA;
  const int64_t row0 = (int64_t)blockIdx.x * BM;
  const int nrow = (int)min((int64_t)BM, rows - row0);
  const uint16_t* W3 = static_cast<const uint16_t*>(pol.W[2]);

  for (int i = tid; i < 2 * HMAX; i += PT_NT)
    bias_s[i] = bf16_to_f32(i < HMAX ? static_cast<const uint16_t*>(pol.b[0])[i]
                                     : static_cast<const uint16_t*>(pol.b[1])[i - HMAX]);

  // One dense tanh layer of HMAX units: out = tanh(in W^T + b) into hs.
  // Layer 1 (tag true) stages observation rows with the weights; layer 2
  // reads its input from hs.
  auto layer = [&](auto l1_tag, const uint16_t* __restrict__ W, const uint16_t* __restrict__ Wp, int K,
                   const float* bias) {
    constexpr bool L1 = decltype(l1_tag)::value;
    const int nsteps = (K + PT_KC - 1) / PT_KC;
    // Weight slices are fetched one step before they are stored to LDS (they
    // come from L2); observation slices, which come from HBM, PX steps
    // before, through a ring of PX register slots (slot = slice % PX).
    constexpr int PX = NB == 3 ? 4 : 1;
    u32x4 wv[WV], xv[PX][XV];
    // per-thread byte offsets of the staged vectors (global) and their LDS
    // slots, fixed for the layer; the slice offset goes in a scalar register
    // PK: weights from the fragment-major copy (1 KB per 16 rows x 32 k),
    // one contiguous 1 KB block per wave-wide load instead of 16 rows x 64 B
    const int S = (K + PT_KC - 1) / PT_KC;
    const __amdgpu_buffer_rsrc_t wres =
        PK ? pt_rsrc(Wp, (uint32_t)(HMAX / 16) * S * 1024) : pt_rsrc(W, (uint32_t)HMAX * K * 2);
    const __amdgpu_buffer_rsrc_t xres = pt_rsrc(obs + (size_t)row0 * D, (uint32_t)nrow * D * 2);
    int wgo[WV], wlo[WV], xgo[XV], xlo[XV];
#pragma unroll
    for (int j = 0; j < WV; ++j) {
      const int v = tid + j * PT_NT;
      if constexpr (PK) {
        const int t = v >> 6, l = v & 63;  // operand block of tile t, lane l: row 16t + l % 16, chunk l / 16
        wgo[j] = (t * S * 64 + l) * 16;
        wlo[j] = pt_slot(16 * t + (l & 15), l >> 4);
      } else {
        const int n = v >> 2, q = v & 3;
        wgo[j] = (n * K + 8 * q) * 2;
        wlo[j] = pt_slot(n, q);
      }
    }
#pragma unroll
    for (int j = 0; j < XV; ++j) {
      const int v = tid + j * PT_NT, r = v >> 2, q = v & 3;
      xgo[j] = (r * D + 8 * q) * 2;  // rows past nrow lie past the resource: read as 0
      xlo[j] = pt_slot(r, q);
    }
    constexpr bool XALL = BM * 4 % PT_NT == 0;  // every thread stages XV observation vectors
    auto fetch_w = [&](int st) {
#pragma unroll
      for (int j = 0; j < WV; ++j)
        wv[j] = __builtin_amdgcn_raw_buffer_load_b128(wres, wgo[j], PK ? st * 1024 : st * PT_KC * 2, 0);
    };
    auto fetch_x = [&](int st, u32x4 (&x)[XV]) {
      if constexpr (L1) {
#pragma unroll
        for (int j = 0; j < XV; ++j)
          if (XALL || tid + j * PT_NT < BM * 4)
            x[j] = __builtin_amdgcn_raw_buffer_load_b128(xres, xgo[j], st * PT_KC * 2, 0);
      }
    };
    // store slice st to LDS buffer st % NB, zeroing what lies past K in the
    // partial last slice (uniform branch; q = tid % 4 for every vector)
    auto stage = [&](int st, u32x4 (&x)[XV]) {
      const int k0 = st * PT_KC;
      const bool part = k0 + PT_KC > K;
      const int left = K - k0 - 8 * (tid & 3);
      uint16_t* wb = wst + (st % NB) * (HMAX * PT_KC);
#pragma unroll
      for (int j = 0; j < WV; ++j)  // (the packed copy already holds zeros past K)
        *reinterpret_cast<u32x4*>(wb + wlo[j]) = (part && !PK) ? pt_mask8(wv[j], left) : wv[j];
      if constexpr (L1) {
        uint16_t* xb = xst + (st % NB) * (BM * PT_KC);
#pragma unroll
        for (int j = 0; j < XV; ++j)
          if (XALL || tid + j * PT_NT < BM * 4)
            *reinterpret_cast<u32x4*>(xb + xlo[j]) = part ? pt_mask8(x[j], left) : x[j];
      }
    };
    // MFMA operands of slice st (staged in buffer st % NB): unit tiles of W
    // and row tiles of the input, at fixed offsets from one lane base each
    const int a_lo = pt_slot(wu * HH + (lane & 15), lane >> 4);
    const int b_lo = L1 ? pt_slot(wr * (BM / 2) + (lane & 15), lane >> 4)
                        : (wr * (BM / 2) + (lane & 15)) * L::LDH + 8 * (lane >> 4);
    auto frags = [&](int st, u32x4 (&a)[UT], u32x4 (&b)[RT]) {
      const uint16_t* wb = wst + (st % NB) * (HMAX * PT_KC) + a_lo;
#pragma unroll
      for (int ut = 0; ut < UT; ++ut) a[ut] = *reinterpret_cast<const u32x4*>(wb + ut * 16 * PT_KC);
      if constexpr (L1) {
        const uint16_t* xb = xst + (st % NB) * (BM * PT_KC) + b_lo;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) b[rt] = *reinterpret_cast<const u32x4*>(xb + rt * 16 * PT_KC);
      } else {
        const uint16_t* hb = hs + b_lo + st * PT_KC;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) b[rt] = *reinterpret_cast<const u32x4*>(hb + rt * 16 * L::LDH);
      }
    };
    f32x4 acc[UT][RT];
#pragma unroll
    for (int ut = 0; ut < UT; ++ut)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[ut][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const u32x4 (&a)[UT], const u32x4 (&b)[RT]) {
#pragma unroll
      for (int ut = 0; ut < UT; ++ut)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[ut][rt] = mfma16<DT_BF16>(a[ut], b[rt], acc[ut][rt]);
    };
    if constexpr (NB == 3) {
      // prologue: slices 0 and 1 in LDS, weights of slice 2 and observations
      // of slices 2 .. PX+1 in flight
      fetch_w(0);
      fetch_x(0, xv[0]);
      stage(0, xv[0]);
      if (1 < nsteps) {
        fetch_w(1);
        fetch_x(1, xv[1]);
        stage(1, xv[1]);
      }
      if (2 < nsteps) fetch_w(2);
#pragma unroll
      for (int u = 2; u < PX + 2; ++u)
        if (u < nsteps) fetch_x(u, xv[u % PX]);
      __syncthreads();
      u32x4 a0[UT], b0[RT], a1[UT], b1[RT];
      frags(0, a0, b0);
      // one step (U = st % PX): store slice st+2 (its buffer was last read at
      // step st-1), fetch the weights of slice st+3 and the observations of
      // slice st+2+PX into the slot just stored, read slice st+1's operands,
      // then run slice st's MFMAs, behind which these memory operations land
      auto step = [&](auto u_tag, int st, const u32x4 (&a)[UT], const u32x4 (&b)[RT], u32x4 (&an)[UT],
                      u32x4 (&bn)[RT]) {
        constexpr int U = decltype(u_tag)::value;
        if (st + 2 < nsteps) stage(st + 2, xv[(U + 2) % PX]);
        if (st + 3 < nsteps) fetch_w(st + 3);
        if (st + 2 + PX < nsteps) fetch_x(st + 2 + PX, xv[(U + 2) % PX]);
        if (st + 1 < nsteps) frags(st + 1, an, bn);
        mma(a, b);
        __syncthreads();
      };
      static_assert(PX % 2 == 0, "operand registers alternate within the unrolled steps");
      for (int st = 0; st < nsteps; st += 4) {
        step(std::integral_constant<int, 0>{}, st, a0, b0, a1, b1);
        if (st + 1 < nsteps) step(std::integral_constant<int, 1>{}, st + 1, a1, b1, a0, b0);
        if (st + 2 < nsteps) step(std::integral_constant<int, 2>{}, st + 2, a0, b0, a1, b1);
        if (st + 3 < nsteps) step(std::integral_constant<int, 3>{}, st + 3, a1, b1, a0, b0);
      }
    } else {
      fetch_w(0);
      fetch_x(0, xv[0]);
      stage(0, xv[0]);
      __syncthreads();
      for (int st = 0; st < nsteps; ++st) {
        if (st + 1 < nsteps) {
          fetch_w(st + 1);
          fetch_x(st + 1, xv[0]);
        }
        u32x4 a[UT], b[RT];
        frags(st, a, b);
        mma(a, b);
        if (st + 1 < nsteps) stage(st + 1, xv[0]);
        __syncthreads();
      }
    }
    // every wave is past its last read of hs (layer 2 input): overwrite it
#pragma unroll
    for (int ut = 0; ut < UT; ++ut) {
      const int u0 = wu * HH + ut * 16 + 4 * (lane >> 4);
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias + u0);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int r = wr * (BM / 2) + rt * 16 + (lane & 15);
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = fast_tanh(acc[ut][rt][q] + b4[q]);
        const uint32_t lo = pack_bf16x2(v[0], v[1]);
        const uint32_t hi = pack_bf16x2(v[2], v[3]);
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u32x2*>(hs + r * L::LDH + u0) = u32x2{lo, hi};
      }
    }
    __syncthreads();
  };
  layer(std::true_type{}, static_cast<const uint16_t*>(pol.W[0]), static_cast<const uint16_t*>(pol.Wp[0]), D, bias_s);
  layer(std::false_type{}, static_cast<const uint16_t*>(pol.W[1]), static_cast<const uint16_t*>(pol.Wp[1]), HMAX,
        bias_s + HMAX);

  // layer 3, transposed: logits^T = W3 h2^T, items (action tile, row tile)
  constexpr int K3 = HMAX / PT_KC;
  const int nat = (NA + 15) >> 4;
  for (int item = wave; item < nat * (BM / 16); item += PT_NT / 64) {
    const int mt = item % nat, rt = item / nat;
    const int a_row = mt * 16 + (lane & 15);
    const uint16_t* w3r = W3 + (size_t)(a_row < NA ? a_row : 0) * HMAX + 8 * (lane >> 4);
    const int r = rt * 16 + (lane & 15);
    u32x4 a3[K3];
#pragma unroll
    for (int ks = 0; ks < K3; ++ks)
      a3[ks] = a_row < NA ? *reinterpret_cast<const u32x4*>(w3r + ks * PT_KC) : u32x4{0u, 0u, 0u, 0u};
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < K3; ++ks)
      acc = mfma16<DT_BF16>(a3[ks], *reinterpret_cast<const u32x4*>(hs + r * L::LDH + ks * PT_KC + 8 * (lane >> 4)),
                            acc);
    if (r < nrow) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int act = mt * 16 + 4 * (lane >> 4) + q;
        if (act < NA) {
          const size_t gi = (size_t)(row0 + r) * NA + act;
          const float lg = acc[q] + bf16_to_f32(static_cast<const uint16_t*>(pol.b[2])[act]);
          logits[gi] = (legal == nullptr || legal[gi] != 0) ? lg : -INFINITY;
        }
      }
    }
  }
}

template <int HMAX, int BM, int NB, int MINB, bool PK>
static hipError_t launch_policy_tiled_pk(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                         float* logits, hipStream_t s) {
  using L = PtLayout<HMAX, BM, NB>;
  static_assert(L::TOTAL <= MAX_LDS_BYTES, "tile fits in LDS");
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute((const void*)policy_fwd_tiled_kernel<HMAX, BM, NB, MINB, PK>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)L::TOTAL);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const unsigned grid = (unsigned)((rows + BM - 1) / BM);
  policy_fwd_tiled_kernel<HMAX, BM, NB, MINB, PK><<<dim3(grid), PT_NT, L::TOTAL, s>>>(
      pol, static_cast<const uint16_t*>(obs), legal, rows, logits);
  return hipGetLastError();
}

template <int HMAX, int BM, int NB, int MINB>
static hipError_t launch_policy_tiled(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                      float* logits, hipStream_t s) {
  return pol.Wp[0] != nullptr ? launch_policy_tiled_pk<HMAX, BM, NB, MINB, true>(pol, obs, legal, rows, logits, s)
                              : launch_policy_tiled_pk<HMAX, BM, NB, MINB, false>(pol, obs, legal, rows, logits, s);
}

// Shapes the tiled kernel serves: bf16, two hidden layers of 256 or of 512
// units, an even input width.
static bool try_launch_policy_tiled(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                    float* logits, hipStream_t s, hipError_t* err) {
  if (pol.dt != DT_BF16 || pol.D % 2 != 0 || pol.H1 != pol.H2 || pol.NA > MAX_NA) return false;
  if (pol.H1 == 256)
    *err = launch_policy_tiled<256, 64, 2, 2>(pol, obs, legal, rows, logits, s);  // two workgroups per CU
  else if (pol.H1 == 512)
    *err = launch_policy_tiled<512, 64, 2, 1>(pol, obs, legal, rows, logits, s);
  else
    return false;
  return true;
}

// ---------------------------------------------------- packed weights ----
//
// Writes the fragment-major copy of one bf16 layer W [N x K] (layout in
// packed_layer_offset): one thread per 16-byte operand block, zero outside W.
__global__ void policy_pack_kernel(const uint16_t* __restrict__ W, int N, int K, uint16_t* __restrict__ out,
                                   int64_t nvec) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nvec) return;
  const int S = (K + 31) / 32;
  const int lane = (int)(v & 63);
  const int64_t ts = v >> 6;
  const int s = (int)(ts % S), t = (int)(ts / S);
  const int n = 16 * t + (lane & 15), k0 = 32 * s + 8 * (lane >> 4);
  uint32_t h[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = (n < N && k0 + 2 * q < K) ? W[(size_t)n * K + k0 + 2 * q] : 0u;
    const uint32_t hi = (n < N && k0 + 2 * q + 1 < K) ? W[(size_t)n * K + k0 + 2 * q + 1] : 0u;
    h[q] = lo | (hi << 16);
  }
  *reinterpret_cast<u32x4*>(out + v * 8) = u32x4{h[0], h[1], h[2], h[3]};
}

hipError_t launch_policy_pack(const PolicyArgs& pol, void* packed, hipStream_t s) {
  const int dims[4] = {pol.D, pol.H1, pol.H2, pol.NA};
  for (int l = 0; l < 3; ++l) {
    const int64_t nvec = (int64_t)(packed_layer_bytes(dims[l + 1], dims[l]) / 16);
    uint16_t* out = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(packed) + packed_layer_offset(dims, l));
    policy_pack_kernel<<<dim3((unsigned)((nvec + 255) / 256)), 256, 0, s>>>(static_cast<const uint16_t*>(pol.W[l]),
                                                                          dims[l + 1], dims[l], out, nvec);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_policy_forward(const PolicyArgs& pol, const void* obs, const uint8_t* legal, int64_t rows,
                                 float* logits, hipStream_t s) {
  hipError_t err;
  if (try_launch_policy_reg(pol, obs, legal, rows, logits, s, &err)) return err;
  if (try_launch_policy_tiled(pol, obs, legal, rows, logits, s, &err)) return err;
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
