// Policy MLP on the gfx950 matrix cores (MFMA), one workgroup per row tile.
//
// A layer computes out[R x N] = act(in[R x K] W^T + b) with the input tile in
// LDS (row-major, leading dimension lda, zero in columns K..Kpad-1) and W in
// the nn.Linear layout [N x K] in global memory.  The R x N output is cut
// into 16 x 16 tiles dealt round-robin to the workgroup's waves; each tile is
// a chain of MFMA instructions over K:
//   float32: v_mfma_f32_16x16x4_f32   (K step 4, one element per lane)
//   bf16:    v_mfma_f32_16x16x32_bf16 (K step 32, eight elements per lane)
// both accumulating in float32.  Operand lanes: A row = lane % 16, B column =
// lane % 16, each lane covering one K slice (lane / 16); the 16 x 16 result
// holds row 4 * (lane / 16) + r, column lane % 16 in accumulator element r.
// Hidden layers apply tanh (fast_tanh) and store in the layer dtype (bf16:
// round to nearest even); the output layer stores float32 logits.
#pragma once
#include <type_traits>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rl {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum { DT_F32 = 0, DT_BF16 = 1 };

// float -> bfloat16 bits, round to nearest even (one v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Two floats -> two bfloat16 in one dword (lo in bits 0-15), round to nearest
// even: one v_cvt_pk_bf16_f32, the same rounding as f32_to_bf16.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

template <int DT>
struct DType;
template <>
struct DType<DT_F32> {
  using T = float;
  static constexpr int KS = 4;
  __device__ static float to_f32(float x) { return x; }
  __device__ static float from_f32(float x) { return x; }
};
template <>
struct DType<DT_BF16> {
  using T = uint16_t;
  static constexpr int KS = 32;
  __device__ static float to_f32(uint16_t x) { return bf16_to_f32(x); }
  __device__ static uint16_t from_f32(float x) { return f32_to_bf16(x); }
};

__host__ __device__ constexpr int round_up(int x, int m) { return (x + m - 1) / m * m; }

// A small non-negative integer (an observation feature) in a layer dtype;
// exact in bf16 up to 256.
template <typename OT>
__device__ __forceinline__ OT small_int_to(uint32_t v);
template <>
__device__ __forceinline__ float small_int_to<float>(uint32_t v) {
  return (float)v;
}
template <>
__device__ __forceinline__ uint16_t small_int_to<uint16_t>(uint32_t v) {
  return (uint16_t)(__float_as_uint((float)v) >> 16);
}

// tanh(x) = 1 - 2 / (exp(2x) + 1) with the hardware exp2 and reciprocal
// (v_exp_f32, v_rcp_f32).  Absolute error is a few 1e-7; +-inf and large
// |x| give +-1 exactly, NaN stays NaN.
__device__ __forceinline__ float fast_tanh(float x) {
  const float e = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);  // 2 / ln(2)
  return 1.f - 2.f * __builtin_amdgcn_rcpf(e + 1.f);
}

// Leading dimension (elements) of an LDS operand tile holding K columns:
// K padded to the MFMA K step, plus 16 bytes so that consecutive rows start
// on different LDS banks.
template <int DT>
__host__ __device__ constexpr int lds_ld(int K) {
  return DT == DT_F32 ? round_up(K, 4) + 4 : round_up(K, 32) + 8;
}

// How weight rows may be loaded 8 bf16 at a time: K % 8 == 0 (16-byte
// aligned rows), K even (4-byte aligned rows: gfx950 global loads of 16 bytes
// need only that), or K odd (2-byte loads).
enum : int { WALIGN_16 = 0, WALIGN_4 = 1, WALIGN_2 = 2 };

__host__ __device__ constexpr int weight_align(int K) { return K % 8 == 0 ? WALIGN_16 : K % 2 == 0 ? WALIGN_4 : WALIGN_2; }

// 8 consecutive bf16 weights starting at p, all inside the row.
template <int AL>
__device__ __forceinline__ u32x4 load_w8(const uint16_t* __restrict__ p) {
  u32x4 b;
  if constexpr (AL == WALIGN_16) {
    b = *reinterpret_cast<const u32x4*>(p);
  } else if constexpr (AL == WALIGN_4) {
    __builtin_memcpy(&b, __builtin_assume_aligned(p, 4), 16);
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = (uint32_t)p[2 * q] | ((uint32_t)p[2 * q + 1] << 16);
  }
  return b;
}

// This lane's B operand of the last, partial k-step: weights at k = kk.. of
// one output row, zero past K.
template <int DT>
__device__ __forceinline__ auto load_b_tail(const typename DType<DT>::T* __restrict__ wrow, int k0, int kk, int K) {
  if constexpr (DT == DT_F32) {
    return kk < K ? wrow[k0] : 0.f;
  } else {
    uint32_t h[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = (kk + 2 * q < K) ? wrow[k0 + 2 * q] : 0u;
      const uint32_t hi = (kk + 2 * q + 1 < K) ? wrow[k0 + 2 * q + 1] : 0u;
      h[q] = lo | (hi << 16);
    }
    return u32x4{h[0], h[1], h[2], h[3]};
  }
}

__device__ __forceinline__ f32x4 mfma_step(float a, float b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_step(u32x4 a, u32x4 b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                 0, 0, 0);
}

// MT x G output tiles of 16 x 16: rows of MT row tiles against G adjacent
// output-column tiles, acc[m][g] = A_m[16 rows, 0:Kpad] * W[n0+16g .. +16, 0:Kpad]^T,
// where a_row[m] points at element 0 of this lane's A row (lane % 16) in row
// tile m.  Every weight fragment loaded from L2 feeds MT MFMAs (one per row
// tile) and every activation fragment G.  The k-steps inside K run
// branch-free (unconditional weight loads; output rows past N read row 0 and
// are zeroed after the load) and software-pipelined: a ring of PF k-steps'
// weight fragments is in flight, each slot consumed and then refilled in
// place, so loads overlap the MFMAs of earlier steps without register copies.
// The loop is kept rolled (these kernels run many different phases per step
// and must stay within the instruction cache).  The one partial step at the
// end is guarded.  Each tile's sum runs over k in the same order whatever G
// and MT are, so results do not depend on them.  PFX > 0 sets the ring depth
// (deeper rings hide more of the weight-load latency in short, long-K chains);
// tile g covers output columns n0 + gstride * g (gstride 16: adjacent tiles;
// n0 and gstride are multiples of 16).  PK (bf16): the B operands come from
// Wp, the layer's fragment-major copy (packed_layer_offset), where each
// operand load is one contiguous 1 KB block instead of 16 rows x 64 bytes;
// the operands, and so the results, are the same as from W.
template <int DT, int G, int MT, int AL, int PFX = 0, bool PK = false>
__device__ __forceinline__ void mma_tiles(const typename DType<DT>::T* const (&a_row)[MT], int Kpad, int K,
                                          const typename DType<DT>::T* __restrict__ W, int n0, int N, int lane,
                                          f32x4 (&acc)[MT][G], int gstride = 16,
                                          const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  using T = typename DType<DT>::T;
  using BT = typename std::conditional<DT == DT_F32, float, u32x4>::type;
  constexpr int KS = DType<DT>::KS;
  constexpr int KL = DT == DT_F32 ? 1 : 8;  // k values per lane per step
  constexpr int PF = PFX > 0 ? PFX : G >= 4 ? 2 : 4;  // k-steps of weights in flight
  constexpr bool PACKED = PK && DT == DT_BF16;
  const T* wrow[G];
  bool nok[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int n = n0 + gstride * g + (lane & 15);
    nok[g] = n < N;
    if constexpr (PACKED) {
      // operand block of this lane in k step 0 of tile (n0 + gstride g) / 16
      // (tiles past the layer read tile 0; nok zeroes them)
      const int tile = n0 + gstride * g < N ? (n0 + gstride * g) >> 4 : 0;
      wrow[g] = Wp + ((size_t)tile * (Kpad / KS) * 64 + lane) * 8;
    } else {
      wrow[g] = W + (size_t)(nok[g] ? n : 0) * K + (lane >> 4) * KL;
    }
  }
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int g = 0; g < G; ++g) acc[m][g] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int koff = (lane >> 4) * KL;
  auto a_at = [&](int m, int k0) -> BT {
    if constexpr (DT == DT_F32)
      return a_row[m][koff + k0];
    else
      return *reinterpret_cast<const u32x4*>(a_row[m] + koff + k0);
  };
  auto b_at = [&](int g, int k0) -> BT {
    if constexpr (DT == DT_F32)
      return wrow[g][k0];
    else if constexpr (PACKED)
      return *reinterpret_cast<const u32x4*>(wrow[g] + (size_t)(k0 / KS) * 512);
    else
      return load_w8<AL>(wrow[g] + k0);
  };
  auto mfma_all = [&](int k0, const BT (&b)[G]) {
    BT a[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) a[m] = a_at(m, k0);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      BT bg;
      if constexpr (DT == DT_F32)
        bg = nok[g] ? b[g] : 0.f;
      else
        bg = nok[g] ? b[g] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m][g] = mfma_step(a[m], bg, acc[m][g]);
    }
  };
  const int nsteps = K / KS, nmain = nsteps / PF * PF;
  if (nmain > 0) {
    BT ring[PF][G];
#pragma unroll
    for (int u = 0; u < PF; ++u)
#pragma unroll
      for (int g = 0; g < G; ++g) ring[u][g] = b_at(g, u * KS);
#pragma nounroll
    for (int s0 = 0; s0 < nmain; s0 += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        mfma_all((s0 + u) * KS, ring[u]);
        const int nxt = min(s0 + PF + u, nmain - 1) * KS;  // past the end: reload the last step (unused)
#pragma unroll
        for (int g = 0; g < G; ++g) ring[u][g] = b_at(g, nxt);
      }
    }
  }
  for (int st = nmain; st < nsteps; ++st) {  // full steps left over from the pipelined groups
    BT b[G];
#pragma unroll
    for (int g = 0; g < G; ++g) b[g] = b_at(g, st * KS);
    mfma_all(st * KS, b);
  }
  if (nsteps * KS < Kpad) {  // the partial last step
    const int k0 = nsteps * KS, kk = k0 + koff;
    BT b[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (PACKED)
        b[g] = b_at(g, k0);  // the copy holds the zeros past K
      else
        b[g] = load_b_tail<DT>(wrow[g], k0, kk, K);
    }
    mfma_all(k0, b);
  }
}

// A dense layer over R = 16 * MT rows in groups of G output tiles per wave;
// each wave's work item covers all MT row tiles.  Row r of the input is
// in[rows ? rows[r] : r].  Hidden layers (LOGITS false) store
// tanh(x W^T + b) in the layer dtype to `out`; the output layer stores
// x W^T + b as float32 to `logits` (columns < N only).
template <int DT, int G, int MT, int AL, bool LOGITS, bool PK = false>
__device__ __forceinline__ void mlp_layer_g(const typename DType<DT>::T* in, int lda, const int* rows, int K,
                                            const typename DType<DT>::T* __restrict__ W,
                                            const typename DType<DT>::T* __restrict__ b, int N,
                                            typename DType<DT>::T* out, float* logits, int ldo, int wave, int nwaves,
                                            int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  using T = typename DType<DT>::T;
  using DTy = DType<DT>;
  const int Kpad = round_up(K, DTy::KS);
  const int nt = (N + 15) >> 4, ng = (nt + G - 1) / G;
  const T* a_row[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = 16 * m + (lane & 15);
    a_row[m] = in + (size_t)(rows ? rows[r] : r) * lda;
  }
  for (int item = wave; item < ng; item += nwaves) {
    const int n0 = item * 16 * G;
    float bias[G];  // loaded before the k loop so that its latency hides behind the MFMAs
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int col = n0 + 16 * g + (lane & 15);
      bias[g] = DTy::to_f32(b[col < N ? col : 0]);
    }
    f32x4 acc[MT][G];
    mma_tiles<DT, G, MT, AL, 0, PK>(a_row, Kpad, K, W, n0, N, lane, acc, 16, Wp);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int col = n0 + 16 * g + (lane & 15);
      if (col < N) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = 16 * m + 4 * (lane >> 4) + q;
            if constexpr (LOGITS)
              logits[(size_t)row * ldo + col] = acc[m][g][q] + bias[g];
            else
              out[(size_t)row * ldo + col] = DTy::from_f32(fast_tanh(acc[m][g][q] + bias[g]));
          }
      }
    }
  }
}

template <int DT, int MT, int AL, bool LOGITS, bool PK = false>
__device__ __forceinline__ void mlp_layer_mt(const typename DType<DT>::T* in, int lda, const int* rows, int K,
                                             const typename DType<DT>::T* __restrict__ W,
                                             const typename DType<DT>::T* __restrict__ b, int N,
                                             typename DType<DT>::T* out, float* logits, int ldo, int wave,
                                             int nwaves, int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  const int nt = (N + 15) >> 4;
  if (nt >= 4 * nwaves && nt % 4 == 0)
    mlp_layer_g<DT, 4, MT, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
  else if (nt >= 2 * nwaves && nt % 2 == 0)
    mlp_layer_g<DT, 2, MT, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
  else
    mlp_layer_g<DT, 1, MT, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
}

// Picks the row-tile count (R = 16, 32, 48 or 64) and the widest tile group
// that still gives every wave work.
template <int DT, int AL, bool LOGITS, bool PK = false>
__device__ __forceinline__ void mlp_layer_al(const typename DType<DT>::T* in, int lda, const int* rows, int R, int K,
                                             const typename DType<DT>::T* __restrict__ W,
                                             const typename DType<DT>::T* __restrict__ b, int N,
                                             typename DType<DT>::T* out, float* logits, int ldo, int wave,
                                             int nwaves, int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  switch (R >> 4) {
    case 1:
      mlp_layer_mt<DT, 1, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
      break;
    case 2:
      mlp_layer_mt<DT, 2, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
      break;
    case 3:
      mlp_layer_mt<DT, 3, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
      break;
    default:
      mlp_layer_mt<DT, 4, AL, LOGITS, PK>(in, lda, rows, K, W, b, N, out, logits, ldo, wave, nwaves, lane, Wp);
  }
}

// The first layer for any input width K (picks the weight-load width at run time).
template <int DT, bool PK = false>
__device__ __forceinline__ void mlp_input_layer(const typename DType<DT>::T* in, int lda, const int* rows, int R,
                                                int K, const typename DType<DT>::T* __restrict__ W,
                                                const typename DType<DT>::T* __restrict__ b, int N,
                                                typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                                int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  const int al = DT == DT_F32 ? WALIGN_16 : weight_align(K);
  if (al == WALIGN_16)
    mlp_layer_al<DT, WALIGN_16, false, PK>(in, lda, rows, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane, Wp);
  else if (al == WALIGN_4)
    mlp_layer_al<DT, WALIGN_4, false, PK>(in, lda, rows, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane, Wp);
  else
    mlp_layer_al<DT, WALIGN_2, false, PK>(in, lda, rows, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane, Wp);
}

// The first layer for an input width KC known at compile time.
template <int DT, int KC, bool PK = false>
__device__ __forceinline__ void mlp_input_layer_const(const typename DType<DT>::T* in, int lda, const int* rows,
                                                      int R, const typename DType<DT>::T* __restrict__ W,
                                                      const typename DType<DT>::T* __restrict__ b, int N,
                                                      typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                                      int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  constexpr int AL = DT == DT_F32 ? WALIGN_16 : weight_align(KC);
  mlp_layer_al<DT, AL, false, PK>(in, lda, rows, R, KC, W, b, N, out, nullptr, ldo, wave, nwaves, lane, Wp);
}

// A hidden layer after the first: K (a hidden width) is a multiple of 16.
// R rows: 16, 32, 48 or 64.
template <int DT, bool PK = false>
__device__ __forceinline__ void mlp_hidden(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N,
                                           typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                           int lane, const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  mlp_layer_al<DT, WALIGN_16, false, PK>(in, lda, nullptr, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane, Wp);
}

// The output layer: logits = in W^T + b as float32, N <= 32 actions, K a multiple of 16.
template <int DT, bool PK = false>
__device__ __forceinline__ void mlp_logits(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N, float* out,
                                           int ldo, int wave, int nwaves, int lane,
                                           const typename DType<DT>::T* __restrict__ Wp = nullptr) {
  mlp_layer_al<DT, WALIGN_16, true, PK>(in, lda, nullptr, R, K, W, b, N, nullptr, out, ldo, wave, nwaves, lane, Wp);
}

}  // namespace rl
