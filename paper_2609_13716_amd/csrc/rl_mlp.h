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

// G adjacent 16 x 16 output tiles of the same 16 rows:
// acc[g] = A[16 rows, 0:Kpad] * W[n0+16g : n0+16g+16, 0:Kpad]^T, where `a_row`
// points at element 0 of A row (lane % 16).  The k-steps inside K run
// branch-free (unconditional weight loads, output rows past N read row 0 and
// are zeroed after the load) so that the loads of several steps and tiles
// are in flight together; the one partial step at the end is guarded.  Each
// tile's sum runs over k in the same order for every G, so results do not
// depend on G.
template <int DT, int G, int AL>
__device__ __forceinline__ void mma_tiles_row(const typename DType<DT>::T* __restrict__ a_row, int Kpad, int K,
                                              const typename DType<DT>::T* __restrict__ W, int n0, int N, int lane,
                                              f32x4 (&acc)[G]) {
  using T = typename DType<DT>::T;
  using BT = typename std::conditional<DT == DT_F32, float, u32x4>::type;
  constexpr int KS = DType<DT>::KS;
  constexpr int KL = DT == DT_F32 ? 1 : 8;  // k values per lane per step
  const T* wrow[G];
  bool nok[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int n = n0 + 16 * g + (lane & 15);
    nok[g] = n < N;
    wrow[g] = W + (size_t)(nok[g] ? n : 0) * K + (lane >> 4) * KL;
  }
  const T* arow = a_row + (lane >> 4) * KL;
  const int kfull = K / KS * KS;
  auto a_at = [&](int k0) -> BT {
    if constexpr (DT == DT_F32)
      return arow[k0];
    else
      return *reinterpret_cast<const u32x4*>(arow + k0);
  };
#pragma unroll(G >= 4 ? 2 : 4)
  for (int k0 = 0; k0 < kfull; k0 += KS) {
    const BT a = a_at(k0);
    BT b[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (DT == DT_F32)
        b[g] = wrow[g][k0];
      else
        b[g] = load_w8<AL>(wrow[g] + k0);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if constexpr (DT == DT_F32)
        b[g] = nok[g] ? b[g] : 0.f;
      else
        b[g] = nok[g] ? b[g] : u32x4{0u, 0u, 0u, 0u};
      acc[g] = mfma_step(a, b[g], acc[g]);
    }
  }
  if (kfull < Kpad) {  // the partial last step
    const int k0 = kfull, kk = k0 + (lane >> 4) * KL;
    const BT a = a_at(k0);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      BT b = load_b_tail<DT>(wrow[g], k0, kk, K);
      if constexpr (DT == DT_F32)
        b = nok[g] ? b : 0.f;
      else
        b = nok[g] ? b : u32x4{0u, 0u, 0u, 0u};
      acc[g] = mfma_step(a, b, acc[g]);
    }
  }
}

// One tile (G = 1).
template <int DT>
__device__ __forceinline__ f32x4 mma_tile_row(const typename DType<DT>::T* __restrict__ a_row, int Kpad, int K,
                                              const typename DType<DT>::T* __restrict__ W, int n0, int N,
                                              int lane) {
  f32x4 acc[1];
  if (DT == DT_F32 || weight_align(K) == WALIGN_16)
    mma_tiles_row<DT, 1, WALIGN_16>(a_row, Kpad, K, W, n0, N, lane, acc);
  else if (weight_align(K) == WALIGN_4)
    mma_tiles_row<DT, 1, WALIGN_4>(a_row, Kpad, K, W, n0, N, lane, acc);
  else
    mma_tiles_row<DT, 1, WALIGN_2>(a_row, Kpad, K, W, n0, N, lane, acc);
  return acc[0];
}

// The same tile for rows m0..m0+15 of a row-major A with leading dimension lda.
template <int DT>
__device__ __forceinline__ f32x4 mma_tile(const typename DType<DT>::T* __restrict__ in, int lda, int m0,
                                          int Kpad, int K, const typename DType<DT>::T* __restrict__ W,
                                          int n0, int N, int lane) {
  return mma_tile_row<DT>(in + (size_t)(m0 + (lane & 15)) * lda, Kpad, K, W, n0, N, lane);
}

// A dense layer over R rows (a multiple of 16) in groups of G output tiles
// per wave.  Row r of the input is in[rows ? rows[r] : r].  Hidden layers
// (LOGITS false) store tanh(x W^T + b) in the layer dtype to `out`; the
// output layer stores x W^T + b as float32 to `logits` (columns < N only).
template <int DT, int G, int AL, bool LOGITS>
__device__ __forceinline__ void mlp_layer_g(const typename DType<DT>::T* in, int lda, const int* rows, int R, int K,
                                            const typename DType<DT>::T* __restrict__ W,
                                            const typename DType<DT>::T* __restrict__ b, int N,
                                            typename DType<DT>::T* out, float* logits, int ldo, int wave, int nwaves,
                                            int lane) {
  using DTy = DType<DT>;
  const int Kpad = round_up(K, DTy::KS);
  const int mt = R >> 4, nt = (N + 15) >> 4, ng = (nt + G - 1) / G;
  for (int item = wave; item < mt * ng; item += nwaves) {
    const int m0 = (item / ng) << 4, n0 = (item % ng) * 16 * G;
    const int r = m0 + (lane & 15);
    f32x4 acc[G];
    mma_tiles_row<DT, G, AL>(in + (size_t)(rows ? rows[r] : r) * lda, Kpad, K, W, n0, N, lane, acc);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int col = n0 + 16 * g + (lane & 15);
      if (col < N) {
        const float bias = DTy::to_f32(b[col]);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = m0 + 4 * (lane >> 4) + q;
          if constexpr (LOGITS)
            logits[(size_t)row * ldo + col] = acc[g][q] + bias;
          else
            out[(size_t)row * ldo + col] = DTy::from_f32(fast_tanh(acc[g][q] + bias));
        }
      }
    }
  }
}

template <int DT, int AL, bool LOGITS>
__device__ __forceinline__ void mlp_layer_al(const typename DType<DT>::T* in, int lda, const int* rows, int R, int K,
                                             const typename DType<DT>::T* __restrict__ W,
                                             const typename DType<DT>::T* __restrict__ b, int N,
                                             typename DType<DT>::T* out, float* logits, int ldo, int wave,
                                             int nwaves, int lane) {
  const int tiles = (R >> 4) * ((N + 15) >> 4);
  if (tiles >= 4 * nwaves && ((N + 15) >> 4) % 4 == 0)
    mlp_layer_g<DT, 4, AL, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
  else if (tiles >= 2 * nwaves && ((N + 15) >> 4) % 2 == 0)
    mlp_layer_g<DT, 2, AL, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
  else
    mlp_layer_g<DT, 1, AL, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
}

// Picks the weight-load width for K and the widest tile group that still
// gives every wave work.
template <int DT, bool LOGITS>
__device__ __forceinline__ void mlp_layer(const typename DType<DT>::T* in, int lda, const int* rows, int R, int K,
                                          const typename DType<DT>::T* __restrict__ W,
                                          const typename DType<DT>::T* __restrict__ b, int N,
                                          typename DType<DT>::T* out, float* logits, int ldo, int wave, int nwaves,
                                          int lane) {
  const int al = DT == DT_F32 ? WALIGN_16 : weight_align(K);
  if (al == WALIGN_16)
    mlp_layer_al<DT, WALIGN_16, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
  else if (al == WALIGN_4)
    mlp_layer_al<DT, WALIGN_4, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
  else
    mlp_layer_al<DT, WALIGN_2, LOGITS>(in, lda, rows, R, K, W, b, N, out, logits, ldo, wave, nwaves, lane);
}

// A hidden layer: out = tanh(in W^T + b), stored in the layer dtype.
// R rows (multiple of 16), N outputs (multiple of 16).
template <int DT>
__device__ __forceinline__ void mlp_hidden(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N,
                                           typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                           int lane) {
  mlp_layer<DT, false>(in, lda, nullptr, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane);
}

// mlp_hidden over the A rows rows[0..R-1] of `in` (row indices in LDS).
template <int DT>
__device__ __forceinline__ void mlp_hidden_rows(const typename DType<DT>::T* in, int lda, const int* rows, int R,
                                                int K, const typename DType<DT>::T* __restrict__ W,
                                                const typename DType<DT>::T* __restrict__ b, int N,
                                                typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                                int lane) {
  mlp_layer<DT, false>(in, lda, rows, R, K, W, b, N, out, nullptr, ldo, wave, nwaves, lane);
}

// The output layer: logits = in W^T + b as float32, N <= 32 actions.
template <int DT>
__device__ __forceinline__ void mlp_logits(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N, float* out,
                                           int ldo, int wave, int nwaves, int lane) {
  mlp_layer<DT, true>(in, lda, nullptr, R, K, W, b, N, nullptr, out, ldo, wave, nwaves, lane);
}

}  // namespace rl
