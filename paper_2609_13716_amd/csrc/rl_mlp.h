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

// One 16 x 16 output tile: acc += A[16 rows, 0:Kpad] * W[n0:n0+16, 0:Kpad]^T,
// where `a` points at element 0 of A row (lane % 16) of the tile.
template <int DT>
__device__ __forceinline__ f32x4 mma_tile_row(const typename DType<DT>::T* __restrict__ a_row, int Kpad, int K,
                                              const typename DType<DT>::T* __restrict__ W, int n0, int N,
                                              int lane) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const int n = n0 + (lane & 15);
  const bool nok = n < N;
  if constexpr (DT == DT_F32) {
    const float* arow = a_row + (lane >> 4);
    const float* wrow = W + (size_t)(nok ? n : 0) * K + (lane >> 4);
    for (int k0 = 0; k0 < Kpad; k0 += 4) {
      const float a = arow[k0];
      const float b = (nok && k0 + (lane >> 4) < K) ? wrow[k0] : 0.f;
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
    }
  } else {
    const uint16_t* arow = a_row + (lane >> 4) * 8;
    const uint16_t* wrow = W + (size_t)(nok ? n : 0) * K + (lane >> 4) * 8;
    const bool vec = (K & 7) == 0;
    for (int k0 = 0; k0 < Kpad; k0 += 32) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(arow + k0);
      u32x4 b = {0u, 0u, 0u, 0u};
      const int kk = k0 + (lane >> 4) * 8;
      if (nok) {
        if (vec) {
          if (kk < K) b = *reinterpret_cast<const u32x4*>(wrow + k0);
        } else {
          uint32_t h[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t lo = (kk + 2 * q < K) ? wrow[k0 + 2 * q] : 0u;
            const uint32_t hi = (kk + 2 * q + 1 < K) ? wrow[k0 + 2 * q + 1] : 0u;
            h[q] = lo | (hi << 16);
          }
          b = u32x4{h[0], h[1], h[2], h[3]};
        }
      }
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    }
  }
  return acc;
}

// The same tile for rows m0..m0+15 of a row-major A with leading dimension lda.
template <int DT>
__device__ __forceinline__ f32x4 mma_tile(const typename DType<DT>::T* __restrict__ in, int lda, int m0,
                                          int Kpad, int K, const typename DType<DT>::T* __restrict__ W,
                                          int n0, int N, int lane) {
  return mma_tile_row<DT>(in + (size_t)(m0 + (lane & 15)) * lda, Kpad, K, W, n0, N, lane);
}

// A hidden layer: out = tanh(in W^T + b), stored in the layer dtype.
// R rows (multiple of 16), N outputs (multiple of 16).
template <int DT>
__device__ __forceinline__ void mlp_hidden(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N,
                                           typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                           int lane) {
  using DTy = DType<DT>;
  const int Kpad = round_up(K, DTy::KS);
  const int mt = R >> 4, nt = N >> 4;
  for (int tile = wave; tile < mt * nt; tile += nwaves) {
    const int m0 = (tile / nt) << 4, n0 = (tile % nt) << 4;
    const f32x4 acc = mma_tile<DT>(in, lda, m0, Kpad, K, W, n0, N, lane);
    const int col = n0 + (lane & 15);
    const float bias = DTy::to_f32(b[col]);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + 4 * (lane >> 4) + r;
      out[(size_t)row * ldo + col] = DTy::from_f32(fast_tanh(acc[r] + bias));
    }
  }
}

// mlp_hidden over the A rows rows[0..R-1] of `in` (row indices in LDS).
template <int DT>
__device__ __forceinline__ void mlp_hidden_rows(const typename DType<DT>::T* in, int lda, const int* rows, int R,
                                                int K, const typename DType<DT>::T* __restrict__ W,
                                                const typename DType<DT>::T* __restrict__ b, int N,
                                                typename DType<DT>::T* out, int ldo, int wave, int nwaves,
                                                int lane) {
  using DTy = DType<DT>;
  const int Kpad = round_up(K, DTy::KS);
  const int mt = R >> 4, nt = N >> 4;
  for (int tile = wave; tile < mt * nt; tile += nwaves) {
    const int m0 = (tile / nt) << 4, n0 = (tile % nt) << 4;
    const f32x4 acc = mma_tile_row<DT>(in + (size_t)rows[m0 + (lane & 15)] * lda, Kpad, K, W, n0, N, lane);
    const int col = n0 + (lane & 15);
    const float bias = DTy::to_f32(b[col]);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + 4 * (lane >> 4) + r;
      out[(size_t)row * ldo + col] = DTy::from_f32(fast_tanh(acc[r] + bias));
    }
  }
}

// The output layer: logits = in W^T + b as float32, N <= 32 actions.
template <int DT>
__device__ __forceinline__ void mlp_logits(const typename DType<DT>::T* in, int lda, int R, int K,
                                           const typename DType<DT>::T* __restrict__ W,
                                           const typename DType<DT>::T* __restrict__ b, int N, float* out,
                                           int ldo, int wave, int nwaves, int lane) {
  using DTy = DType<DT>;
  const int Kpad = round_up(K, DTy::KS);
  const int mt = R >> 4, nt = (N + 15) >> 4;
  for (int tile = wave; tile < mt * nt; tile += nwaves) {
    const int m0 = (tile / nt) << 4, n0 = (tile % nt) << 4;
    const f32x4 acc = mma_tile<DT>(in, lda, m0, Kpad, K, W, n0, N, lane);
    const int col = n0 + (lane & 15);
    if (col < N) {
      const float bias = DTy::to_f32(b[col]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + 4 * (lane >> 4) + r;
        out[(size_t)row * ldo + col] = acc[r] + bias;
      }
    }
  }
}

}  // namespace rl
