// Policy layers whose weights stay in registers for a whole rollout.
//
// A layer's N outputs are cut into 16-column tiles; tile j belongs to wave
// j % NW.  At kernel start each wave loads the MFMA B operands of its tiles
// for every K step into VGPRs (W in the nn.Linear layout [N x K]), so the
// per-step matrix products read only the LDS activation tile and registers.
// Same MFMA shapes and operand layouts as rl_mlp.h.
#pragma once
#include <type_traits>

#include "rl_mlp.h"

namespace rl {

template <int DT>
struct BOperand {
  using type = float;  // f32: one K element per lane per K step of 4
};
template <>
struct BOperand<DT_BF16> {
  using type = u32x4;  // bf16: eight K elements per lane per K step of 32
};

template <int DT>
__device__ __forceinline__ f32x4 mfma16(const typename BOperand<DT>::type& a, const typename BOperand<DT>::type& b,
                                        f32x4 acc) {
  if constexpr (DT == DT_F32) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                   0, 0, 0);
  }
}

// The B operand (or an A operand read from a row) of one lane for K step ks:
// f32 lanes hold element ks*4 + lane/16, bf16 lanes hold elements
// ks*32 + (lane/16)*8 .. +7.  Elements at or beyond K read as zero.
template <int DT, int KC = 0>
__device__ __forceinline__ typename BOperand<DT>::type load_operand_global(const typename DType<DT>::T* row, int K,
                                                                           int ks, int lane, bool valid) {
  if constexpr (KC > 0 && KC % DType<DT>::KS == 0) {
    // K a multiple of the K step (known at compile time): every element is
    // in range, one vector load per lane
    if constexpr (DT == DT_F32) {
      return valid ? row[ks * 4 + (lane >> 4)] : 0.f;
    } else {
      return valid ? *reinterpret_cast<const u32x4*>(row + ks * 32 + (lane >> 4) * 8) : u32x4{0u, 0u, 0u, 0u};
    }
  } else if constexpr (DT == DT_F32) {
    const int k = ks * 4 + (lane >> 4);
    return (valid && k < K) ? row[k] : 0.f;
  } else {
    const int k0 = ks * 32 + (lane >> 4) * 8;
    uint32_t h[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = (valid && k0 + 2 * q < K) ? row[k0 + 2 * q] : 0u;
      const uint32_t hi = (valid && k0 + 2 * q + 1 < K) ? row[k0 + 2 * q + 1] : 0u;
      h[q] = lo | (hi << 16);
    }
    return u32x4{h[0], h[1], h[2], h[3]};
  }
}

template <int DT>
__device__ __forceinline__ typename BOperand<DT>::type load_operand_lds(const typename DType<DT>::T* tile, int ld,
                                                                        int row, int ks, int lane) {
  if constexpr (DT == DT_F32) {
    return tile[row * ld + ks * 4 + (lane >> 4)];
  } else {
    return *reinterpret_cast<const u32x4*>(tile + row * ld + ks * 32 + (lane >> 4) * 8);
  }
}

// BL: the bias lives in an fp32 LDS array of N entries (filled by the caller
// before the first store_tanh) instead of registers, for layers whose
// resident weights leave no room for it.
template <int DT, int K, int N, int NW, bool BL = false>
struct RegLayer {
  using T = typename DType<DT>::T;
  using B = typename BOperand<DT>::type;
  static constexpr int KS = DType<DT>::KS;
  static constexpr int KSTEPS = round_up(K, KS) / KS;
  static constexpr int NT = N / 16;
  static constexpr int OWN = (NT + NW - 1) / NW;
  // VGPRs per lane that the resident operands take
  static constexpr int WREGS = OWN * KSTEPS * (int)(sizeof(B) / 4) + (BL ? 0 : 4 * OWN);
  // operand reads in flight ahead of the MFMAs in run (fewer where the
  // resident weights already crowd the register file)
  static constexpr int PFMAX = BL ? 2 : 6;
  static_assert(N % 16 == 0, "layer width must be a multiple of 16");

  B w[OWN][KSTEPS];                 // operand of output units tile*16 + lane%16
  float bias[BL ? 1 : OWN][4];      // bias of output units tile*16 + 4*(lane/16) + r

  __device__ __forceinline__ void load(const T* __restrict__ W, const T* __restrict__ b, int wave, int lane) {
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
      const int tile = wave + o * NW;
      const bool valid = tile < NT;
      const int n = tile * 16 + (lane & 15);
      const T* row = W + (size_t)(valid ? n : 0) * K;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) w[o][ks] = load_operand_global<DT, K>(row, K, ks, lane, valid);
      if constexpr (!BL) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          bias[o][r] = valid ? DType<DT>::to_f32(b[tile * 16 + 4 * (lane >> 4) + r]) : 0.f;
      }
    }
  }

  // Transposed products, out^T = W in^T: acc[m][o] element r holds output
  // unit tile(o)*16 + 4*(lane/16) + r of row m*16 + lane%16.  (Each sum is
  // the same MFMA chain as the untransposed product, so the values are
  // bit-identical to it.)
  template <int MT>
  __device__ __forceinline__ void run(const T* in, int ld, f32x4 (&acc)[MT][OWN], int wave, int lane) const {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int o = 0; o < OWN; ++o) acc[m][o] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (NT % NW == 0) {
      // every wave owns OWN full tiles: a branch-free chain.  The LDS operand
      // of step s (K step s / MT, row tile s % MT) is read PF steps ahead of
      // its MFMAs into a register of its own, so that the reads are in flight
      // together; with one operand register reused, each read would wait for
      // the MFMAs of the previous one and the chain would pay the LDS latency
      // once per K step.
      constexpr int STEPS = KSTEPS * MT;
      constexpr int PF = STEPS < PFMAX ? STEPS : PFMAX;
      B a[STEPS];
#pragma unroll
      for (int s = 0; s < PF; ++s) a[s] = load_operand_lds<DT>(in, ld, (s % MT) * 16 + (lane & 15), s / MT, lane);
      __builtin_amdgcn_sched_barrier(0);  // (the scheduler would sink these reads below the first MFMAs)
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        if (s + PF < STEPS)
          a[s + PF] = load_operand_lds<DT>(in, ld, ((s + PF) % MT) * 16 + (lane & 15), (s + PF) / MT, lane);
        const int ks = s / MT, m = s % MT;
#pragma unroll
        for (int o = 0; o < OWN; ++o) acc[m][o] = mfma16<DT>(w[o][ks], a[s], acc[m][o]);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const B a = load_operand_lds<DT>(in, ld, m * 16 + (lane & 15), ks, lane);
#pragma unroll
          for (int o = 0; o < OWN; ++o)
            if (wave + o * NW < NT) acc[m][o] = mfma16<DT>(w[o][ks], a, acc[m][o]);
        }
      }
    }
  }

  // out = tanh(acc + bias) in the layer dtype for one accumulator (row tile
  // m, owned tile o): four consecutive units of one row per lane, stored with
  // one 8-byte (bf16) or 16-byte (f32) LDS write.
  __device__ __forceinline__ void store_block(const f32x4& acc, T* out, int ld, int m, int o, int wave, int lane,
                                              const float* bias_lds) const {
    const int row = m * 16 + (lane & 15);
    const int col = (wave + o * NW) * 16 + 4 * (lane >> 4);
    float bo[4];
    if constexpr (BL) {
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias_lds + col);
#pragma unroll
      for (int r = 0; r < 4; ++r) bo[r] = b4[r];
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) bo[r] = bias[o][r];
    }
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = fast_tanh(acc[r] + bo[r]);
    if constexpr (DT == DT_F32) {
      *reinterpret_cast<f32x4*>(out + row * ld + col) = f32x4{v[0], v[1], v[2], v[3]};
    } else {
      const uint32_t lo = pack_bf16x2(v[0], v[1]);
      const uint32_t hi = pack_bf16x2(v[2], v[3]);
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      *reinterpret_cast<u32x2*>(out + row * ld + col) = u32x2{lo, hi};
    }
  }

  template <int MT>
  __device__ __forceinline__ void store_tanh(const f32x4 (&acc)[MT][OWN], T* out, int ld, int wave, int lane,
                                             const float* bias_lds = nullptr) const {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int o = 0; o < OWN; ++o) {
        if (NT % NW != 0 && wave + o * NW >= NT) continue;
        store_block(acc[m][o], out, ld, m, o, wave, lane, bias_lds);
      }
  }

  // Software-pipelined layer step for a wave that owns whole tiles: acc gets
  // W in^T of a new row tile (the same MFMA chains as run, so the same bits),
  // while the epilogue of acc's previous contents (store_tanh into out) is
  // spread between the matrix instructions.  The wave's transcendental and
  // conversion work then issues while its own MFMAs execute, instead of
  // after them.
  template <int MT>
  __device__ __forceinline__ void run_overlapped(const T* in, int ld, f32x4 (&acc)[MT][OWN], T* out, int ldo,
                                                 int wave, int lane) const {
    static_assert(NT % NW == 0, "every wave owns whole tiles");
    constexpr int STEPS = KSTEPS * MT, EB = MT * OWN;
    f32x4 prev[MT][OWN];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int o = 0; o < OWN; ++o) {
        prev[m][o] = acc[m][o];
        acc[m][o] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    B a = load_operand_lds<DT>(in, ld, lane & 15, 0, lane);
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int ks = s / MT, m = s % MT;
      B an = a;
      if (s + 1 < STEPS) an = load_operand_lds<DT>(in, ld, ((s + 1) % MT) * 16 + (lane & 15), (s + 1) / MT, lane);
#pragma unroll
      for (int o = 0; o < OWN; ++o) acc[m][o] = mfma16<DT>(w[o][ks], a, acc[m][o]);
#pragma unroll
      for (int e = 0; e < EB; ++e)
        if (e * STEPS / EB == s) store_block(prev[e / OWN][e % OWN], out, ldo, e / OWN, e % OWN, wave, lane, nullptr);
      a = an;
    }
  }
};

// A bf16 layer with the same interface, MFMA chains and outputs as RegLayer
// whose weights are streamed instead of held: each K step's B operands of the
// wave's tiles are read from global memory (L2) PD steps ahead of their MFMAs,
// from the fragment-major packed copy (one contiguous 1 KB block per
// wave-wide load; the caller must supply it).  It holds PD operand sets
// instead of all KSTEPS, for shapes whose resident weights would not fit the
// register file.
template <int DT, int K, int N, int NW, bool BL = false, int PD = 4>
struct StreamLayer {
  static_assert(DT == DT_BF16, "streamed resident-interface layer: bf16");
  using T = typename DType<DT>::T;
  using B = typename BOperand<DT>::type;
  static constexpr int KS = DType<DT>::KS;
  static constexpr int KSTEPS = round_up(K, KS) / KS;
  static constexpr int NT = N / 16;
  static constexpr int OWN = (NT + NW - 1) / NW;
  static constexpr int P = PD < KSTEPS ? PD : KSTEPS;  // operand sets in flight
  static constexpr int WREGS = OWN * P * (int)(sizeof(B) / 4) + (BL ? 0 : 4 * OWN);
  static_assert(N % 16 == 0, "layer width must be a multiple of 16");

  const T* Wp;  // fragment-major copy (rl_policy_pack layout)
  float bias[BL ? 1 : OWN][4];

  __device__ __forceinline__ void load(const T* __restrict__ b, int wave, int lane, const T* __restrict__ Wp_) {
    Wp = Wp_;
    if constexpr (!BL) {
#pragma unroll
      for (int o = 0; o < OWN; ++o) {
        const int tile = wave + o * NW;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          bias[o][r] = tile < NT ? DType<DT>::to_f32(b[tile * 16 + 4 * (lane >> 4) + r]) : 0.f;
      }
    }
  }

  __device__ __forceinline__ void fetch(int ks, B (&dst)[OWN], int wave, int lane) const {
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
      const int tile = wave + o * NW;
      // tile t, K step s at block (t * KSTEPS + s), lane l's 16 bytes
      dst[o] = tile < NT ? *reinterpret_cast<const B*>(Wp + ((size_t)(tile * KSTEPS + ks) * 64 + lane) * 8)
                         : B{0u, 0u, 0u, 0u};
    }
  }

  // Same products and accumulation order as RegLayer::run.
  template <int MT>
  __device__ __forceinline__ void run(const T* in, int ld, f32x4 (&acc)[MT][OWN], int wave, int lane) const {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int o = 0; o < OWN; ++o) acc[m][o] = f32x4{0.f, 0.f, 0.f, 0.f};
    // (the lane index is made opaque here, so that the weight addresses are
    // formed inside each call rather than hoisted out of the caller's step
    // loop into registers that would stay live for the whole rollout)
    int ln = lane;
    asm volatile("" : "+v"(ln));
    B ring[P][OWN];
#pragma unroll
    for (int q = 0; q < P; ++q) fetch(q, ring[q], wave, ln);
    // the LDS operands of K step ks + 1 are read while the MFMAs of step ks
    // run (two register sets), so each step does not wait out an LDS latency
    B a[2][MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) a[0][m] = load_operand_lds<DT>(in, ld, m * 16 + (lane & 15), 0, lane);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
          a[(ks + 1) & 1][m] = load_operand_lds<DT>(in, ld, m * 16 + (lane & 15), ks + 1, lane);
      }
      __builtin_amdgcn_sched_barrier(0);  // (keeps those reads ahead of this step's MFMAs)
#pragma unroll
      for (int m = 0; m < MT; ++m) {
#pragma unroll
        for (int o = 0; o < OWN; ++o)
          if (NT % NW == 0 || wave + o * NW < NT) acc[m][o] = mfma16<DT>(ring[ks % P][o], a[ks & 1][m], acc[m][o]);
      }
      if (ks + P < KSTEPS) fetch(ks + P, ring[ks % P], wave, ln);
    }
  }

  __device__ __forceinline__ void store_block(const f32x4& acc, T* out, int ld, int m, int o, int wave, int lane,
                                              const float* bias_lds) const {
    const int row = m * 16 + (lane & 15);
    const int col = (wave + o * NW) * 16 + 4 * (lane >> 4);
    float bo[4];
    if constexpr (BL) {
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(bias_lds + col);
#pragma unroll
      for (int r = 0; r < 4; ++r) bo[r] = b4[r];
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) bo[r] = bias[o][r];
    }
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = fast_tanh(acc[r] + bo[r]);
    const uint32_t lo = pack_bf16x2(v[0], v[1]);
    const uint32_t hi = pack_bf16x2(v[2], v[3]);
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    *reinterpret_cast<u32x2*>(out + row * ld + col) = u32x2{lo, hi};
  }

  template <int MT>
  __device__ __forceinline__ void store_tanh(const f32x4 (&acc)[MT][OWN], T* out, int ld, int wave, int lane,
                                             const float* bias_lds = nullptr) const {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int o = 0; o < OWN; ++o) {
        if (NT % NW != 0 && wave + o * NW >= NT) continue;
        store_block(acc[m][o], out, ld, m, o, wave, lane, bias_lds);
      }
  }
};

// Cross-lane argmax within each 16-lane row of a wave: lexicographic max of
// (score, -index), i.e. the first index of the largest score.  Uses DPP lane
// permutations (no LDS traffic): swap neighbours, swap pairs, mirror each
// half-row, mirror the row; after the four steps every lane of the row holds
// the result.
template <int CTRL>
__device__ __forceinline__ void argmax_dpp_step(float& score, int& idx) {
  const float os = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(score), CTRL, 0xf, 0xf, false));
  const int oi = __builtin_amdgcn_update_dpp(0, idx, CTRL, 0xf, 0xf, false);
  const bool take = (os > score) | ((os == score) & (oi < idx));
  score = take ? os : score;
  idx = take ? oi : idx;
}

__device__ __forceinline__ void row16_argmax(float& score, int& idx) {
  argmax_dpp_step<0xB1>(score, idx);   // quad_perm [1,0,3,2]
  argmax_dpp_step<0x4E>(score, idx);   // quad_perm [2,3,0,1]
  argmax_dpp_step<0x141>(score, idx);  // row_half_mirror
  argmax_dpp_step<0x140>(score, idx);  // row_mirror
}

}  // namespace rl
