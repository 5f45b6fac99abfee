// Recurrent S5 actor-critic in the rollout loop (LBF), bfloat16 dense layers.
//
// The ego agent of the paper's experiments: observations through a dense
// encoder into an S5 layer (model width H, complex diagonal state of size P),
// then separate actor and critic heads of three F-wide tanh layers.  S5
// (Smith et al., ICLR 2023): zero-order hold of x' = Lambda x + B u gives
// Lambda_bar = exp(Lambda Delta), B_bar = Lambda^-1 (Lambda_bar - 1) B; a step
// is x_t = Lambda_bar x_{t-1} + B_bar u_t, y_t = Re(C x_t) + D u_t, with the
// state zeroed at an episode's first step (as Lu et al., NeurIPS 2023, do
// for reinforcement learning).
//
// One rollout step is six launches on one stream:
//   front  per 32 rows: observation tile -> encoder (bf16 MFMA, tanh) -> the
//          S5 step in float32 MFMA (B_bar u as two real products, the
//          complex diagonal update with the reset, Re(C x) as two real
//          products) -> y in bf16, the carried state updated in place;
//   heads  three grouped GEMMs (actor and critic in one launch, 128 x 128
//          tiles, LDS double buffering, bias + tanh epilogue in bf16);
//   out    output layers (logits, value), Gumbel-max sampling with the
//          rollout's Philox draws, log pi of the sampled action;
//   env    one LBF step with the sampled actions (the env-only kernels).
// The heads dominate (2 x (H F + 2 F F) MACs per row): they are the GEMMs
// that the MFMA roofline is taken on.
#include <mutex>
#include "rl_internal.h"
#include "rl_mlp.h"
#include "rl_sample.h"

namespace rl {

// ------------------------------------------------------- discretisation ----

// Zero-order hold in float64 (rounded once to float32 at the end):
// lambda_bar = exp(lambda dt), b_bar[p, h] = (lambda_bar - 1) / lambda * b[p, h].
__global__ void s5_discretize_kernel(int P, int H, const float* __restrict__ lam, const float* __restrict__ log_dt,
                                     const float* __restrict__ b, float* __restrict__ lbar,
                                     float* __restrict__ bbar) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;  // p * H + h
  if (i >= P * H) return;
  const int p = i / H;
  const double lr = lam[p], li = lam[P + p], dt = exp((double)log_dt[p]);
  const double mag = exp(lr * dt);
  const double er = mag * cos(li * dt), ei = mag * sin(li * dt);  // lambda_bar
  // (lambda_bar - 1) / lambda
  const double nr = er - 1.0, ni = ei, den = lr * lr + li * li;
  const double qr = (nr * lr + ni * li) / den, qi = (ni * lr - nr * li) / den;
  const double br = b[i], bi = b[(size_t)P * H + i];
  bbar[i] = (float)(qr * br - qi * bi);
  bbar[(size_t)P * H + i] = (float)(qr * bi + qi * br);
  if (i % H == 0) {
    lbar[p] = (float)er;
    lbar[P + p] = (float)ei;
  }
}

hipError_t launch_s5_discretize(int P, int H, const float* lam, const float* log_dt, const float* b, float* lbar,
                                float* bbar, hipStream_t s) {
  const int n = P * H;
  s5_discretize_kernel<<<dim3((unsigned)((n + 255) / 256)), 256, 0, s>>>(P, H, lam, log_dt, b, lbar, bbar);
  return hipGetLastError();
}

// ---------------------------------------------------------------- front ----

constexpr int S5_RT = 32;    // rows per front workgroup
constexpr int S5F_NT = 512;  // front: 8 waves, one 16-column item each per phase (latency hiding)
constexpr int S5F_NW = S5F_NT / 64;
constexpr int S5_NT = 256;  // threads of the head and output kernels
constexpr int S5_NW = S5_NT / 64;

constexpr int S5_WK = 32;       // K slice of the float32 weights staged in LDS
constexpr int S5_WLD = S5_WK + 2;  // its row stride in words: 16 rows x 2 k of a half-wave on 32 banks
constexpr int S5_WROWS = 256;     // rows of a staged slice: at most 2P (B_bar) and H (C)

struct S5Lds {
  int ldx, ldu, ldf, ldxf;
  size_t off_u, off_xf, off_keep, off_w, total;  // region 0 (obs tile, then u as float) at 0
};

__host__ __device__ inline S5Lds s5_lds(int D, int H, int P) {
  S5Lds L;
  L.ldx = lds_ld<DT_BF16>(D);
  L.ldu = lds_ld<DT_BF16>(H);
  // float32 operand rows: a stride of 2 (mod 32) words puts the 16 rows x 2 k
  // of each half-wave's MFMA operand reads on 32 distinct banks
  L.ldf = round_up(H, 32) + 2;
  L.ldxf = round_up(2 * P, 32) + 2;  // state tile: real parts, then imaginary parts
  const size_t r0 = (size_t)S5_RT * (L.ldx * 2 > L.ldf * 4 ? L.ldx * 2 : L.ldf * 4);
  L.off_u = (r0 + 15) / 16 * 16;
  L.off_xf = (L.off_u + (size_t)S5_RT * L.ldu * 2 + 15) / 16 * 16;
  L.off_keep = L.off_xf + (size_t)S5_RT * L.ldxf * 4;
  L.off_w = (L.off_keep + S5_RT * 4 + 15) / 16 * 16;
  L.total = L.off_w + (size_t)2 * S5_WROWS * S5_WLD * 4;  // two slice buffers
  return L;
}

size_t s5_front_lds_bytes(int D, int H, int P) { return s5_lds(D, H, P).total; }

struct S5FrontArgs {
  const uint16_t* obs;   // [R, D] bf16
  const int32_t* state;  // env state planes; an episode starts where plane step_plane is 0
  int step_plane, E, A, R, D, H, P;
  float* carry;  // [R, 2P]: real parts, then imaginary parts
  int commit;    // write the new state back (0: value of the final observation only)
  const uint16_t* w_enc;
  const uint16_t* b_enc;
  const float* lbar;  // [2, P]
  const float* bbar;  // [2, P, H]
  const float* wcat;  // [H, 2P]: C_re | -C_im, so that Re(C x) is one product with [x_re | x_im]
  const float* d;     // [H]
  uint16_t* y;        // [R, H] bf16
};

// [C_re | -C_im] as one [H, 2P] matrix.
__global__ void s5_cat_kernel(int H, int P, const float* __restrict__ c, float* __restrict__ wcat) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;  // h * 2P + k
  if (i >= H * 2 * P) return;
  const int h = i / (2 * P), k = i - h * 2 * P;
  wcat[i] = k < P ? c[(size_t)h * P + k] : -c[(size_t)H * P + (size_t)h * P + (k - P)];
}

// float32 MFMA tiles acc[m][g] = A[16 m + r][0:K] . W[nb[g] + c][0:K] for
// r, c < 16, where W ([N, K] row-major, N <= 256, K a multiple of 32) is read
// from global memory with 16-byte loads in K slices of 32, all N rows of a
// slice staged by the whole workgroup into LDS (double-buffered; the loads
// of slice s + 1 are issued before slice s is multiplied).  Every wave must
// call it (it holds barriers).  A rows are in LDS with stride lda.
template <int MT, int G>
__device__ __forceinline__ void s5_lds_mma(const float* A, int lda, const float* __restrict__ W, int N, int K,
                                           const int (&nb)[G], float* wsl, int tid, int lane, f32x4 (&acc)[MT][G]) {
  constexpr int CPT = S5_WROWS * (S5_WK / 4) / S5F_NT;  // 16-byte chunks per thread per slice (at most)
  const int nchunk = N * (S5_WK / 4);
  f32x4 reg[CPT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int q = tid + S5F_NT * j;
      if (q < nchunk) reg[j] = *reinterpret_cast<const f32x4*>(W + (size_t)(q >> 3) * K + k0 + (q & 7) * 4);
    }
  };
  auto lstore = [&](int buf) {
    float* w = wsl + buf * S5_WROWS * S5_WLD;
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int q = tid + S5F_NT * j;
      if (q < nchunk) {
        float* d = w + (q >> 3) * S5_WLD + (q & 7) * 4;
        *reinterpret_cast<float2*>(d) = float2{reg[j][0], reg[j][1]};
        *reinterpret_cast<float2*>(d + 2) = float2{reg[j][2], reg[j][3]};
      }
    }
  };
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int g = 0; g < G; ++g) acc[m][g] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int ns = K / S5_WK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int sl = 0; sl < ns; ++sl) {
    if (sl + 1 < ns) gload((sl + 1) * S5_WK);
    const float* w = wsl + (sl & 1) * S5_WROWS * S5_WLD;
#pragma unroll
    for (int kk = 0; kk < S5_WK; kk += 4) {
      const int k = kk + (lane >> 4);
      float av[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) av[m] = A[(16 * m + (lane & 15)) * lda + sl * S5_WK + k];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float bv = w[(nb[g] + (lane & 15)) * S5_WLD + k];
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[m][g] = mfma_step(av[m], bv, acc[m][g]);
      }
    }
    if (sl + 1 < ns) lstore((sl + 1) & 1);
    __syncthreads();
  }
}

__global__ __launch_bounds__(S5F_NT) void s5_front_kernel(S5FrontArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  constexpr int MT = S5_RT / 16;
  const S5Lds L = s5_lds(a.D, a.H, a.P);
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  float* uf = reinterpret_cast<float*>(smem);  // replaces xs once the encoder is done
  uint16_t* us = reinterpret_cast<uint16_t*>(smem + L.off_u);
  float* xf = reinterpret_cast<float*>(smem + L.off_xf);
  float* wsl = reinterpret_cast<float*>(smem + L.off_w);
  int* keep_s = reinterpret_cast<int*>(smem + L.off_keep);  // 1: the row's episode continues (carry used)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = blockIdx.x * S5_RT;
  const int D = a.D, H = a.H, P = a.P;

  if (tid < S5_RT) {
    const int row = r0 + tid;
    keep_s[tid] = row < a.R && a.state[(size_t)a.step_plane * a.E + row / a.A] != 0;
  }
  // observation tile (zero past D and past the last row): 16-byte chunks
  // when rows are whole chunks (all loads issued before the stores)
  if (D % 8 == 0) {
    const int cpr = L.ldx / 8;  // chunks per LDS row (the K padding included)
    constexpr int CI = 4;
    for (int i0 = tid; i0 < S5_RT * cpr; i0 += CI * S5F_NT) {
      u32x4 v[CI];
#pragma unroll
      for (int j = 0; j < CI; ++j) {
        const int i = i0 + j * S5F_NT, r = i / cpr, c = (i - r * cpr) * 8;
        v[j] = (i < S5_RT * cpr && r0 + r < a.R && c < D)
                   ? *reinterpret_cast<const u32x4*>(a.obs + (size_t)(r0 + r) * D + c)
                   : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int j = 0; j < CI; ++j) {
        const int i = i0 + j * S5F_NT, r = i / cpr, c = (i - r * cpr) * 8;
        if (i < S5_RT * cpr) *reinterpret_cast<u32x4*>(xs + r * L.ldx + c) = v[j];
      }
    }
  } else {
    for (int i = tid; i < S5_RT * L.ldx; i += S5F_NT) {
      const int r = i / L.ldx, c = i - r * L.ldx;
      xs[i] = (r0 + r < a.R && c < D) ? a.obs[(size_t)(r0 + r) * D + c] : (uint16_t)0;
    }
  }
  __syncthreads();
  // u = tanh(W_enc o + b_enc), rounded to bf16
  mlp_input_layer<DT_BF16>(xs, L.ldx, nullptr, S5_RT, D, a.w_enc, a.b_enc, H, us, L.ldu, wave, S5F_NW, lane);
  __syncthreads();
  for (int i = tid; i < S5_RT * H; i += S5F_NT) {
    const int r = i / H, h = i - r * H;
    uf[r * L.ldf + h] = bf16_to_f32(us[r * L.ldu + h]);
  }
  __syncthreads();

  // x_new = Lambda_bar x (zeroed at an episode start) + B_bar u: wave w takes
  // states 16 w.. (P <= 16 waves' worth): its real and imaginary rows of B_bar
  // ([2P, H] rows 16 w.. and P + 16 w..) as two tiles
  {
    const int item = wave < P / 16 ? wave : 0;
    const int n0 = item * 16;
    const int p = n0 + (lane & 15);
    // previous states of this lane's rows, loaded ahead of the product (rows past the end read the last row)
    float xo[MT][4][2];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const size_t row = (size_t)min(r0 + 16 * m + 4 * (lane >> 4) + q, a.R - 1);
        xo[m][q][0] = a.carry[row * 2 * P + p];
        xo[m][q][1] = a.carry[row * 2 * P + P + p];
      }
    const float lr = a.lbar[p], li = a.lbar[P + p];
    f32x4 bu[MT][2];
    const int nb[2] = {n0, P + n0};
    s5_lds_mma<MT, 2>(uf, L.ldf, a.bbar, 2 * P, H, nb, wsl, tid, lane, bu);
    if (wave < P / 16)
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rl = 16 * m + 4 * (lane >> 4) + q, row = r0 + rl;
        const bool keep = keep_s[rl] != 0;
        const float xr = keep ? xo[m][q][0] : 0.f, xi = keep ? xo[m][q][1] : 0.f;
        const float nr = lr * xr - li * xi + bu[m][0][q];
        const float ni = lr * xi + li * xr + bu[m][1][q];
        xf[rl * L.ldxf + p] = nr;
        xf[rl * L.ldxf + P + p] = ni;
        if (a.commit && row < a.R) {
          a.carry[(size_t)row * 2 * P + p] = nr;
          a.carry[(size_t)row * 2 * P + P + p] = ni;
        }
      }
  }
  __syncthreads();

  // y = Re(C x) + D u = [C_re | -C_im] [x_re | x_im] + D u, rounded to bf16:
  // wave w takes outputs 16 w.. and 16 (w + 8).. (H <= 256)
  {
    f32x4 cy[MT][2];
    const int nb[2] = {(16 * wave) % H, (16 * (wave + S5F_NW)) % H};
    s5_lds_mma<MT, 2>(xf, L.ldxf, a.wcat, H, 2 * P, nb, wsl, tid, lane, cy);
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      if (16 * (wave + S5F_NW * g) >= H) continue;
      const int h = 16 * (wave + S5F_NW * g) + (lane & 15);
      const float dh = a.d[h];
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rl = 16 * m + 4 * (lane >> 4) + q, row = r0 + rl;
          const float yv = cy[m][g][q] + dh * uf[rl * L.ldf + h];
          if (row < a.R) a.y[(size_t)row * H + h] = f32_to_bf16(yv);
        }
    }
  }
}

// ---------------------------------------------------------------- heads ----
//
// out[z] = tanh(in[z] W[z]^T + b[z]) in bf16 for the two heads z (grouped in
// one launch).  128 x 128 output tiles, 4 waves of 64 x 64, K in stages of 64
// through double-buffered LDS (16-byte chunks XOR-swizzled by row so that
// each 8-lane group of a fragment read covers all 32 banks).  The product is
// taken transposed (W rows as the MFMA A operand), so each lane ends with
// four consecutive outputs of one row: 8-byte stores.  Tiles are dealt so that
// each XCD gets a contiguous range of one head's row blocks: that XCD's L2
// then holds one head's weights and each input row block once.

constexpr int HG_BM = 128, HG_BN = 128, HG_BK = 64;

struct HeadGemmArgs {
  const uint16_t* in[2];
  int lda;
  const uint16_t* w[2];  // [N, K]
  const uint16_t* b[2];  // [N]
  uint16_t* out[2];
  int ldo, M, N, K;
};

__device__ __forceinline__ int hg_off(int row, int chunk) { return row * HG_BK + ((chunk ^ (row & 7)) << 3); }

__global__ __launch_bounds__(S5_NT, 2) void s5_head_gemm_kernel(HeadGemmArgs g) {
  __shared__ __align__(16) uint16_t sa[2][HG_BM * HG_BK];
  __shared__ __align__(16) uint16_t sb[2][HG_BN * HG_BK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int mt = (g.M + HG_BM - 1) / HG_BM, nt = g.N / HG_BN;
  const int total = 2 * mt * nt;
  const int L = blockIdx.x;
  const int T = (total % 8 == 0) ? (L % 8) * (total / 8) + L / 8 : L;  // XCD-contiguous tile ranges
  const int z = T / (mt * nt), rem = T - z * mt * nt;
  const int m0 = (rem / nt) * HG_BM, n0 = (rem % nt) * HG_BN;
  const uint16_t* __restrict__ A = g.in[z];
  const uint16_t* __restrict__ W = g.w[z];
  const int wm = wave >> 1, wn = wave & 1;

  // Two register stages: the global loads of stage s + 2 are issued before
  // stage s's MFMAs and reach LDS after stage s + 1's, so each load has two
  // stages of MFMA work to arrive in.
  u32x4 ra0[4], rb0[4], ra1[4], rb1[4];
  auto gload = [&](int k0, u32x4(&A4)[4], u32x4(&B4)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int q = tid + S5_NT * i, row = q >> 3, c = q & 7;
      const int ar = min(m0 + row, g.M - 1);
      A4[i] = *reinterpret_cast<const u32x4*>(A + (size_t)ar * g.lda + k0 + c * 8);
      B4[i] = *reinterpret_cast<const u32x4*>(W + (size_t)(n0 + row) * g.K + k0 + c * 8);
    }
  };
  auto lstore = [&](int buf, const u32x4(&A4)[4], const u32x4(&B4)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int q = tid + S5_NT * i, row = q >> 3, c = q & 7;
      *reinterpret_cast<u32x4*>(&sa[buf][hg_off(row, c)]) = A4[i];
      *reinterpret_cast<u32x4*>(&sb[buf][hg_off(row, c)]) = B4[i];
    }
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int c = kk * 4 + (lane >> 4);
      u32x4 fw[4], fx[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int nr = wn * 64 + j * 16 + (lane & 15);
        fw[j] = *reinterpret_cast<const u32x4*>(&sb[buf][hg_off(nr, c)]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mr = wm * 64 + i * 16 + (lane & 15);
        fx[i] = *reinterpret_cast<const u32x4*>(&sa[buf][hg_off(mr, c)]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = mfma_step(fw[j], fx[i], acc[j][i]);
    }
  };

  const int nk = g.K / HG_BK;  // >= 1
  gload(0, ra0, rb0);
  if (nk > 1) gload(HG_BK, ra1, rb1);
  lstore(0, ra0, rb0);
  __syncthreads();
  for (int s = 0; s < nk; s += 2) {
    // LDS buffer 0 holds stage s, registers 1 stage s + 1
    if (s + 2 < nk) gload((s + 2) * HG_BK, ra0, rb0);
    compute(0);
    if (s + 1 < nk) lstore(1, ra1, rb1);
    __syncthreads();
    if (s + 1 < nk) {
      if (s + 3 < nk) gload((s + 3) * HG_BK, ra1, rb1);
      compute(1);
      if (s + 2 < nk) lstore(0, ra0, rb0);
      __syncthreads();
    }
  }

  const uint16_t* __restrict__ bias = g.b[z];
  uint16_t* __restrict__ out = g.out[z];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int nb = n0 + wn * 64 + j * 16 + 4 * (lane >> 4);
    const uint2 bw = *reinterpret_cast<const uint2*>(bias + nb);
    const float b0 = bf16_to_f32((uint16_t)(bw.x & 0xffffu)), b1 = bf16_to_f32((uint16_t)(bw.x >> 16));
    const float b2 = bf16_to_f32((uint16_t)(bw.y & 0xffffu)), b3 = bf16_to_f32((uint16_t)(bw.y >> 16));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + wm * 64 + i * 16 + (lane & 15);
      if (m < g.M) {
        uint2 v;
        v.x = pack_bf16x2(fast_tanh(acc[j][i][0] + b0), fast_tanh(acc[j][i][1] + b1));
        v.y = pack_bf16x2(fast_tanh(acc[j][i][2] + b2), fast_tanh(acc[j][i][3] + b3));
        *reinterpret_cast<uint2*>(out + (size_t)m * g.ldo + nb) = v;
      }
    }
  }
}

// --------------------------------------------------------------- output ----

struct S5OutArgs {
  const uint16_t* ha;  // [R, F] last actor hidden layer
  const uint16_t* hc;  // [R, F] last critic hidden layer
  const uint16_t* wa;  // [nA, F]
  const uint16_t* ba;
  const uint16_t* wc;  // [1, F]
  const uint16_t* bc;
  int R, F, NA, A;
  uint64_t seed, t;
  int64_t env_base;
  int sample;  // 0: value only (into value)
  int32_t* actions;
  float* logits;  // [R, nA] or null
  float* value;   // [R] or null
  float* logp;    // [R] or null
};

// 16 rows per workgroup: wave w takes the K slice [w F / 4, (w + 1) F / 4)
// of both output layers (MFMA chains over 16-byte fragments), the four
// partial sums meet in LDS and lanes 0-15 of wave 0 finish and sample a row.
__global__ __launch_bounds__(S5_NT) void s5_out_kernel(S5OutArgs o) {
  __shared__ float lp[S5_NW][16][17];
  __shared__ float vp[S5_NW][16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = blockIdx.x * 16;
  const int rr = min(r0 + (lane & 15), o.R - 1);
  const int n = lane & 15;
  const int kq = o.F / S5_NW, kb = wave * kq;
  const uint16_t* xa = o.ha + (size_t)rr * o.F + kb + 8 * (lane >> 4);
  const uint16_t* xc = o.hc + (size_t)rr * o.F + kb + 8 * (lane >> 4);
  const uint16_t* wa = o.wa + (size_t)(n < o.NA ? n : 0) * o.F + kb + 8 * (lane >> 4);
  const uint16_t* wc = o.wc + kb + 8 * (lane >> 4);
  const u32x4 zero = {0u, 0u, 0u, 0u};
  f32x4 acc_a = {0.f, 0.f, 0.f, 0.f}, acc_c = {0.f, 0.f, 0.f, 0.f};
  // groups of 4 k-steps: every load of a group issued before its MFMAs
  constexpr int KG = 4;
  if (o.sample) {
    for (int k0 = 0; k0 < kq; k0 += 32 * KG) {
      u32x4 fc[KG], gc[KG], fa[KG], ga[KG];
#pragma unroll
      for (int j = 0; j < KG; ++j) {
        const int k = min(k0 + 32 * j, kq - 32);  // (kq is a multiple of 32; a repeat past the end is not used)
        fc[j] = *reinterpret_cast<const u32x4*>(xc + k);
        gc[j] = *reinterpret_cast<const u32x4*>(wc + k);
        fa[j] = *reinterpret_cast<const u32x4*>(xa + k);
        ga[j] = *reinterpret_cast<const u32x4*>(wa + k);
      }
#pragma unroll
      for (int j = 0; j < KG; ++j)
        if (k0 + 32 * j < kq) {
          acc_c = mfma_step(fc[j], n == 0 ? gc[j] : zero, acc_c);
          acc_a = mfma_step(fa[j], n < o.NA ? ga[j] : zero, acc_a);
        }
    }
  } else {
    for (int k0 = 0; k0 < kq; k0 += 32 * KG) {
      u32x4 fc[KG], gc[KG];
#pragma unroll
      for (int j = 0; j < KG; ++j) {
        const int k = min(k0 + 32 * j, kq - 32);
        fc[j] = *reinterpret_cast<const u32x4*>(xc + k);
        gc[j] = *reinterpret_cast<const u32x4*>(wc + k);
      }
#pragma unroll
      for (int j = 0; j < KG; ++j)
        if (k0 + 32 * j < kq) acc_c = mfma_step(fc[j], n == 0 ? gc[j] : zero, acc_c);
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    lp[wave][4 * (lane >> 4) + q][n] = acc_a[q];
    if (n == 0) vp[wave][4 * (lane >> 4) + q] = acc_c[q];
  }
  __syncthreads();
  // logits and Gumbel scores: thread t takes action t % 16 of row t / 16 (the
  // noise draws, the costly part, run on all lanes instead of one per row)
  __shared__ float lgs[16][17], scs[16][17];
  if (o.sample) {
    const int rl = tid >> 4, k = tid & 15, row = r0 + rl;
    if (k < o.NA && row < o.R) {
      float x = bf16_to_f32(o.ba[k]);
#pragma unroll
      for (int w = 0; w < S5_NW; ++w) x += lp[w][rl][k];
      lgs[rl][k] = x;
      const int e = row / o.A, ag = row - e * o.A;
      // noise of action k: draw k % 8 of Philox block (env, t, agent * 256 + k / 8, action tag), top 24 bits
      const Block4 b = draw_block(o.seed, (uint64_t)(o.env_base + e), o.t, (uint64_t)ag * 256u + (uint64_t)(k >> 3),
                                  TAG_ACTION);
      scs[rl][k] = action_score(x, gumbel24(block_u32(b, k & 7) >> 8), true);
    }
    __syncthreads();
  }
  const int row = r0 + tid;
  if (tid < 16 && row < o.R) {
    float v = bf16_to_f32(o.bc[0]);
#pragma unroll
    for (int w = 0; w < S5_NW; ++w) v += vp[w][tid];
    if (o.value) o.value[row] = v;
    if (o.sample) {
      int best = 0;
      float bs = -INFINITY;
      for (int k = 0; k < o.NA; ++k)
        if (scs[tid][k] > bs) {
          bs = scs[tid][k];
          best = k;
        }
      o.actions[row] = best;
      if (o.logits)
        for (int k = 0; k < o.NA; ++k) o.logits[(size_t)row * o.NA + k] = lgs[tid][k];
      if (o.logp) o.logp[row] = log_softmax_at(lgs[tid], o.NA, best);
    }
  }
}

// ------------------------------------------------------------- the loop ----

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Workspace of the allocation-free S5 rollout: one copy of this array per GPU
// the library runs on, held until the process ends.  Host code never uses the
// array's name as an address: s5_scratch_ptr() resolves the device copy of the
// current GPU once and the kernels receive that pointer.
static __device__ __align__(256) uint8_t s5_scratch[S5_SCRATCH_BYTES];

namespace {
constexpr int S5_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch[S5_MAX_DEVICES] = {};
}  // namespace

hipError_t s5_scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= S5_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(s5_scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

S5Workspace s5_workspace(const LbfParams& p, const S5Net& net) {
  S5Workspace w;
  const size_t R = (size_t)p.E * p.A;
  size_t off = 0;
  w.off_obs = off;
  off += align256(2 * R * p.D * 2);
  w.off_y = off;
  off += align256(R * net.H * 2);
  w.off_h = off;
  off += align256(4 * R * net.F * 2);
  w.off_act = off;
  off += align256(R * 4);
  w.off_wcat = off;
  off += align256((size_t)net.H * 2 * net.P * 4);
  w.bytes = off;
  return w;
}

hipError_t launch_s5_rollout(const LbfParams& p, const S5Net& net, int32_t* state, float* carry, uint64_t t0,
                             int n_steps, const TrajArgs& out, void* workspace, hipStream_t s) {
  const S5Workspace W = s5_workspace(p, net);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const int E = p.E, A = p.A, D = p.D, R = E * A, H = net.H, F = net.F, NA = net.NA;
  const size_t obs_stride = (size_t)R * D;
  uint16_t* obs_ws = reinterpret_cast<uint16_t*>(ws + W.off_obs);
  uint16_t* ybuf = reinterpret_cast<uint16_t*>(ws + W.off_y);
  uint16_t* hbuf = reinterpret_cast<uint16_t*>(ws + W.off_h);
  uint16_t* ha[2] = {hbuf, hbuf + (size_t)R * F};
  uint16_t* hc[2] = {hbuf + 2 * (size_t)R * F, hbuf + 3 * (size_t)R * F};
  int32_t* act_ws = reinterpret_cast<int32_t*>(ws + W.off_act);
  auto obs_slot = [&](int k) -> uint16_t* {
    if (k < n_steps && out.obs) return static_cast<uint16_t*>(out.obs) + (size_t)k * obs_stride;
    if (k == n_steps && out.obs_last) return static_cast<uint16_t*>(out.obs_last);
    return obs_ws + (size_t)(k & 1) * obs_stride;
  };
  const size_t front_lds = s5_front_lds_bytes(D, H, net.P);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)s5_front_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)MAX_LDS_BYTES);
    if (e != hipSuccess) return e;
    attr = true;
  }
  S5FrontArgs fa{};
  fa.state = state;
  fa.step_plane = 2 * A + 2 * p.F + 1;
  fa.E = E;
  fa.A = A;
  fa.R = R;
  fa.D = D;
  fa.H = H;
  fa.P = net.P;
  fa.carry = carry;
  fa.w_enc = static_cast<const uint16_t*>(net.w_enc);
  fa.b_enc = static_cast<const uint16_t*>(net.b_enc);
  fa.lbar = net.lbar;
  fa.bbar = net.bbar;
  fa.wcat = reinterpret_cast<const float*>(ws + W.off_wcat);
  fa.d = net.d;
  fa.y = ybuf;
  const dim3 front_grid((unsigned)((R + S5_RT - 1) / S5_RT));
  const int mtiles = (R + HG_BM - 1) / HG_BM;
  const dim3 head_grid((unsigned)(2 * mtiles * (F / HG_BN)));
  const dim3 out_grid((unsigned)((R + 15) / 16));

  // the policy on the observations in obs_slot(k): y, the three head layers, then the output kernel
  auto policy = [&](int k, int commit, const S5OutArgs& oa) -> hipError_t {
    fa.obs = obs_slot(k);
    fa.commit = commit;
    s5_front_kernel<<<front_grid, S5F_NT, front_lds, s>>>(fa);
    HeadGemmArgs g{};
    g.M = R;
    g.N = F;
    g.ldo = F;
    for (int l = 0; l < 3; ++l) {
      const int src = (l + 1) & 1, dst = l & 1;  // layer 0 -> buffer 0, 1 -> 1, 2 -> 0
      g.K = l == 0 ? H : F;
      g.lda = g.K;
      g.in[0] = l == 0 ? ybuf : ha[src];
      g.in[1] = l == 0 ? ybuf : hc[src];
      g.w[0] = static_cast<const uint16_t*>(net.actor_w[l]);
      g.w[1] = static_cast<const uint16_t*>(net.critic_w[l]);
      g.b[0] = static_cast<const uint16_t*>(net.actor_b[l]);
      g.b[1] = static_cast<const uint16_t*>(net.critic_b[l]);
      g.out[0] = ha[dst];
      g.out[1] = hc[dst];
      s5_head_gemm_kernel<<<head_grid, S5_NT, 0, s>>>(g);
    }
    s5_out_kernel<<<out_grid, S5_NT, 0, s>>>(oa);
    return hipGetLastError();
  };
  S5OutArgs oa{};
  oa.ha = ha[0];
  oa.hc = hc[0];
  oa.wa = static_cast<const uint16_t*>(net.actor_w[3]);
  oa.ba = static_cast<const uint16_t*>(net.actor_b[3]);
  oa.wc = static_cast<const uint16_t*>(net.critic_w[3]);
  oa.bc = static_cast<const uint16_t*>(net.critic_b[3]);
  oa.R = R;
  oa.F = F;
  oa.NA = NA;
  oa.A = A;
  oa.seed = p.seed;
  oa.env_base = p.env_base;

  s5_cat_kernel<<<dim3((unsigned)((H * 2 * net.P + 255) / 256)), 256, 0, s>>>(
      H, net.P, net.c, reinterpret_cast<float*>(ws + W.off_wcat));
  hipError_t err = launch_lbf_observe(p, state, obs_slot(0), s);
  if (err != hipSuccess) return err;
  for (int k = 0; k < n_steps; ++k) {
    const size_t ko = (size_t)k * R;
    oa.t = t0 + (uint64_t)k;
    oa.sample = 1;
    oa.actions = out.actions ? out.actions + ko : act_ws;
    oa.logits = out.logits ? out.logits + ko * NA : nullptr;
    oa.value = out.value ? out.value + ko : nullptr;
    oa.logp = out.logp ? out.logp + ko : nullptr;
    if ((err = policy(k, 1, oa)) != hipSuccess) return err;
    err = launch_lbf_step(p, state, t0 + (uint64_t)k, 1, oa.actions, obs_slot(k + 1), DT_BF16,
                          out.reward ? out.reward + (size_t)k * E : nullptr,
                          out.done ? out.done + (size_t)k * E : nullptr, nullptr, s);
    if (err != hipSuccess) return err;
  }
  if (out.value_last) {  // V(o_{t0+T}) from the state the next call would start from (not committed)
    oa.sample = 0;
    oa.actions = nullptr;
    oa.logits = nullptr;
    oa.logp = nullptr;
    oa.value = out.value_last;
    if ((err = policy(n_steps, 0, oa)) != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace rl
