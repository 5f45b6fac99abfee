// Two-player Hanabi kernels: init (deal), env-only steps with injected
// actions, and the fused rollout.
//
// Env lane e of wave 0 holds its game in registers (rl_hanabi.h) and, after
// every move, publishes what the observation needs to LDS.  The 26 fields of
// each player's 658-feature observation are computed by many threads at once
// (hn_field_bits) and ORed into bit vectors, which are expanded into 0 / 1
// values only where they are written: the trajectory rows (16 bytes per
// store, through a 256-entry expansion table) and, in the fused rollout, the
// mover's row of the layer-1 operand tile (the other player has no legal
// action), whose MLP is the streaming MFMA MLP of rl_mlp.h.  The env-only
// kernel keeps a move's rows in one flat bit array (row r's feature f at bit
// r * 658 + f), where an output vector of 8 bf16 is one byte.  When games
// end, the waves shuffle the new decks (one wave per deck) before the env
// lanes deal them.
#include "rl_hanabi.h"
#include "rl_internal.h"
#include "rl_sample.h"

namespace rl {

RL_STAMP_TABLE


struct HnTile {
  uint64_t bits[2][HN_OBS_WORDS];  // both players' observations as bit vectors (zero between steps)
  HnPub pub;                       // the game as of the last move
  uint32_t legal;                  // mover's 20-bit legal mask
};

// Assemble the observation bit vectors of every row of the tile: thread t
// computes field t / (2 TE) of row t % (2 TE) (consecutive lanes take the
// same field of different rows, so a wave runs few of the field branches) and
// ORs it into the row's words (LDS atomics; the words are zero beforehand).
// Needs the published games.  `rows`: the bit vectors row by row (row
// 2 el + me at rows + (2 el + me) * HN_OBS_WORDS), or null for the vectors
// inside the HnTiles.
template <class G, int TE, int NT>
__device__ __forceinline__ void hn_build_bits(HnTile* envs, int te_valid, int tid, uint64_t* rows = nullptr) {
  for (int t = tid; t < 2 * TE * G::NFIELDS; t += NT) {
    const int f = t / (2 * TE), row = t - f * (2 * TE), el = row >> 1, me = row & 1;
    if (el >= te_valid) continue;
    int off;
    const uint64_t v = hn_field_bits<G>(envs[el].pub, me, f, off);
    if (v) {
      unsigned long long* w =
          reinterpret_cast<unsigned long long*>(rows ? rows + row * HN_OBS_WORDS : envs[el].bits[me]);
      const int i = off >> 6, sh = off & 63;
      atomicOr(w + i, (unsigned long long)(v << sh));
      if (sh && (v >> (64 - sh))) atomicOr(w + i + 1, (unsigned long long)(v >> (64 - sh)));
    }
  }
}

// Paint rows 2*el + me (el < te_valid) of the observation tile from the
// assembled bit vectors, one row per wave at a time (lane l writes features
// l, l + 64, ...), and clear the vectors for the next step.
template <class G, typename T, int NW>
__device__ __forceinline__ void hn_paint(HnTile* envs, int te_valid, T* tile, int ld, int wave, int lane) {
  for (int r = wave; r < 2 * te_valid; r += NW) {
    uint64_t* wp = envs[r >> 1].bits[r & 1];
    uint64_t w[HN_OBS_WORDS];
#pragma unroll
    for (int i = 0; i < HN_OBS_WORDS; ++i) w[i] = wp[i];
    if (lane == 0)  // after every lane's read (one wave's LDS operations complete in order)
#pragma unroll
      for (int i = 0; i < HN_OBS_WORDS; ++i) wp[i] = 0;
    T* row = tile + (size_t)r * ld;
#pragma unroll
    for (int i = 0; i < HN_OBS_WORDS; ++i) {
      const int f = 64 * i + lane;
      if (f < G::OBS) row[f] = small_int_to<T>((uint32_t)(w[i] >> lane) & 1u);
    }
  }
}

// Write `nrows` observation rows of G::OBS features, held as bit vectors
// (row r at rows + r * HN_OBS_WORDS; the bits past G::OBS are 0), to
// consecutive global rows as 0 / 1 values, straight from the bits, by one
// wave.  Each lane expands VE features (16 bytes of output) at a time; a
// vector may run from the end of one row into the next.  All the LDS words a
// lane needs are read before any of its stores (three independent 32-bit
// reads per vector, no branches; batches of up to six vectors), so the wave
// waits on LDS once a batch.  Rows at a destination that is not 16-byte
// aligned, or a total that is not a whole number of vectors, go one 4-byte
// word at a time.
template <class G, typename OT, int MAXROWS>
__device__ __forceinline__ void hn_write_obs(const uint64_t* rows, int nrows, OT* __restrict__ dst, int lane,
                                             const u32x4* lut) {
  constexpr int VE = 16 / sizeof(OT), WE = 4 / sizeof(OT);  // features per 16-byte vector, per word
  const uint32_t one = sizeof(OT) == 2 ? 0x3f80u : 0x3f800000u;  // 1.0 in OT
  auto word = [&](uint32_t b, int q) -> uint32_t {  // output word q of a vector with feature bits b
    if constexpr (sizeof(OT) == 2)
      return (((b >> (2 * q)) & 1u) ? one : 0u) | (((b >> (2 * q + 1)) & 1u) ? one << 16 : 0u);
    else
      return ((b >> q) & 1u) ? one : 0u;
  };
  // features f0 .. f0+n-1 (n <= 8) of the flat rows from three 32-bit words:
  // the row's word holding feature f0 (lo) and the word after it (hi), and
  // the next row's first word (nx)
  const uint32_t* rw32 = reinterpret_cast<const uint32_t*>(rows);
  constexpr int W32 = 2 * HN_OBS_WORDS;  // 32-bit words per row
  auto load = [&](int f0, uint32_t& lo, uint32_t& hi, uint32_t& nx) {
    const int r = f0 / G::OBS, j = f0 - r * G::OBS, wi = j >> 5;
    const uint32_t* w = rw32 + r * W32;
    lo = w[wi];
    hi = w[min(wi + 1, W32 - 1)];
    nx = rw32[min(r + 1, nrows - 1) * W32];
  };
  auto bits = [&](int f0, int n, uint32_t lo, uint32_t hi, uint32_t nx) -> uint32_t {
    const int j = f0 % G::OBS, sh = j & 31, n0 = G::OBS - j;  // n0 features left in the row
    uint32_t x = lo >> sh;
    if ((j >> 5) + 1 < W32 && sh) x |= hi << (32 - sh);
    if (n0 < n) x |= nx << n0;
    return x & ((1u << n) - 1u);
  };
  const int total = nrows * G::OBS;
  if ((reinterpret_cast<uintptr_t>(dst) & 15) == 0 && total % VE == 0) {
    constexpr int IT = (MAXROWS * G::OBS / VE + 63) / 64, B = IT < 6 ? IT : 6;  // vectors per lane, per batch
    const int nv = total / VE;
    u32x4* g4 = reinterpret_cast<u32x4*>(dst);
#pragma unroll
    for (int i0 = 0; i0 < IT; i0 += B) {
      uint32_t lo[B], hi[B], nx[B];
#pragma unroll
      for (int it = 0; it < B; ++it) load(min(lane + 64 * (i0 + it), nv - 1) * VE, lo[it], hi[it], nx[it]);
      u32x4 val[B];  // the vectors' 16 bytes from the expansion table
#pragma unroll
      for (int it = 0; it < B; ++it) val[it] = lut[bits(min(lane + 64 * (i0 + it), nv - 1) * VE, VE, lo[it], hi[it], nx[it])];
#pragma unroll
      for (int it = 0; it < B; ++it) {
        const int v = lane + 64 * (i0 + it);
        if (i0 + it < IT && v < nv) g4[v] = val[it];
      }
    }
  } else {
    uint32_t* g = reinterpret_cast<uint32_t*>(dst);
    for (int v = lane; v < total / WE; v += 64) {
      uint32_t lo, hi, nx;
      load(v * WE, lo, hi, nx);
      g[v] = word(bits(v * WE, WE, lo, hi, nx), 0);
    }
  }
}

// The flat bit layout of a tile's observation rows: row r's feature f is bit
// r * G::OBS + f of one bit array (64-bit words), so that the 8 features of
// an output vector of 8 bf16 (or the 4 of a vector of 4 float32) are one
// byte (one nibble) of it when a wave's first row starts on a byte.  The
// expansion table maps such a byte (nibble) to the vector's 16 bytes of 0 / 1
// values.
template <typename OT>
struct HnExpand {
  static constexpr int N = sizeof(OT) == 2 ? 256 : 16;  // table entries
  __device__ static u32x4 entry(uint32_t i) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (sizeof(OT) == 2)
        w[q] = (((i >> (2 * q)) & 1u) ? 0x3f80u : 0u) | (((i >> (2 * q + 1)) & 1u) ? 0x3f800000u : 0u);
      else
        w[q] = ((i >> q) & 1u) ? 0x3f800000u : 0u;
    }
    return u32x4{w[0], w[1], w[2], w[3]};
  }
};

// Write a tile's `total` observation features, held in the flat layout
// (from bit 0 of `bytes`), to consecutive global elements from `dst` as
// 0 / 1 values, and clear the bytes written out.  Wave w of the NW taking
// part writes its share, a contiguous run of whole 16-byte vectors (or of
// 4-byte words when `dst` is not 16-byte aligned or `total` is not a whole
// number of vectors) that starts and ends on a byte of the bit array, so no
// two waves clear the same byte.  Per vector: one LDS byte (or nibble) read
// and one table read, in batches of up to eight whose reads are all issued
// before their stores.
template <class G, typename OT, int MAXF, int NW>
__device__ __forceinline__ void hn_write_flat(uint8_t* bytes, int total, OT* __restrict__ dst, int w, int lane,
                                              const u32x4* lut) {
  constexpr int VE = 16 / sizeof(OT), WE = 4 / sizeof(OT);  // features per 16-byte vector, per word
  static_assert(G::OBS % 2 == 0, "rows of whole 4-byte words");
  if ((reinterpret_cast<uintptr_t>(dst) & 15) == 0 && total % VE == 0) {
    constexpr int VB = 8 / VE;                                   // vectors per byte of bits
    constexpr int CMAX = ((MAXF / VE + NW - 1) / NW + VB - 1) / VB * VB;
    constexpr int IT = (CMAX + 63) / 64, B = IT < 8 ? IT : 8;  // vectors per lane, per batch
    const int nv = total / VE, c = ((nv + NW - 1) / NW + VB - 1) / VB * VB;
    const int v0 = min(nv, w * c), v1 = min(nv, v0 + c);
    u32x4* g4 = reinterpret_cast<u32x4*>(dst);
#pragma unroll
    for (int i0 = 0; i0 < IT; i0 += B) {
      uint32_t b[B];
#pragma unroll
      for (int it = 0; it < B; ++it) {
        const int v = max(0, min(v0 + lane + 64 * (i0 + it), v1 - 1));
        if constexpr (VE == 8)
          b[it] = bytes[v];
        else
          b[it] = ((uint32_t)bytes[v >> 1] >> (4 * (v & 1))) & 15u;
      }
      u32x4 val[B];
#pragma unroll
      for (int it = 0; it < B; ++it) val[it] = lut[b[it]];
#pragma unroll
      for (int it = 0; it < B; ++it) {
        const int v = v0 + lane + 64 * (i0 + it);
        if (i0 + it < IT && v < v1) g4[v] = val[it];
      }
    }
    wave_lds_sync();
    for (int j = v0 / VB + lane; j < (v1 + VB - 1) / VB; j += 64) bytes[j] = 0;
  } else {
    constexpr int WB = 8 / WE;  // words per byte of bits
    const int nw = total / WE, c = ((nw + NW - 1) / NW + WB - 1) / WB * WB;
    const int w0 = min(nw, w * c), w1 = min(nw, w0 + c);
    uint32_t* g = reinterpret_cast<uint32_t*>(dst);
    for (int x = w0 + lane; x < w1; x += 64) {
      const int f = x * WE;  // first feature of the word (its bits never straddle a byte)
      const uint32_t bb = ((uint32_t)bytes[f >> 3] >> (f & 7)) & ((1u << WE) - 1u);
      g[x] = lut[bb][0];  // (entry bb's first word holds features 0 .. WE-1 of bb)
    }
    wave_lds_sync();
    for (int j = w0 / WB + lane; j < (w1 + WB - 1) / WB; j += 64) bytes[j] = 0;
  }
}

// Paint the mover's observation of envs 0..te_valid-1 (bit-vector row
// 2 el + cur, rows as in hn_build_bits) into row el of the layer-1 operand
// tile as 0 / 1 values, 16 bytes (VE features) per store, by all NT threads.
// The tile's row stride holds whole vectors (the features past G::OBS come
// out 0, the K padding they fall in).
template <class G, typename T, int NT>
__device__ __forceinline__ void hn_paint_movers(const HnTile* __restrict__ envs, int te_valid,
                                                const uint64_t* __restrict__ rows, T* __restrict__ tile, int ld,
                                                int tid) {
  constexpr int VE = 16 / sizeof(T), NV = (G::OBS + VE - 1) / VE;  // vectors per row
  const uint32_t one = sizeof(T) == 2 ? 0x3f80u : 0x3f800000u;
  for (int i = tid; i < te_valid * NV; i += NT) {
    const int el = i / NV, v = i - el * NV, j = v * VE;
    const uint64_t* w = rows + (2 * el + envs[el].pub.cur) * HN_OBS_WORDS;
    const int wi = j >> 6, sh = j & 63;  // VE divides 64: a vector never straddles two words
    const uint32_t b = (uint32_t)(w[wi] >> sh) & ((1u << VE) - 1u);
    uint32_t q[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if constexpr (sizeof(T) == 2)
        q[c] = (((b >> (2 * c)) & 1u) ? one : 0u) | (((b >> (2 * c + 1)) & 1u) ? one << 16 : 0u);
      else
        q[c] = ((b >> c) & 1u) ? one : 0u;
    }
    *reinterpret_cast<u32x4*>(tile + (size_t)el * ld + j) = u32x4{q[0], q[1], q[2], q[3]};
  }
}

// Legal masks of both players of envs 0..te_valid-1 ([env][agent][20] bytes).
template <class G, int NT>
__device__ __forceinline__ void hn_write_legal(const HnTile* __restrict__ envs, int te_valid, uint8_t* __restrict__ g,
                                               int tid) {
  for (int i = tid; i < te_valid * 2 * G::NACT; i += NT) {
    const int el = i / (2 * G::NACT), rem = i - el * 2 * G::NACT, ag = rem / G::NACT, a = rem - ag * G::NACT;
    g[i] = (ag == envs[el].pub.cur) ? (uint8_t)((envs[el].legal >> a) & 1u) : (uint8_t)0;
  }
}

// What the workgroup reads of a game after each move: the packed game and
// the mover's legal actions.
template <class G>
__device__ __forceinline__ void hn_publish(const HnEnv& s, HnTile& t) {
  hn_pub(s, t.pub);
  t.legal = hn_legal<G>(s);
}

// Shuffles for the envs of the tile flagged in need[] (drawn at step t):
// wave w takes envs w, w + NW, ...
template <class G, int NW>
__device__ __forceinline__ void hn_shuffle_flagged(const HnParams& p, int e0, int te_valid, uint64_t t,
                                                   const uint32_t* need, uint32_t (*words)[HN_DECK_WORDS], int wave,
                                                   int lane) {
  for (int el = wave; el < te_valid; el += NW)
    if (need[el]) hn_wave_shuffle<G>(p.seed, (uint64_t)(p.env_base + e0 + el), t, lane, words[el]);
}

// need[TE] = whether any env lane (all in wave 0) has d != 0; read after a barrier.
__device__ __forceinline__ void hn_flag_any(uint32_t* need, int TE, uint32_t d, int wave, int lane) {
  if (wave == 0) {
    const bool any = __builtin_amdgcn_ballot_w64(d != 0) != 0;
    if (lane == 0) need[TE] = any ? 1u : 0u;
  }
}

// -------------------------------------------------------------- init ----

template <class G, typename OT, int TE>
__global__ __launch_bounds__(NTHREADS) void hn_init_kernel(HnParams p, int32_t* __restrict__ state,
                                                           OT* __restrict__ obs, uint8_t* __restrict__ legal) {
  constexpr int NW = NTHREADS / 64;
  __shared__ HnTile envs[TE];
  __shared__ uint32_t words[TE][HN_DECK_WORDS];
  __shared__ __align__(16) OT tile[2 * TE * G::OBS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0);
  zero_lds<NTHREADS>(envs, sizeof(envs), tid);  // the bit vectors start clear
  for (int el = wave; el < te_valid; el += NW)
    hn_wave_shuffle<G>(p.seed, (uint64_t)(p.env_base + e0 + el), 0, lane, words[el]);
  __syncthreads();
  if (tid < te_valid) {
    HnEnv s;
    hn_deal<G>(s, words[tid]);
    hn_store(state, p.E, e0 + tid, s);
    hn_publish<G>(s, envs[tid]);
  }
  __syncthreads();
  if (obs) {
    hn_build_bits<G, TE, NTHREADS>(envs, te_valid, tid);
    __syncthreads();
    hn_paint<G, OT, NW>(envs, te_valid, tile, G::OBS, wave, lane);
    __syncthreads();
    copy_tile(tile, obs + (size_t)e0 * 2 * G::OBS, 2 * te_valid * G::OBS, tid, NTHREADS);
  }
  if (legal) hn_write_legal<G, NTHREADS>(envs, te_valid, legal + (size_t)e0 * 2 * G::NACT, tid);
}

// ---------------------------------------------------------- env-only ----

// Legal masks ([env][agent][NACT] bytes, the mover's row only) of the n
// published games at `envs`, computed from the snapshots: one 4-byte word
// per lane (NACT is a multiple of 4, so a word never straddles an agent).
template <class G>
__device__ __forceinline__ void hn_write_legal_pub(const HnTile* __restrict__ envs, int n, uint8_t* __restrict__ g,
                                                   int lane) {
  static_assert(G::NACT % 4 == 0, "word-wise mask rows");
  constexpr int WPE = 2 * G::NACT / 4;  // words per env
  for (int w = lane; w < n * WPE; w += 64) {
    const int el = w / WPE, b0 = 4 * (w - el * WPE), ag = b0 / G::NACT, a0 = b0 - ag * G::NACT;
    const HnPub& v = envs[el].pub;
    const uint32_t m = ag == v.cur ? hn_legal<G>(v) >> a0 : 0u;
    reinterpret_cast<uint32_t*>(g)[w] = (m & 1u) | ((m & 2u) << 7) | ((m & 4u) << 14) | ((m & 8u) << 21);
  }
}

// Env-only steps, the workgroup run as a three-stage pipeline, one barrier
// per iteration.  In iteration i wave 0, which holds the TE games (one lane
// each), plays move i and publishes a snapshot of the games; waves 1..OW
// assemble the observation bit vectors of move i - 1 from the snapshot of the
// iteration before and write out those of move i - 2 (snapshots and bit
// vectors are double-buffered), so moves, field computation and stores
// overlap.  The field computations of a move are spread over the
// observation waves a pass of 64 (field, row) items at a time, field-major,
// so one pass takes few distinct fields (a wave runs the branch of every
// field its lanes hold); each observation wave writes out, then clears, its
// own rows.  A game that ends is re-dealt by the env wave itself: the whole
// wave shuffles the new decks one at a time (hn_wave_deck) and the owning
// lane picks its words up with readlane.  The actions are read straight
// from global memory one move ahead (the env wave stores only rewards and
// done flags, so those loads wait on little).
template <class G, typename OT, int TE, int OW>
__global__ __launch_bounds__(64 * (OW + 1)) __attribute__((amdgpu_waves_per_eu(sizeof(OT) == 2 ? 4 : 3))) void hn_env_kernel(HnParams p, int32_t* __restrict__ state, uint64_t t0,
                                                                int n_steps, const int32_t* __restrict__ actions,
                                                                OT* __restrict__ obs, float* __restrict__ reward,
                                                                uint8_t* __restrict__ done, uint8_t* __restrict__ legal) {
  static_assert(TE <= 64, "one env wave");
  constexpr int RB = 2 * TE;                                     // rows per workgroup
  constexpr int NPASS = (RB * G::NFIELDS + 63) / 64;            // field passes per move
  constexpr int LPW = (TE + OW - 1) / OW;                        // envs whose legal masks a wave writes
  constexpr int FW = (RB * G::OBS + 63) / 64;                    // words of a move's flat bit array
  __shared__ HnTile snap[2][TE];
  __shared__ __align__(16) uint64_t rows[2][FW];                 // move k's rows, flat, in rows[k % 2]
  __shared__ u32x4 lut[HnExpand<OT>::N];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, ow = wave - 1;
  const int e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0), E = p.E;
  const bool envlane = wave == 0 && lane < te_valid;
  const int e = e0 + lane;
  HnEnv s;
  int act0 = 0, act1 = 0;  // both agents' actions of the move about to be played
  if (envlane) {
    hn_load(state, E, e, s);
    if (n_steps > 0) {
      act0 = actions[(size_t)e * 2];
      act1 = actions[(size_t)e * 2 + 1];
    }
  }
  zero_lds<64 * (OW + 1)>(rows, sizeof(rows), tid);  // the bit vectors start clear
  for (int j = tid; j < HnExpand<OT>::N; j += 64 * (OW + 1)) lut[j] = HnExpand<OT>::entry((uint32_t)j);
  // the env wave's serial chain sets the pace: it goes first when the waves
  // sharing its SIMD are ready to issue too
  if (wave == 0) __builtin_amdgcn_s_setprio(3);
  RL_STAMP_BEGIN
  for (int i = 0; i < n_steps + 2; ++i) {
    if (wave == 0) {
      if (i < n_steps) {  // move i
        const uint64_t t = t0 + (uint64_t)i;
        uint32_t d = 0;
        if (envlane) {
          float r;
          hn_transition<G>(p, s, s.cur ? act1 : act0, r, d);
          if (reward) reward[(size_t)i * E + e] = r;
          if (done) done[(size_t)i * E + e] = (uint8_t)d;
          if (i + 1 < n_steps) {
            act0 = actions[((size_t)(i + 1) * E + e) * 2];
            act1 = actions[((size_t)(i + 1) * E + e) * 2 + 1];
          }
        }
        RL_STAMP(0)
        // an ended game restarts with the deal drawn at t + 1
        uint64_t ended = __builtin_amdgcn_ballot_w64(d != 0);
        while (ended) {
          const int el = __builtin_ctzll(ended);
          ended &= ended - 1;
          const uint32_t v = hn_wave_deck<G>(p.seed, (uint64_t)(p.env_base + e0 + el), t + 1, lane);
#pragma unroll
          for (int w = 0; w < HN_DECK_WORDS; ++w) {
            const uint32_t x = (uint32_t)__builtin_amdgcn_readlane((int)v, 4 * w);
            s.deck[w] = lane == el ? x : s.deck[w];
          }
        }
        RL_STAMP(1)
        if (d) hn_deal_deck<G>(s);
        if (envlane) hn_pub(s, snap[i & 1][lane].pub);
        RL_STAMP(2)
      }
    } else {
      if (i >= 1 && i <= n_steps) {  // the fields of move i - 1
        const int k = i - 1;
        const HnTile* sn = snap[k & 1];
        if (obs) {
          uint64_t* rw = rows[k & 1];
          for (int q = ow; q < NPASS; q += OW) {
            const int j = q * 64 + lane, f = j / RB, r = j - f * RB;
            if (f >= G::NFIELDS || (r >> 1) >= te_valid) continue;
            int off;
            const uint64_t v = hn_field_bits<G>(sn[r >> 1].pub, r & 1, f, off);
            if (v) {
              unsigned long long* w = reinterpret_cast<unsigned long long*>(rw);
              const int b = r * G::OBS + off, wi = b >> 6, sh = b & 63;
              atomicOr(w + wi, (unsigned long long)(v << sh));
              if (sh && (v >> (64 - sh))) atomicOr(w + wi + 1, (unsigned long long)(v >> (64 - sh)));
            }
          }
        }
        RL_STAMP(4)
        if (legal) {
          const int l0 = ow * LPW, nl = max(0, min(LPW, te_valid - l0));
          if (nl > 0) hn_write_legal_pub<G>(sn + l0, nl, legal + ((size_t)k * E + e0 + l0) * 2 * G::NACT, lane);
        }
      }
      RL_STAMP(5)
      if (obs && i >= 2) {  // write out and clear this wave's share of the rows of move i - 2
        const int k = i - 2;
        hn_write_flat<G, OT, RB * G::OBS, OW>(reinterpret_cast<uint8_t*>(rows[k & 1]), 2 * te_valid * G::OBS,
                                              obs + ((size_t)k * E + e0) * 2 * G::OBS, ow, lane, lut);
      }
    }
    RL_STAMP(6)
    __syncthreads();  // snapshot i and the fields of move i - 1 are in; the rows of move i - 2 are out
    RL_STAMP(7)
  }
  RL_STAMP_END(wave == 0 ? 0 : 1)
  if (envlane) hn_store(state, E, e, s);
}

// ----------------------------------------------------- fused rollout ----

constexpr int HN_RUN_TE = 16;   // envs (and mover rows) per workgroup
constexpr int HN_RUN_NT = 512;  // 8 waves: the MLP's weight-streaming chains of a workgroup spread over twice the waves

struct HnRunLayout {
  int ldx, ld1, ld2;
  size_t off_x, off_h1, off_h2, off_lg, off_sc, off_env, off_words, off_need, off_bits, off_lut, off_nz, total;
};

__host__ __device__ inline HnRunLayout hn_run_layout(int H1, int H2, int dt, int obs) {
  HnRunLayout L;
  const size_t es = dt == DT_F32 ? 4 : 2;
  L.ldx = dt == DT_F32 ? lds_ld<DT_F32>(obs) : lds_ld<DT_BF16>(obs);
  L.ld1 = dt == DT_F32 ? lds_ld<DT_F32>(H1) : lds_ld<DT_BF16>(H1);
  L.ld2 = dt == DT_F32 ? lds_ld<DT_F32>(H2) : lds_ld<DT_BF16>(H2);
  size_t o = 0;
  L.off_x = o;     o += (size_t)HN_RUN_TE * L.ldx * es;
  L.off_h1 = o;    o += (size_t)HN_RUN_TE * L.ld1 * es;
  L.off_h2 = o;    o += (size_t)HN_RUN_TE * L.ld2 * es;
  L.off_lg = o;    o += (size_t)HN_RUN_TE * MAX_NA * 4;
  L.off_sc = o;    o += (size_t)HN_RUN_TE * MAX_NA * 4;
  o = (o + 15) & ~(size_t)15;
  L.off_env = o;   o += (size_t)HN_RUN_TE * sizeof(HnTile);
  L.off_words = o; o += (size_t)HN_RUN_TE * HN_DECK_WORDS * 4;
  L.off_need = o;  o += (size_t)(HN_RUN_TE + 1) * 4;
  o = (o + 15) & ~(size_t)15;
  L.off_bits = o;  o += (size_t)2 * HN_RUN_TE * HN_OBS_WORDS * 8;
  L.off_lut = o;   o += (size_t)HnExpand<uint16_t>::N * 16;  // (the larger expansion table)
  L.off_nz = o;    o += (size_t)HN_RUN_TE * (MAX_NA + 2) * 4;  // next step's noise, its agent, the mover
  L.total = o;
  return L;
}

size_t hn_run_lds_bytes(const PolicyArgs& pol) { return hn_run_layout(pol.H1, pol.H2, pol.dt, pol.D).total; }

template <class G, int DT, bool PK>
__global__ __launch_bounds__(HN_RUN_NT) void hn_run_kernel(HnParams p, PolicyArgs pol, int32_t* __restrict__ state,
                                                          uint64_t t0, int n_steps, TrajArgs out) {
  using T = typename DType<DT>::T;
  constexpr int TE = HN_RUN_TE, NA = G::NACT, NW = HN_RUN_NT / 64;
  constexpr int LDX = lds_ld<DT>(G::OBS);
  extern __shared__ __align__(16) uint8_t smem[];
  const HnRunLayout L = hn_run_layout(pol.H1, pol.H2, DT, G::OBS);
  T* xs = reinterpret_cast<T*>(smem + L.off_x);
  T* h1 = reinterpret_cast<T*>(smem + L.off_h1);
  T* h2 = reinterpret_cast<T*>(smem + L.off_h2);
  float* lg = reinterpret_cast<float*>(smem + L.off_lg);
  float* sc = reinterpret_cast<float*>(smem + L.off_sc);
  HnTile* envs = reinterpret_cast<HnTile*>(smem + L.off_env);
  uint32_t(*words)[HN_DECK_WORDS] = reinterpret_cast<uint32_t(*)[HN_DECK_WORDS]>(smem + L.off_words);
  uint32_t* need = reinterpret_cast<uint32_t*>(smem + L.off_need);
  uint64_t* bits = reinterpret_cast<uint64_t*>(smem + L.off_bits);  // the observation bit vectors, row by row
  u32x4* lut = reinterpret_cast<u32x4*>(smem + L.off_lut);
  float* nz = reinterpret_cast<float*>(smem + L.off_nz);  // [env][action]: the next step's noise
  int* nz_ag = reinterpret_cast<int*>(nz + TE * MAX_NA);  // [env]: the agent nz was drawn for
  int* mover = nz_ag + TE;                                // [env]: this step's mover

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = blockIdx.x * TE, te_valid = min(TE, p.E - e0), E = p.E;
  const T* W1 = static_cast<const T*>(pol.W[0]);
  const T* W2 = static_cast<const T*>(pol.W[1]);
  const T* W3 = static_cast<const T*>(pol.W[2]);
  const T* b1 = static_cast<const T*>(pol.b[0]);
  const T* b2 = static_cast<const T*>(pol.b[1]);
  const T* b3 = static_cast<const T*>(pol.b[2]);
  const T* Wp1 = static_cast<const T*>(pol.Wp[0]);
  const T* Wp2 = static_cast<const T*>(pol.Wp[1]);
  const T* Wp3 = static_cast<const T*>(pol.Wp[2]);
  zero_lds<HN_RUN_NT>(smem, L.off_lut, tid);  // (all but the expansion table, which is written here)
  for (int j = tid; j < HnExpand<T>::N; j += HN_RUN_NT) lut[j] = HnExpand<T>::entry((uint32_t)j);
  __syncthreads();
  const bool envlane = tid < te_valid;
  const int e = e0 + tid;
  HnEnv s;
  if (envlane) {
    hn_load(state, E, e, s);
    hn_publish<G>(s, envs[tid]);
  }
  // the noise of step kn for agent ag(el) of every game, threads i0, i0 +
  // stride, ...  The next step's mover is known only after the move; the
  // turn passes to the other player unless the game ends, so that player's
  // noise is drawn ahead, and a step whose mover differs (a new game)
  // draws its own in the score loop.
  auto draw_noise = [&](int kn, int i0, int stride, auto ag_of) {
    for (int idx = i0; idx < te_valid * NA; idx += stride) {
      const int el = idx / NA, a = idx - el * NA, ag = ag_of(el);
      nz[el * MAX_NA + a] = action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t0 + (uint64_t)kn, ag, a);
      if (a == 0) nz_ag[el] = ag;
    }
  };
  __syncthreads();  // the games are published
  if (n_steps > 0) draw_noise(0, tid, HN_RUN_NT, [&](int el) { return envs[el].pub.cur; });
  RL_STAMP_BEGIN
  for (int k = 0; k < n_steps; ++k) {
    const uint64_t t = t0 + (uint64_t)k;
    __syncthreads();  // the previous move's games are published
    RL_STAMP(0)
    hn_build_bits<G, TE, HN_RUN_NT>(envs, te_valid, tid, bits);
    __syncthreads();
    RL_STAMP(1)
    hn_paint_movers<G, T, HN_RUN_NT>(envs, te_valid, bits, xs, LDX, tid);  // row el: the mover of env el
    __syncthreads();
    RL_STAMP(2)
    mlp_input_layer_const<DT, G::OBS, PK>(xs, LDX, nullptr, TE, W1, b1, pol.H1, h1, L.ld1, wave, NW, lane, Wp1);
    __syncthreads();
    RL_STAMP(3)
    mlp_hidden<DT, PK>(h1, L.ld1, TE, pol.H1, W2, b2, pol.H2, h2, L.ld2, wave, NW, lane, Wp2);
    __syncthreads();
    RL_STAMP(4)
    mlp_logits<DT, PK>(h2, L.ld2, TE, pol.H2, W3, b3, NA, lg, MAX_NA, wave, NW, lane, Wp3);
    __syncthreads();
    RL_STAMP(5)
    for (int idx = tid; idx < te_valid * NA; idx += HN_RUN_NT) {
      const int el = idx / NA, a = idx - el * NA;
      const int cur = envs[el].pub.cur;
      const bool ok = (envs[el].legal >> a) & 1u;
      const float g = nz_ag[el] == cur ? nz[el * MAX_NA + a]
                                       : action_noise(p.seed, (uint64_t)(p.env_base + e0 + el), t, cur, a);
      sc[el * MAX_NA + a] = action_score(lg[el * MAX_NA + a], g, ok);
      if (a == 0) mover[el] = cur;
      if (out.logits) {
        float* lo = out.logits + ((size_t)k * E + e0 + el) * 2 * NA;
        lo[cur * NA + a] = ok ? lg[el * MAX_NA + a] : -INFINITY;
        lo[(1 - cur) * NA + a] = -INFINITY;
      }
    }
    RL_STAMP(6)
    // o_t to the trajectory straight from the bit vectors, each wave its own
    // rows, which it then clears for the next step; issued after the step's
    // weight loads (a wave's loads wait for its earlier stores: one in-order
    // counter).
    {
      constexpr int RPW = 2 * TE / NW;  // rows per wave
      const int r0 = wave * RPW, nr = max(0, min(RPW, 2 * te_valid - r0));
      uint64_t* rw = bits + r0 * HN_OBS_WORDS;
      if (nr > 0) {
        if (out.obs)
          hn_write_obs<G, T, RPW>(rw, nr, static_cast<T*>(out.obs) + (((size_t)k * E + e0) * 2 + r0) * G::OBS, lane,
                                  lut);
        wave_lds_sync();
        for (int j = lane; j < nr * HN_OBS_WORDS; j += 64) rw[j] = 0;
      }
    }
    __syncthreads();
    RL_STAMP(7)
    uint32_t d = 0;
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
      hn_transition<G>(p, s, best, r, d);
      need[tid] = d;
      if (!d) hn_publish<G>(s, envs[tid]);
      if (out.reward) out.reward[(size_t)k * E + e] = r;
      if (out.done) out.done[(size_t)k * E + e] = (uint8_t)d;
    } else if (wave > 0 && k + 1 < n_steps) {
      // the other waves draw the next step's noise (for the player whose turn
      // it will be if the game goes on) while the env lanes move
      draw_noise(k + 1, tid - 64, HN_RUN_NT - 64, [&](int el) { return 1 - mover[el]; });
    }
    hn_flag_any(need, TE, d, wave, lane);
    __syncthreads();
    RL_STAMP(8)
    if (need[TE]) {
      hn_shuffle_flagged<G, NW>(p, e0, te_valid, t + 1, need, words, wave, lane);
      __syncthreads();
      if (d) {
        hn_deal<G>(s, words[tid]);
        hn_publish<G>(s, envs[tid]);
      }
    }
    RL_STAMP(9)
  }
  RL_STAMP_END(wave)
  __syncthreads();
  if (out.obs_last) {
    hn_build_bits<G, TE, HN_RUN_NT>(envs, te_valid, tid, bits);
    __syncthreads();
    constexpr int RPW = 2 * TE / NW;
    const int r0 = wave * RPW, nr = max(0, min(RPW, 2 * te_valid - r0));
    if (nr > 0)
      hn_write_obs<G, T, RPW>(bits + r0 * HN_OBS_WORDS, nr, static_cast<T*>(out.obs_last) + ((size_t)e0 * 2 + r0) * G::OBS,
                              lane, lut);
  }
  if (envlane) hn_store(state, E, e, s);
}

// ---------------------------------------------------------- launchers ----

constexpr int HN_ENV_TE = 8;  // envs per workgroup of the init and env-only kernels

static dim3 hn_tiles(int E, int te) { return dim3((unsigned)((E + te - 1) / te)); }

template <class G>
static hipError_t launch_hn_init_g(const HnParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal,
                                   hipStream_t s) {
  if (obs_dt == DT_F32)
    hn_init_kernel<G, float, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(
        p, state, static_cast<float*>(obs), legal);
  else
    hn_init_kernel<G, uint16_t, HN_ENV_TE><<<hn_tiles(p.E, HN_ENV_TE), NTHREADS, 0, s>>>(
        p, state, static_cast<uint16_t*>(obs), legal);
  return hipGetLastError();
}

constexpr int HN_STEP_TE = 4;  // envs per workgroup of the env-only kernel
// its observation waves: three for bf16 (four waves of at most 128 VGPRs, four
// workgroups per CU), two for float32 (whose kernel needs more registers)
constexpr int HN_STEP_OW_BF16 = 3, HN_STEP_OW_F32 = 2;

template <class G>
static hipError_t launch_hn_step_g(const HnParams& p, int32_t* state, uint64_t t0, int n_steps,
                                   const int32_t* actions, void* obs, int obs_dt, float* reward, uint8_t* done,
                                   uint8_t* legal, hipStream_t s) {
  constexpr int TE = HN_STEP_TE, OWF = HN_STEP_OW_F32, OWB = HN_STEP_OW_BF16;
  if (obs_dt == DT_F32)
    hn_env_kernel<G, float, TE, OWF><<<hn_tiles(p.E, TE), 64 * (OWF + 1), 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<float*>(obs), reward, done, legal);
  else
    hn_env_kernel<G, uint16_t, TE, OWB><<<hn_tiles(p.E, TE), 64 * (OWB + 1), 0, s>>>(
        p, state, t0, n_steps, actions, static_cast<uint16_t*>(obs), reward, done, legal);
  return hipGetLastError();
}

template <class G>
static hipError_t launch_hn_run_g(const HnParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0,
                                  int n_steps, const TrajArgs& out, hipStream_t s) {
  const size_t lds = hn_run_lds_bytes(pol);
  const bool pk = pol.dt == DT_BF16 && pol.Wp[0] != nullptr;  // fragment-major weights
  const void* fn = pol.dt == DT_F32 ? (const void*)hn_run_kernel<G, DT_F32, false>
                   : pk             ? (const void*)hn_run_kernel<G, DT_BF16, true>
                                    : (const void*)hn_run_kernel<G, DT_BF16, false>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  if (pol.dt == DT_F32)
    hn_run_kernel<G, DT_F32, false><<<hn_tiles(p.E, HN_RUN_TE), HN_RUN_NT, lds, s>>>(p, pol, state, t0, n_steps, out);
  else if (pk)
    hn_run_kernel<G, DT_BF16, true><<<hn_tiles(p.E, HN_RUN_TE), HN_RUN_NT, lds, s>>>(p, pol, state, t0, n_steps, out);
  else
    hn_run_kernel<G, DT_BF16, false><<<hn_tiles(p.E, HN_RUN_TE), HN_RUN_NT, lds, s>>>(p, pol, state, t0, n_steps, out);
  return hipGetLastError();
}

hipError_t launch_hn_init(const HnParams& p, int32_t* state, void* obs, int obs_dt, uint8_t* legal, hipStream_t s) {
  return p.mini ? launch_hn_init_g<HnMini>(p, state, obs, obs_dt, legal, s)
                : launch_hn_init_g<HnStd>(p, state, obs, obs_dt, legal, s);
}

hipError_t launch_hn_step(const HnParams& p, int32_t* state, uint64_t t0, int n_steps, const int32_t* actions,
                          void* obs, int obs_dt, float* reward, uint8_t* done, uint8_t* legal, hipStream_t s) {
  return p.mini ? launch_hn_step_g<HnMini>(p, state, t0, n_steps, actions, obs, obs_dt, reward, done, legal, s)
                : launch_hn_step_g<HnStd>(p, state, t0, n_steps, actions, obs, obs_dt, reward, done, legal, s);
}

hipError_t launch_hn_run(const HnParams& p, const PolicyArgs& pol, int32_t* state, uint64_t t0, int n_steps,
                         const TrajArgs& out, hipStream_t s) {
  return p.mini ? launch_hn_run_g<HnMini>(p, pol, state, t0, n_steps, out, s)
                : launch_hn_run_g<HnStd>(p, pol, state, t0, n_steps, out, s);
}

}  // namespace rl

RL_STAMP_EXPORT(hn)
