// Level-Based Foraging device logic: reset (rho) and transition (P, r) of one
// env held in the registers of one lane.
//
// Rules (the environment of Section 4 / environment table, run as the
// Dec-POMDP step of Section 3), with the readings the paper leaves open:
//   reset   A agent levels, F food levels capped by the agents' level sum, F
//           food cells on interior cells, A agent cells on free cells, each a
//           uniform index among the free candidates in row-major order;
//   moves   legal iff the target is on the grid and holds neither uneaten
//           food nor an agent before the step; legal movers sharing a
//           target all stay;
//   loads   a food is eaten iff the 4-adjacent loaders' levels sum to at
//           least its level (a loader counts for every adjacent food);
//   reward  float32(eaten levels) / float32(total food levels of the episode);
//   done    bit 0 all food eaten, bit 1 step limit reached.
// Every loop runs over compile-time bounds (MAXA, MAXF) with runtime guards,
// so all per-env arrays stay in registers.
#pragma once
#include "rl_philox.h"

namespace rl {

constexpr int LBF_MAXA = 4;
constexpr int LBF_MAXF = 8;
constexpr int LBF_MAXCELLS = 256;
constexpr int LBF_NACT = 6;

struct LbfParams {
  int E, A, F, H, W, HW, D, Lmax, Fmax, max_steps;
  int const_levels;  // 1: agents at Lmax and foods at Fmax (level draws made and ignored)
  uint32_t wmagic;  // ceil(2^32 / W): x / W == umulhi(x, wmagic) for 0 <= x < 2^16
  int64_t env_base;
  uint64_t seed;
};

__device__ __forceinline__ int lbf_row(const LbfParams& p, int cell) {
  return (int)__umulhi((uint32_t)cell, p.wmagic);
}

// Grid row of a cell when the width WC is known at compile time (0 = use p).
template <int WC>
__device__ __forceinline__ int lbf_row_ct(const LbfParams& p, int cell) {
  if constexpr (WC > 0)
    return (int)((uint32_t)cell / (uint32_t)WC);
  else
    return lbf_row(p, cell);
}

struct LbfEnv {
  int acell[LBF_MAXA];
  int alevel[LBF_MAXA];
  int fcell[LBF_MAXF];
  int flevel[LBF_MAXF];
  uint32_t eaten;  // bit j = food j eaten
  int steps;       // steps taken in the episode
  int den;         // sum of the episode's food levels
};

// Number of int32 state planes: A cells, A levels, F cells, F levels, eaten, steps, den.
__host__ __device__ inline int lbf_planes(int A, int F) { return 2 * A + 2 * F + 3; }

// AC / FC: agent and food counts when known at compile time (0 = read from p).
template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_load(const int32_t* __restrict__ st, const LbfParams& p, int e,
                                         LbfEnv& s) {
  const int E = p.E, A = AC ? AC : p.A, F = FC ? FC : p.F;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A) {
      s.acell[i] = st[(size_t)i * E + e];
      s.alevel[i] = st[(size_t)(A + i) * E + e];
    }
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F) {
      s.fcell[j] = st[(size_t)(2 * A + j) * E + e];
      s.flevel[j] = st[(size_t)(2 * A + F + j) * E + e];
    }
  s.eaten = (uint32_t)st[(size_t)(2 * A + 2 * F) * E + e];
  s.steps = st[(size_t)(2 * A + 2 * F + 1) * E + e];
  s.den = st[(size_t)(2 * A + 2 * F + 2) * E + e];
}

template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_store(int32_t* __restrict__ st, const LbfParams& p, int e,
                                          const LbfEnv& s) {
  const int E = p.E, A = AC ? AC : p.A, F = FC ? FC : p.F;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A) {
      st[(size_t)i * E + e] = s.acell[i];
      st[(size_t)(A + i) * E + e] = s.alevel[i];
    }
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F) {
      st[(size_t)(2 * A + j) * E + e] = s.fcell[j];
      st[(size_t)(2 * A + F + j) * E + e] = s.flevel[j];
    }
  st[(size_t)(2 * A + 2 * F) * E + e] = (int32_t)s.eaten;
  st[(size_t)(2 * A + 2 * F + 1) * E + e] = s.steps;
  st[(size_t)(2 * A + 2 * F + 2) * E + e] = s.den;
}

// The idx-th (0-based) free candidate among 0, 1, 2, ..., where count_le(x)
// is the number of occupied candidates <= x: the least fixed point of
// x = idx + count_le(x), reached by iterating from x = idx (at most n_occ + 1
// iterations, count_le being monotone).
template <typename CountLE>
__device__ __forceinline__ int lbf_kth_free(int idx, int n_occ, CountLE count_le) {
  int x = idx;
  for (int it = 0; it <= n_occ; ++it) {
    const int nx = idx + count_le(x);
    if (nx == x) break;
    x = nx;
  }
  return x;
}

// Number of 32-bit reset draws (and Philox blocks) an episode of this config uses.
__host__ __device__ inline int lbf_reset_draws(int A, int F) { return 2 * A + 2 * F; }
constexpr int LBF_MAX_DRAWS = 2 * LBF_MAXA + 2 * LBF_MAXF;  // 24 = 3 blocks

// Build a fresh episode from its reset draws dw[0..2A+2F-1] (draw k = 32-bit
// word k of the reset stream of (env, t)).
template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_reset_from_draws(const LbfParams& p, const uint32_t (&dw)[LBF_MAX_DRAWS],
                                                     LbfEnv& s) {
  const int A = AC ? AC : p.A, F = FC ? FC : p.F, W = p.W;
  // draw(k) selects with compares so that a runtime k never turns the
  // array into scratch memory.
  auto draw = [&](int k) -> uint32_t {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < LBF_MAX_DRAWS; ++q) v = (q == k) ? dw[q] : v;
    return v;
  };
  int lsum = 0;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A) {
      s.alevel[i] = p.const_levels ? p.Lmax : 1 + (int)range_map(draw(i), (uint32_t)p.Lmax);
      lsum += s.alevel[i];
    }
  const int fcap = p.Fmax < lsum ? p.Fmax : lsum;
  int den = 0;
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F) {
      s.flevel[j] = p.const_levels ? p.Fmax : 1 + (int)range_map(draw(A + j), (uint32_t)fcap);
      den += s.flevel[j];
    }
  // Food on interior cells, indexed row-major over the (H-2) x (W-2) interior.
  const int IW = W - 2;
  const int NI = (p.H - 2) * IW;
  int fint[LBF_MAXF];
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F) {
      const int idx = (int)range_map(draw(A + F + j), (uint32_t)(NI - j));
      fint[j] = lbf_kth_free(idx, j, [&](int x) {
        int c = 0;
#pragma unroll
        for (int q = 0; q < LBF_MAXF; ++q) c += (q < j && fint[q] <= x) ? 1 : 0;
        return c;
      });
      const int fr = fint[j] / IW;
      s.fcell[j] = (1 + fr) * W + 1 + (fint[j] - fr * IW);
    }
  // Agents on cells free of food and of earlier agents.
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A) {
      const int idx = (int)range_map(draw(A + 2 * F + i), (uint32_t)(p.HW - F - i));
      s.acell[i] = lbf_kth_free(idx, F + i, [&](int x) {
        int c = 0;
#pragma unroll
        for (int q = 0; q < LBF_MAXF; ++q) c += (q < F && s.fcell[q] <= x) ? 1 : 0;
#pragma unroll
        for (int r = 0; r < LBF_MAXA; ++r) c += (r < i && s.acell[r] <= x) ? 1 : 0;
        return c;
      });
    }
  s.eaten = 0;
  s.steps = 0;
  s.den = den;
}

// Draw a fresh episode for global env id `env` from the reset stream at step t.
template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_reset(const LbfParams& p, uint64_t env, uint64_t t, LbfEnv& s) {
  const int nd = lbf_reset_draws(AC ? AC : p.A, FC ? FC : p.F);
  const Block4 b0 = draw_block(p.seed, env, t, 0, TAG_RESET);
  Block4 b1 = b0, b2 = b0;
  if (nd > 8) b1 = draw_block(p.seed, env, t, 1, TAG_RESET);
  if (nd > 16) b2 = draw_block(p.seed, env, t, 2, TAG_RESET);
  uint32_t dw[LBF_MAX_DRAWS];
#pragma unroll
  for (int q = 0; q < LBF_MAX_DRAWS; ++q) dw[q] = block_u32(q < 8 ? b0 : (q < 16 ? b1 : b2), q & 7);
  lbf_reset_from_draws<AC, FC>(p, dw, s);
}

template <int AC, int FC>
__device__ __forceinline__ void lbf_start_cells(const LbfParams& p, uint64_t env, uint64_t t, const LbfEnv& s,
                                                int (&start)[LBF_MAXA]) {
  LbfEnv s0{};
  lbf_reset<AC, FC>(p, env, t - (uint64_t)s.steps, s0);
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) start[i] = s0.acell[i];
}

// Heuristic teammates (the paper's Greedy and Sequential LBF agents, read as
// deterministic policies).  Kinds: 0-2 Greedy closest to self / to the
// teammate (agent (i + 1) mod A) / to both (sum of distances); 3-4 Greedy
// lowest / highest food level (then closest to self); 5-8 Sequential in
// row-major, reverse row-major, column-major, reverse column-major order of
// the food cells; 9-10 Sequential nearest / farthest first from the agent's
// cell at the start of its episode (`start`).  The target is the uneaten food
// of least key (the lowest index on ties).  Next to it the agent loads;
// otherwise it steps along the axis with more distance left (rows on ties),
// or along the other axis when that cell holds an uneaten food or another
// agent and the other axis also closes in.
constexpr int LBF_NHEUR = 11;

// Agent cells at the start of the episode a state is in: the episode began at
// step t - steps, and its first state is the reset drawn for that step.
template <int AC = 0, int FC = 0>
__device__ __forceinline__ void lbf_start_cells(const LbfParams& p, uint64_t env, uint64_t t, const LbfEnv& s,
                                                int (&start)[LBF_MAXA]);

__device__ __forceinline__ int lbf_heuristic_action(const LbfParams& p, const LbfEnv& s, int agent, int kind,
                                                    int start) {
  const int A = p.A, F = p.F, W = p.W;
  const int me = s.acell[agent], mate = s.acell[agent + 1 < A ? agent + 1 : 0];
  const int mr = lbf_row(p, me), mc = me - mr * W;
  const int tr_ = lbf_row(p, mate), tc_ = mate - tr_ * W;
  const int sr = lbf_row(p, start), sc = start - sr * W;
  int best = -1, b1 = 0, b2 = 0, bcell = 0;
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j) {
    if (j < F && !((s.eaten >> j) & 1u)) {
      const int fcell = s.fcell[j];
      const int fr = lbf_row(p, fcell), fc = fcell - fr * W;
      const int dme = abs(fr - mr) + abs(fc - mc), dmate = abs(fr - tr_) + abs(fc - tc_);
      int k1, k2 = 0;
      switch (kind) {
        case 0: k1 = dme; break;
        case 1: k1 = dmate; break;
        case 2: k1 = dme + dmate; break;
        case 3: k1 = s.flevel[j]; k2 = dme; break;
        case 4: k1 = -s.flevel[j]; k2 = dme; break;
        case 5: k1 = fcell; break;
        case 6: k1 = -fcell; break;
        case 7: k1 = fc * 64 + fr; break;
        case 8: k1 = -(fc * 64 + fr); break;
        case 9: k1 = abs(fr - sr) + abs(fc - sc); break;
        default: k1 = -(abs(fr - sr) + abs(fc - sc)); break;
      }
      if (best < 0 || k1 < b1 || (k1 == b1 && k2 < b2)) {
        best = j;
        b1 = k1;
        b2 = k2;
        bcell = fcell;
      }
    }
  }
  if (best < 0) return 0;  // (no uneaten food: the episode has ended)
  const int tr = lbf_row(p, bcell), tc = bcell - tr * W;
  const int dr = tr - mr, dc = tc - mc;
  if (abs(dr) + abs(dc) == 1) return 5;  // LOAD
  const int vert = dr < 0 ? 1 : 2, horiz = dc < 0 ? 3 : 4;  // NORTH / SOUTH, WEST / EAST
  const bool rows_first = abs(dr) >= abs(dc);
  const int first = rows_first ? vert : horiz, other = rows_first ? horiz : vert;
  const bool other_closes = rows_first ? dc != 0 : dr != 0;
  const int next = me + (first == 1 ? -W : first == 2 ? W : first == 3 ? -1 : 1);
  bool blocked = false;
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    if (j < F && !((s.eaten >> j) & 1u) && s.fcell[j] == next) blocked = true;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i)
    if (i < A && i != agent && s.acell[i] == next) blocked = true;
  return (blocked && other_closes) ? other : first;
}

// The end of a transition: apply the moves and the eaten foods, the reward
// (one IEEE division, skipped when no env of the wave ate: the quotient is
// then +0), the step count and the done bits.
template <int FC = 0>
__device__ __forceinline__ void lbf_finish(const LbfParams& p, LbfEnv& s, const int (&newcell)[LBF_MAXA],
                                           uint32_t eaten, int eaten_sum, float& reward, uint32_t& done) {
  const int F = FC ? FC : p.F;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) s.acell[i] = newcell[i];
  s.eaten = eaten;
  reward = __builtin_amdgcn_ballot_w64(eaten_sum != 0) ? (float)eaten_sum / (float)s.den : 0.f;
  s.steps += 1;
  const uint32_t all = (F >= 32) ? 0xffffffffu : ((1u << F) - 1u);
  done = ((eaten & all) == all ? 1u : 0u) | (s.steps >= p.max_steps ? 2u : 0u);
}

// The transition on grids of at most 64 cells, with the grid as a 64-bit
// occupancy mask (bit c = cell c): a move is legal iff its target is on the
// grid and its bit is clear in the mask of uneaten foods and agents before
// the step; a loader's 4-neighbourhood is one more mask, and food j is
// adjacent to it iff bit fcell[j] is set there.  The same rules as
// lbf_transition_rc in fewer, mostly independent instructions.
template <int AC = 0, int FC = 0, int HC = 0, int WC = 0>
__device__ __forceinline__ void lbf_transition_bb(const LbfParams& p, LbfEnv& s, const int (&act_in)[LBF_MAXA],
                                                  float& reward, uint32_t& done) {
  const int A = AC ? AC : p.A, F = FC ? FC : p.F, W = WC ? WC : p.W, H = HC ? HC : p.H;
  const int HW = H * W;
  int act[LBF_MAXA], col[LBF_MAXA];
  uint64_t occ = 0;  // uneaten foods and agents before the step
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j)
    occ |= ((j < F) & !((s.eaten >> j) & 1u)) ? (1ull << (s.fcell[j] & 63)) : 0ull;
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    act[i] = ((unsigned)act_in[i] < (unsigned)LBF_NACT) ? act_in[i] : 0;
    col[i] = s.acell[i] - lbf_row_ct<WC>(p, s.acell[i]) * W;
    occ |= (i < A) ? (1ull << (s.acell[i] & 63)) : 0ull;
  }
  // 1. moves: the target of a legal move, else -1
  int tgt[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    const int a = act[i], c = s.acell[i];
    const bool inb = ((a == 1) & (c >= W)) | ((a == 2) & (c < HW - W)) | ((a == 3) & (col[i] > 0)) |
                     ((a == 4) & (col[i] < W - 1));
    const int t = c + (a == 1 ? -W : a == 2 ? W : a == 3 ? -1 : 1);
    const bool ok = (i < A) & inb & !((occ >> (t & 63)) & 1ull);
    tgt[i] = ok ? t : -1;
  }
  int newcell[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    bool contested = false;
#pragma unroll
    for (int k = 0; k < LBF_MAXA; ++k)
      if (k != i) contested |= (k < A) & (tgt[k] == tgt[i]);
    newcell[i] = ((tgt[i] >= 0) & !contested) ? tgt[i] : s.acell[i];
  }
  // 2. loads, with the pre-step positions: the loaders' 4-neighbourhoods
  uint64_t nb[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    const uint64_t b = 1ull << (s.acell[i] & 63);
    const uint64_t n = (b << W) | (b >> W) | (col[i] > 0 ? b >> 1 : 0ull) | (col[i] < W - 1 ? b << 1 : 0ull);
    nb[i] = ((i < A) & (act[i] == 5)) ? n : 0ull;
  }
  int eaten_sum = 0;
  uint32_t eaten = s.eaten;
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j) {
    int lsum = 0;
#pragma unroll
    for (int i = 0; i < LBF_MAXA; ++i) lsum += ((nb[i] >> (s.fcell[j] & 63)) & 1ull) ? s.alevel[i] : 0;
    const bool eat = (j < F) & !((s.eaten >> j) & 1u) & (lsum > 0) & (lsum >= s.flevel[j]);
    eaten |= eat ? (1u << j) : 0u;
    eaten_sum += eat ? s.flevel[j] : 0;
  }
  lbf_finish<FC>(p, s, newcell, eaten, eaten_sum, reward, done);
}

// The occupancy-mask transition resolved by a group of 8 consecutive lanes
// per env (a wave holds 8 groups), every lane of the group holding the env
// state and the actions: lane q of the group evaluates the move of agent
// q mod 4 (when < A) and the cooperative load of food q (when < F); the
// agents' targets reach every lane by quad broadcasts (DPP), the contested
// targets are resolved in every lane, and the eaten foods are gathered with
// one ballot.  Every lane of the group ends with the same post-step state,
// reward and done.  All 64 lanes of the wave must be active.
template <int A, int F, int GH, int GW>
__device__ __forceinline__ void lbf_transition_group(const LbfParams& p, LbfEnv& s, const int (&act_in)[LBF_MAXA],
                                                     float& reward, uint32_t& done) {
  constexpr int W = GW, HW = GH * GW;
  static_assert(HW <= 64 && A <= 4 && F <= 8, "one occupancy word; agents in a quad; foods in a group");
  const int lane = (int)(threadIdx.x & 63u), q = lane & 7, me = q & 3;
  int act[LBF_MAXA], col[LBF_MAXA];
  uint64_t occ = 0;  // uneaten foods and agents before the step
#pragma unroll
  for (int j = 0; j < F; ++j) occ |= !((s.eaten >> j) & 1u) ? (1ull << (s.fcell[j] & 63)) : 0ull;
#pragma unroll
  for (int i = 0; i < A; ++i) {
    act[i] = ((unsigned)act_in[i] < (unsigned)LBF_NACT) ? act_in[i] : 0;
    col[i] = s.acell[i] % W;
    occ |= 1ull << (s.acell[i] & 63);
  }
  // 1. this lane's agent: the target of a legal move, else -1
  int a = act[0], c = s.acell[0], cl = col[0];
#pragma unroll
  for (int i = 1; i < A; ++i) {
    a = me == i ? act[i] : a;
    c = me == i ? s.acell[i] : c;
    cl = me == i ? col[i] : cl;
  }
  const bool inb = ((a == 1) & (c >= W)) | ((a == 2) & (c < HW - W)) | ((a == 3) & (cl > 0)) | ((a == 4) & (cl < W - 1));
  const int t = c + (a == 1 ? -W : a == 2 ? W : a == 3 ? -1 : 1);
  const int mytgt = ((me < A) & inb & !((occ >> (t & 63)) & 1ull)) ? t : -1;
  int tgt[LBF_MAXA];
  tgt[0] = __builtin_amdgcn_mov_dpp(mytgt, 0x00, 0xf, 0xf, false);  // quad_perm [0,0,0,0]
  if constexpr (A > 1) tgt[1] = __builtin_amdgcn_mov_dpp(mytgt, 0x55, 0xf, 0xf, false);
  if constexpr (A > 2) tgt[2] = __builtin_amdgcn_mov_dpp(mytgt, 0xaa, 0xf, 0xf, false);
  if constexpr (A > 3) tgt[3] = __builtin_amdgcn_mov_dpp(mytgt, 0xff, 0xf, 0xf, false);
  int newcell[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    if (i >= A) {
      newcell[i] = s.acell[i];
      continue;
    }
    bool contested = false;
#pragma unroll
    for (int k = 0; k < A; ++k)
      if (k != i) contested |= tgt[k] == tgt[i];
    newcell[i] = ((tgt[i] >= 0) & !contested) ? tgt[i] : s.acell[i];
  }
  // 2. this lane's food: the levels of the loaders 4-adjacent to it, with the pre-step positions
  int fc = s.fcell[0], fl = s.flevel[0];
#pragma unroll
  for (int j = 1; j < F; ++j) {
    fc = q == j ? s.fcell[j] : fc;
    fl = q == j ? s.flevel[j] : fl;
  }
  const uint64_t fb = 1ull << (fc & 63);
  int lsum = 0;
#pragma unroll
  for (int i = 0; i < A; ++i) {
    const uint64_t b = 1ull << (s.acell[i] & 63);
    const uint64_t n = (b << W) | (b >> W) | (col[i] > 0 ? b >> 1 : 0ull) | (col[i] < W - 1 ? b << 1 : 0ull);
    lsum += ((act[i] == 5) & ((n & fb) != 0ull)) ? s.alevel[i] : 0;
  }
  const bool eat = (q < F) & !((s.eaten >> q) & 1u) & (lsum > 0) & (lsum >= fl);
  const uint32_t got = (uint32_t)(__builtin_amdgcn_ballot_w64(eat) >> (lane & ~7)) & 0xffu;
  int eaten_sum = 0;
#pragma unroll
  for (int j = 0; j < F; ++j) eaten_sum += ((got >> j) & 1u) ? s.flevel[j] : 0;
  lbf_finish<F>(p, s, newcell, s.eaten | got, eaten_sum, reward, done);
}

// One transition with actions act[0..A-1] (out-of-range -> noop).
// Writes reward and done; `s` becomes the post-transition state (no reset).
// Written without data-dependent branches: every candidate move and load is
// evaluated and the outcome selected, so the lanes of a wave never diverge.
// Grids of at most 64 cells take the occupancy-mask form above.
template <int AC = 0, int FC = 0, int HC = 0, int WC = 0>
__device__ __forceinline__ void lbf_transition_rc(const LbfParams& p, LbfEnv& s, const int (&act_in)[LBF_MAXA],
                                                  float& reward, uint32_t& done);

template <int AC = 0, int FC = 0, int HC = 0, int WC = 0>
__device__ __forceinline__ void lbf_transition(const LbfParams& p, LbfEnv& s, const int (&act_in)[LBF_MAXA],
                                               float& reward, uint32_t& done) {
  if constexpr (HC > 0 && WC > 0) {
    if constexpr (HC * WC <= 64)
      lbf_transition_bb<AC, FC, HC, WC>(p, s, act_in, reward, done);
    else
      lbf_transition_rc<AC, FC, HC, WC>(p, s, act_in, reward, done);
  } else {
    if (p.HW <= 64)
      lbf_transition_bb<AC, FC, HC, WC>(p, s, act_in, reward, done);
    else
      lbf_transition_rc<AC, FC, HC, WC>(p, s, act_in, reward, done);
  }
}

// The transition by rows and columns (any grid size).
template <int AC, int FC, int HC, int WC>
__device__ __forceinline__ void lbf_transition_rc(const LbfParams& p, LbfEnv& s, const int (&act_in)[LBF_MAXA],
                                                  float& reward, uint32_t& done) {
  const int A = AC ? AC : p.A, F = FC ? FC : p.F, W = WC ? WC : p.W, H = HC ? HC : p.H;
  int act[LBF_MAXA], ar[LBF_MAXA], ac[LBF_MAXA], fr[LBF_MAXF], fc[LBF_MAXF];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    act[i] = ((unsigned)act_in[i] < (unsigned)LBF_NACT) ? act_in[i] : 0;
    ar[i] = lbf_row_ct<WC>(p, s.acell[i]);
    ac[i] = s.acell[i] - ar[i] * W;
  }
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j) {
    fr[j] = lbf_row_ct<WC>(p, s.fcell[j]);
    fc[j] = s.fcell[j] - fr[j] * W;
  }

  // 1. moves against the pre-step state: tgt[i] = target cell of a legal move, else -1
  int tgt[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    const int r2 = ar[i] + (act[i] == 1 ? -1 : 0) + (act[i] == 2 ? 1 : 0);
    const int c2 = ac[i] + (act[i] == 3 ? -1 : 0) + (act[i] == 4 ? 1 : 0);
    const int cell = r2 * W + c2;
    bool ok = (i < A) & (act[i] >= 1) & (act[i] <= 4) & (r2 >= 0) & (r2 < H) & (c2 >= 0) & (c2 < W);
#pragma unroll
    for (int j = 0; j < LBF_MAXF; ++j)
      ok &= !((j < F) & !((s.eaten >> j) & 1u) & (s.fcell[j] == cell));
#pragma unroll
    for (int k = 0; k < LBF_MAXA; ++k) ok &= !((k < A) & (s.acell[k] == cell));
    tgt[i] = ok ? cell : -1;
  }
  int newcell[LBF_MAXA];
#pragma unroll
  for (int i = 0; i < LBF_MAXA; ++i) {
    bool contested = false;
#pragma unroll
    for (int k = 0; k < LBF_MAXA; ++k)
      if (k != i) contested |= (k < A) & (tgt[k] == tgt[i]);
    newcell[i] = ((tgt[i] >= 0) & !contested) ? tgt[i] : s.acell[i];
  }

  // 2. loads, with the pre-step positions (loaders do not move)
  int eaten_sum = 0;
  uint32_t eaten = s.eaten;
#pragma unroll
  for (int j = 0; j < LBF_MAXF; ++j) {
    int lsum = 0;
#pragma unroll
    for (int i = 0; i < LBF_MAXA; ++i) {
      const bool adj = (abs(ar[i] - fr[j]) + abs(ac[i] - fc[j])) == 1;
      lsum += ((i < A) & (act[i] == 5) & adj) ? s.alevel[i] : 0;
    }
    const bool eat = (j < F) & !((s.eaten >> j) & 1u) & (lsum > 0) & (lsum >= s.flevel[j]);
    eaten |= eat ? (1u << j) : 0u;
    eaten_sum += eat ? s.flevel[j] : 0;
  }
  lbf_finish<FC>(p, s, newcell, eaten, eaten_sum, reward, done);
}

}  // namespace rl
