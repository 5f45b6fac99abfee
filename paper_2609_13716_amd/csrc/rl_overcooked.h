// Overcooked-style kitchen device logic: layout generation, reset (rho) and
// transition (P, r) of one env held in the registers of one lane.
//
// The kitchen is an environment of Section 4 (environment table), run as the
// Dec-POMDP step of Section 3; its dynamics, the synthetic layout generator
// and the observation are readings of the paper's description, documented in
// include/rollout.h.  A kitchen lives on a fixed 5 x 9 canvas (cell id =
// row * 9 + col); every cell set is a 45-bit mask, so neighbourhoods,
// connectivity and "the k-th free cell" are a few 64-bit operations.
#pragma once
#include "rl_philox.h"

namespace rl {

constexpr int OC_CH = 5, OC_CW = 9, OC_NCELL = 45;
constexpr int OC_NACT = 6, OC_PLANES = 26, OC_D = OC_PLANES * OC_NCELL;  // 1170
constexpr int OC_MAX_ATTEMPTS = 64;
constexpr uint64_t OC_ALL = (1ull << OC_NCELL) - 1;
constexpr uint64_t OC_COL0 = (1ull << 0) | (1ull << 9) | (1ull << 18) | (1ull << 27) | (1ull << 36);
constexpr uint64_t OC_COL8 = OC_COL0 << 8;
enum : int { OC_HELD_NONE = 0, OC_HELD_ONION = 1, OC_HELD_PLATE = 2, OC_HELD_SOUP = 3 };

struct OcParams {
  int E, cook_time, soup_reward, max_steps;
  int64_t env_base;
  uint64_t seed;
};

struct OcEnv {
  uint64_t floor, counter, onion, plate, pot, serve;  // cell-type masks (counter: non-floor, non-station)
  uint64_t it_onion, it_plate, it_soup;               // items lying on counters
  int W, H;
  int acell[2], face[2], held[2];                     // facing 0 N, 1 S, 2 W, 3 E
  int pcell[2], pon[2], ptm[2];                       // pots in row-major order (cell -1: none)
  int steps;
};

constexpr int OC_PLANES_STATE = 32;  // int32 state planes per env

__device__ __forceinline__ uint64_t bit64(int c) { return 1ull << c; }

// Cells 4-adjacent to any cell of m (within the canvas).
__device__ __forceinline__ uint64_t oc_nb(uint64_t m) {
  return ((m << OC_CW) | (m >> OC_CW) | ((m << 1) & ~OC_COL0) | ((m >> 1) & ~OC_COL8)) & OC_ALL;
}

// The k-th (0-based) set bit of m, in increasing cell order.
__device__ __forceinline__ int oc_select(uint64_t m, int k) {
  for (int i = 0; i < k; ++i) m &= m - 1;
  return __builtin_ctzll(m);
}

// Sequential 32-bit draws of one (env, t, tag) stream (draw k: block k / 8,
// word (k % 8) / 2, high half first).
struct DrawCursor {
  uint64_t seed, env, t, tag, sub;
  Block4 b;
  int pos;
  __device__ DrawCursor(uint64_t seed_, uint64_t env_, uint64_t t_, uint64_t tag_)
      : seed(seed_), env(env_), t(t_), tag(tag_), sub(0), b{0, 0, 0, 0}, pos(8) {}
  __device__ __forceinline__ uint32_t next() {
    if (pos == 8) {
      b = draw_block(seed, env, t, sub++, tag);
      pos = 0;
    }
    return block_u32(b, pos++);
  }
  __device__ __forceinline__ int u(int n) { return (int)range_map(next(), (uint32_t)n); }
};

__device__ __forceinline__ bool oc_layout_attempt(const OcParams& p, uint64_t env, int attempt, bool force,
                                                  OcEnv& s) {
  DrawCursor d(p.seed, env, (uint64_t)attempt, TAG_LAYOUT);
  const int W = 5 + d.u(5), H = 4 + d.u(2);
  uint64_t interior = 0, grid = 0;
  for (int r = 0; r < H; ++r)
    for (int q = 0; q < W; ++q) {
      grid |= bit64(r * OC_CW + q);
      if (r > 0 && r < H - 1 && q > 0 && q < W - 1) interior |= bit64(r * OC_CW + q);
    }
  uint64_t floor = interior, counter = OC_ALL & ~interior;
  int n_ic = d.u((H - 2) * (W - 2) / 4 + 1);
  if (force) n_ic = 0;
  for (int i = 0; i < n_ic; ++i) {
    const int c = oc_select(floor, d.u(__builtin_popcountll(floor)));
    floor &= ~bit64(c);
    counter |= bit64(c);
  }
  const int n_onion = 1 + d.u(2), n_pot = 1 + d.u(2);
  const uint64_t corners = bit64(0) | bit64(W - 1) | bit64((H - 1) * OC_CW) | bit64((H - 1) * OC_CW + W - 1);
  const uint64_t border = grid & ~interior & ~corners;
  uint64_t kinds[4] = {0, 0, 0, 0};  // onion, pot, plate, serve
  bool ok = true;
  for (int st = 0; st < n_onion + n_pot + 2 && ok; ++st) {
    const uint64_t cand = border & counter & oc_nb(floor);
    if (!cand) {
      ok = false;
    } else {
      const int c = oc_select(cand, d.u(__builtin_popcountll(cand)));
      counter &= ~bit64(c);
      const int kind = st < n_onion ? 0 : st < n_onion + n_pot ? 1 : st == n_onion + n_pot ? 2 : 3;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q == kind) kinds[q] |= bit64(c);
    }
  }
  if (ok) {
    ok = __builtin_popcountll(floor) >= 2;
    uint64_t reach = floor & (~floor + 1);  // lowest floor cell
    for (int it = 0; it < OC_NCELL && ok; ++it) {
      const uint64_t nr = (reach | oc_nb(reach)) & floor;
      if (nr == reach) break;
      reach = nr;
    }
    ok = ok && reach == floor;
  }
  s.W = W;
  s.H = H;
  s.floor = floor;
  s.counter = counter;
  s.onion = kinds[0];
  s.pot = kinds[1];
  s.plate = kinds[2];
  s.serve = kinds[3];
  return ok;
}

// env's kitchen: the first valid attempt, else the counter-free fallback.
__device__ __forceinline__ void oc_layout(const OcParams& p, uint64_t env, OcEnv& s) {
  for (int a = 0; a < OC_MAX_ATTEMPTS; ++a)
    if (oc_layout_attempt(p, env, a, false, s)) return;
  oc_layout_attempt(p, env, OC_MAX_ATTEMPTS, true, s);
}

// A fresh episode on the kept kitchen, from the reset stream at step t.
__device__ __forceinline__ void oc_reset(const OcParams& p, uint64_t env, uint64_t t, OcEnv& s) {
  DrawCursor d(p.seed, env, t, TAG_RESET);
  const int nf = __builtin_popcountll(s.floor);
  s.acell[0] = oc_select(s.floor, d.u(nf));
  s.acell[1] = oc_select(s.floor & ~bit64(s.acell[0]), d.u(nf - 1));
  s.face[0] = s.face[1] = 0;
  s.held[0] = s.held[1] = OC_HELD_NONE;
  s.it_onion = s.it_plate = s.it_soup = 0;
  uint64_t pots = s.pot;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    s.pcell[j] = pots ? __builtin_ctzll(pots) : -1;
    pots &= pots - 1;
    s.pon[j] = 0;
    s.ptm[j] = 0;
  }
  s.steps = 0;
}

__device__ __forceinline__ int oc_faced(int cell, int face) {
  const int r = cell / OC_CW, q = cell - r * OC_CW;
  const int r2 = r + (face == 0 ? -1 : face == 1 ? 1 : 0);
  const int q2 = q + (face == 2 ? -1 : face == 3 ? 1 : 0);
  return (r2 >= 0 && r2 < OC_CH && q2 >= 0 && q2 < OC_CW) ? r2 * OC_CW + q2 : -1;
}

__device__ __forceinline__ int oc_item_at(const OcEnv& s, int c) {
  return ((s.it_onion >> c) & 1) ? OC_HELD_ONION : ((s.it_plate >> c) & 1) ? OC_HELD_PLATE
                                                 : ((s.it_soup >> c) & 1) ? OC_HELD_SOUP : 0;
}

__device__ __forceinline__ void oc_set_item(OcEnv& s, int c, int item) {
  const uint64_t m = bit64(c);
  s.it_onion = (s.it_onion & ~m) | (item == OC_HELD_ONION ? m : 0);
  s.it_plate = (s.it_plate & ~m) | (item == OC_HELD_PLATE ? m : 0);
  s.it_soup = (s.it_soup & ~m) | (item == OC_HELD_SOUP ? m : 0);
}

// One joint action (out-of-range -> noop); `s` becomes the post-transition
// state (no reset).  `changed` receives the counter cells whose item changed.
__device__ __forceinline__ void oc_transition(const OcParams& p, OcEnv& s, const int (&act_in)[2], float& reward,
                                              uint32_t& done, uint64_t& changed) {
  int act[2];
  act[0] = ((unsigned)act_in[0] < (unsigned)OC_NACT) ? act_in[0] : 0;
  act[1] = ((unsigned)act_in[1] < (unsigned)OC_NACT) ? act_in[1] : 0;
  int tgt[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    tgt[i] = -1;
    if (act[i] >= 1 && act[i] <= 4) {
      s.face[i] = act[i] - 1;
      const int n = oc_faced(s.acell[i], s.face[i]);
      if (n >= 0 && ((s.floor >> n) & 1) && n != s.acell[0] && n != s.acell[1]) tgt[i] = n;
    }
  }
  const int nc0 = (tgt[0] >= 0 && tgt[0] != tgt[1]) ? tgt[0] : s.acell[0];
  const int nc1 = (tgt[1] >= 0 && tgt[1] != tgt[0]) ? tgt[1] : s.acell[1];
  s.acell[0] = nc0;
  s.acell[1] = nc1;
  bool cooking[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) cooking[j] = s.pcell[j] >= 0 && s.pon[j] == 3 && s.ptm[j] > 0;
  int rew = 0;
  changed = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    if (act[i] != 5) continue;
    const int c = oc_faced(s.acell[i], s.face[i]);
    if (c < 0) continue;
    const uint64_t m = bit64(c);
    const int h = s.held[i];
    if ((s.onion & m) && h == OC_HELD_NONE) {
      s.held[i] = OC_HELD_ONION;
    } else if ((s.plate & m) && h == OC_HELD_NONE) {
      s.held[i] = OC_HELD_PLATE;
    } else if (s.pot & m) {
      const int j = s.pcell[0] == c ? 0 : 1;
      if (h == OC_HELD_ONION && s.pon[j] < 3) {
        s.held[i] = OC_HELD_NONE;
        s.pon[j] += 1;
        if (s.pon[j] == 3) s.ptm[j] = p.cook_time;
      } else if (h == OC_HELD_PLATE && s.pon[j] == 3 && s.ptm[j] == 0) {
        s.held[i] = OC_HELD_SOUP;
        s.pon[j] = 0;
      }
    } else if ((s.serve & m) && h == OC_HELD_SOUP) {
      s.held[i] = OC_HELD_NONE;
      rew += p.soup_reward;
    } else if (s.counter & m) {
      const int it = oc_item_at(s, c);
      if (h != OC_HELD_NONE && it == 0) {
        oc_set_item(s, c, h);
        s.held[i] = OC_HELD_NONE;
        changed |= m;
      } else if (h == OC_HELD_NONE && it != 0) {
        s.held[i] = it;
        oc_set_item(s, c, 0);
        changed |= m;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j)
    if (cooking[j]) s.ptm[j] -= 1;
  s.steps += 1;
  reward = (float)rew;
  done = s.steps >= p.max_steps ? 2u : 0u;
}

// State planes (int32, E entries each): 0-17 the nine cell masks as lo/hi
// words (floor, counter, onion, plate, pot, serve, item onion, item plate,
// item soup), 18 W | H << 8, 19-20 agent cells, 21-22 facings, 23-24 held,
// 25-26 pot cells, 27-28 pot onions, 29-30 pot timers, 31 steps.
__device__ __forceinline__ void oc_load(const int32_t* __restrict__ st, int E, int e, OcEnv& s) {
  auto w = [&](int pl) { return (uint32_t)st[(size_t)pl * E + e]; };
  auto m = [&](int pl) { return (uint64_t)w(pl) | ((uint64_t)w(pl + 1) << 32); };
  s.floor = m(0);
  s.counter = m(2);
  s.onion = m(4);
  s.plate = m(6);
  s.pot = m(8);
  s.serve = m(10);
  s.it_onion = m(12);
  s.it_plate = m(14);
  s.it_soup = m(16);
  s.W = (int)(w(18) & 0xff);
  s.H = (int)((w(18) >> 8) & 0xff);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    s.acell[i] = (int)w(19 + i);
    s.face[i] = (int)w(21 + i);
    s.held[i] = (int)w(23 + i);
    s.pcell[i] = (int)w(25 + i);
    s.pon[i] = (int)w(27 + i);
    s.ptm[i] = (int)w(29 + i);
  }
  s.steps = (int)w(31);
}

__device__ __forceinline__ void oc_store(int32_t* __restrict__ st, int E, int e, const OcEnv& s) {
  auto w = [&](int pl, uint32_t v) { st[(size_t)pl * E + e] = (int32_t)v; };
  auto m = [&](int pl, uint64_t v) {
    w(pl, (uint32_t)v);
    w(pl + 1, (uint32_t)(v >> 32));
  };
  m(0, s.floor);
  m(2, s.counter);
  m(4, s.onion);
  m(6, s.plate);
  m(8, s.pot);
  m(10, s.serve);
  m(12, s.it_onion);
  m(14, s.it_plate);
  m(16, s.it_soup);
  w(18, (uint32_t)s.W | ((uint32_t)s.H << 8));
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    w(19 + i, (uint32_t)s.acell[i]);
    w(21 + i, (uint32_t)s.face[i]);
    w(23 + i, (uint32_t)s.held[i]);
    w(25 + i, (uint32_t)s.pcell[i]);
    w(27 + i, (uint32_t)s.pon[i]);
    w(29 + i, (uint32_t)s.ptm[i]);
  }
  w(31, (uint32_t)s.steps);
}

}  // namespace rl
