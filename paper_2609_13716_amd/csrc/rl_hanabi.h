// Two-player Hanabi device logic: one game held in the registers of one lane
// as packed bit fields, plus the observation feature function.
//
// Hanabi is an environment of Section 4 (environment table), run as the
// Dec-POMDP step of Section 3 with the standard game: 5 colours x 5 ranks,
// 50 cards, hands of 5, 8 info tokens, 3 lives, 20 actions.  Rules, the
// state-buffer layout and the observation are documented in
// include/rollout.h.  Hands and per-card knowledge are arrays of small
// fields in one 32-bit word each, so closing up a hand after a play is two
// masks and a shift; the deck is 13 words of 4 card bytes, read with a
// select chain (no dynamically indexed registers).  A reset's Fisher-Yates
// shuffle runs across a whole wave, one deck position per lane, and the
// observation is assembled from fields computed by many threads.
#pragma once
#include "rl_philox.h"

namespace rl {

constexpr int HN_INFO = 8, HN_LIVES = 3;
constexpr int HN_DECK_WORDS = 13;     // deck words of the state (the standard game's 50 cards; smaller games use fewer)
constexpr int HN_PLANES_STATE = 35;  // int32 state planes per env (the same layout for every game size)

// Game sizes: C colours, R ranks (copies 3, 2, ..., 2, 1 per colour), hands
// of H (H <= 5, C * R <= 25: card ids fit the 5-bit fields), 8 tokens, 3 lives.
template <int C_, int R_, int H_>
struct HnGame {
  static constexpr int C = C_, R = R_, H = H_;
  static_assert(C >= 1 && C <= 5 && R >= 2 && R <= 5 && H >= 1 && H <= 5, "packed fields hold 5 slots of 5 bits");
  static constexpr int PER_COLOUR = 3 + 2 * (R - 2) + 1;
  static constexpr int CARDS = C * PER_COLOUR, KINDS = C * R, NACT = 2 * H + C + R;
  static constexpr int DW = (CARDS + 3) / 4;  // deck words in use
  static constexpr int LASTW = 2 + 4 + 2 + C + R + H + H + KINDS + 1 + 1;
  // observation sections, in order
  static constexpr int O_FLAGS = H * KINDS, O_DECK = O_FLAGS + 2, O_FW = O_DECK + CARDS - 2 * H,
                       O_INFO = O_FW + KINDS, O_LIVES = O_INFO + HN_INFO, O_DISC = O_LIVES + HN_LIVES,
                       O_LAST = O_DISC + CARDS, O_KNOW = O_LAST + LASTW;
  static constexpr int KNOW_SLOT = KINDS + C + R;
  static constexpr int OBS = O_KNOW + 2 * H * KNOW_SLOT;
  static constexpr int NFIELDS = 3 * H + C + 6;  // field computations per observation row (hn_field_bits)
  static constexpr int OBS_WORDS = (OBS + 63) / 64;
  static constexpr uint32_t FW_FULL = []() {
    uint32_t m = 0;
    for (int c = 0; c < C; ++c) m |= (uint32_t)R << (3 * c);
    return m;
  }();
};
using HnStd = HnGame<5, 5, 5>;   // the standard game: 50 cards, 20 actions, 658 features
using HnMini = HnGame<3, 3, 5>;  // 3 colours x 3 ranks: 18 cards, 16 actions
static_assert(HnStd::OBS == 658 && HnStd::NACT == 20 && HnStd::CARDS == 50 && HnStd::NFIELDS == 26, "standard game");
constexpr int HN_OBS = HnStd::OBS, HN_NACT = HnStd::NACT;  // the largest game's sizes
enum : int { HN_PLAY = 0, HN_DISCARD = 1, HN_HINT_COLOUR = 2, HN_HINT_RANK = 3 };

struct HnParams {
  int E, max_steps;
  int mini;  // 1: the 3 x 3 game (HnMini), 0: the standard game (HnStd)
  int64_t env_base;
  uint64_t seed;
};

struct HnEnv {
  uint32_t deck[HN_DECK_WORDS];  // card k in byte k % 4 of word k / 4
  uint32_t hand[2];              // 5-bit card id per slot (slot s at bit 5s); unused slots 0
  uint32_t kc[2], kr[2];         // possible colours / ranks, 5 bits per slot
  uint32_t hc[2], hr[2];         // hinted colour + 1 / hinted rank, 3 bits per slot (0: none)
  int n[2];                      // cards held
  uint32_t fw;                   // firework heights, 3 bits per colour
  uint32_t disc0, disc1;         // discarded copies, 2 bits per card id (ids 0-15, 16-24)
  int info, lives, cur, turns_left, next, steps;
  uint32_t last;                 // packed last action, 0 before the first move
};

// Packed last action: bit 0 present, 1 actor, 2-3 kind, 4 hint target,
// 5-7 hinted colour + 1, 8-10 hinted rank, 11-15 revealed slots,
// 16-18 acted slot + 1, 19-23 acted card + 1, 24 play succeeded, 25 token gained.

__device__ __forceinline__ uint32_t hn_field(uint32_t w, int width, int i) {
  return (w >> (width * i)) & ((1u << width) - 1u);
}

// Remove field i of a packed array of `width`-bit fields; later fields move down one.
__device__ __forceinline__ uint32_t hn_remove(uint32_t w, int width, int i) {
  const uint32_t low = (1u << (width * i)) - 1u;
  return (w & low) | ((w >> width) & ~low);
}

__device__ __forceinline__ int hn_deck_card(const HnEnv& s, int k) {
  uint32_t w = 0;
#pragma unroll
  for (int i = 0; i < HN_DECK_WORDS; ++i) w = (i == (k >> 2)) ? s.deck[i] : w;
  return (int)((w >> (8 * (k & 3))) & 0xffu);
}

__device__ __forceinline__ int hn_disc(const HnEnv& s, int card) {
  return card < 16 ? (int)((s.disc0 >> (2 * card)) & 3u) : (int)((s.disc1 >> (2 * (card - 16))) & 3u);
}

__device__ __forceinline__ void hn_add_disc(HnEnv& s, int card) {
  if (card < 16)
    s.disc0 += 1u << (2 * card);
  else
    s.disc1 += 1u << (2 * (card - 16));
}

// The deck of a fresh game at step t, shuffled by one whole wave (all lanes
// call this with the same env and t): Fisher-Yates from the ordered deck (per
// colour: rank 1 x3, middle ranks x2, the top rank x1) for i = CARDS-1 down to
// 1 swaps positions i and j_i = u(i + 1), with draw k = CARDS-1 - i of the
// reset stream.  Each lane l < CARDS finds the card that ends at position l
// without moving any card: the swaps applied in that order leave at l the
// card that started at S_{CARDS-1}( ... S_1(l)), S_i exchanging i and j_i, so
// the lane follows its position through S_1, S_2, ... (two compares and two
// selects per swap, j_i in scalar registers) and reads the ordered deck
// there.  The first lanes evaluate the Philox blocks of the draws.  Returns
// the packed deck words (card k in byte k % 4 of word k / 4; the words past
// the game's deck are 0): lane 4 w holds word w.
template <class G>
__device__ __forceinline__ uint32_t hn_wave_deck(uint64_t seed, uint64_t env, uint64_t t, int lane) {
  constexpr int NB = (G::CARDS - 1 + 7) / 8;
  Block4 b{0, 0, 0, 0};
  if (lane < NB) b = draw_block(seed, env, t, (uint64_t)lane, TAG_RESET);
  int x = lane;
#pragma unroll
  for (int i = 1; i < G::CARDS; ++i) {
    const int k = G::CARDS - 1 - i;  // the draw of the swap at position i
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)block_u32(b, k & 7), k >> 3);
    const int j = (int)range_map(d, (uint32_t)(i + 1));
    x = x == i ? j : x == j ? i : x;
  }
  const int c = x / G::PER_COLOUR, o = x - c * G::PER_COLOUR;
  const int rk = o < 3 ? 0 : min((o - 3) / 2 + 1, G::R - 1);
  const int a = c * G::R + rk;
  uint32_t v = lane < G::CARDS ? (uint32_t)a << (8 * (lane & 3)) : 0u;
  v |= (uint32_t)__shfl_xor((int)v, 1);
  v |= (uint32_t)__shfl_xor((int)v, 2);
  return v;
}

// hn_wave_deck with the words written to `words` (LDS).
template <class G>
__device__ __forceinline__ void hn_wave_shuffle(uint64_t seed, uint64_t env, uint64_t t, int lane,
                                                uint32_t* __restrict__ words) {
  const uint32_t v = hn_wave_deck<G>(seed, env, t, lane);
  if ((lane & 3) == 0 && lane < 4 * HN_DECK_WORDS) words[lane >> 2] = v;
}

// A fresh game on the shuffled deck `words`: player 0 holds cards 0..H-1 in
// slots 0..H-1, player 1 cards H..2H-1, card 2H is drawn next; player 0 moves
// first with all tokens and lives, blank knowledge, no fireworks or discards.
// hn_deal_deck deals from the deck already in s.deck.
template <class G>
__device__ __forceinline__ void hn_deal_deck(HnEnv& s) {
  constexpr int HN_HAND = G::H;
#pragma unroll
  for (int pl = 0; pl < 2; ++pl) {
    uint32_t h = 0;
#pragma unroll
    for (int q = 0; q < HN_HAND; ++q) {
      const int k = pl * HN_HAND + q;  // compile-time position: a fixed byte of a fixed word
      h |= ((s.deck[k >> 2] >> (8 * (k & 3))) & 0xffu) << (5 * q);
    }
    s.hand[pl] = h;
    s.n[pl] = HN_HAND;
    s.kc[pl] = s.kr[pl] = 0x1ffffffu & ((1u << (5 * HN_HAND)) - 1u);  // every colour and rank possible
    s.kc[pl] &= 0x108421u * ((1u << G::C) - 1u);  // (only the game's colours and ranks)
    s.kr[pl] &= 0x108421u * ((1u << G::R) - 1u);
    s.hc[pl] = s.hr[pl] = 0;
  }
  s.fw = 0;
  s.disc0 = s.disc1 = 0;
  s.info = HN_INFO;
  s.lives = HN_LIVES;
  s.cur = 0;
  s.turns_left = -1;
  s.next = 2 * HN_HAND;
  s.steps = 0;
  s.last = 0;
}

template <class G>
__device__ __forceinline__ void hn_deal(HnEnv& s, const uint32_t* __restrict__ words) {
#pragma unroll
  for (int w = 0; w < HN_DECK_WORDS; ++w) s.deck[w] = words[w];
  hn_deal_deck<G>(s);
}

// Legal actions of the player to move as a 20-bit mask, from a game or its
// published copy.  (Player-indexed fields are picked with selects, not
// indexed by the mover: a register array indexed at run time would live in
// scratch memory.)
template <class G, class S>
__device__ __forceinline__ uint32_t hn_legal(const S& s) {
  constexpr int HN_HAND = G::H, HN_RANKS = G::R, HN_COLOURS = G::C;
  const bool one = s.cur == 1;
  const int np = one ? s.n[1] : s.n[0], nq = one ? s.n[0] : s.n[1];
  const uint32_t hq = one ? s.hand[0] : s.hand[1];
  const uint32_t held = (1u << np) - 1u;
  uint32_t m = held << HN_HAND;                   // play
  if (s.info < HN_INFO) m |= held;                // discard
  if (s.info > 0) {
    uint32_t cols = 0, ranks = 0;
#pragma unroll
    for (int i = 0; i < HN_HAND; ++i)
      if (i < nq) {
        const int card = (int)hn_field(hq, 5, i);
        cols |= 1u << (card / HN_RANKS);
        ranks |= 1u << (card % HN_RANKS);
      }
    m |= cols << (2 * HN_HAND);
    m |= ranks << (2 * HN_HAND + HN_COLOURS);
  }
  return m;
}

// Exchange the two players' hands and knowledge when `sw` (so that the mover
// can be addressed as player 0 with constant indices).
__device__ __forceinline__ void hn_orient(HnEnv& s, bool sw) {
  auto x = [sw](uint32_t& a, uint32_t& b) {
    const uint32_t t0 = sw ? b : a, t1 = sw ? a : b;
    a = t0;
    b = t1;
  };
  x(s.hand[0], s.hand[1]);
  x(s.kc[0], s.kc[1]);
  x(s.kr[0], s.kr[1]);
  x(s.hc[0], s.hc[1]);
  x(s.hr[0], s.hr[1]);
  const int n0 = sw ? s.n[1] : s.n[0], n1 = sw ? s.n[0] : s.n[1];
  s.n[0] = n0;
  s.n[1] = n1;
}

// One move of the player to move (an illegal or out-of-range action acts as
// its lowest legal one); `s` becomes the post-transition state (no reset).
template <class G>
__device__ __forceinline__ void hn_transition(const HnParams& p, HnEnv& s, int a_in, float& reward, uint32_t& done) {
  constexpr int HN_HAND = G::H, HN_RANKS = G::R, HN_COLOURS = G::C, HN_CARDS = G::CARDS, HN_NACT = G::NACT;
  const uint32_t legal = hn_legal<G>(s);
  const int a = ((unsigned)a_in < (unsigned)HN_NACT && ((legal >> a_in) & 1u)) ? a_in : __builtin_ctz(legal);
  const int mover = s.cur;
  hn_orient(s, mover == 1);
  constexpr int pl = 0, q = 1;  // the mover and its partner after hn_orient
  int rew = 0;
  bool drew_last = false;
  int fw_total_before = 0;
#pragma unroll
  for (int c = 0; c < HN_COLOURS; ++c) fw_total_before += (int)hn_field(s.fw, 3, c);
  if (a < 2 * HN_HAND) {
    const int slot = a % HN_HAND;
    const bool play = a >= HN_HAND;
    const int card = (int)hn_field(s.hand[pl], 5, slot);
    uint32_t last = 1u | ((uint32_t)mover << 1) | ((uint32_t)(play ? HN_PLAY : HN_DISCARD) << 2) |
                    ((uint32_t)(slot + 1) << 16) | ((uint32_t)(card + 1) << 19);
    if (!play) {
      hn_add_disc(s, card);
      s.info += 1;
      last |= 1u << 25;
    } else {
      const int c = card / HN_RANKS, r = card % HN_RANKS + 1;
      if ((int)hn_field(s.fw, 3, c) + 1 == r) {
        s.fw += 1u << (3 * c);
        rew = 1;
        last |= 1u << 24;
        if (r == HN_RANKS && s.info < HN_INFO) {
          s.info += 1;
          last |= 1u << 25;
        }
      } else {
        hn_add_disc(s, card);
        s.lives -= 1;
      }
    }
    s.hand[pl] = hn_remove(s.hand[pl], 5, slot);
    s.kc[pl] = hn_remove(s.kc[pl], 5, slot);
    s.kr[pl] = hn_remove(s.kr[pl], 5, slot);
    s.hc[pl] = hn_remove(s.hc[pl], 3, slot);
    s.hr[pl] = hn_remove(s.hr[pl], 3, slot);
    s.n[pl] -= 1;
    if (s.next < HN_CARDS) {
      const int sh = 5 * s.n[pl];
      s.hand[pl] |= (uint32_t)hn_deck_card(s, s.next) << sh;
      s.kc[pl] |= ((1u << HN_COLOURS) - 1u) << sh;
      s.kr[pl] |= ((1u << HN_RANKS) - 1u) << sh;
      s.n[pl] += 1;
      s.next += 1;
      drew_last = s.next == HN_CARDS;
    }
    s.last = last;
  } else {
    const int h = a - 2 * HN_HAND;
    const bool colour = h < HN_COLOURS;
    const int v = colour ? h : h - HN_COLOURS;  // colour, or rank - 1
    uint32_t revealed = 0;
    uint32_t mask = colour ? s.kc[q] : s.kr[q];  // the knowledge words the hint updates
    uint32_t hint = colour ? s.hc[q] : s.hr[q];
#pragma unroll
    for (int i = 0; i < HN_HAND; ++i)
      if (i < s.n[q]) {
        const int card = (int)hn_field(s.hand[q], 5, i);
        const bool match = colour ? card / HN_RANKS == v : card % HN_RANKS == v;
        if (match) {
          mask = (mask & ~(31u << (5 * i))) | ((1u << v) << (5 * i));
          hint = (hint & ~(7u << (3 * i))) | ((uint32_t)(v + 1) << (3 * i));
          revealed |= 1u << i;
        } else {
          mask &= ~((1u << v) << (5 * i));
        }
      }
    s.kc[q] = colour ? mask : s.kc[q];
    s.hc[q] = colour ? hint : s.hc[q];
    s.kr[q] = colour ? s.kr[q] : mask;
    s.hr[q] = colour ? s.hr[q] : hint;
    s.info -= 1;
    s.last = 1u | ((uint32_t)mover << 1) | ((uint32_t)(colour ? HN_HINT_COLOUR : HN_HINT_RANK) << 2) |
             ((uint32_t)(1 - mover) << 4) | (colour ? (uint32_t)(v + 1) << 5 : (uint32_t)(v + 1) << 8) |
             (revealed << 11);
  }
  hn_orient(s, mover == 1);
  if (s.turns_left > 0) s.turns_left -= 1;
  if (drew_last) s.turns_left = 2;
  bool terminated = false;
  if (s.lives == 0) {
    terminated = true;
    rew = -fw_total_before;
  } else if (s.fw == G::FW_FULL /* every firework complete */ || s.turns_left == 0) {
    terminated = true;
  }
  s.cur = 1 - mover;
  s.steps += 1;
  reward = (float)rew;
  done = (terminated ? 1u : 0u) | (s.steps >= p.max_steps ? 2u : 0u);
}

// State planes (int32, E entries each); see include/rollout.h.
__device__ __forceinline__ void hn_load(const int32_t* __restrict__ st, int E, int e, HnEnv& s) {
  auto w = [&](int pl) { return (uint32_t)st[(size_t)pl * E + e]; };
#pragma unroll
  for (int i = 0; i < HN_DECK_WORDS; ++i) s.deck[i] = w(i);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    s.hand[i] = w(13 + i);
    s.n[i] = (int)w(15 + i);
    s.kc[i] = w(17 + i);
    s.kr[i] = w(19 + i);
    s.hc[i] = w(21 + i);
    s.hr[i] = w(23 + i);
  }
  s.fw = w(25);
  s.disc0 = w(26);
  s.disc1 = w(27);
  s.info = (int)w(28);
  s.lives = (int)w(29);
  s.cur = (int)w(30);
  s.turns_left = (int)w(31);
  s.next = (int)w(32);
  s.steps = (int)w(33);
  s.last = w(34);
}

__device__ __forceinline__ void hn_store(int32_t* __restrict__ st, int E, int e, const HnEnv& s) {
  auto w = [&](int pl, uint32_t v) { st[(size_t)pl * E + e] = (int32_t)v; };
#pragma unroll
  for (int i = 0; i < HN_DECK_WORDS; ++i) w(i, s.deck[i]);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    w(13 + i, s.hand[i]);
    w(15 + i, (uint32_t)s.n[i]);
    w(17 + i, s.kc[i]);
    w(19 + i, s.kr[i]);
    w(21 + i, s.hc[i]);
    w(23 + i, s.hr[i]);
  }
  w(25, s.fw);
  w(26, s.disc0);
  w(27, s.disc1);
  w(28, (uint32_t)s.info);
  w(29, (uint32_t)s.lives);
  w(30, (uint32_t)s.cur);
  w(31, (uint32_t)s.turns_left);
  w(32, (uint32_t)s.next);
  w(33, (uint32_t)s.steps);
  w(34, s.last);
}

// The observation as a bit vector in 64-bit words (bit f = feature f),
// assembled from G::NFIELDS fields per row that different threads compute
// in parallel (hn_field_bits) and OR into the row's words.
constexpr int HN_OBS_WORDS = (HN_OBS + 63) / 64;  // (the largest game)
constexpr int HN_NFIELDS = HnStd::NFIELDS;

// What the field computations read of one game (published to LDS after each move).
struct HnPub {
  uint32_t hand[2], kc[2], kr[2], hc[2], hr[2];
  int n[2];
  uint32_t fw, disc0, disc1, last;
  int info, lives, next, cur;
};

__device__ __forceinline__ void hn_pub(const HnEnv& s, HnPub& v) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    v.hand[i] = s.hand[i];
    v.kc[i] = s.kc[i];
    v.kr[i] = s.kr[i];
    v.hc[i] = s.hc[i];
    v.hr[i] = s.hr[i];
    v.n[i] = s.n[i];
  }
  v.fw = s.fw;
  v.disc0 = s.disc0;
  v.disc1 = s.disc1;
  v.last = s.last;
  v.info = s.info;
  v.lives = s.lives;
  v.next = s.next;
  v.cur = s.cur;
}

__device__ __forceinline__ uint64_t hn_therm(int n, int width) {  // n ones (clamped to width) from bit 0
  const int k = n < 0 ? 0 : n > width ? width : n;
  return k >= 64 ? ~0ull : ((1ull << k) - 1ull);
}

// Field f (0..NFIELDS-1) of player me's observation: its bits, and in `off`
// the feature index of its bit 0.  Fields: 0..H-1 partner slots (one-hot
// card id), H short hands, H+1 deck thermometer, H+2 fireworks, H+3 tokens,
// H+4 lives, then C fields of one colour's discard thermometers, the last
// move, and 2H fields of the knowledge of one slot (observer's hand, then the
// partner's).  `v` is normally in LDS; player indices are plain memory
// indices there.
template <class G>
__device__ __forceinline__ uint64_t hn_field_bits(const HnPub& v, int me, int f, int& off) {
  constexpr int H = G::H, C = G::C, R = G::R, K = G::KINDS;
  const int pt = 1 - me;
  if (f < H) {
    off = K * f;
    return f < v.n[pt] ? (1ull << hn_field(v.hand[pt], 5, f)) : 0ull;
  }
  if (f == H) {
    off = G::O_FLAGS;
    return (v.n[me] < H ? 1ull : 0ull) | (v.n[pt] < H ? 2ull : 0ull);
  }
  if (f == H + 1) {
    off = G::O_DECK;
    return hn_therm(G::CARDS - v.next, G::CARDS - 2 * H);
  }
  if (f == H + 2) {
    off = G::O_FW;
    uint64_t fw = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const uint32_t h = hn_field(v.fw, 3, c);
      fw |= h ? (1ull << (R * c + h - 1)) : 0ull;
    }
    return fw;
  }
  if (f == H + 3) {
    off = G::O_INFO;
    return hn_therm(v.info, HN_INFO);
  }
  if (f == H + 4) {
    off = G::O_LIVES;
    return hn_therm(v.lives, HN_LIVES);
  }
  if (f < H + 5 + C) {  // one colour's discards: thermometers of 3, 2, ..., 2, 1 copies
    const int c = f - (H + 5);
    off = G::O_DISC + G::PER_COLOUR * c;
    uint64_t d = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int card = c * R + r;
      const uint32_t cnt = card < 16 ? (v.disc0 >> (2 * card)) & 3u : (v.disc1 >> (2 * (card - 16))) & 3u;
      d |= hn_therm((int)cnt, r == 0 ? 3 : r == R - 1 ? 1 : 2) << (r == 0 ? 0 : 2 * r + 1);
    }
    return d;
  }
  if (f == H + 5 + C) {  // last move: actor 2, kind 4, target 2, colour C, rank R, revealed H, slot H,
                         // card C * R, success, token
    off = G::O_LAST;
    const uint32_t L = v.last;
    if (!(L & 1u)) return 0ull;
    const int actor = (int)((L >> 1) & 1u), kind = (int)((L >> 2) & 3u), target = (int)((L >> 4) & 1u);
    const uint32_t hcol = (L >> 5) & 7u, hrank = (L >> 8) & 7u, slot = (L >> 16) & 7u, card = (L >> 19) & 31u;
    constexpr int B_COL = 8, B_RANK = B_COL + C, B_REV = B_RANK + R, B_SLOT = B_REV + H, B_CARD = B_SLOT + H,
                  B_OK = B_CARD + K;
    uint64_t a = (1ull << ((actor - me) & 1)) | (1ull << (2 + kind));
    if (kind >= HN_HINT_COLOUR) a |= 1ull << (6 + ((target - me) & 1));
    if (hcol) a |= 1ull << (B_COL + hcol - 1);
    if (hrank) a |= 1ull << (B_RANK + hrank - 1);
    a |= (uint64_t)((L >> 11) & ((1u << H) - 1u)) << B_REV;
    if (slot) a |= 1ull << (B_SLOT + slot - 1);
    if (card) a |= 1ull << (B_CARD + card - 1);
    a |= (uint64_t)((L >> 24) & 3u) << B_OK;
    return a;
  }
  // knowledge of one card: C * R plausible cards, hinted colour, hinted rank
  const int f0 = f - (H + 6 + C);
  const int j = f0 / H, sl = f0 - H * j, who = j ? pt : me;
  off = G::O_KNOW + H * G::KNOW_SLOT * j + G::KNOW_SLOT * sl;
  if (sl >= v.n[who]) return 0ull;
  const uint32_t kc = hn_field(v.kc[who], 5, sl), kr = hn_field(v.kr[who], 5, sl);
  const uint32_t hc = hn_field(v.hc[who], 3, sl), hr = hn_field(v.hr[who], 3, sl);
  uint64_t spread = 0;  // colour bits at the bottom of R-bit groups; times the rank mask fills each group
#pragma unroll
  for (int c = 0; c < C; ++c) spread |= (uint64_t)((kc >> c) & 1u) << (R * c);
  const uint64_t plaus = spread * (uint64_t)kr;
  return plaus | ((hc ? 1ull << (hc - 1) : 0ull) << K) | ((hr ? 1ull << (hr - 1) : 0ull) << (K + C));
}

}  // namespace rl
