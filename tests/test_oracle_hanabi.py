"""Pins of the oracle's two-player Hanabi.

* The deck: composition, and Fisher-Yates checked as a bijection between draw
  sequences and permutations and against the standard library's shuffle driven
  by the same choices.
* A hand-worked game on a fixed deck: plays, a failed play, hints with
  negative information, discards, token limits and the illegal-action rule.
* Each way a game ends: lives lost (the game scores 0), all fireworks
  complete, the last round after the deck runs out, and truncation.
* Invariants over many random games: card conservation, token and life
  bounds, knowledge that never excludes the true card, final score.
* The 658-feature observation, section by section.
"""

import itertools
import math
import random
from collections import Counter

import numpy as np
import pytest
from scipy import stats

from oracle import hanabi as hn
from oracle import philox, rollout

CFG = hn.Config()
C, R, H = CFG.colours, CFG.ranks, CFG.hand_size


def card(c, r):
    return c * R + r - 1


def draw_for(j, n):
    """A 32-bit draw that uniform_int maps to j of n."""
    return -(-(j << 32) // n)


# ---------------------------------------------------------------- deck

def test_deck_composition():
    deck = hn.ordered_deck(CFG)
    assert len(deck) == CFG.n_cards == 50
    cnt = Counter(deck)
    for c in range(C):
        assert [cnt[card(c, r)] for r in range(1, 6)] == [3, 2, 2, 2, 1]
    assert deck == sorted(deck)
    assert CFG.n_actions == 20 and CFG.obs_dim == 658


def test_fisher_yates_is_a_bijection_of_choices():
    """Every sequence of choices (j_i in 0..i) yields a different permutation: n! sequences, n! permutations."""
    for n in (2, 3, 4, 5):
        items = list(range(n))
        seen = set()
        for js in itertools.product(*[range(i + 1) for i in range(n - 1, 0, -1)]):
            draws = [draw_for(j, i + 1) for j, i in zip(js, range(n - 1, 0, -1))]
            seen.add(tuple(hn.fisher_yates(items, draws)))
        assert len(seen) == math.factorial(n)


def test_fisher_yates_matches_library_shuffle():
    """random.shuffle is the same top-down algorithm; feed it the same choices."""

    class Scripted(random.Random):
        choices = []

        def _randbelow(self, n):
            j = self.choices.pop(0)
            assert 0 <= j < n
            return j

    rng = np.random.default_rng(5)
    for _ in range(50):
        items = list(range(12))
        draws = [int(x) for x in rng.integers(0, 1 << 32, size=11)]
        js = [philox.uniform_int(d, i + 1) for d, i in zip(draws, range(11, 0, -1))]
        lib = list(items)
        scripted = Scripted(0)
        scripted.choices = list(js)
        scripted.shuffle(lib)
        assert not scripted.choices
        assert hn.fisher_yates(items, draws) == lib


def test_fisher_yates_uniform_over_permutations():
    rng = np.random.default_rng(11)
    counts = Counter()
    n_trials = 24000
    for _ in range(n_trials):
        draws = [int(x) for x in rng.integers(0, 1 << 32, size=3)]
        counts[tuple(hn.fisher_yates([0, 1, 2, 3], draws))] += 1
    assert len(counts) == 24
    _, p = stats.chisquare(list(counts.values()))
    assert p > 1e-3


def test_reset_deal_and_keying():
    s = hn.reset(CFG, 3, 17, 5)
    assert sorted(s.deck) == hn.ordered_deck(CFG)
    assert s.hands == [s.deck[0:5], s.deck[5:10]] and s.next_card == 10
    assert (s.info, s.lives, s.cur, s.turns_left, s.last, s.step_count) == (8, 3, 0, -1, None, 0)
    assert all(k.colours == 31 and k.ranks == 31 and k.hint_colour == -1 and k.hint_rank == -1
               for ks in s.know for k in ks)
    draws = philox.u32_draws(3, 17, 5, philox.TAG_RESET, 49)
    assert s.deck == hn.fisher_yates(hn.ordered_deck(CFG), draws)
    assert hn.reset(CFG, 3, 17, 5).deck == s.deck
    assert hn.reset(CFG, 3, 17, 6).deck != s.deck
    assert hn.reset(CFG, 3, 18, 5).deck != s.deck
    assert hn.reset(CFG, 4, 17, 5).deck != s.deck


# ---------------------------------------------------------- hand-worked game

def fixed_state(hand0, hand1, first=(), **kw):
    """A fresh game whose deck deals hand0, hand1, then the cards `first`, then the rest in order."""
    pool = Counter(hn.ordered_deck(CFG))
    for x in list(hand0) + list(hand1) + list(first):
        pool[x] -= 1
        assert pool[x] >= 0
    rest = list(first)
    for x, n in sorted(pool.items()):
        rest += [x] * n
    deck = list(hand0) + list(hand1) + rest
    s = hn.State(deck, 10, [list(hand0), list(hand1)], [[hn._blank(CFG) for _ in range(5)] for _ in range(2)],
                 [0] * C, [0] * (C * R), 8, 3, 0, -1, None, 0)
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def act(s, a, cfg=CFG):
    acts = [0, 0]
    acts[s.cur] = a
    return hn.transition(cfg, s, acts)


DISCARD, PLAY, HINT_C, HINT_R = 0, 5, 10, 15


def test_hand_worked_game():
    h0 = [card(0, 1), card(0, 2), card(1, 1), card(4, 5), card(2, 3)]
    h1 = [card(0, 1), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    nxt = [card(3, 2), card(1, 3), card(2, 2), card(4, 1)]
    s = fixed_state(h0, h1, first=nxt)
    # 1. player 0 plays slot 0 (red 1): success, hand closes up, the new card enters slot 4
    s, r, d = act(s, PLAY + 0)
    assert (float(r), d, s.fireworks, s.cur, s.info, s.lives) == (1.0, 0, [1, 0, 0, 0, 0], 1, 8, 3)
    assert s.hands[0] == [card(0, 2), card(1, 1), card(4, 5), card(2, 3), nxt[0]]
    assert s.last.kind == hn.LAST_PLAY and s.last.success and not s.last.token and s.last.card == card(0, 1)
    # 2. player 1 hints colour 0 to player 0: slot 0 (red 2) learns red, the others lose red
    s, r, d = act(s, HINT_C + 0)
    assert (float(r), s.info, s.cur) == (0.0, 7, 0)
    assert s.last.revealed == 0b00001 and s.last.target == 0 and s.last.colour == 0
    k = s.know[0]
    assert (k[0].colours, k[0].hint_colour) == (0b00001, 0)
    assert all(x.colours == 0b11110 and x.hint_colour == -1 for x in k[1:])
    # 3. player 0 plays slot 0 (red 2): success
    s, r, d = act(s, PLAY + 0)
    assert (float(r), s.fireworks[0]) == (1.0, 2)
    assert s.know[0][0].colours == 0b11110  # the yellow 1 moved into slot 0 with its knowledge
    # 4. player 1 plays slot 0 (red 1): fails, a life is lost, the card is discarded
    s, r, d = act(s, PLAY + 0)
    assert (float(r), d, s.lives, s.discards[card(0, 1)], s.fireworks[0]) == (0.0, 0, 2, 1, 2)
    assert not s.last.success
    # 5. player 0 hints rank 1 to player 1; its hand closed up and drew the third card (green 2):
    #    [white 1, yellow 2, red 3, green 1, green 2]
    assert s.hands[0][4] == nxt[1] and s.hands[1] == [card(3, 1), card(1, 2), card(0, 3), card(2, 1), nxt[2]]
    s, r, d = act(s, HINT_R + 0)
    assert s.last.revealed == 0b01001 and s.last.rank == 1
    assert [(k.ranks, k.hint_rank) for k in s.know[1]] == [(0b00001, 1), (0b11110, -1), (0b11110, -1),
                                                             (0b00001, 1), (0b11110, -1)]
    assert s.info == 6
    # 6. player 1 discards slot 2 (red 3): +1 token
    s, r, d = act(s, DISCARD + 2)
    assert (s.info, s.discards[card(0, 3)], s.last.kind, s.last.token, s.last.slot) == (7, 1, hn.LAST_DISCARD,
                                                                                       True, 2)
    assert s.step_count == 6 and s.cur == 0


def test_legality_and_illegal_action_rule():
    h0 = [card(0, 1), card(0, 2), card(1, 1), card(4, 5), card(2, 3)]
    h1 = [card(0, 4), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1)
    m = hn.legal_mask(CFG, s, 0)
    # 8 tokens: no discard; every play; colour hints for colours 0,1,2,3 (partner holds no blue); ranks 1..4
    assert m[:5] == [False] * 5 and m[5:10] == [True] * 5
    assert m[10:15] == [True, True, True, True, False]
    assert m[15:20] == [True, True, True, True, False]
    assert not any(hn.legal_mask(CFG, s, 1))
    # an illegal action (discard at 8 tokens) and out-of-range ones act as the lowest legal one: play slot 0
    for bad in (0, 3, 14, 19, -1, 20, 1 << 20):
        t, _, _ = act(s, bad)
        ref, _, _ = act(s, PLAY + 0)
        assert t.hands == ref.hands and t.fireworks == ref.fireworks, bad
    # no tokens: no hints, discards allowed
    s.info = 0
    m = hn.legal_mask(CFG, s, 0)
    assert m[:10] == [True] * 10 and not any(m[10:])
    # the non-mover's action is ignored
    a, _, _ = hn.transition(CFG, s, [PLAY + 1, 7])
    b, _, _ = hn.transition(CFG, s, [PLAY + 1, 0])
    assert a.hands == b.hands


def test_completing_a_firework_returns_a_token():
    h0 = [card(4, 5), card(0, 2), card(1, 1), card(4, 4), card(2, 3)]
    h1 = [card(0, 4), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1, fireworks=[0, 0, 0, 0, 4], info=5)
    t, r, d = act(s, PLAY + 0)
    assert (float(r), t.info, t.fireworks[4], t.last.token, d) == (1.0, 6, 5, True, 0)
    s.info = 8
    t, r, d = act(s, PLAY + 0)
    assert (t.info, t.last.token) == (8, False)


# ---------------------------------------------------------------- endings

def test_losing_the_last_life_scores_zero():
    h0 = [card(0, 4), card(0, 2), card(1, 1), card(4, 4), card(2, 3)]
    h1 = [card(0, 5), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1, fireworks=[2, 1, 0, 0, 0], lives=1)
    t, r, d = act(s, PLAY + 0)  # red 4 on red 2: fails
    assert (float(r), d, t.lives) == (-3.0, 1, 0)
    # a failed play with lives left is an ordinary step
    s.lives = 2
    t, r, d = act(s, PLAY + 0)
    assert (float(r), d, t.lives) == (0.0, 0, 1)


def test_all_fireworks_complete_ends_the_game():
    h0 = [card(4, 5), card(0, 2), card(1, 1), card(4, 4), card(2, 3)]
    h1 = [card(0, 4), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1, fireworks=[5, 5, 5, 5, 4])
    t, r, d = act(s, PLAY + 0)
    assert (float(r), d, sum(t.fireworks)) == (1.0, 1, 25)


def test_last_round_after_the_deck_runs_out():
    h0 = [card(0, 1), card(0, 2), card(1, 1), card(4, 4), card(2, 3)]
    h1 = [card(0, 4), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1, info=3)
    s.next_card = len(s.deck) - 1  # one card left
    s, r, d = act(s, DISCARD + 4)  # draws the last card
    assert (d, s.turns_left, s.next_card) == (0, 2, 50)
    s, r, d = act(s, HINT_R + 0)  # player 1's last move
    assert (d, s.turns_left) == (0, 1)
    s, r, d = act(s, DISCARD + 0)  # player 0's last move: hand shrinks, nothing to draw
    assert (d, s.turns_left, len(s.hands[0])) == (1, 0, 4)


def test_truncation_and_auto_reset():
    cfg = hn.Config(max_steps=3)
    s = hn.reset(cfg, 1, 2, 0)
    for t in range(3):
        acts = [0, 0]
        acts[s.cur] = hn.legal_mask(cfg, s, s.cur).index(True)
        s2, r, d = hn.step(cfg, 1, 2, t, s, acts)
        if t < 2:
            assert d == 0
            s = s2
    assert d == 2
    assert s2.deck == hn.reset(cfg, 1, 2, 3).deck and s2.step_count == 0


# --------------------------------------------------------------- invariants

def _check_invariants(cfg, s):
    played = [card(c, r) for c in range(cfg.colours) for r in range(1, s.fireworks[c] + 1)]
    discarded = [x for x in range(cfg.colours * cfg.ranks) for _ in range(s.discards[x])]
    everything = s.deck[s.next_card:] + s.hands[0] + s.hands[1] + played + discarded
    assert sorted(everything) == hn.ordered_deck(cfg)
    assert 0 <= s.info <= cfg.info_tokens and 0 < s.lives <= cfg.life_tokens
    for p in range(2):
        assert len(s.hands[p]) == len(s.know[p]) <= cfg.hand_size
        assert len(s.hands[p]) >= cfg.hand_size - 1
        for x, k in zip(s.hands[p], s.know[p]):
            c, r = hn.colour_of(cfg, x), hn.rank_of(cfg, x)
            assert (k.colours >> c) & 1 and (k.ranks >> (r - 1)) & 1
            assert k.hint_colour in (-1, c) and k.hint_rank in (-1, r)
    assert any(hn.legal_mask(cfg, s, s.cur)) and not any(hn.legal_mask(cfg, s, 1 - s.cur))


def test_invariants_over_random_games():
    rng = np.random.default_rng(0)
    finished = 0
    for e in range(40):
        s = hn.reset(CFG, 9, e, 0)
        ret = 0.0
        for t in range(300):
            _check_invariants(CFG, s)
            legal = [a for a, ok in enumerate(hn.legal_mask(CFG, s, s.cur)) if ok]
            acts = [0, 0]
            acts[s.cur] = int(rng.choice(legal))
            prev = s
            s, r, d = hn.step(CFG, 9, e, t, s, acts)
            ret += float(r)
            if d:
                assert d == 1
                end, _, _ = hn.transition(CFG, prev, acts)
                assert ret == (sum(end.fireworks) if end.lives > 0 else 0)
                assert end.step_count <= 50 + 8 + 40 + 5 + 2
                finished += 1
                ret = 0.0
    assert finished >= 40


def test_rollout_loop_plays_only_legal_moves():
    dims = (658, 32, 32, 20)
    rng = np.random.default_rng(1)
    ws = [(rng.standard_normal((dims[i + 1], dims[i])) / np.sqrt(dims[i])).astype(np.float32) for i in range(3)]
    bs = [np.zeros(dims[i + 1], np.float32) for i in range(3)]
    out = rollout.rollout(hn, CFG, 4, range(3), 0, 90, ws, bs, "f32")
    mask, acts = out["mask"], out["actions"]
    T, n = acts.shape[:2]
    for k in range(T):
        for i in range(n):
            movers = [a for a in range(2) if mask[k, i, a].any()]
            assert len(movers) == 1
            p = movers[0]
            assert mask[k, i, p, acts[k, i, p]]
            assert acts[k, i, 1 - p] == 0  # all masked: action 0, ignored
    assert (out["done"] == 1).any()


# ------------------------------------------------------------- observation

SECTIONS = [("partner", 125), ("missing", 2), ("deck", 40), ("fireworks", 25), ("info", 8), ("lives", 3),
            ("discards", 50), ("last", 55), ("know", 350)]


def split(o):
    out, i = {}, 0
    for name, n in SECTIONS:
        out[name] = o[i:i + n]
        i += n
    assert i == len(o) == 658
    return out


def test_observation_sections():
    rng = np.random.default_rng(2)
    s = hn.reset(CFG, 5, 0, 0)
    for t in range(120):
        for me in range(2):
            o = hn.observe(CFG, s, me)
            assert set(np.unique(o)) <= {0.0, 1.0}
            v = split(o)
            ph = v["partner"].reshape(5, 25)
            other = s.hands[1 - me]
            assert ph.sum() == len(other)
            for i, x in enumerate(other):
                assert ph[i, x] == 1
            assert list(v["missing"]) == [len(s.hands[me]) < 5, len(other) < 5]
            assert v["deck"].sum() == min(40, 50 - s.next_card)
            assert np.all(np.diff(v["deck"]) <= 0)  # thermometer
            fw = v["fireworks"].reshape(5, 5)
            assert [int(np.argmax(row)) + 1 if row.any() else 0 for row in fw] == s.fireworks
            assert v["info"].sum() == s.info and np.all(np.diff(v["info"]) <= 0)
            assert v["lives"].sum() == s.lives
            i = 0
            for x in range(25):  # one thermometer per card id, as long as its number of copies
                n = CFG.copies[x % 5]
                seg = v["discards"][i:i + n]
                assert seg.sum() == s.discards[x] and np.all(np.diff(seg) <= 0)
                i += n
            kn = v["know"].reshape(2, 5, 35)
            for j, who in enumerate((me, 1 - me)):
                for i in range(5):
                    if i >= len(s.hands[who]):
                        assert not kn[j, i].any()
                        continue
                    x = s.hands[who][i]
                    assert kn[j, i, x] == 1  # the true card is always plausible
                    k = s.know[who][i]
                    assert kn[j, i, :25].sum() == bin(k.colours).count("1") * bin(k.ranks).count("1")
            if s.last is None:
                assert not v["last"].any()
            else:
                la = v["last"]
                assert la[:2].sum() == 1 and la[(s.last.actor - me) % 2] == 1
                assert la[2:6].sum() == 1 and la[2 + s.last.kind] == 1
        legal = [a for a, ok in enumerate(hn.legal_mask(CFG, s, s.cur)) if ok]
        acts = [0, 0]
        acts[s.cur] = int(rng.choice(legal))
        s, _, _ = hn.step(CFG, 5, 0, t, s, acts)
    # the two agents see each other's hands
    o0, o1 = split(hn.observe(CFG, s, 0)), split(hn.observe(CFG, s, 1))
    assert not np.array_equal(o0["partner"], o1["partner"])
    assert np.array_equal(o0["know"][:175], o1["know"][175:]) and np.array_equal(o0["know"][175:], o1["know"][:175])


def test_last_action_encoding_of_a_hint():
    h0 = [card(0, 1), card(0, 2), card(1, 1), card(4, 5), card(2, 3)]
    h1 = [card(0, 4), card(3, 1), card(1, 2), card(0, 3), card(2, 1)]
    s = fixed_state(h0, h1)
    s, _, _ = act(s, HINT_C + 0)  # player 0 hints red to player 1: slots 0 and 3
    for me in range(2):
        la = split(hn.observe(CFG, s, me))["last"]
        exp = np.zeros(55)
        exp[(0 - me) % 2] = 1                 # actor
        exp[2 + hn.LAST_HINT_COLOUR] = 1      # kind
        exp[6 + (1 - me) % 2] = 1             # target
        exp[8 + 0] = 1                        # colour red
        exp[18 + 0] = exp[18 + 3] = 1         # revealed slots 0 and 3
        assert np.array_equal(la, exp), me
    s, _, _ = act(s, PLAY + 2)  # player 1 plays yellow 2 on an empty yellow pile: fails
    la = split(hn.observe(CFG, s, 0))["last"]
    exp = np.zeros(55)
    exp[1] = 1
    exp[2 + hn.LAST_PLAY] = 1
    exp[23 + 2] = 1                           # slot 2
    exp[28 + card(1, 2)] = 1                  # the card
    assert np.array_equal(la, exp)
