"""Pins of the oracle's mini Hanabi (3 colours x 3 ranks, the paper's environment table).

The oracle is parametric in colours, ranks and hand size; these pins fix the
3 x 3 game: a deck of 18 cards with copies (3, 2, 1) per colour, 16 actions
(discard / play 5 slots, 3 colour and 3 rank hints), a 278-feature
observation whose sections have the sizes the game implies, card conservation
and knowledge invariants over random games, finished games scoring their
fireworks (9 at most), completing every firework ending the game, and the
observation's knowledge section leaving no plausible card outside the 3 x 3
kinds.
"""

from collections import Counter

import numpy as np

from oracle import hanabi as hn
from oracle import rollout

MINI = hn.Config(colours=3, ranks=3)
SECTIONS = [("partner", 5 * 9), ("missing", 2), ("deck", 18 - 10), ("fireworks", 9), ("info", 8), ("lives", 3),
            ("discards", 18), ("last", 2 + 4 + 2 + 3 + 3 + 5 + 5 + 9 + 1 + 1), ("know", 2 * 5 * (9 + 3 + 3))]


def test_mini_sizes_and_deck():
    deck = hn.ordered_deck(MINI)
    assert len(deck) == MINI.n_cards == 18 and deck == sorted(deck)
    cnt = Counter(deck)
    for c in range(3):
        assert [cnt[c * 3 + r] for r in range(3)] == [3, 2, 1]
    assert MINI.n_actions == 16
    assert MINI.obs_dim == sum(n for _, n in SECTIONS) == 278


def _invariants(s):
    played = [c * 3 + r - 1 for c in range(3) for r in range(1, s.fireworks[c] + 1)]
    discarded = [x for x in range(9) for _ in range(s.discards[x])]
    assert sorted(s.deck[s.next_card:] + s.hands[0] + s.hands[1] + played + discarded) == hn.ordered_deck(MINI)
    for p in range(2):
        for x, k in zip(s.hands[p], s.know[p]):
            assert k.colours < 8 and k.ranks < 8
            assert (k.colours >> (x // 3)) & 1 and (k.ranks >> (x % 3)) & 1


def test_mini_random_games():
    rng = np.random.default_rng(3)
    finished = 0
    for e in range(60):
        s = hn.reset(MINI, 4, e, 0)
        ret = 0.0
        for t in range(200):
            _invariants(s)
            o = hn.observe(MINI, s, s.cur)
            assert len(o) == 278
            know = np.asarray(o[-150:]).reshape(10, 15)
            assert know[:, :9].sum() >= 0 and (know >= 0).all()
            legal = [a for a, ok in enumerate(hn.legal_mask(MINI, s, s.cur)) if ok]
            assert legal and max(legal) < 16
            acts = [0, 0]
            acts[s.cur] = int(rng.choice(legal))
            prev = s
            s, r, d = hn.step(MINI, 4, e, t, s, acts)
            ret += float(r)
            if d:
                end, _, _ = hn.transition(MINI, prev, acts)
                assert ret == (sum(end.fireworks) if end.lives > 0 else 0) <= 9
                finished += 1
                ret = 0.0
    assert finished >= 60


def test_mini_complete_fireworks_end_the_game():
    s = hn.reset(MINI, 1, 0, 0)
    s.fireworks = [3, 3, 2]
    s.hands[s.cur][0] = 2 * 3 + 2  # the last card of colour 2, rank 3
    s.know[s.cur][0] = hn.Knowledge(7, 7)
    acts = [0, 0]
    acts[s.cur] = 5  # play slot 0
    end, r, d = hn.transition(MINI, s, acts)
    assert (float(r), d & 1, sum(end.fireworks)) == (1.0, 1, 9)


def test_mini_rollout_plays_legal_moves():
    dims = (278, 32, 32, 16)
    rng = np.random.default_rng(5)
    ws = [(rng.standard_normal((dims[i + 1], dims[i])) / np.sqrt(dims[i])).astype(np.float32) for i in range(3)]
    bs = [np.zeros(dims[i + 1], np.float32) for i in range(3)]
    out = rollout.rollout(hn, MINI, 2, range(4), 0, 60, ws, bs, "f32")
    mask, acts = out["mask"], out["actions"]
    for k in range(60):
        for i in range(4):
            p = [a for a in range(2) if mask[k, i, a].any()][0]
            assert mask[k, i, p, acts[k, i, p]]
    assert (out["done"] == 1).any()
