"""Pins of the oracle's Overcooked-style kitchen.

* A scripted episode on a hand-built 5x4 kitchen: three onions into the pot,
  cooking for exactly cook_time steps, plating, and +20 exactly at the serve.
* One hand-worked case per interact rule and per move rule.
* The layout law: sizes, border, station placement and connectivity, the last
  checked with scipy's connected-component labelling.
* Invariants along random-action rollouts on many generated kitchens.
"""

import numpy as np
import pytest

from oracle import overcooked as oc
from oracle import rollout

CFG = oc.Config()
C, F, O, P, K, S = oc.COUNTER, oc.FLOOR, oc.ONION, oc.PLATE, oc.POT, oc.SERVE


def kitchen(rows):
    """State on a hand-drawn kitchen; rows are strings over 'C.OPKS' (K = pot)."""
    H, W = len(rows), len(rows[0])
    cells = [C] * oc.NCELL
    code = {"C": C, ".": F, "O": O, "P": P, "K": K, "S": S}
    for r, row in enumerate(rows):
        for q, ch in enumerate(row):
            cells[r * oc.CW + q] = code[ch]
    pots = [c for c in range(oc.NCELL) if cells[c] == K]
    return oc.State(W, H, cells, [0] * oc.NCELL, [0, 0], [0, 0], [0, 0], {c: 0 for c in pots},
                    {c: 0 for c in pots}, 0)


def rc(r, q):
    return r * oc.CW + q


ROOM = ["COCKC",
        "C...C",
        "C...C",
        "CPCSC"]


def run(state, script, cfg=CFG):
    rewards = []
    for a in script:
        state, r, d = oc.transition(cfg, state, a)
        rewards.append(float(r))
    return state, rewards


def test_scripted_soup():
    s = kitchen(ROOM)
    s.agent_cell = [rc(1, 1), rc(2, 1)]
    N, So, W, E, I, Z = 1, 2, 3, 4, 5, 0
    one_onion = [(N, Z), (I, Z), (E, Z), (E, Z), (N, Z), (I, Z), (W, Z), (W, Z), (N, Z)]
    # the first trip starts facing north at (1,1): take, walk to (1,3), face the pot, drop, walk back
    s, rw = run(s, [(I, Z), (E, Z), (E, Z), (N, Z), (I, Z), (W, Z), (W, Z), (N, Z)])
    assert s.pot_onions[rc(0, 3)] == 1 and s.agent_cell[0] == rc(1, 1)
    s, rw = run(s, [(I, Z), (E, Z), (E, Z), (N, Z), (I, Z), (W, Z), (W, Z), (N, Z)])
    assert s.pot_onions[rc(0, 3)] == 2
    s, rw = run(s, [(I, Z), (E, Z), (E, Z), (N, Z)])
    s, rw = run(s, [(I, Z)])  # third onion: cooking starts
    assert s.pot_onions[rc(0, 3)] == 3 and s.pot_timer[rc(0, 3)] == CFG.cook_time
    # fetch a plate: walk to (2,1) is blocked by agent 1, so agent 1 steps aside east first
    s, rw = run(s, [(W, E), (W, Z), (So, Z), (So, Z)])
    assert s.agent_cell == [rc(2, 1), rc(2, 2)] and s.facing[0] == 1
    s, rw = run(s, [(I, Z)])  # take a plate from (3,1)
    assert s.held[0] == oc.HELD_PLATE
    s, rw = run(s, [(N, W), (E, Z), (E, Z), (N, Z)])  # back under the pot, agent 1 out of the way
    assert s.agent_cell[0] == rc(1, 3) and s.facing[0] == 0
    cooked = CFG.cook_time - s.pot_timer[rc(0, 3)]
    # wait until one step before ready: plating must fail while the timer runs
    while s.pot_timer[rc(0, 3)] > 0:
        s, rw = run(s, [(I, Z)])
        if s.pot_timer[rc(0, 3)] > 0 or s.held[0] == oc.HELD_PLATE:
            assert s.held[0] == oc.HELD_PLATE
    assert cooked > 0
    s, rw = run(s, [(I, Z)])
    assert s.held[0] == oc.HELD_SOUP and s.pot_onions[rc(0, 3)] == 0
    s, rw = run(s, [(So, Z)])
    assert s.agent_cell[0] == rc(2, 3)
    s, rw = run(s, [(I, Z)])  # serve at (3,3)
    assert rw == [float(CFG.soup_reward)] and s.held[0] == oc.HELD_NONE


def test_cook_time_exact():
    """The third onion at step k makes the soup plateable from step k + cook_time + 1."""
    s = kitchen(ROOM)
    s.agent_cell = [rc(1, 3), rc(2, 1)]
    s.pot_onions[rc(0, 3)] = 2
    s.held = [oc.HELD_ONION, 0]
    s, _ = run(s, [(5, 0)])  # step k: third onion
    s.held = [oc.HELD_PLATE, 0]
    for j in range(CFG.cook_time):  # steps k+1 .. k+cook_time: not yet plateable
        s, _ = run(s, [(5, 0)])
        assert s.held[0] == oc.HELD_PLATE, j
    assert s.pot_timer[rc(0, 3)] == 0
    s, _ = run(s, [(5, 0)])  # step k + cook_time + 1
    assert s.held[0] == oc.HELD_SOUP


@pytest.mark.parametrize("name,setup,acts,check", [
    ("take_onion", dict(cells=[rc(1, 1), rc(2, 3)], face=[0, 0], held=[0, 0]), (5, 0),
     lambda s, r: s.held[0] == oc.HELD_ONION),
    ("take_plate_needs_empty_hand", dict(cells=[rc(2, 1), rc(1, 3)], face=[1, 0], held=[oc.HELD_ONION, 0]), (5, 0),
     lambda s, r: s.held[0] == oc.HELD_ONION),
    ("take_plate", dict(cells=[rc(2, 1), rc(1, 3)], face=[1, 0], held=[0, 0]), (5, 0),
     lambda s, r: s.held[0] == oc.HELD_PLATE),
    ("serve_needs_soup", dict(cells=[rc(2, 3), rc(1, 1)], face=[1, 0], held=[oc.HELD_PLATE, 0]), (5, 0),
     lambda s, r: s.held[0] == oc.HELD_PLATE and r == 0),
    ("serve_soup", dict(cells=[rc(2, 3), rc(1, 1)], face=[1, 0], held=[oc.HELD_SOUP, 0]), (5, 0),
     lambda s, r: s.held[0] == 0 and r == 20),
    ("place_on_counter", dict(cells=[rc(1, 1), rc(2, 3)], face=[2, 0], held=[oc.HELD_PLATE, 0]), (5, 0),
     lambda s, r: s.held[0] == 0 and s.items[rc(1, 0)] == oc.HELD_PLATE),
    ("interact_with_floor_does_nothing", dict(cells=[rc(1, 1), rc(2, 3)], face=[3, 0], held=[oc.HELD_ONION, 0]),
     (5, 0), lambda s, r: s.held[0] == oc.HELD_ONION),
    ("both_serve", dict(cells=[rc(2, 3), rc(1, 3)], face=[1, 0], held=[oc.HELD_SOUP, oc.HELD_SOUP]), (5, 0),
     lambda s, r: r == 20 and s.held == [0, oc.HELD_SOUP]),
    ("move_blocked_by_counter_turns", dict(cells=[rc(1, 1), rc(2, 3)], face=[0, 0], held=[0, 0]), (3, 0),
     lambda s, r: s.agent_cell[0] == rc(1, 1) and s.facing[0] == 2),
    ("move_blocked_by_agent", dict(cells=[rc(1, 1), rc(1, 2)], face=[0, 0], held=[0, 0]), (4, 0),
     lambda s, r: s.agent_cell == [rc(1, 1), rc(1, 2)] and s.facing[0] == 3),
    ("same_target_both_stay", dict(cells=[rc(1, 1), rc(1, 3)], face=[0, 0], held=[0, 0]), (4, 3),
     lambda s, r: s.agent_cell == [rc(1, 1), rc(1, 3)] and s.facing == [3, 2]),
    ("no_follow", dict(cells=[rc(1, 1), rc(1, 2)], face=[0, 0], held=[0, 0]), (4, 4),
     lambda s, r: s.agent_cell == [rc(1, 1), rc(1, 3)]),
    ("move_then_nothing_else", dict(cells=[rc(2, 2), rc(1, 1)], face=[0, 0], held=[0, 0]), (2, 0),
     lambda s, r: s.agent_cell[0] == rc(2, 2) and s.facing[0] == 1),
])
def test_rules(name, setup, acts, check):
    s = kitchen(ROOM)
    s.agent_cell, s.facing, s.held = list(setup["cells"]), list(setup["face"]), list(setup["held"])
    nxt, r, d = oc.transition(CFG, s, acts)
    assert check(nxt, float(r)), name


def test_counter_pick_and_agent_order():
    s = kitchen(ROOM)
    # agent 0 at (1,1) facing west onto counter (1,0) holding an onion; agent 1 at (2,1) facing west onto (2,0)
    s.agent_cell, s.facing, s.held = [rc(1, 1), rc(2, 1)], [2, 2], [oc.HELD_ONION, 0]
    s.items[rc(2, 0)] = oc.HELD_SOUP
    nxt, _, _ = oc.transition(CFG, s, (5, 5))
    assert nxt.items[rc(1, 0)] == oc.HELD_ONION and nxt.held == [0, oc.HELD_SOUP] and nxt.items[rc(2, 0)] == 0
    # occupied counter: placing does nothing
    s2 = nxt.copy()
    s2.held[0] = oc.HELD_PLATE
    n2, _, _ = oc.transition(CFG, s2, (5, 0))
    assert n2.held[0] == oc.HELD_PLATE and n2.items[rc(1, 0)] == oc.HELD_ONION


def test_pot_rules():
    s = kitchen(ROOM)
    s.agent_cell, s.facing = [rc(1, 3), rc(2, 1)], [0, 0]
    # a plate on an idle pot does nothing; an onion into a cooking pot does nothing
    s.held = [oc.HELD_PLATE, 0]
    n, _, _ = oc.transition(CFG, s, (5, 0))
    assert n.held[0] == oc.HELD_PLATE and n.pot_onions[rc(0, 3)] == 0
    s.pot_onions[rc(0, 3)], s.pot_timer[rc(0, 3)] = 3, 5
    s.held = [oc.HELD_ONION, 0]
    n, _, _ = oc.transition(CFG, s, (5, 0))
    assert n.held[0] == oc.HELD_ONION and n.pot_onions[rc(0, 3)] == 3 and n.pot_timer[rc(0, 3)] == 4


def test_truncation_and_reset():
    cfg = oc.Config(max_steps=7)
    s = oc.reset(cfg, 3, 11, 0)
    for t in range(7):
        nxt, r, d = oc.step(cfg, 3, 11, t, s, (0, 0))
        if t < 6:
            assert d == 0
            s = nxt
    assert d == 2
    fresh = oc.reset(cfg, 3, 11, 7)
    assert nxt.agent_cell == fresh.agent_cell and nxt.cells == s.cells and nxt.step_count == 0


def _check_layout(W, H, cells):
    from scipy import ndimage
    assert 5 <= W <= 9 and 4 <= H <= 5
    grid = np.array(cells).reshape(oc.CH, oc.CW)
    assert (grid[H:, :] == C).all() and (grid[:, W:] == C).all()
    border = np.zeros_like(grid, dtype=bool)
    border[0, :W] = border[H - 1, :W] = True
    border[:H, 0] = border[:H, W - 1] = True
    assert (grid[border] != F).all()
    for r, q in [(0, 0), (0, W - 1), (H - 1, 0), (H - 1, W - 1)]:
        assert grid[r, q] == C
    stations = np.isin(grid, [O, P, K, S])
    assert not (stations & ~border).any()
    for r, q in zip(*np.nonzero(stations)):
        nb = [(r + dr, q + dq) for dr, dq in ((-1, 0), (1, 0), (0, -1), (0, 1))]
        assert any(0 <= a < oc.CH and 0 <= b < oc.CW and grid[a, b] == F for a, b in nb)
    assert 1 <= (grid == O).sum() <= 2 and 1 <= (grid == K).sum() <= 2
    assert (grid == P).sum() == 1 and (grid == S).sum() == 1
    labels, n = ndimage.label(grid == F)
    assert n == 1 and (grid == F).sum() >= 2
    n_ic = ((grid[1:H - 1, 1:W - 1]) != F).sum()
    assert n_ic <= (H - 2) * (W - 2) // 4


def test_layout_law():
    seen_w, seen_h = set(), set()
    for e in range(600):
        W, H, cells = oc.layout(5, e)
        _check_layout(W, H, cells)
        seen_w.add(W)
        seen_h.add(H)
    assert seen_w == {5, 6, 7, 8, 9} and seen_h == {4, 5}
    # the fallback (no interior counters) is always a valid kitchen
    for e in range(50):
        ok, W, H, cells = oc._attempt(5, e, oc.MAX_ATTEMPTS, True)
        assert ok
        _check_layout(W, H, cells)


def test_reset_places_agents_on_distinct_floor():
    for e in range(200):
        s = oc.reset(CFG, 9, e, 0)
        assert s.agent_cell[0] != s.agent_cell[1]
        assert all(s.cells[c] == F for c in s.agent_cell)
        assert s.facing == [0, 0] and s.held == [0, 0] and not any(s.items)


def test_invariants_random_rollout():
    n, T = 24, 300
    rng = np.random.default_rng(2)
    acts = rng.integers(0, 6, size=(T, n, 2))
    states = rollout.initial_states(oc, CFG, 4, range(n))
    layouts = [(s.W, s.H, list(s.cells)) for s in states]
    total = 0.0
    picked = 0
    for t in range(T):
        for i in range(n):
            s = states[i]
            nxt, r, d = oc.transition(CFG, s, acts[t, i])
            assert (nxt.W, nxt.H, nxt.cells) == layouts[i]
            assert nxt.agent_cell[0] != nxt.agent_cell[1]
            assert all(nxt.cells[c] == F for c in nxt.agent_cell)
            assert all(0 <= h <= 3 for h in nxt.held)
            assert all(nxt.items[c] == 0 or nxt.cells[c] == C for c in range(oc.NCELL))
            for c in nxt.pots():
                assert 0 <= nxt.pot_onions[c] <= 3 and 0 <= nxt.pot_timer[c] <= CFG.cook_time
                assert nxt.pot_timer[c] == 0 or nxt.pot_onions[c] == 3
            assert float(r) in (0.0, 20.0, 40.0)
            total += float(r)
            picked += sum(1 for h0, h1 in zip(s.held, nxt.held) if h0 == 0 and h1 != 0)
            states[i] = oc.step(CFG, 4, i, t, s, acts[t, i])[0]
    assert picked > 0


def test_observation_planes():
    s = kitchen(ROOM)
    s.agent_cell, s.facing, s.held = [rc(1, 1), rc(2, 3)], [2, 1], [oc.HELD_ONION, oc.HELD_SOUP]
    s.items[rc(1, 4)] = oc.HELD_PLATE
    s.pot_onions[rc(0, 3)], s.pot_timer[rc(0, 3)] = 3, 7
    o = oc.observe(CFG, s, 0).reshape(oc.N_PLANES, oc.NCELL)
    assert o[0, rc(1, 1)] == 1 and o[0].sum() == 1 and o[1, rc(2, 3)] == 1
    assert o[2 + 2, rc(1, 1)] == 1 and o[6 + 1, rc(2, 3)] == 1 and o[2:10].sum() == 2
    assert o[18, rc(1, 1)] == 1 and o[23, rc(2, 3)] == 1 and o[18:24].sum() == 2
    assert o[16, rc(1, 4)] == 1 and o[15:18].sum() == 1
    assert o[24, rc(0, 3)] == 3 and o[25, rc(0, 3)] == 7
    assert o[11, rc(0, 1)] == 1 and o[12, rc(3, 1)] == 1 and o[13, rc(0, 3)] == 1 and o[14, rc(3, 3)] == 1
    assert o[10].sum() == sum(1 for c in s.cells if c == C)
    o1 = oc.observe(CFG, s, 1).reshape(oc.N_PLANES, oc.NCELL)
    assert o1[0, rc(2, 3)] == 1 and o1[1, rc(1, 1)] == 1 and o1[20, rc(2, 3)] == 1 and o1[21, rc(1, 1)] == 1
