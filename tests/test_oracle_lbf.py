"""Pins of the oracle's Level-Based Foraging environment.

* Hand-worked transitions (tests/golden/lbf_cases.json), one per rule reading.
* The reset law: ranges, placement constraints and chi-square uniformity.
* Invariants along long random-action rollouts at 8x8 and 12x12.
* Brute force over every 3x3 state (food at the single interior cell) and all
  36 joint actions, each checked against a second, reason-by-reason statement
  of the movement and load rules.
"""

import itertools
import json
import os

import numpy as np
import pytest

from oracle import lbf, rollout

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lbf_cases.json")


def _load_cases():
    with open(GOLDEN) as f:
        return json.load(f)


def _cell(cfg, rc):
    return rc[0] * cfg.grid_w + rc[1]


def _state(cfg, case):
    return lbf.State([_cell(cfg, a) for a in case["agents"]], list(case["levels"]),
                     [_cell(cfg, f) for f in case["foods"]], list(case["food_levels"]),
                     list(case["eaten"]), case["step_count"], sum(case["food_levels"]))


@pytest.mark.parametrize("case", _load_cases()["cases"], ids=lambda c: c["name"])
def test_hand_worked_case(case):
    cfg = lbf.Config(**_load_cases()["config"])
    nxt, reward, done = lbf.transition(cfg, _state(cfg, case), case["actions"])
    exp = case["expect"]
    assert nxt.agent_cell == [_cell(cfg, a) for a in exp["agents"]]
    assert nxt.food_eaten == exp["eaten"]
    assert int(np.array([reward], np.float32).view(np.uint32)[0]) == int(exp["reward_bits"], 16)
    assert done == exp["done"]
    assert nxt.step_count == exp["step_count"]


def test_auto_reset_draws_from_next_step():
    cfg = lbf.Config(8, 8, 2, 3, 2, 3)
    case = [c for c in _load_cases()["cases"] if c["name"] == "step_limit_truncates"][0]
    st = _state(cfg, case)
    nxt, _, done = lbf.step(cfg, 11, 5, 200, st, case["actions"])
    assert done == 2
    fresh = lbf.reset(cfg, 11, 5, 201)
    assert nxt == fresh and nxt.step_count == 0
    assert nxt != lbf.reset(cfg, 11, 5, 200)


def _check_reset(cfg, s):
    H, W, A, F = cfg.grid_h, cfg.grid_w, cfg.n_agents, cfg.n_food
    assert all(1 <= l <= cfg.max_agent_level for l in s.agent_level)
    cap = min(cfg.max_food_level, sum(s.agent_level))
    assert all(1 <= f <= cap for f in s.food_level)
    assert len(set(s.food_cell)) == F
    for c in s.food_cell:
        r, q = divmod(c, W)
        assert 1 <= r <= H - 2 and 1 <= q <= W - 2
    assert len(set(s.agent_cell)) == A
    assert not set(s.agent_cell) & set(s.food_cell)
    assert all(0 <= c < H * W for c in s.agent_cell)
    assert s.den == sum(s.food_level) and s.step_count == 0 and not any(s.food_eaten)


@pytest.mark.parametrize("cfg", [lbf.Config(8, 8, 2, 3, 2, 3), lbf.Config(12, 12, 3, 6, 3, 6)])
def test_reset_law(cfg):
    from scipy.stats import chisquare
    n = 3000
    states = [lbf.reset(cfg, 1, e, 0) for e in range(n)]
    for s in states:
        _check_reset(cfg, s)
    lv = np.bincount([l for s in states for l in s.agent_level], minlength=cfg.max_agent_level + 1)[1:]
    assert chisquare(lv).pvalue > 1e-4
    # food level uniform on 1..min(Fmax, sum of levels), given that sum
    by_cap = {}
    for s in states:
        cap = min(cfg.max_food_level, sum(s.agent_level))
        by_cap.setdefault(cap, []).extend(s.food_level)
    for cap, vals in by_cap.items():
        if cap > 1 and len(vals) > 50 * cap:
            assert chisquare(np.bincount(vals, minlength=cap + 1)[1:]).pvalue > 1e-4
    # food cells uniform over the interior
    fc = np.bincount([c for s in states for c in s.food_cell], minlength=cfg.grid_h * cfg.grid_w)
    interior = [r * cfg.grid_w + c for r in range(1, cfg.grid_h - 1) for c in range(1, cfg.grid_w - 1)]
    assert chisquare(fc[interior]).pvalue > 1e-4


def test_reset_is_keyed_by_env_and_step():
    cfg = lbf.Config(8, 8, 2, 3, 2, 3)
    a = lbf.reset(cfg, 1, 3, 0)
    assert a == lbf.reset(cfg, 1, 3, 0)
    distinct = {repr(lbf.reset(cfg, 1, 3, t)) for t in range(20)}
    assert len(distinct) > 15
    assert repr(lbf.reset(cfg, 2, 3, 0)) != repr(a)


@pytest.mark.parametrize("cfg,T", [(lbf.Config(8, 8, 2, 3, 2, 3), 300), (lbf.Config(12, 12, 3, 6, 3, 6), 200)])
def test_invariants_random_rollout(cfg, T):
    n = 24
    rng = np.random.default_rng(7)
    # mostly load/moves so that food gets eaten; a few out-of-range actions
    acts = rng.integers(0, 6, size=(T, n, cfg.n_agents))
    acts[rng.random(acts.shape) < 0.02] = 9
    states = rollout.initial_states(lbf, cfg, 3, range(n))
    ep_return = np.zeros(n)
    n_term = 0
    n_eaten = 0
    for t in range(T):
        for i in range(n):
            s = states[i]
            nxt, r, d = lbf.transition(cfg, s, acts[t, i])
            # each agent moves at most one cell, never onto food or another agent
            for a in range(cfg.n_agents):
                r0, c0 = divmod(s.agent_cell[a], cfg.grid_w)
                r1, c1 = divmod(nxt.agent_cell[a], cfg.grid_w)
                assert abs(r0 - r1) + abs(c0 - c1) <= 1
            assert len(set(nxt.agent_cell)) == cfg.n_agents
            uneaten = {c for c, e in zip(nxt.food_cell, nxt.food_eaten) if not e}
            assert not uneaten & set(nxt.agent_cell)
            # food never reappears; levels and cells are constant in an episode
            assert all(e1 or not e0 for e0, e1 in zip(s.food_eaten, nxt.food_eaten))
            assert nxt.agent_level == s.agent_level and nxt.food_cell == s.food_cell
            newly = sum(f for f, e0, e1 in zip(s.food_level, s.food_eaten, nxt.food_eaten) if e1 and not e0)
            assert r == np.float32(newly) / np.float32(s.den)
            ep_return[i] += float(r)
            n_eaten += newly > 0
            assert bool(d & 1) == all(nxt.food_eaten)
            assert bool(d & 2) == (nxt.step_count == cfg.max_steps)
            if d:
                assert ep_return[i] <= 1.0 + 1e-6
                if d & 1:
                    assert abs(ep_return[i] - 1.0) < 1e-5
                    n_term += 1
                ep_return[i] = 0.0
            states[i] = lbf.step(cfg, 3, i, t, s, acts[t, i])[0]
            if d:
                _check_reset(cfg, states[i])
    assert n_eaten > 0
    if cfg.n_food <= 3:
        assert n_term > 0


def test_observation_planes():
    cfg = lbf.Config(8, 8, 2, 3, 2, 3)
    case = _load_cases()["cases"][0]
    st = _state(cfg, case)
    st.food_eaten = [False, True, False]
    for a in range(2):
        o = lbf.observe(cfg, st, a).reshape(3, 8, 8)
        assert o[0, 3, 2] == 1 and o[0, 3, 4] == 2 and o[0].sum() == 3
        assert o[1, 3, 3] == 3 and o[1, 1, 6] == 2 and o[1, 5, 5] == 0 and o[1].sum() == 5
        assert o[2].sum() == 1 and o[2].reshape(-1)[st.agent_cell[a]] == 1


def _brute_force_expect(cfg, cells, levels, food, flevel, acts):
    """Second statement of the rules, reason by reason, for the 3x3 enumeration."""
    H, W = cfg.grid_h, cfg.grid_w
    step = {1: (-1, 0), 2: (1, 0), 3: (0, -1), 4: (0, 1)}
    targets = []
    for c, a in zip(cells, acts):
        if a not in step:
            targets.append(None)
            continue
        r, q = divmod(c, W)
        r, q = r + step[a][0], q + step[a][1]
        targets.append((r, q))
    final = []
    for i, c in enumerate(cells):
        t = targets[i]
        if t is None:
            final.append(c)
            continue
        r, q = t
        off_grid = not (0 <= r < H and 0 <= q < W)
        cell = r * W + q
        blocked = off_grid or cell == food or cell in cells
        contested = any(j != i and targets[j] == t for j in range(len(cells)))
        final.append(c if (blocked or contested) else cell)
    fr, fq = divmod(food, W)
    lsum = sum(l for c, l, a in zip(cells, levels, acts)
               if a == 5 and abs(c // W - fr) + abs(c % W - fq) == 1)
    eaten = lsum >= flevel and lsum > 0
    return final, eaten


def test_brute_force_3x3():
    cfg = lbf.Config(3, 3, 2, 1, 2, 3)
    food = 4  # the only interior cell, (1, 1)
    free = [c for c in range(9) if c != food]
    n = 0
    for c0, c1 in itertools.permutations(free, 2):
        for l0, l1 in itertools.product((1, 2), repeat=2):
            for f in (1, 2, 3):
                st = lbf.State([c0, c1], [l0, l1], [food], [f], [False], 0, f)
                for a0, a1 in itertools.product(range(6), repeat=2):
                    nxt, r, d = lbf.transition(cfg, st, [a0, a1])
                    final, eaten = _brute_force_expect(cfg, [c0, c1], [l0, l1], food, f, [a0, a1])
                    assert nxt.agent_cell == final, (c0, c1, a0, a1)
                    assert nxt.food_eaten == [eaten]
                    assert r == (np.float32(1.0) if eaten else np.float32(0.0))
                    assert d == (1 if eaten else 0)
                    n += 1
    assert n == 24192
