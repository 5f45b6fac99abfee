"""Pins of the oracle's LBF constant-levels variant (the 7x7 "constant levels"
task of the paper's environment table).

* A constant-levels reset puts agents and foods on the same cells as the
  drawn-levels reset of the same (seed, env, step): only the levels differ,
  and they are the configured constants (agents at max_agent_level, foods at
  max_food_level), so the return normaliser is n_food * max_food_level.
* With agents at level 1 and foods at level 2, a food is eaten only when both
  agents load it in the same step: brute force over every placement of two
  agents next to an interior food on a 5x5 grid and every joint action.
* Over a random rollout the levels never change, every positive reward is a
  multiple of 2 / (3 * 2) (one food of level 2 out of three), and an episode's
  return never exceeds 1.
"""

import itertools

import numpy as np

from oracle import lbf, rollout

CFG7 = lbf.Config(7, 7, 2, 3, 1, 2, max_steps=50, const_levels=True)


def test_constant_levels_keep_the_drawn_cells():
    drawn = lbf.Config(7, 7, 2, 3, 3, 5, max_steps=50)
    const = lbf.Config(7, 7, 2, 3, 3, 5, max_steps=50, const_levels=True)
    for env in range(200):
        a = lbf.reset(drawn, 17, env, env % 5)
        b = lbf.reset(const, 17, env, env % 5)
        assert a.agent_cell == b.agent_cell and a.food_cell == b.food_cell
        assert b.agent_level == [3, 3] and b.food_level == [5, 5, 5] and b.den == 15
        assert b.food_eaten == [False] * 3 and b.step_count == 0


def test_level_two_food_needs_both_agents():
    cfg = lbf.Config(5, 5, 2, 1, 1, 2, max_steps=50, const_levels=True)
    food = 2 * 5 + 2  # the centre
    around = [food - 5, food + 5, food - 1, food + 1]
    seen_eaten = 0
    for c0, c1 in itertools.permutations(around, 2):
        for a0, a1 in itertools.product(range(6), repeat=2):
            s = lbf.State([c0, c1], [1, 1], [food], [2], [False], 0, 2)
            nxt, rew, done = lbf.transition(cfg, s, [a0, a1])
            both_load = a0 == lbf.LOAD and a1 == lbf.LOAD
            assert nxt.food_eaten == [both_load]
            assert rew == (np.float32(1.0) if both_load else np.float32(0.0))
            seen_eaten += both_load
    assert seen_eaten == 12  # 4 * 3 ordered placements, one joint action each


def test_random_rollout_keeps_constant_levels():
    rng = np.random.default_rng(3)
    T, envs = 150, list(range(12))
    acts = rng.integers(0, 6, size=(T, len(envs), 2))
    out = rollout.env_only(lbf, CFG7, 5, envs, 0, acts)
    for s in out["states"]:
        assert s.agent_level == [1, 1] and s.food_level == [2, 2, 2]
    r = out["reward"].astype(np.float64)
    assert set(np.round(r[r > 0] * 3, 6)) <= {1.0, 2.0, 3.0}
    ret = np.zeros(len(envs))
    for t in range(T):
        ret += r[t]
        assert (ret <= 1.0 + 1e-6).all()
        ret[out["done"][t] != 0] = 0.0
    assert CFG7.obs_dim == 147
