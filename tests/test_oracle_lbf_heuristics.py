"""Pins of the oracle's heuristic LBF teammates (Greedy and Sequential agents).

* Targets against independent formulations over random states: Greedy
  closest_self / closest_teammate / closest_avg are numpy argmins over the
  uneaten foods' distance arrays (first minimum = lowest index);
  Sequential lexicographic is the uneaten food with the smallest row-major
  cell id, column_major the smallest column-major id, their reverses the
  largest; nearest/farthest agent are numpy argmin/argmax of the distance
  from the start cell; lowest/highest level is the extreme level, ties to the
  closest.
* Start cells in a rollout: every nearest/farthest-agent action is the
  heuristic's for the agent's cell at its episode's first step, read back
  from the rollout's own observations and dones; a rollout split in two
  (the second part recovering the start cells from the reset draws of step
  t0 - step_count) equals the whole.
* Actions: LOAD exactly when next to the target; otherwise a move along the
  longer axis that brings the agent one cell closer to it.
* Behaviour: Greedy agents able to eat alone clear the board (episodes end
  terminated); two closest_avg agents of level 1 meet at level-2 foods and
  eat them together; every heuristic agent of a rollout takes the heuristic's
  action whatever the network says, and with no heuristic agent the rollout
  is the plain one.
"""

import numpy as np
import pytest

from oracle import lbf, lbf_heuristics as H, rollout
from paper_2609_13716_amd import workloads

CFG = lbf.Config(7, 7, 2, 4, 2, 3, max_steps=40)


def _states(n=300, seed=0, cfg=CFG):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        s = lbf.reset(cfg, 5, i, int(rng.integers(0, 50)))
        eaten = list(rng.random(cfg.n_food) < 0.4)
        if all(eaten):
            eaten[int(rng.integers(0, cfg.n_food))] = False
        s.food_eaten = eaten
        out.append(s)
    return out


def _rows_cols(cfg, cells):
    cells = np.asarray(cells)
    return cells // cfg.grid_w, cells % cfg.grid_w


def test_greedy_distance_targets():
    for s in _states():
        fr, fc = _rows_cols(CFG, s.food_cell)
        live = ~np.array(s.food_eaten)
        for a in range(2):
            ar, ac = _rows_cols(CFG, [s.agent_cell[a]])
            mr, mc = _rows_cols(CFG, [s.agent_cell[1 - a]])
            d_me = np.abs(fr - ar) + np.abs(fc - ac)
            d_mate = np.abs(fr - mr) + np.abs(fc - mc)
            for kind, d in ((0, d_me), (1, d_mate), (2, d_me + d_mate)):
                assert H.target(CFG, s, a, kind) == int(np.argmin(np.where(live, d, 10 ** 6)))


def test_level_targets():
    for s in _states(seed=1):
        live = [j for j in range(CFG.n_food) if not s.food_eaten[j]]
        for a in range(2):
            for kind, pick in ((3, min), (4, max)):
                lv = pick(s.food_level[j] for j in live)
                cand = [j for j in live if s.food_level[j] == lv]
                dist = [abs(s.food_cell[j] // 7 - s.agent_cell[a] // 7) + abs(s.food_cell[j] % 7 - s.agent_cell[a] % 7)
                        for j in cand]
                assert H.target(CFG, s, a, kind) == cand[int(np.argmin(dist))]


def test_sequential_orders_are_cell_orders():
    for s in _states(seed=2):
        live = [j for j in range(CFG.n_food) if not s.food_eaten[j]]
        row_major = {j: s.food_cell[j] for j in live}
        col_major = {j: (s.food_cell[j] % 7) * 7 + s.food_cell[j] // 7 for j in live}
        for a in range(2):
            assert H.target(CFG, s, a, 5) == min(live, key=row_major.get)
            assert H.target(CFG, s, a, 6) == max(live, key=row_major.get)
            assert H.target(CFG, s, a, 7) == min(live, key=col_major.get)
            assert H.target(CFG, s, a, 8) == max(live, key=col_major.get)


def test_sequential_agent_orders_rank_by_distance_from_the_start_cell():
    rng = np.random.default_rng(7)
    for s in _states(seed=4):
        fr, fc = _rows_cols(CFG, s.food_cell)
        live = ~np.array(s.food_eaten)
        for a in range(2):
            start = int(rng.integers(0, 49))
            sr, sc = divmod(start, 7)
            d = np.abs(fr - sr) + np.abs(fc - sc)
            assert H.target(CFG, s, a, 9, start) == int(np.argmin(np.where(live, d, 10 ** 6)))
            assert H.target(CFG, s, a, 10, start) == int(np.argmax(np.where(live, d, -1)))
    with pytest.raises(ValueError):
        H.target(CFG, _states(1)[0], 0, 9)


def test_actions_load_next_to_the_target_else_close_in():
    delta = {lbf.NORTH: (-1, 0), lbf.SOUTH: (1, 0), lbf.WEST: (0, -1), lbf.EAST: (0, 1)}
    for s in _states(seed=3):
        for a in range(2):
            for kind in range(len(H.KINDS)):
                j = H.target(CFG, s, a, kind, s.agent_cell[1 - a])
                r, c = divmod(s.agent_cell[a], 7)
                tr, tc = divmod(s.food_cell[j], 7)
                d = abs(tr - r) + abs(tc - c)
                act = H.action(CFG, s, a, kind, s.agent_cell[1 - a])
                if d == 1:
                    assert act == lbf.LOAD
                    continue
                assert act in delta
                nr, nc = r + delta[act][0], c + delta[act][1]
                assert abs(tr - nr) + abs(tc - nc) == d - 1
                longer = abs(tr - r) >= abs(tc - c) if act in (lbf.NORTH, lbf.SOUTH) else abs(tc - c) > abs(tr - r)
                if not longer:  # the longer axis was blocked by a food or the other agent
                    lr, lc = (r + (1 if tr > r else -1), c) if act in (lbf.WEST, lbf.EAST) else (r, c + (1 if tc > c else -1))
                    cell = lr * 7 + lc
                    foods = {x for x, e in zip(s.food_cell, s.food_eaten) if not e}
                    assert cell in foods or cell == s.agent_cell[1 - a]
                lg = H.logits(CFG, s, a, kind, s.agent_cell[1 - a])
                assert lg[act] == 0 and np.isneginf(np.delete(lg, act)).all()


def _net(cfg):
    dims = (cfg.obs_dim, 16, 16, 6)
    return workloads.policy_weights(dims, seed=3, bias_scale=0.3)


def test_greedy_agents_that_can_eat_alone_clear_the_board():
    cfg = lbf.Config(7, 7, 2, 3, 3, 3, max_steps=60, const_levels=True)
    ws, bs = _net(cfg)
    envs = list(range(10))
    out = rollout.rollout(lbf, cfg, 2, envs, 0, 60, ws, bs, "f32", teammates=np.zeros((10, 2), int))
    cleared = [(out["done"][:, i] & 1).sum() for i in range(10)]  # terminated: every food eaten
    assert sum(c >= 2 for c in cleared) >= 8


def test_closest_avg_pairs_cooperate():
    cfg = lbf.Config(7, 7, 2, 3, 1, 2, max_steps=50, const_levels=True)
    ws, bs = _net(cfg)
    envs = list(range(12))
    avg = rollout.rollout(lbf, cfg, 4, envs, 0, 50, ws, bs, "f32", teammates=np.full((12, 2), 2))
    own = rollout.rollout(lbf, cfg, 4, envs, 0, 50, ws, bs, "f32", teammates=np.full((12, 2), 0))
    # agreeing on the food closest to both lets level-1 pairs eat level-2 foods; each heading for
    # its own closest food rarely does
    assert (avg["reward"] > 0).any(axis=0).mean() >= 0.5
    assert (avg["reward"] > 0).sum() >= 4 * max(1, (own["reward"] > 0).sum())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rollout_with_heuristic_teammates(dtype):
    ws, bs = _net(CFG)
    envs = list(range(9))
    tm = np.array([[-1, k] for k in range(9)])
    out = rollout.rollout(lbf, CFG, 6, envs, 0, 30, ws, bs, dtype, teammates=tm)
    assert np.isneginf(out["logits"][:, :, 1]).sum(axis=-1).max() == 5
    # replay: each heuristic agent's action is the heuristic's on the state it acted in
    states = rollout.initial_states(lbf, CFG, 6, envs)
    for k in range(30):
        for i in range(9):
            assert out["actions"][k, i, 1] == H.action(CFG, states[i], 1, i)
            states[i], _, _ = lbf.step(CFG, 6, envs[i], k, states[i], list(out["actions"][k, i]))
    plain = rollout.rollout(lbf, CFG, 6, envs, 0, 30, ws, bs, dtype)
    same = rollout.rollout(lbf, CFG, 6, envs, 0, 30, ws, bs, dtype, teammates=np.full((9, 2), -1))
    for key in ("obs", "actions", "reward", "done", "logits"):
        assert np.array_equal(plain[key], same[key]), key


def _own_cell(cfg, obs_row):
    """The agent's cell from its observation (plane 2 is 1 at its own cell)."""
    hw = cfg.grid_h * cfg.grid_w
    return int(np.flatnonzero(obs_row[2 * hw:])[0])


def test_agent_order_teammates_plan_from_the_episode_start():
    cfg = lbf.Config(7, 7, 2, 4, 2, 3, max_steps=12)
    ws, bs = _net(cfg)
    envs = list(range(8))
    tm = np.array([[9 + (i % 2), 10 - (i % 2)] for i in envs])  # both agents heuristic, both new orders
    T = 40
    out = rollout.rollout(lbf, cfg, 3, envs, 0, T, ws, bs, "f32", teammates=tm)
    states = rollout.initial_states(lbf, cfg, 3, envs)
    for i in range(len(envs)):
        starts = [None, None]
        for k in range(T):
            if k == 0 or out["done"][k - 1, i]:
                starts = [_own_cell(cfg, out["obs"][k, i, a]) for a in range(2)]
            for a in range(2):
                assert out["actions"][k, i, a] == H.action(cfg, states[i], a, int(tm[i, a]), starts[a])
            states[i], _, _ = lbf.step(cfg, 3, envs[i], k, states[i], list(out["actions"][k, i]))
    assert (out["done"] != 0).sum() >= 2 * len(envs)
    # a split rollout recovers the start cells of the running episodes from the reset draws
    a = rollout.rollout(lbf, cfg, 3, envs, 0, 17, ws, bs, "f32", teammates=tm)
    b = rollout.rollout(lbf, cfg, 3, envs, 17, T - 17, ws, bs, "f32", states=a["states"], teammates=tm)
    for key in ("obs", "actions", "reward", "done"):
        assert np.array_equal(out[key], np.concatenate([a[key], b[key]])), key
