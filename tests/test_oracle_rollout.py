"""Oracle rollout loop: determinism, env independence, resume, and the policy's effect."""

import numpy as np

from oracle import lbf, rollout


def _policy(dims, seed):
    rng = np.random.default_rng(seed)
    ws = [(rng.standard_normal((dims[i + 1], dims[i])) / np.sqrt(dims[i])).astype(np.float32)
          for i in range(3)]
    bs = [np.zeros(dims[i + 1], np.float32) for i in range(3)]
    return ws, bs


CFG = lbf.Config(8, 8, 2, 3, 2, 3)


def test_subset_matches_batch_and_is_deterministic():
    ws, bs = _policy((192, 64, 64, 6), 1000)
    full = rollout.rollout(lbf, CFG, 0, range(6), 0, 60, ws, bs, "f32")
    sub = rollout.rollout(lbf, CFG, 0, [4, 1], 0, 60, ws, bs, "f32")
    for k in ("obs", "actions", "reward", "done"):
        assert np.array_equal(full[k][:, [4, 1]], sub[k])
    again = rollout.rollout(lbf, CFG, 0, range(6), 0, 60, ws, bs, "f32")
    assert np.array_equal(full["actions"], again["actions"])
    # episodes end by the 50-step limit at the latest
    assert (full["done"] != 0).any(axis=0).all()


def test_split_run_equals_single_run():
    ws, bs = _policy((192, 64, 64, 6), 1001)
    one = rollout.rollout(lbf, CFG, 2, range(4), 0, 40, ws, bs, "bf16")
    a = rollout.rollout(lbf, CFG, 2, range(4), 0, 25, ws, bs, "bf16")
    b = rollout.rollout(lbf, CFG, 2, range(4), 25, 15, ws, bs, "bf16", states=a["states"])
    assert np.array_equal(one["actions"], np.concatenate([a["actions"], b["actions"]]))
    assert np.array_equal(one["obs_last"], b["obs_last"])


def test_actions_follow_logits():
    # a policy whose last-layer bias strongly prefers action 5 (load) picks it almost always
    ws, bs = _policy((192, 64, 64, 6), 1002)
    ws[2] = np.zeros_like(ws[2])
    bs[2] = np.array([0, 0, 0, 0, 0, 8.0], np.float32)
    out = rollout.rollout(lbf, CFG, 0, range(4), 0, 30, ws, bs, "f32")
    assert (out["actions"] == 5).mean() > 0.98


def test_env_only_matches_rollout_transitions():
    ws, bs = _policy((192, 64, 64, 6), 1003)
    ro = rollout.rollout(lbf, CFG, 5, range(3), 0, 30, ws, bs, "f32")
    eo = rollout.env_only(lbf, CFG, 5, range(3), 0, ro["actions"])
    assert np.array_equal(eo["reward"], ro["reward"])
    assert np.array_equal(eo["done"], ro["done"])
    assert np.array_equal(eo["obs"][:-1], ro["obs"][1:])
    assert np.array_equal(eo["obs"][-1], ro["obs_last"])
