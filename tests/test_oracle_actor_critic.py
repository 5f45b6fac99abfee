"""Pins of the oracle's actor-critic outputs (log pi of sampled actions, GAE, value head).

log pi: probabilities sum to one over the legal actions, softmax shift
invariance, illegal actions excluded, stable at extreme logits.
GAE: lambda = 0 is the one-step TD error, lambda = 1 the discounted Monte-Carlo
return minus the value (bootstrapped at the end), gamma = 0 is r - V; an episode
end cuts the dependence on everything after it; and the backward scan equals an
explicit double sum of discounted TD errors.
Value head: a zero-weight head with bias c reads V = c and leaves the
trajectory exactly as without it.
"""

import math

import numpy as np
import pytest

from oracle import actor_critic as ac
from oracle import lbf, rollout
from paper_2609_13716_amd import workloads


def test_log_prob_normalises_and_is_shift_invariant():
    rng = np.random.default_rng(0)
    for _ in range(50):
        x = rng.standard_normal(6) * 3
        lp = [ac.log_prob(x, a) for a in range(6)]
        assert abs(sum(math.exp(v) for v in lp) - 1.0) < 1e-12
        assert all(v <= 0 for v in lp)
        assert all(abs(ac.log_prob(x + 37.5, a) - lp[a]) < 1e-12 for a in range(6))


def test_log_prob_masks_and_extremes():
    x = np.array([0.3, 5.0, -1.0, 2.0])
    mask = [True, False, True, True]
    sub = np.array([0.3, -1.0, 2.0])
    ref = sub - (sub.max() + math.log(np.exp(sub - sub.max()).sum()))
    assert [ac.log_prob(x, a, mask) for a in (0, 2, 3)] == pytest.approx(list(ref), abs=1e-13)
    assert ac.log_prob([0.0] * 5, 3) == pytest.approx(math.log(1 / 5), abs=1e-15)
    assert ac.log_prob([1000.0, 0.0], 0) == pytest.approx(0.0, abs=1e-300)
    assert ac.log_prob([1000.0, 0.0], 1) == pytest.approx(-1000.0, rel=1e-15)


def _traj(T=7, n=3, A=2, seed=1, done_p=0.0):
    rng = np.random.default_rng(seed)
    r = rng.standard_normal((T, n)).astype(np.float32)
    d = (rng.random((T, n)) < done_p).astype(np.uint8)
    v = rng.standard_normal((T, n, A))
    vl = rng.standard_normal((n, A))
    return r, d, v, vl


def test_gae_special_cases():
    r, d, v, vl = _traj()
    T = r.shape[0]
    g = 0.9
    adv0, ret0 = ac.gae(r, d, v, vl, g, 0.0)
    nxt = np.concatenate([v[1:], vl[None]])
    assert np.allclose(adv0, r[:, :, None] + g * nxt - v, atol=1e-12)
    assert np.allclose(ret0, adv0 + v, atol=1e-15)
    adv1, _ = ac.gae(r, d, v, vl, g, 1.0)
    for t in range(T):
        mc = sum(g ** (k - t) * r[k] for k in range(t, T))[:, None] + g ** (T - t) * vl
        assert np.allclose(adv1[t], mc - v[t], atol=1e-12)
    advg0, _ = ac.gae(r, d, v, vl, 0.0, 0.7)
    assert np.allclose(advg0, r[:, :, None] - v, atol=1e-15)


def test_gae_episode_end_cuts_the_future():
    r, d, v, vl = _traj(T=9, n=4, seed=3)
    d[4, :] = 1  # every episode ends at the transition of step 4
    a, _ = ac.gae(r, d, v, vl, 0.95, 0.9)
    r2, v2, vl2 = r.copy(), v.copy(), vl + 100.0
    r2[5:] += 10.0
    v2[5:] -= 7.0
    b, _ = ac.gae(r2, d, v2, vl2, 0.95, 0.9)
    assert np.array_equal(a[:5], b[:5])
    assert np.allclose(a[4], r[4][:, None] - v[4], atol=1e-15)


def test_gae_equals_the_explicit_sum():
    r, d, v, vl = _traj(T=8, n=5, A=3, seed=7, done_p=0.25)
    g, lam = 0.97, 0.8
    adv, _ = ac.gae(r, d, v, vl, g, lam)
    T = r.shape[0]
    vnext = np.concatenate([v[1:], vl[None]])
    keep = (d == 0).astype(np.float64)[:, :, None]
    delta = r[:, :, None] + g * keep * vnext - v
    for t in range(T):
        tot = np.zeros_like(v[0])
        w = np.ones_like(v[0])
        for k in range(t, T):
            tot += w * delta[k]
            w = w * g * lam * keep[k]
        assert np.allclose(adv[t], tot, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_value_head_does_not_change_the_trajectory(dtype):
    cfg = lbf.Config(6, 6, 2, 2, 2, 3, max_steps=12)
    dims = (108, 16, 16, 6)
    ws, bs = workloads.policy_weights(dims, seed=5, bias_scale=0.3)
    wv = [w.copy() for w in ws]
    bv = [b.copy() for b in bs]
    wv[2] = np.concatenate([ws[2], np.zeros((1, 16), dtype=np.float32)])
    bv[2] = np.concatenate([bs[2], np.array([0.5], dtype=np.float32)])
    envs = list(range(4))
    a = rollout.rollout(lbf, cfg, 9, envs, 0, 20, ws, bs, dtype)
    b = rollout.rollout(lbf, cfg, 9, envs, 0, 20, wv, bv, dtype, value_head=True)
    for k in ("obs", "actions", "reward", "done", "logits", "obs_last"):
        assert np.array_equal(a[k], b[k]), k
    assert a["states"] == b["states"]
    assert (b["value"] == 0.5).all() and (b["value_last"] == 0.5).all()
    assert b["value"].shape == (20, 4, 2) and b["logp"].shape == (20, 4, 2)
    lp = b["logp"]
    for k in range(20):
        for i in range(4):
            for ag in range(2):
                assert lp[k, i, ag] == ac.log_prob(b["logits"][k, i, ag].astype(np.float32),
                                                   b["actions"][k, i, ag])
