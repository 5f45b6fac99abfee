"""GPU parity of the recurrent S5 actor-critic rollout (rollout_run_s5, rl_s5_discretize) against the oracle.

Discretisation: float64 on the device rounded once to float32, so within a
few float32 ulps of the oracle's float64 values (1e-6 relative to the
array's largest entry).  Rollouts are checked like rollout_run_ac's: env
outputs bit-exact, actions in lockstep (certified near-ties adopted) and
strictly (the oracle sampling from the GPU's logits), logits and values
within the bf16 tolerance (2e-2 of the row scale, the value checked as one
more output of its row), log pi against the oracle's float64 log-softmax of
the GPU's logits (1e-5 relative plus 1e-6), and the carried S5 state at the
end within 2e-2 of its row scale (the state is float32 on the device and
float64 in the oracle, fed by bf16 encoder outputs on both sides).
A rollout split into two calls is bit-identical to one call.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import actor_critic, lbf, rollout, s5
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import RTOL, NearTieLockstep, assert_logits_close, oracle_cfg, require_gpu, states_from_device

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_discretize_matches_the_oracle():
    require_gpu()
    P, H = 128, 96
    cont = workloads.s5_params(192, H, P, 128, 6, seed=3)
    pol = R.S5Policy(cont)
    torch.cuda.synchronize()
    lbar, bbar = s5.discretize(cont["lam_re"], cont["lam_im"], cont["log_dt"], cont["b_re"], cont["b_im"])
    g_l = pol.lambda_bar.cpu().numpy().astype(np.float64)
    g_b = pol.b_bar.cpu().numpy().astype(np.float64)
    for got, ref in ((g_l[0], lbar.real), (g_l[1], lbar.imag), (g_b[0], bbar.real), (g_b[1], bbar.imag)):
        assert np.abs(got - ref).max() <= 1e-6 * np.abs(ref).max()
    assert (np.abs(lbar) < 1).all()


def _run(cfg, pol, T, t0=0, state=None, carry=None):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    if state is None:
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
    if carry is None:
        carry = torch.full((E * A, 2, pol.P), 7.0, device="cuda")  # every agent starts an episode at t = 0
    out = dict(obs=torch.empty(T, E, A, D, dtype=torch.bfloat16, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=torch.bfloat16, device="cuda"),
               value=torch.empty(T, E, A, device="cuda"), logp=torch.empty(T, E, A, device="cuda"),
               value_last=torch.empty(E, A, device="cuda"))
    R.rollout_run_s5(cfg, pol, state, carry, t0, T, **out)
    torch.cuda.synchronize()
    return state, carry, {k: v.cpu() for k, v in out.items()}


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("cfgkw,sizes,T", [
    (dict(n_envs=37, max_steps=15), (64, 32, 128), 40),
    (dict(n_envs=64, max_steps=8), (128, 128, 1024), 12),
    # the benchmarked widths over 600 agent rows: five 128-row head tiles, the last one ragged (88 rows)
    (dict(n_envs=300, max_steps=20), (128, 128, 1024), 60),
])
def test_s5_rollout_parity(cfgkw, sizes, T):
    require_gpu()
    H, P, F = sizes
    cfg = R.EnvConfig(seed=29, env_base=3, **cfgkw)
    D = R.rl_obs_dim(cfg)
    _note(f"rollout_run_s5 {cfgkw} H={H} P={P} F={F} T={T}")
    cont = workloads.s5_params(D, H, P, F, 6, seed=41)
    pol = R.S5Policy(cont)
    state, carry, g = _run(cfg, pol, T)
    net = s5.from_continuous(cont)
    oc = oracle_cfg(cfg)
    env_ids = list(range(3, 3 + cfg.n_envs))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, None, None, "bf16", action_hook=hook, recurrent=net)
    assert np.array_equal(_obs_np(g["obs"]), ref["obs"])
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(g["obs_last"]), ref["obs_last"])
    assert states_from_device(cfg, state) == ref["states"]
    assert ref["done"].any()
    lg_ref = np.concatenate([ref["logits"], ref["value"][..., None]], axis=-1)
    lg_gpu = np.concatenate([g["logits"].numpy(), g["value"].numpy()[..., None]], axis=-1)
    assert_logits_close(lg_gpu, lg_ref, RTOL["bf16"])
    # V(o_last) is checked as the last output of its row, scaled like the steps' values by the row's logits
    last_ref = np.concatenate([ref["logits_last"], ref["value_last"][..., None]], axis=-1)
    last_gpu = np.concatenate([ref["logits_last"], g["value_last"].numpy()[..., None]], axis=-1)
    assert_logits_close(last_gpu, last_ref, RTOL["bf16"])
    c = carry.cpu().numpy().astype(np.float64)
    assert_logits_close(c[:, 0], ref["carry"].real, RTOL["bf16"])
    assert_logits_close(c[:, 1], ref["carry"].imag, RTOL["bf16"])
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, None, None, "bf16", recurrent=net,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())
    lp = np.array([[[actor_critic.log_prob(g["logits"][k, i, a].numpy(), int(g["actions"][k, i, a]))
                     for a in range(cfg.n_agents)] for i in range(cfg.n_envs)] for k in range(T)])
    assert np.allclose(g["logp"].numpy(), lp, rtol=1e-5, atol=1e-6)


def test_s5_split_rollout_is_identical():
    require_gpu()
    cfg = R.EnvConfig(n_envs=50, seed=5, max_steps=11)
    cont = workloads.s5_params(R.rl_obs_dim(cfg), 64, 48, 256, 6, seed=9)
    pol = R.S5Policy(cont)
    s1, c1, a = _run(cfg, pol, 24)
    s2, c2, b1 = _run(cfg, pol, 10)
    s2, c2, b2 = _run(cfg, pol, 14, t0=10, state=s2, carry=c2)
    for k in ("obs", "actions", "logits", "reward", "done", "value", "logp"):
        assert torch.equal(a[k], torch.cat([b1[k], b2[k]])), k
    for k in ("obs_last", "value_last"):
        assert torch.equal(a[k], b2[k]), k
    assert torch.equal(s1, s2) and torch.equal(c1, c2)


def test_s5_rollout_4096_sampled_envs():
    """The benchmarked S5 rollout at full size (4096 envs x 128 steps, 8192 agent rows = 64 head tiles, the
    bench's parameters); the oracle replays 12 sampled envs, whose rows lie in different head tiles and
    workgroups."""
    require_gpu()
    name = "lbf8_4096_s5"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=0, **w["env"])
    D, nA = R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    x = w["s5"]
    cont = workloads.s5_params(D, x["d_model"], x["d_state"], x["head_width"], nA, seed=1000)
    pol = R.S5Policy(cont)
    T = w["n_steps"]
    _note(f"rollout_run_s5 {name} full size")
    state, carry, g = _run(cfg, pol, T)
    sample = [0, 1, 63, 64, 65, 1000, 2047, 2048, 3333, 4031, 4094, 4095]
    net = s5.from_continuous(cont)
    oc = oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"][:, sample].numpy(), cfg.seed, sample, RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, sample, 0, T, None, None, "bf16", action_hook=hook, recurrent=net)
    assert np.array_equal(_obs_np(g["obs"][:, sample]), ref["obs"])
    assert np.array_equal(g["reward"][:, sample].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"][:, sample].numpy(), ref["done"])
    assert np.array_equal(g["actions"][:, sample].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(g["obs_last"][sample]), ref["obs_last"])
    final = states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]
    lg_ref = np.concatenate([ref["logits"], ref["value"][..., None]], axis=-1)
    lg_gpu = np.concatenate([g["logits"][:, sample].numpy(), g["value"][:, sample].numpy()[..., None]], axis=-1)
    assert_logits_close(lg_gpu, lg_ref, RTOL["bf16"])
    last_ref = np.concatenate([ref["logits_last"], ref["value_last"][..., None]], axis=-1)
    last_gpu = np.concatenate([ref["logits_last"], g["value_last"][sample].numpy()[..., None]], axis=-1)
    assert_logits_close(last_gpu, last_ref, RTOL["bf16"])
    rows = np.array([[e * cfg.n_agents + a for a in range(cfg.n_agents)] for e in sample]).reshape(-1)
    c = carry.cpu().numpy().astype(np.float64)[rows]
    assert_logits_close(c[:, 0], ref["carry"].real, RTOL["bf16"])
    assert_logits_close(c[:, 1], ref["carry"].imag, RTOL["bf16"])
    # properties over every env
    done = g["done"].numpy()
    assert set(np.unique(done)) <= {0, 1, 2, 3}
    assert ((done != 0).sum(axis=0) >= 2).all()
    assert torch.isfinite(g["logits"]).all() and torch.isfinite(g["value"]).all()
