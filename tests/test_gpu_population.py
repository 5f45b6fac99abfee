"""GPU parity of the population rollout (rollout_run_pop) against the oracle, through the C ABI.

Agent a of env e acts with policy policy_index[e, a] of a population (the ego
agent and its teammates of the ad hoc teamwork objective).  Trajectories are
checked like rollout_run's: bit-exact env outputs, logits within the dtype's
tolerance, actions in lockstep (certified near-ties adopted) and strictly
(the oracle sampling from the GPU's logits).  GPU-internal checks: a
one-policy population is rollout_run with that policy, and every row's logits
are policy_forward with the row's own policy (both bit-exact, on layer shapes
that take the same MFMA path in each call).
"""

import sys

import numpy as np
import pytest
import torch

from oracle import lbf, rollout
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import RTOL, NearTieLockstep, assert_logits_close, oracle_cfg, require_gpu, states_from_device

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _pop(dims, n, seed):
    ws, bs = [], []
    for p in range(n):
        w, b = workloads.policy_weights(dims, seed=seed + 17 * p, bias_scale=0.2)
        ws.append(w)
        bs.append(b)
    return ws, bs


def _run(cfg, pop, idx, T):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pop.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pop.torch_dtype, device="cuda"))
    R.rollout_run_pop(cfg, pop, torch.as_tensor(idx, dtype=torch.int32).cuda(), state, 0, T, **out)
    torch.cuda.synchronize()
    return state, {k: v.cpu() for k, v in out.items()}


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("cfgkw,dims,npol,T,dtype", [
    (dict(n_envs=37), (192, 64, 64, 6), 3, 60, "f32"),
    (dict(n_envs=37), (192, 64, 64, 6), 3, 60, "bf16"),
    (dict(n_envs=21, grid_h=12, grid_w=12, n_agents=3, n_food=6, max_agent_level=3, max_food_level=6,
          max_steps=20), (432, 32, 48, 6), 5, 40, "bf16"),
])
def test_population_rollout_parity(cfgkw, dims, npol, T, dtype):
    require_gpu()
    cfg = R.EnvConfig(seed=17, env_base=5, **cfgkw)
    _note(f"rollout_run_pop {cfgkw} {dims} P={npol} {dtype}")
    E, A = cfg.n_envs, cfg.n_agents
    ws, bs = _pop(dims, npol, seed=300)
    rng = np.random.default_rng(npol + E)
    idx = rng.integers(0, npol, size=(E, A))
    idx[0, 0], idx[1, -1], idx[2, 0] = -1, npol, 1000  # out of range: policy 0
    pop = R.Population(ws, bs, dtype)
    state, g = _run(cfg, pop, idx, T)
    oc = oracle_cfg(cfg)
    env_ids = list(range(5, 5 + E))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook, policy_index=idx)
    assert np.array_equal(_obs_np(g["obs"]), ref["obs"])
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(g["obs_last"]), ref["obs_last"])
    assert_logits_close(g["logits"].numpy(), ref["logits"], RTOL[dtype])
    assert states_from_device(cfg, state) == ref["states"]
    assert ref["done"].any()
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, policy_index=idx,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_one_policy_population_is_rollout_run(dtype):
    """Every agent on policy 1 of a population == rollout_run with that policy (generic-kernel shape)."""
    require_gpu()
    cfg = R.EnvConfig(n_envs=45, seed=3)
    dims = (192, 48, 32, 6)
    ws, bs = _pop(dims, 3, seed=11)
    T = 40
    _, g = _run(cfg, R.Population(ws, bs, dtype), np.ones((45, 2), dtype=np.int64), T)
    pol = R.Policy(ws[1], bs[1], dtype)
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    ref = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"), reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"))
    R.rollout_run(cfg, pol, state, 0, T, **ref)
    torch.cuda.synchronize()
    for k in ref:
        assert torch.equal(g[k], ref[k].cpu()), k


def test_rows_use_their_own_policy():
    """Each row's logits are exactly policy_forward of its observation with its own policy."""
    require_gpu()
    cfg = R.EnvConfig(n_envs=64, seed=8)
    dims = (192, 48, 32, 6)
    ws, bs = _pop(dims, 4, seed=90)
    idx = np.array([[e % 4, (e // 16) % 4] for e in range(64)])
    _, g = _run(cfg, R.Population(ws, bs, "bf16"), idx, 20)
    obs = g["obs"]  # [T, E, A, D]
    for p in range(4):
        sel = torch.as_tensor(idx == p)
        rows = obs[:, sel].reshape(-1, dims[0]).cuda()
        pf = R.policy_forward(R.Policy(ws[p], bs[p], "bf16"), rows).cpu()
        assert torch.equal(pf, g["logits"][:, sel].reshape(-1, 6)), p
