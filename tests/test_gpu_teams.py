"""GPU parity of rollouts with heuristic LBF teammates (rollout_run_teams) against the oracle, through the C ABI.

Every heuristic kind drives some agent (kind = env index mod 11 on agent 1,
plus out-of-range kinds that fall back to the policy); agent 0 runs the
policy.  Env outputs and actions are bit-exact; a heuristic agent's logits
(0 for its action, -inf elsewhere) are exact; policy logits are within the
dtype tolerance; a strict run samples the oracle's actions from the GPU's
logits.
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


@pytest.mark.parametrize("cfgkw,hidden,dtype", [
    (dict(grid_h=7, grid_w=7, max_agent_level=1, max_food_level=2, const_levels=True), (64, 64), "bf16"),
    (dict(), (64, 64), "f32"),
    (dict(n_agents=3, n_food=4, max_agent_level=2, max_food_level=4), (32, 48), "bf16"),
    # the register-resident 128-wide kernels with teammates: the benchmarked 7x7 one and its 8x8 sibling
    (dict(grid_h=7, grid_w=7, max_agent_level=1, max_food_level=2, const_levels=True), (128, 128), "bf16"),
    (dict(), (128, 128), "bf16"),
])
def test_heuristic_teammates_parity(cfgkw, hidden, dtype):
    require_gpu()
    cfg = R.EnvConfig(n_envs=41, seed=13, env_base=9, max_steps=25, **cfgkw)
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    _note(f"rollout_run_teams {cfgkw} {hidden} {dtype}")
    tm = np.full((E, A), -1, dtype=np.int32)
    tm[:, 1] = np.arange(E) % 11
    tm[3, 1], tm[4, 1] = 11, -5  # out of range: the policy
    if A > 2:
        tm[:, 2] = (np.arange(E) * 5 + 2) % 11
    ws, bs = workloads.policy_weights((D, *hidden, 6), seed=77, bias_scale=0.2)
    pol = R.Policy(ws, bs, dtype)
    T = 60
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"), done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run_teams(cfg, pol, torch.from_numpy(tm).cuda(), state, 0, T, **out)
    torch.cuda.synchronize()
    g = {k: v.cpu() for k, v in out.items()}
    oc = oracle_cfg(cfg)
    env_ids = list(range(9, 9 + E))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook, teammates=tm)
    assert np.array_equal(g["obs"].float().numpy().astype(np.float64), ref["obs"])
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(g["obs_last"].float().numpy().astype(np.float64), ref["obs_last"])
    assert states_from_device(cfg, state) == ref["states"]
    heur = (tm >= 0) & (tm < 11)
    gl, rl_ = g["logits"].numpy().astype(np.float64), ref["logits"]
    assert np.array_equal(gl[:, heur], rl_[:, heur])
    assert_logits_close(gl[:, ~heur], rl_[:, ~heur], RTOL[dtype])
    assert ref["done"].any()
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, teammates=tm,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())


def test_teams_4096_sampled_envs():
    """The benchmarked teammate rollout at full size (7x7 constant levels, 4096 envs x 128 steps, policy
    147-128-128-6 bf16 on agent 0, heuristic kind e mod 11 on agent 1); the oracle replays 22 sampled envs,
    two of every heuristic kind."""
    require_gpu()
    name = "lbf7_teams_4096"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=0, **w["env"])
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, "bf16")
    T = w["n_steps"]
    tm = np.full((E, A), -1, dtype=np.int32)
    tm[:, 1] = np.arange(E) % 11
    _note(f"rollout_run_teams {name} full size")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"), done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run_teams(cfg, pol, torch.from_numpy(tm).cuda(), state, 0, T, **out)
    torch.cuda.synchronize()
    g = {k: v.cpu() for k, v in out.items()}
    sample = list(range(11)) + [1001 + k for k in range(11)]
    sample[-1] = E - 1  # the last env (kind 4095 mod 11 = 3)
    oc = oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"][:, sample].numpy(), cfg.seed, sample, RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, sample, 0, T, ws, bs, "bf16", action_hook=hook, teammates=tm[sample])
    assert np.array_equal(g["obs"][:, sample].float().numpy().astype(np.float64), ref["obs"])
    assert np.array_equal(g["reward"][:, sample].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"][:, sample].numpy(), ref["done"])
    assert np.array_equal(g["actions"][:, sample].numpy(), ref["actions"])
    assert np.array_equal(g["obs_last"][sample].float().numpy().astype(np.float64), ref["obs_last"])
    final = states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]
    gl, rl_ = g["logits"][:, sample].numpy().astype(np.float64), ref["logits"]
    assert np.array_equal(gl[:, :, 1], rl_[:, :, 1])
    assert_logits_close(gl[:, :, 0], rl_[:, :, 0], RTOL["bf16"])


@pytest.mark.parametrize("cfgkw,hidden", [
    (dict(grid_h=7, grid_w=7, max_agent_level=1, max_food_level=2, const_levels=True), (128, 128)),
    (dict(n_agents=3, n_food=4, max_agent_level=2, max_food_level=4), (32, 48)),
])
def test_split_teams_rollout_is_identical(cfgkw, hidden):
    """A rollout with nearest/farthest-agent teammates split in two calls equals one call: the second call
    recovers the running episodes' start cells from the reset draws (register-resident and generic kernels)."""
    require_gpu()
    cfg = R.EnvConfig(n_envs=70, seed=31, max_steps=17, **cfgkw)
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    tm = np.full((E, A), -1, dtype=np.int32)
    tm[:, 1] = 9 + np.arange(E) % 2
    if A > 2:
        tm[:, 2] = 10 - np.arange(E) % 2
    tmd = torch.from_numpy(tm).cuda()
    ws, bs = workloads.policy_weights((D, *hidden, 6), seed=8, bias_scale=0.2)
    pol = R.Policy(ws, bs, "bf16")

    def run(state, t0, T):
        out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
                   actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
                   logits=torch.empty(T, E, A, 6, device="cuda"),
                   reward=torch.empty(T, E, device="cuda"), done=torch.empty(T, E, dtype=torch.uint8, device="cuda"))
        R.rollout_run_teams(cfg, pol, tmd, state, t0, T, **out)
        torch.cuda.synchronize()
        return {k: v.cpu() for k, v in out.items()}

    s1 = R.new_state(cfg)
    R.rollout_init(cfg, s1)
    whole = run(s1, 0, 60)
    s2 = R.new_state(cfg)
    R.rollout_init(cfg, s2)
    a = run(s2, 0, 25)
    b = run(s2, 25, 35)
    for k in whole:
        assert torch.equal(whole[k], torch.cat([a[k], b[k]])), k
    assert torch.equal(s1.cpu(), s2.cpu())
    assert (whole["done"] != 0).any()
