"""Edge cases of the GPU path against the oracle, through the C ABI: a single env, episodes truncated at every
step (max_steps 1), one-step rollouts, and a batch of 65,537 envs (16 times the benchmark's, plus a ragged
workgroup) checked on sampled envs at both ends of the batch; for Hanabi and the kitchen, single envs and
ragged tiles with every game truncated after one or two moves (a re-deal at nearly every move)."""

import sys

import numpy as np
import pytest
import torch

from oracle import lbf, rollout, s5
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import RTOL, NearTieLockstep, assert_logits_close, oracle_cfg, require_gpu, states_from_device

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run(cfg, pol, T):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"), reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run(cfg, pol, state, 0, T, **out)
    torch.cuda.synchronize()
    return state, out


def _check(cfg, g, idx, env_ids, ws, bs, dtype, T, state=None):
    oc = oracle_cfg(cfg)
    # select on the host (bounds-checked): [T, E, ...] outputs along dim 1, obs_last [E, A, D] along dim 0
    ga = {k: (v.cpu()[idx] if k == "obs_last" else v.cpu()[:, idx]) for k, v in g.items()}
    hook = NearTieLockstep(ga["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook)
    assert np.array_equal(ga["obs"].float().numpy().astype(np.float64), ref["obs"])
    assert np.array_equal(ga["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(ga["done"].numpy(), ref["done"])
    assert np.array_equal(ga["actions"].numpy(), ref["actions"])
    assert np.array_equal(ga["obs_last"].float().numpy().astype(np.float64), ref["obs_last"])
    assert_logits_close(ga["logits"].numpy(), ref["logits"], RTOL[dtype])
    return ref


@pytest.mark.parametrize("hidden,dtype", [((128, 128), "bf16"), ((128, 128), "f32"), ((48, 32), "bf16")])
def test_single_env_and_every_step_truncated(hidden, dtype):
    require_gpu()
    for E, max_steps, T in ((1, 50, 60), (1, 1, 5), (9, 1, 7), (1, 50, 1)):
        cfg = R.EnvConfig(n_envs=E, seed=3, env_base=11, max_steps=max_steps)
        _note(f"edge E={E} max_steps={max_steps} T={T} {hidden} {dtype}")
        ws, bs = workloads.policy_weights((192, *hidden, 6), seed=21, bias_scale=0.1)
        pol = R.Policy(ws, bs, dtype)
        state, g = _run(cfg, pol, T)
        ref = _check(cfg, g, slice(None), list(range(11, 11 + E)), ws, bs, dtype, T)
        assert states_from_device(cfg, state) == ref["states"]
        if max_steps == 1:
            assert (ref["done"] != 0).all()


def test_65537_envs_sampled():
    require_gpu()
    E, T = 65537, 12
    cfg = R.EnvConfig(n_envs=E, seed=9)
    _note(f"edge E={E} T={T}")
    ws, bs = workloads.policy_weights((192, 128, 128, 6), seed=31, bias_scale=0.1)
    pol = R.Policy(ws, bs, "bf16")
    state, g = _run(cfg, pol, T)
    idx = np.array([0, 1, 7, 8, 32767, 40000, 65528, 65535, 65536])
    _check(cfg, g, torch.as_tensor(idx), [int(i) for i in idx], ws, bs, "bf16", T)


def test_s5_single_env():
    require_gpu()
    cfg = R.EnvConfig(n_envs=1, seed=5, max_steps=7)
    D = R.rl_obs_dim(cfg)
    cont = workloads.s5_params(D, 64, 32, 128, 6, seed=4)
    pol = R.S5Policy(cont)
    T = 20
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    carry = torch.zeros(2, 2, 32, device="cuda")
    out = dict(obs=torch.empty(T, 1, 2, D, dtype=torch.bfloat16, device="cuda"),
               actions=torch.empty(T, 1, 2, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, 1, 2, 6, device="cuda"), reward=torch.empty(T, 1, device="cuda"),
               done=torch.empty(T, 1, dtype=torch.uint8, device="cuda"),
               value=torch.empty(T, 1, 2, device="cuda"), value_last=torch.empty(1, 2, device="cuda"))
    R.rollout_run_s5(cfg, pol, state, carry, 0, T, **out)
    torch.cuda.synchronize()
    g = {k: v.cpu() for k, v in out.items()}
    oc = oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, [0], RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, [0], 0, T, None, None, "bf16", action_hook=hook,
                          recurrent=s5.from_continuous(cont))
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert ref["done"].any()
    lg_ref = np.concatenate([ref["logits"], ref["value"][..., None]], axis=-1)
    lg_gpu = np.concatenate([g["logits"].numpy(), g["value"].numpy()[..., None]], axis=-1)
    assert_logits_close(lg_gpu, lg_ref, RTOL["bf16"])


# ------------------------------------------------- Hanabi and the kitchen

@pytest.mark.parametrize("E,max_steps,dtype", [(1, 1, "f32"), (5, 2, "bf16"), (9, 1, "bf16")])
def test_hanabi_env_only_every_move_truncated(E, max_steps, dtype):
    """Env-only Hanabi where every game is truncated after one or two moves, so the env wave re-deals
    every tile's games at (nearly) every move; a single env and ragged workgroup tiles."""
    require_gpu()
    from oracle import hanabi as hn
    from parity import hn_oracle_cfg, hn_states_from_device
    from test_gpu_hanabi import _actions, _check_env_only, _env_only_gpu
    cfg = R.hanabi_config(E, max_steps=max_steps, seed=E + 40, env_base=7)
    _note(f"hanabi env-only E={E} max_steps={max_steps} {dtype}")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    T = 24
    actions = _actions(T, E, seed=E + 3)
    g = _env_only_gpu(cfg, state, 0, actions, dtype)
    ref = rollout.env_only(hn, hn_oracle_cfg(cfg), cfg.seed, range(7, 7 + E), 0, actions)
    _check_env_only(cfg, g, ref, state)
    assert (g["done"].numpy() & 2).sum() >= T * E // max_steps - E


@pytest.mark.parametrize("E,max_steps,dtype", [(1, 1, "bf16"), (17, 2, "f32")])
def test_hanabi_rollout_every_move_truncated(E, max_steps, dtype):
    """The fused Hanabi rollout with every game truncated after one or two moves (a re-deal of most of the
    workgroup's games at every move), a single env and a ragged second workgroup."""
    require_gpu()
    from oracle import hanabi as hn
    from parity import hn_oracle_cfg, hn_states_from_device
    from test_gpu_hanabi import D, NA, _check_traj, _run_gpu
    cfg = R.hanabi_config(E, max_steps=max_steps, seed=E + 50, env_base=11)
    _note(f"hanabi rollout_run E={E} max_steps={max_steps} {dtype}")
    dims = (D, 64, 64, NA)
    ws, bs = workloads.policy_weights(dims, seed=5, bias_scale=0.1)
    pol = R.Policy(ws, bs, dtype)
    T = 20
    state, g = _run_gpu(cfg, pol, T)
    ids = list(range(11, 11 + E))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, ids, RTOL[dtype])
    ref = rollout.rollout(hn, hn_oracle_cfg(cfg), cfg.seed, ids, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL[dtype])
    assert hn_states_from_device(cfg, state) == ref["states"]


def test_overcooked_single_env_every_step_truncated():
    """The fused kitchen rollout with one env whose episode is truncated at every step."""
    require_gpu()
    from oracle import overcooked as oc
    from parity import oc_oracle_cfg, oc_states_from_device
    from test_gpu_overcooked import D, NA, _check_traj, _run_gpu, _tuples
    cfg = R.overcooked_config(1, cook_time=3, max_steps=1, seed=4, env_base=2)
    _note("overcooked rollout_run E=1 max_steps=1")
    dims = (D, 64, 64, NA)
    ws, bs = workloads.policy_weights(dims, seed=6, bias_scale=0.1)
    pol = R.Policy(ws, bs, "bf16")
    T = 16
    state, g = _run_gpu(cfg, pol, T)
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, [2], RTOL["bf16"])
    ref = rollout.rollout(oc, oc_oracle_cfg(cfg), cfg.seed, [2], 0, T, ws, bs, "bf16", action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL["bf16"])
    assert (g["done"].numpy() & 2).all()
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref["states"])
