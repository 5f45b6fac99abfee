"""Edge cases of the GPU path against the oracle, through the C ABI: a single env, episodes truncated at every
step (max_steps 1), one-step rollouts, and a batch of 65,537 envs (16 times the benchmark's, plus a ragged
workgroup) checked on sampled envs at both ends of the batch."""

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
