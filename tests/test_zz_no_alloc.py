"""The allocation-free S5 rollout (rollout_run_s5_noalloc) against rollout_run_s5 with a caller-owned workspace.

Both run the same kernels on the same inputs, so every output (trajectory,
values, log pi, carried state, env state) must be bit-identical.  Two calls
in a row, the second on a smaller batch, check that the built-in scratch
keeps no state between calls that matters.  A batch whose workspace exceeds
the scratch is rejected before any launch.
"""

import sys

import numpy as np
import pytest
import torch

from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import require_gpu

pytestmark = pytest.mark.gpu


def _outs(cfg, T):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    f = dict(device="cuda")
    return dict(obs=torch.empty(T, E, A, D, dtype=torch.bfloat16, **f),
                actions=torch.empty(T, E, A, dtype=torch.int32, **f), logits=torch.empty(T, E, A, 6, **f),
                reward=torch.empty(T, E, **f), done=torch.empty(T, E, dtype=torch.uint8, **f),
                obs_last=torch.empty(E, A, D, dtype=torch.bfloat16, **f), value=torch.empty(T, E, A, **f),
                logp=torch.empty(T, E, A, **f), value_last=torch.empty(E, A, **f))


def _both(cfg, pol, T):
    E, A = cfg.n_envs, cfg.n_agents
    res = []
    for noalloc in (False, True):
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
        carry = torch.zeros(E * A, 2, pol.P, device="cuda")
        out = _outs(cfg, T)
        if noalloc:
            R.rollout_run_s5_noalloc(cfg, pol, state, carry, 0, T, **out)
        else:
            R.rollout_run_s5(cfg, pol, state, carry, 0, T, **out)
        torch.cuda.synchronize()
        res.append((state.cpu(), carry.cpu(), {k: v.cpu() for k, v in out.items()}))
    return res


def test_noalloc_matches_workspace_rollout_twice():
    require_gpu()
    cont = workloads.s5_params(192, 128, 128, 1024, 6, seed=71)
    pol = R.S5Policy(cont)
    for E, T in ((300, 24), (70, 16)):  # the second call on a smaller batch
        print(f"rollout_run_s5_noalloc vs rollout_run_s5: {E} envs x {T} steps", flush=True)
        sys.stdout.flush()
        cfg = R.EnvConfig(n_envs=E, seed=19, env_base=2, max_steps=10)
        (s_ws, c_ws, o_ws), (s_na, c_na, o_na) = _both(cfg, pol, T)
        assert torch.equal(s_ws, s_na)
        assert torch.equal(c_ws, c_na)
        for k in o_ws:
            assert torch.equal(o_ws[k], o_na[k]), k
        assert o_ws["done"].numpy().any()


def test_noalloc_rejects_oversize_batch():
    require_gpu()
    cont = workloads.s5_params(192, 128, 128, 4096, 6, seed=3)
    pol = R.S5Policy(cont)
    cfg = R.EnvConfig(n_envs=2048, seed=1)
    need = R.s5_workspace_bytes(cfg, pol)
    assert need > 80 << 20
    state = R.new_state(cfg)
    carry = torch.zeros(cfg.n_envs * 2, 2, pol.P, device="cuda")
    with pytest.raises(R.RolloutError, match="scratch"):
        R.rollout_run_s5_noalloc(cfg, pol, state, carry, 0, 4)
