"""GPU parity of the mini Hanabi game (3 colours x 3 ranks, 18 cards, 16 actions, 278 features) against the
oracle, through the C ABI: deals, moves, knowledge, rewards, dones, legal masks and observations bit-exact;
rollouts with the mover's legal logits within the dtype tolerance (the rest exactly -inf), actions in
lockstep and strictly.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import hanabi as hn
from oracle import rollout
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import RTOL, NearTieLockstep, hn_oracle_cfg, hn_states_from_device, logit_tol, require_gpu

pytestmark = pytest.mark.gpu

D, NA = 278, 16
_TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


def _cfg(E, **kw):
    return R.hanabi_config(E, colours=3, ranks=3, **kw)


def test_mini_sizes():
    cfg = _cfg(4)
    assert R.rl_obs_dim(cfg) == D and R.rl_num_actions(cfg) == NA


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mini_init_matches_oracle(dtype):
    require_gpu()
    cfg = _cfg(70, seed=3, env_base=500)
    _note(f"mini hanabi init {dtype}")
    state = R.new_state(cfg)
    obs = torch.empty(70, 2, D, dtype=_TDT[dtype], device="cuda")
    legal = torch.empty(70, 2, NA, dtype=torch.uint8, device="cuda")
    R.rollout_init(cfg, state, obs, legal)
    torch.cuda.synchronize()
    ocfg = hn_oracle_cfg(cfg)
    ref = rollout.initial_states(hn, ocfg, cfg.seed, range(500, 570))
    assert hn_states_from_device(cfg, state) == ref
    ref_obs, ref_mask = rollout.observe_all(hn, ocfg, ref)
    assert np.array_equal(_obs_np(obs), ref_obs)
    assert np.array_equal(legal.cpu().numpy().astype(bool), ref_mask)


@pytest.mark.parametrize("E,T,max_steps,dtype", [(77, 90, 1000, "bf16"), (40, 70, 21, "f32")])
def test_mini_env_only_parity(E, T, max_steps, dtype):
    require_gpu()
    cfg = _cfg(E, max_steps=max_steps, seed=E, env_base=2 * E)
    _note(f"mini hanabi env-only E={E} T={T} {dtype}")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    rng = np.random.default_rng(T)
    acts = rng.integers(0, NA, size=(T, E, 2))
    bad = rng.random(acts.shape) < 0.1
    acts[bad] = rng.choice(np.array([-1, NA, 99]), size=int(bad.sum()))
    acts = acts.astype(np.int32)
    out = dict(obs_out=torch.empty(T, E, 2, D, dtype=_TDT[dtype], device="cuda"),
               reward=torch.empty(T, E, device="cuda"), done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               legal_out=torch.empty(T, E, 2, NA, dtype=torch.uint8, device="cuda"))
    R.rollout_step(cfg, state, 0, torch.as_tensor(acts).cuda(), **out)
    torch.cuda.synchronize()
    g = {k: v.cpu() for k, v in out.items()}
    ref = rollout.env_only(hn, hn_oracle_cfg(cfg), cfg.seed, range(cfg.env_base, cfg.env_base + E), 0, acts)
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["legal_out"].numpy().astype(bool), ref["mask"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    assert hn_states_from_device(cfg, state) == ref["states"]
    assert (g["done"].numpy() & 1).any()


@pytest.mark.parametrize("dims,dtype", [((D, 64, 64, NA), "f32"), ((D, 128, 128, NA), "bf16")])
def test_mini_rollout_lockstep_and_strict(dims, dtype):
    require_gpu()
    cfg = _cfg(37, seed=11, env_base=60)
    _note(f"mini hanabi rollout_run {dims} {dtype}")
    ws, bs = workloads.policy_weights(dims, seed=19, bias_scale=0.1)
    pol = R.Policy(ws, bs, dtype)
    T, E = 80, 37
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, 2, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, 2, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, 2, NA, device="cuda"), reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, 2, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run(cfg, pol, state, 0, T, **out)
    torch.cuda.synchronize()
    g = {k: v.cpu() for k, v in out.items()}
    ocfg = hn_oracle_cfg(cfg)
    ids = list(range(60, 60 + E))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, ids, RTOL[dtype])
    ref = rollout.rollout(hn, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype, action_hook=hook)
    assert np.array_equal(_obs_np(g["obs"]), ref["obs"])
    assert np.array_equal(g["reward"].numpy(), ref["reward"])
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(g["obs_last"]), ref["obs_last"])
    lg, mask = g["logits"].numpy().astype(np.float64), ref["mask"]
    assert np.all(np.isneginf(lg[~mask]))
    tol = np.broadcast_to(logit_tol(ref["logits"], RTOL[dtype]), mask.shape)
    assert np.all(np.abs(lg[mask] - ref["logits"][mask]) <= tol[mask])
    assert hn_states_from_device(cfg, state) == ref["states"]
    assert (g["done"].numpy() == 1).any()
    strict = rollout.rollout(hn, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())
