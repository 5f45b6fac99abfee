"""GPU parity of two-player Hanabi against the CPU oracle, through the C ABI.

Deals, moves, knowledge, rewards, dones, legal masks and observations must be
bit-exact.  In the fused rollout only the mover's policy row counts: its legal
logits must agree with the oracle's float64 logits within 1e-4 (float32) /
2e-2 (bf16), every illegal logit (and every logit of the other player) is
-inf, and actions are checked in lockstep and strictly as for the other envs.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import hanabi as hn
from oracle import rollout
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import (RTOL, NearTieLockstep, hn_oracle_cfg, hn_states_from_device, hn_states_to_device, logit_tol,
                    require_gpu)

pytestmark = pytest.mark.gpu

D, NA = 658, 20
_TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_init_matches_oracle(dtype):
    require_gpu()
    cfg = R.hanabi_config(300, seed=7, env_base=1000)  # ragged last tile
    _note(f"hanabi init {dtype}")
    state = R.new_state(cfg)
    obs = torch.empty(300, 2, D, dtype=_TDT[dtype], device="cuda")
    legal = torch.empty(300, 2, NA, dtype=torch.uint8, device="cuda")
    R.rollout_init(cfg, state, obs, legal)
    torch.cuda.synchronize()
    ocfg = hn_oracle_cfg(cfg)
    ref = rollout.initial_states(hn, ocfg, cfg.seed, range(1000, 1300))
    assert hn_states_from_device(cfg, state) == ref
    ref_obs, ref_mask = rollout.observe_all(hn, ocfg, ref)
    assert np.array_equal(_obs_np(obs), ref_obs)
    assert np.array_equal(legal.cpu().numpy().astype(bool), ref_mask)


def _actions(T, E, seed, p_illegal=0.1):
    """Actions for both players: mostly uniform over 0..19 (often illegal), some out of range."""
    rng = np.random.default_rng(seed)
    a = rng.integers(0, NA, size=(T, E, 2))
    bad = rng.random(a.shape) < p_illegal
    a[bad] = rng.choice(np.array([-1, 20, 99, 1 << 20]), size=int(bad.sum()))
    return a.astype(np.int32)


def _env_only_gpu(cfg, state, t0, actions, dtype):
    T, E = actions.shape[:2]
    out = dict(obs_out=torch.empty(T, E, 2, D, dtype=_TDT[dtype], device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               legal_out=torch.empty(T, E, 2, NA, dtype=torch.uint8, device="cuda"))
    R.rollout_step(cfg, state, t0, torch.as_tensor(actions).cuda(), **out)
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in out.items()}


def _check_env_only(cfg, g, ref, state):
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["legal_out"].numpy().astype(bool), ref["mask"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    assert hn_states_from_device(cfg, state) == ref["states"]


@pytest.mark.parametrize("E,T,max_steps,dtype", [(200, 120, 1000, "f32"), (77, 60, 23, "bf16"), (5, 40, 1000, "bf16")])
def test_env_only_parity(E, T, max_steps, dtype):
    require_gpu()
    cfg = R.hanabi_config(E, max_steps=max_steps, seed=E + 1, env_base=3 * E)
    _note(f"hanabi env-only E={E} T={T} max_steps={max_steps} {dtype}")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    actions = _actions(T, E, seed=T)
    g = _env_only_gpu(cfg, state, 0, actions, dtype)
    ref = rollout.env_only(hn, hn_oracle_cfg(cfg), cfg.seed, range(cfg.env_base, cfg.env_base + E), 0, actions)
    _check_env_only(cfg, g, ref, state)
    done = g["done"].numpy()
    assert (done & 1).any()
    if max_steps < T:
        assert (done & 2).any()


def _near_end_states(ocfg, seed, ids, rng):
    """Oracle games played by discarding whenever tokens allow (else the lowest legal hint) for up to 60..84
    moves, stopping before the game ends: no life is lost and the deck is nearly or fully drawn."""
    out = []
    for e in ids:
        s = hn.reset(ocfg, seed, e, 0)
        for t in range(int(rng.integers(60, 85))):
            m = hn.legal_mask(ocfg, s, s.cur)
            a = [0, 0]
            a[s.cur] = 0 if m[0] else m.index(True, 10) if any(m[10:]) else m.index(True)
            nxt, _, d = hn.step(ocfg, seed, e, t, s, a)
            if d:
                break
            s = nxt
        out.append(s)
    return out


def test_env_only_last_round_and_resume():
    """Games that run the deck out (final round, plays with nothing to draw), resumed from oracle states."""
    require_gpu()
    cfg = R.hanabi_config(48, seed=21)
    ocfg = hn_oracle_cfg(cfg)
    ids = list(range(48))
    pre = _near_end_states(ocfg, cfg.seed, ids, np.random.default_rng(1))
    assert sum(s.next_card == 50 for s in pre) >= 5 and all(s.lives == 3 for s in pre)
    state = hn_states_to_device(cfg, pre)
    # alternate rank-1 hints and slot-0 discards (illegal ones fall back to the lowest legal action)
    actions = np.zeros((40, 48, 2), np.int32)
    actions[0::2] = 15
    g = _env_only_gpu(cfg, state, 100, actions, "f32")
    ref = rollout.env_only(hn, ocfg, cfg.seed, ids, 100, actions, states=pre)
    _check_env_only(cfg, g, ref, state)
    assert (g["done"].numpy() == 1).sum() >= 40  # nearly every game reached its end


def test_env_only_4096_sampled_envs():
    """Env-only steps at the full 4096-env, 80-step size in one launch (bf16 observations); sampled envs,
    across workgroup tiles, replayed in the oracle."""
    require_gpu()
    w = workloads.WORKLOADS["hn_4096"]
    cfg = R.hanabi_config(w["n_envs"], seed=5, **w["env"])
    E, T = cfg.n_envs, 80
    _note(f"hanabi env-only E={E} T={T} bf16 (sampled)")
    sample = [0, 1, 2, 3, 4, 5, 7, 8, 1023, 1024, 2050, 3071, 4092, 4095]
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    actions = _actions(T, E, seed=17)
    out = dict(obs_out=torch.empty(T, E, 2, D, dtype=torch.bfloat16, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               legal_out=torch.empty(T, E, 2, NA, dtype=torch.uint8, device="cuda"))
    R.rollout_step(cfg, state, 0, torch.as_tensor(actions).cuda(), **out)
    torch.cuda.synchronize()
    g = {k: v[:, sample].cpu() for k, v in out.items()}
    ref = rollout.env_only(hn, hn_oracle_cfg(cfg), cfg.seed, sample, 0, actions[:, sample])
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["legal_out"].numpy().astype(bool), ref["mask"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    final = hn_states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]


# ------------------------------------------------------------- full rollout

def _run_gpu(cfg, pol, T, t0=0, state=None):
    E = cfg.n_envs
    if state is None:
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, 2, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, 2, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, 2, NA, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, 2, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run(cfg, pol, state, t0, T, **out)
    torch.cuda.synchronize()
    return state, {k: v.cpu() for k, v in out.items()}


def _check_masked_logits(gpu, ref, mask, rtol):
    """Legal logits within tolerance of the oracle's; illegal ones (the non-mover's included) exactly -inf."""
    gpu = np.asarray(gpu, np.float64)
    assert np.all(np.isneginf(gpu[~mask]))
    tol = np.broadcast_to(logit_tol(ref, rtol), ref.shape)
    err = np.abs(gpu[mask] - ref[mask])
    assert np.all(err <= tol[mask]), f"worst excess {np.max(err - tol[mask]):.3g}"


def _check_traj(gpu, ref, env_idx, rtol):
    assert np.array_equal(_obs_np(gpu["obs"][:, env_idx]), ref["obs"])
    assert np.array_equal(gpu["reward"][:, env_idx].numpy(), ref["reward"])
    assert np.array_equal(gpu["done"][:, env_idx].numpy(), ref["done"])
    assert np.array_equal(gpu["actions"][:, env_idx].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(gpu["obs_last"][env_idx]), ref["obs_last"])
    _check_masked_logits(gpu["logits"][:, env_idx].numpy(), ref["logits"], ref["mask"], rtol)


@pytest.mark.parametrize("dims,dtype", [((D, 64, 64, NA), "f32"), ((D, 64, 64, NA), "bf16"),
                                        ((D, 512, 512, NA), "bf16"), ((D, 512, 512, NA), "f32")])
def test_rollout_run_small_lockstep_and_strict(dims, dtype):
    require_gpu()
    cfg = R.hanabi_config(21, seed=9, env_base=40)
    _note(f"hanabi rollout_run {dims} {dtype}")
    ws, bs = workloads.policy_weights(dims, seed=31, bias_scale=0.1)
    pol = R.Policy(ws, bs, dtype)
    T = 90
    state, g = _run_gpu(cfg, pol, T)
    ocfg = hn_oracle_cfg(cfg)
    ids = list(range(40, 61))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, ids, RTOL[dtype])
    ref = rollout.rollout(hn, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL[dtype])
    assert hn_states_from_device(cfg, state) == ref["states"]
    assert (g["done"].numpy() == 1).any()
    if dtype == "f32":
        assert hook.mismatches == 0
    strict = rollout.rollout(hn, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())


def test_rollout_run_4096_sampled_envs_and_resume():
    """The 4096-env Hanabi workload at full size in two launches of 40 steps; 10 sampled envs replayed."""
    require_gpu()
    name = "hn_4096"
    w = workloads.WORKLOADS[name]
    cfg = R.hanabi_config(w["n_envs"], seed=0, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, "bf16")
    E = cfg.n_envs
    sample = [0, 1, 15, 16, 1001, 2047, 2048, 3000, 4080, 4095]
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    gs = []
    for t0 in (0, 40):
        _note(f"rollout_run {name} bf16, steps {t0}..{t0 + 39}")
        out = dict(actions=torch.empty(40, E, 2, dtype=torch.int32, device="cuda"),
                   logits=torch.empty(40, E, 2, NA, device="cuda"),
                   reward=torch.empty(40, E, device="cuda"),
                   done=torch.empty(40, E, dtype=torch.uint8, device="cuda"))
        R.rollout_run(cfg, pol, state, t0, 40, **out)
        torch.cuda.synchronize()
        gs.append({k: v[:, sample].cpu().numpy() for k, v in out.items()})
    g = {k: np.concatenate([gs[0][k], gs[1][k]]) for k in gs[0]}
    ocfg = hn_oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"], cfg.seed, sample, RTOL["bf16"])
    ref = rollout.rollout(hn, ocfg, cfg.seed, sample, 0, 80, ws, bs, "bf16", action_hook=hook)
    assert np.array_equal(g["reward"], ref["reward"])
    assert np.array_equal(g["done"], ref["done"])
    assert np.array_equal(g["actions"], ref["actions"])
    _check_masked_logits(g["logits"], ref["logits"], ref["mask"], RTOL["bf16"])
    final = hn_states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]


def test_rollout_logits_equal_policy_forward():
    """The mover's logits in a rollout are exactly policy_forward of the recorded observation."""
    require_gpu()
    cfg = R.hanabi_config(64, seed=13)
    for dims, dtype in (((D, 64, 64, NA), "f32"), ((D, 512, 512, NA), "bf16")):
        ws, bs = workloads.policy_weights(dims, seed=77, bias_scale=0.2)
        pol = R.Policy(ws, bs, dtype)
        _, g = _run_gpu(cfg, pol, 30)
        pf = R.policy_forward(pol, g["obs"].reshape(-1, D).cuda()).cpu().reshape(g["logits"].shape)
        lg = g["logits"]
        fin = torch.isfinite(lg)
        assert fin.any(dim=-1).sum() == lg.shape[0] * lg.shape[1]  # exactly one mover row per env and step
        assert torch.equal(lg[fin], pf[fin]), dtype
