"""GPU parity of the Overcooked-style kitchen against the CPU oracle, through the C ABI.

Kitchens (layouts), resets, transitions, rewards, dones and observations must
be bit-exact; logits within 1e-4 (float32) / 2e-2 (bf16) relative to the
oracle's float64 logits.  Trajectories are checked in lockstep (a differing
action must be a certified near-tie, then adopted by the oracle) and strictly
(the oracle samples from the GPU's logits).
"""

import sys

import numpy as np
import pytest
import torch

from oracle import overcooked as oc
from oracle import rollout
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import (RTOL, NearTieLockstep, assert_logits_close, oc_oracle_cfg, oc_state_tuple, oc_states_from_device,
                    oc_states_to_device, require_gpu)

pytestmark = pytest.mark.gpu

D, NA = oc.N_PLANES * oc.NCELL, oc.N_ACTIONS
_TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


def _tuples(states):
    return [oc_state_tuple(s) for s in states]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_init_matches_oracle(dtype):
    require_gpu()
    cfg = R.overcooked_config(300, seed=7, env_base=1000)  # 300 = 37 tiles of 8 + a ragged 4
    _note(f"overcooked init {dtype}")
    state = R.new_state(cfg)
    obs = torch.empty(300, 2, D, dtype=_TDT[dtype], device="cuda")
    legal = torch.zeros(300, 2, NA, dtype=torch.uint8, device="cuda")
    R.rollout_init(cfg, state, obs, legal)
    torch.cuda.synchronize()
    ocfg = oc_oracle_cfg(cfg)
    ref = rollout.initial_states(oc, ocfg, cfg.seed, range(1000, 1300))
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref)
    ref_obs, ref_mask = rollout.observe_all(oc, ocfg, ref)
    assert np.array_equal(_obs_np(obs), ref_obs)
    assert np.array_equal(legal.cpu().numpy().astype(bool), ref_mask)


def test_layouts_at_scale():
    """4096 kitchens: every one decodes to a valid partition; 256 sampled ones equal the oracle's."""
    require_gpu()
    cfg = R.overcooked_config(4096, seed=123)
    _note("overcooked layouts 4096")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    torch.cuda.synchronize()
    dev = oc_states_from_device(cfg, state)
    rng = np.random.default_rng(0)
    for e in sorted(rng.choice(4096, 256, replace=False).tolist()):
        W, H, cells = oc.layout(cfg.seed, e)
        assert (dev[e].W, dev[e].H, dev[e].cells) == (W, H, cells), e
    sizes = {(s.W, s.H) for s in dev}
    assert sizes == {(w, h) for w in range(5, 10) for h in (4, 5)}


def _random_actions(T, E, seed, p_interact=0.45, p_invalid=0.02):
    rng = np.random.default_rng(seed)
    p = np.array([0.05] + [(1 - 0.05 - p_interact) / 4] * 4 + [p_interact])
    a = rng.choice(6, size=(T, E, 2), p=p)
    bad = rng.random(a.shape) < p_invalid
    a[bad] = rng.choice(np.array([-1, 6, 99, 1 << 20]), size=int(bad.sum()))
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


@pytest.mark.parametrize("kw,E,T,dtype", [
    # ragged last workgroups (the env-only kernel takes 8 float32 or 16 bf16
    # kitchens per workgroup) and more than one 64-step chunk of actions
    (dict(cook_time=2, soup_reward=20, max_steps=37, seed=3), 203, 120, "f32"),
    (dict(cook_time=20, soup_reward=20, max_steps=400, seed=5, env_base=5000), 77, 70, "bf16"),
    (dict(cook_time=1, soup_reward=7, max_steps=9, seed=8), 9, 40, "bf16"),
])
def test_env_only_parity(kw, E, T, dtype):
    require_gpu()
    cfg = R.overcooked_config(E, **kw)
    _note(f"overcooked env-only {kw} E={E} T={T} {dtype}")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    actions = _random_actions(T, E, seed=E + T)
    g = _env_only_gpu(cfg, state, 0, actions, dtype)
    ocfg = oc_oracle_cfg(cfg)
    ids = range(cfg.env_base, cfg.env_base + E)
    ref = rollout.env_only(oc, ocfg, cfg.seed, ids, 0, actions)
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    assert np.array_equal(g["legal_out"].numpy().astype(bool), ref["mask"])
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref["states"])
    if cfg.max_steps < T:
        assert (g["done"].numpy() == 2).any()


def test_env_only_resume_from_oracle_states():
    """Mid-episode states built by the oracle (items on counters, pots cooking, soups in hand) step identically."""
    require_gpu()
    cfg = R.overcooked_config(64, cook_time=4, soup_reward=20, max_steps=300, seed=21)
    ocfg = oc_oracle_cfg(cfg)
    ids = list(range(64))
    pre = rollout.env_only(oc, ocfg, cfg.seed, ids, 0, _random_actions(150, 64, seed=1, p_invalid=0))["states"]
    # random play rarely fills a pot: give the pots and hands random contents a kitchen can reach
    rng = np.random.default_rng(3)
    for s in pre:
        for c in s.pots():
            s.pot_onions[c] = int(rng.integers(0, 4))
            s.pot_timer[c] = int(rng.integers(0, cfg.extra["oc_cook_time"] + 1)) if s.pot_onions[c] == 3 else 0
        s.held = [int(x) for x in rng.integers(0, 4, size=2)]
    assert any(any(s.items) for s in pre) and any(v > 0 for s in pre for v in s.pot_timer.values())
    assert any(3 in s.held for s in pre)
    state = oc_states_to_device(cfg, pre)
    actions = _random_actions(60, 64, seed=2)
    g = _env_only_gpu(cfg, state, 150, actions, "f32")
    ref = rollout.env_only(oc, ocfg, cfg.seed, ids, 150, actions, states=pre)
    assert np.array_equal(g["reward"].numpy(), ref["reward"])
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref["states"])


def _soup_kitchen():
    """A 5x4 kitchen (onion and pot on the top wall, plate and serving cell at the bottom)."""
    rows = ["COCKC", "C...C", "C...C", "CPCSC"]
    code = {"C": oc.COUNTER, ".": oc.FLOOR, "O": oc.ONION, "P": oc.PLATE, "K": oc.POT, "S": oc.SERVE}
    cells = [oc.COUNTER] * oc.NCELL
    for r, row in enumerate(rows):
        for q, ch in enumerate(row):
            cells[r * oc.CW + q] = code[ch]
    pot = 3
    return oc.State(5, 4, cells, [0] * oc.NCELL, [10, 19], [0, 0], [0, 0], {pot: 0}, {pot: 0}, 0)


def test_scripted_soup_on_device():
    """Three onions, cooking, plating and serving, stepped on the GPU: exactly one reward of 20 and
    the oracle's state after every step."""
    require_gpu()
    N, S, W, E, I, Z = 1, 2, 3, 4, 5, 0
    trip = [(I, Z), (E, Z), (E, Z), (N, Z), (I, Z), (W, Z), (W, Z), (N, Z)]
    script = trip + trip + [(I, Z), (E, Z), (E, Z), (N, Z), (I, Z)]
    script += [(W, E), (W, Z), (S, Z), (S, Z), (I, Z), (N, W), (E, Z), (E, Z), (N, Z)]
    script += [(I, Z)] * 20  # wait by the pot, then plate the soup
    script += [(S, Z), (S, Z), (I, Z)]  # down to (2,3), face the serving cell below, deliver
    cfg = R.overcooked_config(9, cook_time=5, soup_reward=20, max_steps=400, seed=1)
    ocfg = oc_oracle_cfg(cfg)
    s0 = _soup_kitchen()
    states = [s0.copy() for _ in range(9)]
    state = oc_states_to_device(cfg, states)
    acts = np.array([[list(a)] * 9 for a in script], dtype=np.int32)
    g = _env_only_gpu(cfg, state, 0, acts, "f32")
    ref = rollout.env_only(oc, ocfg, cfg.seed, range(9), 0, acts, states=states)
    assert np.array_equal(g["reward"].numpy(), ref["reward"])
    assert np.array_equal(_obs_np(g["obs_out"]), ref["obs"])
    assert (g["reward"].numpy().sum(axis=0) == 20).all()
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref["states"])


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


def _check_traj(gpu, ref, env_idx, rtol):
    assert np.array_equal(_obs_np(gpu["obs"][:, env_idx]), ref["obs"])
    assert np.array_equal(gpu["reward"][:, env_idx].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(gpu["done"][:, env_idx].numpy(), ref["done"])
    assert np.array_equal(gpu["actions"][:, env_idx].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(gpu["obs_last"][env_idx]), ref["obs_last"])
    assert_logits_close(gpu["logits"][:, env_idx].numpy(), ref["logits"], rtol)


@pytest.mark.parametrize("dims,dtype", [((D, 64, 64, NA), "f32"), ((D, 64, 64, NA), "bf16"),
                                        ((D, 256, 256, NA), "bf16")])
def test_rollout_run_small_lockstep_and_strict(dims, dtype):
    require_gpu()
    cfg = R.overcooked_config(21, cook_time=3, soup_reward=20, max_steps=25, seed=9, env_base=40)
    _note(f"overcooked rollout_run {dims} {dtype}")
    ws, bs = workloads.policy_weights(dims, seed=31, bias_scale=0.1)
    pol = R.Policy(ws, bs, dtype)
    T = 60
    state, g = _run_gpu(cfg, pol, T)
    ocfg = oc_oracle_cfg(cfg)
    ids = list(range(40, 61))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, ids, RTOL[dtype])
    ref = rollout.rollout(oc, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL[dtype])
    assert _tuples(oc_states_from_device(cfg, state)) == _tuples(ref["states"])
    if dtype == "f32":
        assert hook.mismatches == 0
    strict = rollout.rollout(oc, ocfg, cfg.seed, ids, 0, T, ws, bs, dtype,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())


def test_rollout_run_4096_sampled_envs_and_resume():
    """The 4096-env kitchen workload at full size (two launches of 200 steps, resumed from the state);
    the oracle replays 8 sampled envs over all 400 steps."""
    require_gpu()
    name = "oc_4096"
    w = workloads.WORKLOADS[name]
    cfg = R.overcooked_config(w["n_envs"], seed=0, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, "bf16")
    E = cfg.n_envs
    sample = [0, 7, 8, 1001, 2048, 3000, 4088, 4095]
    _note(f"rollout_run {name} bf16, steps 0..199")
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    gs = []
    for t0 in (0, 200):
        actions = torch.empty(200, E, 2, dtype=torch.int32, device="cuda")
        logits = torch.empty(200, E, 2, NA, device="cuda")
        reward = torch.empty(200, E, device="cuda")
        done = torch.empty(200, E, dtype=torch.uint8, device="cuda")
        R.rollout_run(cfg, pol, state, t0, 200, actions=actions, logits=logits, reward=reward, done=done)
        torch.cuda.synchronize()
        gs.append({k: v[:, sample].cpu().numpy() for k, v in
                   dict(actions=actions, logits=logits, reward=reward, done=done).items()})
        _note(f"rollout_run {name} bf16, steps {t0}..{t0 + 199} done")
    g = {k: np.concatenate([gs[0][k], gs[1][k]]) for k in gs[0]}
    ocfg = oc_oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"], cfg.seed, sample, RTOL["bf16"])
    ref = rollout.rollout(oc, ocfg, cfg.seed, sample, 0, 400, ws, bs, "bf16", action_hook=hook)
    assert np.array_equal(g["reward"], ref["reward"])
    assert np.array_equal(g["done"], ref["done"])
    assert np.array_equal(g["actions"], ref["actions"])
    assert_logits_close(g["logits"], ref["logits"], RTOL["bf16"])
    final = oc_states_from_device(cfg, state)
    assert [oc_state_tuple(final[e]) for e in sample] == _tuples(ref["states"])
    assert (g["done"][-1] == 2).all() and (g["done"][:-1] == 0).all()  # one 400-step episode each


def test_rollout_logits_equal_policy_forward():
    """The logits a kitchen rollout samples from are exactly policy_forward of the recorded observations."""
    require_gpu()
    cfg = R.overcooked_config(100, cook_time=3, soup_reward=20, max_steps=30, seed=13)
    for dtype in ("f32", "bf16"):
        dims = (D, 64, 64, NA)
        ws, bs = workloads.policy_weights(dims, seed=77, bias_scale=0.2)
        pol = R.Policy(ws, bs, dtype)
        _, g = _run_gpu(cfg, pol, 20)
        pf = R.policy_forward(pol, g["obs"].reshape(-1, D).cuda()).cpu().reshape(g["logits"].shape)
        assert torch.equal(pf, g["logits"]), dtype
