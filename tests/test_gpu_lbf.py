"""GPU parity of the LBF path against the CPU oracle, through the C ABI.

Environment transitions, observations, rewards, dones, resets and the
sampler's noise must be bit-exact; policy logits must agree within 1e-4
(float32) or 2e-2 (bf16) relative to the oracle's float64 logits, with the
row rms as a floor.  Full trajectories are checked in lockstep (a differing
action is accepted only as a certified near-tie and then adopted by the
oracle) and in strict mode (the oracle samples from the GPU's logits: every
action must then match).
"""

import json
import os
import sys

import numpy as np
import pytest
import torch

from oracle import lbf, mlp, rollout, sampling
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import (RTOL, NearTieLockstep, assert_logits_close, oracle_cfg, require_gpu, states_from_device,
                    states_to_device)

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


# ------------------------------------------------------------------ sampler

def test_gumbel_noise_exhaustive():
    require_gpu()
    _note("gumbel: all 2^24 inputs")
    u = torch.arange(1 << 24, dtype=torch.int32, device="cuda")
    g = R.rl_gumbel_noise(u).cpu().numpy()
    ref = sampling.gumbel_table()
    diff = np.nonzero(g.view(np.uint32) != ref.view(np.uint32))[0]
    assert diff.size == 0, f"{diff.size} inputs differ, first {diff[:5]}"


def test_sample_strict_matches_oracle():
    require_gpu()
    rng = np.random.default_rng(0)
    cfg = R.EnvConfig(n_envs=97, seed=1234, env_base=5)
    E, A, nA = 97, 2, 6
    logits = rng.standard_normal((E, A, nA)).astype(np.float32) * 2
    logits[3, 1, 2] = np.nan
    logits[4, 0, :] = 0.0
    legal = (rng.random((E, A, nA)) < 0.8).astype(np.uint8)
    legal[7, 1, :] = 0
    for t in (0, 17, 1 << 40):
        got = R.rollout_sample(cfg, t, torch.from_numpy(logits).cuda(), torch.from_numpy(legal).cuda()).cpu().numpy()
        for e in range(E):
            for a in range(A):
                ref = sampling.sample_action(1234, 5 + e, t, a, list(logits[e, a]), list(legal[e, a]))
                assert got[e, a] == ref, (t, e, a)
    assert got[7, 1] == 0


# ------------------------------------------------------------ env: init/step

@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_init_matches_oracle(dtype):
    require_gpu()
    cfg = R.EnvConfig(n_envs=100, seed=3, env_base=7)
    oc = oracle_cfg(cfg)
    state = R.new_state(cfg)
    obs = torch.empty(100, 2, 192, dtype=dtype, device="cuda")
    legal = torch.zeros(100, 2, 6, dtype=torch.uint8, device="cuda")
    R.rollout_init(cfg, state, obs, legal)
    torch.cuda.synchronize()
    got = states_from_device(cfg, state)
    ref = [lbf.reset(oc, 3, 7 + e, 0) for e in range(100)]
    assert got == ref
    ro, _ = rollout.observe_all(lbf, oc, ref)
    assert np.array_equal(_obs_np(obs), ro)
    assert (legal.cpu().numpy() == 1).all()


@pytest.mark.parametrize("cfgkw,T,dtype", [
    (dict(n_envs=37), 150, torch.float32),
    (dict(n_envs=37), 120, torch.bfloat16),
    (dict(n_envs=21, grid_h=12, grid_w=12, n_agents=3, n_food=6, max_agent_level=3, max_food_level=6), 110,
     torch.bfloat16),
    (dict(n_envs=13, grid_h=12, grid_w=12, n_agents=3, n_food=6, max_agent_level=3, max_food_level=6), 70,
     torch.float32),
    (dict(n_envs=19, grid_h=5, grid_w=7, n_agents=4, n_food=2, max_agent_level=3, max_food_level=9,
          max_steps=13), 60, torch.float32),
    (dict(n_envs=5, grid_h=3, grid_w=3, n_agents=2, n_food=1, max_steps=7), 40, torch.float32),
    (dict(n_envs=23, grid_h=7, grid_w=7, n_agents=2, n_food=3, max_agent_level=1, max_food_level=2,
          const_levels=True), 90, torch.bfloat16),
    (dict(n_envs=19, grid_h=7, grid_w=7, n_agents=2, n_food=3, max_agent_level=2, max_food_level=3), 70,
     torch.float32),
])
def test_env_only_parity(cfgkw, T, dtype):
    require_gpu()
    cfg = R.EnvConfig(seed=11, env_base=3, **cfgkw)
    _note(f"env-only parity {cfgkw} T={T} {dtype}")
    oc = oracle_cfg(cfg)
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    acts = workloads.injected_actions(T, E, A, 6, seed=99, p_invalid=0.03)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    obs = torch.empty(T, E, A, D, dtype=dtype, device="cuda")
    rew = torch.empty(T, E, dtype=torch.float32, device="cuda")
    done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
    legal = torch.zeros(T, E, A, 6, dtype=torch.uint8, device="cuda")
    R.rollout_step(cfg, state, 0, torch.from_numpy(acts).cuda(), obs, rew, done, legal)
    torch.cuda.synchronize()
    ref = rollout.env_only(lbf, oc, cfg.seed, range(cfg.env_base, cfg.env_base + E), 0, acts)
    assert np.array_equal(rew.cpu().numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(done.cpu().numpy(), ref["done"])
    assert np.array_equal(_obs_np(obs), ref["obs"])
    assert states_from_device(cfg, state) == ref["states"]
    assert (legal.cpu().numpy() == 1).all()
    assert (ref["done"] != 0).any()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_env_only_4096_sampled_envs(dtype):
    """Env-only steps of the 4096-env, 128-step 8x8 workload in one launch (the benchmarked launch, for both
    observation dtypes); sampled envs, across workgroup tiles, replayed in the oracle."""
    require_gpu()
    w = workloads.WORKLOADS["lbf8_4096"]
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=9, **w["env"])
    E, T, A, D = cfg.n_envs, w["n_steps"], cfg.n_agents, R.rl_obs_dim(cfg)
    _note(f"env-only E={E} T={T} {dtype} (sampled)")
    sample = [0, 1, 7, 8, 15, 16, 2047, 2048, 4088, 4095]
    acts = workloads.injected_actions(T, E, A, 6, seed=41, p_invalid=0.02)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    obs = torch.empty(T, E, A, D, dtype=dtype, device="cuda")
    rew = torch.empty(T, E, dtype=torch.float32, device="cuda")
    done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
    R.rollout_step(cfg, state, 0, torch.from_numpy(acts).cuda(), obs, rew, done)
    torch.cuda.synchronize()
    ref = rollout.env_only(lbf, oracle_cfg(cfg), cfg.seed, sample, 0, acts[:, sample])
    assert np.array_equal(rew[:, sample].cpu().numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(done[:, sample].cpu().numpy(), ref["done"])
    assert np.array_equal(_obs_np(obs[:, sample]), ref["obs"])
    final = states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]


def test_env_only_resume_is_bit_identical():
    require_gpu()
    cfg = R.EnvConfig(n_envs=300, seed=5)
    acts = torch.from_numpy(workloads.injected_actions(128, 300, 2, 6, seed=1)).cuda()
    s1 = R.new_state(cfg)
    R.rollout_init(cfg, s1)
    o1 = torch.empty(128, 300, 2, 192, device="cuda")
    R.rollout_step(cfg, s1, 0, acts, o1)
    s2 = R.new_state(cfg)
    R.rollout_init(cfg, s2)
    o2 = torch.empty(128, 300, 2, 192, device="cuda")
    R.rollout_step(cfg, s2, 0, acts[:64].contiguous(), o2[:64])
    host = s2.cpu()  # checkpoint through host memory
    s2 = host.cuda()
    R.rollout_step(cfg, s2, 64, acts[64:].contiguous(), o2[64:])
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(o1, o2)


def test_hand_worked_cases_gpu():
    require_gpu()
    path = os.path.join(os.path.dirname(__file__), "golden", "lbf_cases.json")
    data = json.load(open(path))
    cases = data["cases"]
    cfg = R.EnvConfig(n_envs=len(cases), seed=21, **{k: v for k, v in data["config"].items()})
    oc = oracle_cfg(cfg)
    W = cfg.grid_w
    states = [lbf.State([r * W + c for r, c in cs["agents"]], list(cs["levels"]), [r * W + c for r, c in cs["foods"]],
                        list(cs["food_levels"]), list(cs["eaten"]), cs["step_count"], sum(cs["food_levels"]))
              for cs in cases]
    state = states_to_device(cfg, states)
    acts = torch.tensor([[cs["actions"]] for cs in cases], dtype=torch.int32).permute(1, 0, 2).contiguous().cuda()
    rew = torch.empty(1, len(cases), device="cuda")
    done = torch.empty(1, len(cases), dtype=torch.uint8, device="cuda")
    R.rollout_step(cfg, state, 40, acts, None, rew, done)
    torch.cuda.synchronize()
    after = states_from_device(cfg, state)
    for i, cs in enumerate(cases):
        exp = cs["expect"]
        assert int(rew[0, i].cpu().numpy().view(np.uint32)) == int(exp["reward_bits"], 16), cs["name"]
        assert int(done[0, i]) == exp["done"], cs["name"]
        if exp["done"]:
            assert after[i] == lbf.reset(oc, 21, i, 41), cs["name"]
        else:
            assert after[i].agent_cell == [r * W + c for r, c in exp["agents"]], cs["name"]
            assert after[i].food_eaten == exp["eaten"], cs["name"]
            assert after[i].step_count == exp["step_count"], cs["name"]


def test_brute_force_3x3_gpu():
    """Every 3x3 state (food at the centre) under every joint action, GPU vs oracle."""
    require_gpu()
    import itertools
    free = [c for c in range(9) if c != 4]
    states = []
    for c0, c1 in itertools.permutations(free, 2):
        for l0, l1 in itertools.product((1, 2), repeat=2):
            for f in (1, 2, 3):
                states.append(lbf.State([c0, c1], [l0, l1], [4], [f], [False], 3, f))
    E = len(states)
    cfg = R.EnvConfig(n_envs=E, grid_h=3, grid_w=3, n_food=1, max_food_level=3, seed=8)
    oc = oracle_cfg(cfg)
    for a0, a1 in itertools.product(range(6), repeat=2):
        state = states_to_device(cfg, states)
        acts = torch.tensor([a0, a1], dtype=torch.int32).repeat(1, E, 1).contiguous().cuda()
        obs = torch.empty(1, E, 2, 27, device="cuda")
        rew = torch.empty(1, E, device="cuda")
        done = torch.empty(1, E, dtype=torch.uint8, device="cuda")
        R.rollout_step(cfg, state, 0, acts, obs, rew, done)
        ref = rollout.env_only(lbf, oc, 8, range(E), 0, np.array([[[a0, a1]] * E]), states=states)
        torch.cuda.synchronize()
        assert states_from_device(cfg, state) == ref["states"], (a0, a1)
        assert np.array_equal(rew.cpu().numpy(), ref["reward"]), (a0, a1)
        assert np.array_equal(done.cpu().numpy(), ref["done"]), (a0, a1)
        assert np.array_equal(_obs_np(obs), ref["obs"]), (a0, a1)


# ------------------------------------------------------------------ policy

@pytest.mark.parametrize("dims", [(192, 64, 64, 6), (192, 128, 128, 6), (147, 128, 128, 6), (432, 256, 256, 6), (27, 16, 32, 6),
                                  (658, 512, 512, 20), (1170, 256, 256, 6), (1170, 64, 96, 6), (300, 512, 32, 20)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_forward_parity(dims, dtype):
    require_gpu()
    _note(f"policy_forward {dims} {dtype}")
    rng = np.random.default_rng(dims[1] + len(dtype))
    ws, bs = workloads.policy_weights(dims, seed=7, bias_scale=0.3)
    rows = 1000
    obs = np.concatenate([rng.integers(0, 4, size=(rows // 2, dims[0])),
                          rng.standard_normal((rows - rows // 2, dims[0]))]).astype(np.float32)
    legal = (rng.random((rows, dims[3])) < 0.9).astype(np.uint8)
    pol = R.Policy(ws, bs, dtype)
    x = torch.from_numpy(obs).to("cuda", pol.torch_dtype)
    got = R.policy_forward(pol, x).cpu().numpy()
    ref = mlp.forward(obs, ws, bs, dtype)
    assert_logits_close(got, ref, RTOL[dtype])
    gm = R.policy_forward(pol, x, torch.from_numpy(legal).cuda()).cpu().numpy()
    assert np.all(np.isneginf(gm[legal == 0]))
    assert np.array_equal(gm[legal == 1], got[legal == 1])


@pytest.mark.parametrize("rows", [256 * 64 + 5, 3 * 256 * 64 + 37])
@pytest.mark.parametrize("dims", [(192, 128, 128, 6), (192, 64, 64, 6), (147, 128, 128, 6)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_forward_many_tiles(rows, dims, dtype):
    """Batches that give every workgroup of the persistent policy kernels several 64-row tiles
    (the first workgroups one more than the rest) and end in a ragged tile."""
    require_gpu()
    _note(f"policy_forward {dims} {dtype} rows={rows}")
    rng = np.random.default_rng(rows + dims[1])
    ws, bs = workloads.policy_weights(dims, seed=11, bias_scale=0.3)
    obs = rng.integers(0, 3, size=(rows, dims[0])).astype(np.float32)
    legal = (rng.random((rows, dims[3])) < 0.9).astype(np.uint8)
    pol = R.Policy(ws, bs, dtype)
    x = torch.from_numpy(obs).to("cuda", pol.torch_dtype)
    got = R.policy_forward(pol, x).cpu().numpy()
    assert_logits_close(got, mlp.forward(obs, ws, bs, dtype), RTOL[dtype])
    gm = R.policy_forward(pol, x, torch.from_numpy(legal).cuda()).cpu().numpy()
    assert np.all(np.isneginf(gm[legal == 0]))
    assert np.array_equal(gm[legal == 1], got[legal == 1])


# ------------------------------------------------------------- full rollout

def _run_gpu(cfg, pol, T, t0=0, state=None):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    if state is None:
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"))
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


@pytest.mark.parametrize("name,dtype", [("lbf8_small", "f32"), ("lbf8_small", "bf16")])
def test_rollout_run_small_lockstep_and_strict(name, dtype):
    require_gpu()
    w = workloads.WORKLOADS[name]
    _note(f"rollout_run {name} {dtype}")
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=2, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1002)
    pol = R.Policy(ws, bs, dtype)
    T = w["n_steps"]
    state, g = _run_gpu(cfg, pol, T)
    oc = oracle_cfg(cfg)
    env_ids = list(range(cfg.n_envs))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL[dtype])
    assert states_from_device(cfg, state) == ref["states"]
    if dtype == "f32":
        assert hook.mismatches == 0
    # strict: sampling from the GPU's own logits must reproduce every action
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rollout_run_4096_sampled_envs(dtype):
    """The 4096-env, 128-step workload at full size; the oracle replays 12 sampled envs."""
    require_gpu()
    name = "lbf8_4096"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=0, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, dtype)
    T = w["n_steps"]
    _note(f"rollout_run {name} {dtype}")
    state, g = _run_gpu(cfg, pol, T)
    sample = [0, 1, 15, 16, 17, 1000, 2047, 2048, 3333, 4079, 4094, 4095]
    oc = oracle_cfg(cfg)
    hook = NearTieLockstep(g["actions"][:, sample].numpy(), cfg.seed, sample, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, sample, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, sample, RTOL[dtype])
    final = states_from_device(cfg, state)
    assert [final[e] for e in sample] == ref["states"]
    # properties over every env: rewards, dones and episode lengths
    done = g["done"].numpy()
    rew = g["reward"].numpy()
    assert set(np.unique(done)) <= {0, 1, 2, 3}
    assert (rew >= 0).all() and (rew <= 1).all()
    assert ((done != 0).sum(axis=0) >= 2).all()  # every env finishes >= 2 episodes in 128 steps


def test_rollout_run_resume_and_env_base():
    require_gpu()
    name = "lbf8_4096"
    w = workloads.WORKLOADS[name]
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, "bf16")
    cfg = R.EnvConfig(n_envs=1000, seed=4, **w["env"])
    s_full, g_full = _run_gpu(cfg, pol, 128)
    s_half, g_a = _run_gpu(cfg, pol, 64)
    s_half = s_half.cpu().cuda()
    s_half, g_b = _run_gpu(cfg, pol, 64, t0=64, state=s_half)
    assert torch.equal(s_full.cpu(), s_half.cpu())
    for k in ("obs", "actions", "logits", "reward", "done"):
        assert torch.equal(g_full[k], torch.cat([g_a[k], g_b[k]])), k
    # a shard of the batch (env ids 600..999) reproduces the same envs
    shard = R.EnvConfig(n_envs=400, seed=4, env_base=600, **w["env"])
    _, g_s = _run_gpu(shard, pol, 128)
    for k in ("obs", "actions", "logits", "reward", "done"):
        assert torch.equal(g_full[k][:, 600:], g_s[k]), k


def test_rollout_run_12x12_sampled_envs():
    require_gpu()
    name = "lbf12_16k"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=w["n_envs"], seed=0, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1000)
    pol = R.Policy(ws, bs, "bf16")
    T = w["n_steps"]
    _note(f"rollout_run {name}")
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    actions = torch.empty(T, E, A, dtype=torch.int32, device="cuda")
    logits = torch.empty(T, E, A, 6, device="cuda")
    reward = torch.empty(T, E, device="cuda")
    done = torch.empty(T, E, dtype=torch.uint8, device="cuda")
    R.rollout_run(cfg, pol, state, 0, T, actions=actions, logits=logits, reward=reward, done=done)
    torch.cuda.synchronize()
    sample = [0, 5, 8191, 8192, 16383]
    oc = oracle_cfg(cfg)
    g_act = actions[:, sample].cpu().numpy()
    hook = NearTieLockstep(g_act, cfg.seed, sample, RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, sample, 0, T, ws, bs, "bf16", action_hook=hook)
    assert np.array_equal(reward[:, sample].cpu().numpy(), ref["reward"])
    assert np.array_equal(done[:, sample].cpu().numpy(), ref["done"])
    assert np.array_equal(g_act, ref["actions"])
    assert_logits_close(logits[:, sample].cpu().numpy(), ref["logits"], RTOL["bf16"])
    assert [states_from_device(cfg, state)[e] for e in sample] == ref["states"]


def test_rollout_run_12x12_small_full_parity():
    """Every env of a 12x12 batch that spans three workgroups and a ragged tail, against the oracle."""
    require_gpu()
    name = "lbf12_16k"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=37, seed=6, env_base=40, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=1003, bias_scale=0.1)
    pol = R.Policy(ws, bs, "bf16")
    T = 70
    _note(f"rollout_run {name} n_envs=37 T={T} bf16")
    state, g = _run_gpu(cfg, pol, T)
    oc = oracle_cfg(cfg)
    env_ids = list(range(40, 77))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL["bf16"])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, "bf16", action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL["bf16"])
    assert states_from_device(cfg, state) == ref["states"]
    assert ref["done"].any(), "the run should cross episode ends (max_steps 50)"
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, "bf16",
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())
    obs = g["obs"].reshape(-1, dims[0]).cuda()
    pf = R.policy_forward(pol, obs).cpu().reshape(g["logits"].shape)
    assert torch.equal(pf, g["logits"])


@pytest.mark.parametrize("name,dtype", [("lbf8_4096", "bf16"), ("lbf8_4096", "f32"), ("lbf8_small", "f32"),
                                        ("lbf12_16k", "bf16"), ("lbf7_const_4096", "bf16")])
def test_rollout_logits_equal_policy_forward(name, dtype):
    """The logits a rollout samples from are exactly policy_forward of the recorded observations."""
    require_gpu()
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=min(w["n_envs"], 1024), seed=9, **w["env"])
    dims = workloads.policy_dims(name)
    ws, bs = workloads.policy_weights(dims, seed=77, bias_scale=0.2)
    pol = R.Policy(ws, bs, dtype)
    _, g = _run_gpu(cfg, pol, 40)
    obs = g["obs"].reshape(-1, dims[0]).cuda()
    pf = R.policy_forward(pol, obs).cpu().reshape(g["logits"].shape)
    assert torch.equal(pf, g["logits"])


def test_rollout_run_generic_shapes():
    """Shapes without a register-resident specialisation (5x7 grid, 4 agents, 2 foods, 32-wide layers)."""
    require_gpu()
    cfg = R.EnvConfig(n_envs=45, grid_h=5, grid_w=7, n_agents=4, n_food=2, max_agent_level=3, max_food_level=9,
                      max_steps=20, seed=31, env_base=1000)
    dims = (105, 32, 48, 6)
    for dtype in ("f32", "bf16"):
        ws, bs = workloads.policy_weights(dims, seed=5, bias_scale=0.1)
        pol = R.Policy(ws, bs, dtype)
        T = 70
        state, g = _run_gpu(cfg, pol, T)
        oc = oracle_cfg(cfg)
        env_ids = list(range(1000, 1045))
        hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
        ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook)
        _check_traj(g, ref, slice(None), RTOL[dtype])
        assert states_from_device(cfg, state) == ref["states"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rollout_run_7x7_constant_levels(dtype):
    """The 7x7 constant-levels variant (agents at level 1, foods at level 2), every env of two workgroups and a
    ragged tail against the oracle; levels in the final states are the constants."""
    require_gpu()
    name = "lbf7_const_4096"
    w = workloads.WORKLOADS[name]
    cfg = R.EnvConfig(n_envs=41, seed=12, env_base=7, **w["env"])
    dims = workloads.policy_dims(name)
    assert dims[0] == 147
    ws, bs = workloads.policy_weights(dims, seed=71, bias_scale=0.1)
    pol = R.Policy(ws, bs, dtype)
    T = 80
    _note(f"rollout_run {name} n_envs=41 T={T} {dtype}")
    state, g = _run_gpu(cfg, pol, T)
    oc = oracle_cfg(cfg)
    env_ids = list(range(7, 48))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook)
    _check_traj(g, ref, slice(None), RTOL[dtype])
    states = states_from_device(cfg, state)
    assert states == ref["states"]
    assert all(s.agent_level == [1, 1] and s.food_level == [2, 2, 2] for s in states)
    assert ref["done"].any()
