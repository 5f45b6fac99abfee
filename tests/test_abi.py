"""The C-ABI library loads, exports every declared symbol, and rejects bad arguments on the host.

No call here reaches a kernel launch: each one fails host-side validation first.
"""

import ctypes
import os
import re

import pytest

from paper_2609_13716_amd import rollout as R

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "rollout.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_symbols_exported():
    names = _declared()
    assert "rollout_run" in names and "policy_forward" in names
    assert sorted(R.EXPORTED) == names
    for n in names:
        assert hasattr(R.lib, n), n


def _cfg(**kw):
    base = dict(n_envs=16)
    base.update(kw)
    return R.EnvConfig(**base)


def _status(cfg):
    return R.lib.rl_obs_dim(ctypes.byref(cfg.c()))


@pytest.mark.parametrize("kw,code", [
    (dict(n_envs=0), R.RL_EINVAL),
    (dict(n_agents=0), R.RL_EINVAL),
    (dict(n_agents=5), R.RL_EINVAL),
    (dict(n_food=9), R.RL_EINVAL),
    (dict(grid_h=2), R.RL_EINVAL),
    (dict(grid_w=17), R.RL_EINVAL),
    (dict(grid_h=3, grid_w=3, n_food=2), R.RL_EINVAL),
    (dict(max_agent_level=0), R.RL_EINVAL),
    (dict(max_food_level=16), R.RL_EINVAL),
    (dict(max_steps=0), R.RL_EINVAL),
    (dict(env_base=-1), R.RL_EINVAL),
    (dict(kind=7), R.RL_EINVAL),
    (dict(kind=R.RL_ENV_OVERCOOKED), R.RL_EINVAL),  # cook_time 0
    (dict(kind=R.RL_ENV_HANABI), R.RL_EINVAL),  # game sizes 0
    (dict(extra={"hn_colors": 5}), R.RL_EINVAL),
    (dict(extra={"lbf_const_levels": 2}), R.RL_EINVAL),
    (dict(const_levels=True, max_agent_level=1, max_food_level=3), R.RL_EINVAL),  # food level 3 > 2 agents * 1
])
def test_bad_config(kw, code):
    cfg = _cfg(**kw)
    assert _status(cfg) == code
    assert R.rl_state_bytes(cfg) == 0
    assert R.lib.rollout_last_error()


@pytest.mark.parametrize("kw,code", [
    (dict(cook_time=0), R.RL_EINVAL),
    (dict(cook_time=256), R.RL_EINVAL),
    (dict(soup_reward=-1), R.RL_EINVAL),
    (dict(max_steps=0), R.RL_EINVAL),
])
def test_bad_overcooked_config(kw, code):
    cfg = R.overcooked_config(16, **kw)
    assert _status(cfg) == code
    assert R.rl_state_bytes(cfg) == 0


def test_overcooked_rejects_other_kinds_fields():
    for name, v in (("n_agents", 3), ("grid_h", 5), ("n_food", 1), ("max_food_level", 2), ("hn_colors", 5),
                    ("lbf_const_levels", 1)):
        c = R.overcooked_config(16).c()
        setattr(c, name, v)
        assert R.lib.rl_obs_dim(ctypes.byref(c)) == R.RL_EINVAL, name


def test_hanabi_config_checks():
    cfg = R.hanabi_config(100)
    assert R.rl_obs_dim(cfg) == 658 and R.rl_num_actions(cfg) == 20
    assert R.rl_state_bytes(cfg) == 35 * 100 * 4
    mini = R.hanabi_config(16, colours=3, ranks=3)
    assert R.rl_obs_dim(mini) == 278 and R.rl_num_actions(mini) == 16 and R.rl_state_bytes(mini) == 35 * 16 * 4
    bad = R.hanabi_config(16, colours=3, ranks=5)
    assert R.rl_obs_dim(bad) == R.RL_EUNSUPPORTED
    for name, v, code in (("hn_colors", 4, R.RL_EUNSUPPORTED), ("hn_hand_size", 4, R.RL_EUNSUPPORTED),
                          ("hn_life_tokens", 0, R.RL_EINVAL), ("n_agents", 3, R.RL_EINVAL),
                          ("grid_w", 3, R.RL_EINVAL), ("oc_cook_time", 20, R.RL_EINVAL),
                          ("lbf_const_levels", 1, R.RL_EINVAL)):
        c = R.hanabi_config(16).c()
        setattr(c, name, v)
        assert R.lib.rl_obs_dim(ctypes.byref(c)) == code, name
    assert _run_status(cfg, _policy_struct(dims=(658, 64, 64, 6))) == R.RL_ESHAPE
    assert _run_status(cfg, _policy_struct(dims=(600, 64, 64, 20))) == R.RL_ESHAPE


def test_overcooked_queries():
    cfg = R.overcooked_config(100)
    assert R.rl_obs_dim(cfg) == 26 * 45
    assert R.rl_num_actions(cfg) == 6
    assert R.rl_state_bytes(cfg) == 32 * 100 * 4
    # the fused rollout checks the policy against the kitchen's sizes
    assert _run_status(cfg, _policy_struct(dims=(192, 64, 64, 6))) == R.RL_ESHAPE
    assert _run_status(cfg, _policy_struct(dims=(1170, 64, 64, 5))) == R.RL_ESHAPE


def test_queries():
    cfg = _cfg(n_envs=100, grid_h=12, grid_w=12, n_agents=3, n_food=6)
    assert R.rl_obs_dim(cfg) == 432
    assert R.rl_num_actions(cfg) == 6
    assert R.rl_state_bytes(cfg) == (2 * 3 + 2 * 6 + 3) * 100 * 4


def _policy_struct(dt=R.RL_F32, dims=(192, 64, 64, 6), layers=3, null_w=False):
    p = R._Policy()
    p.dtype, p.n_layers = dt, layers
    for i, d in enumerate(dims):
        p.dims[i] = d
    for i in range(3):
        p.W[i] = None if null_w else 0x1000
        p.b[i] = 0x1000
    return p


def _run_status(cfg, pol, state=0x1000, n_steps=4, t0=0):
    tr = R._Traj()
    return R.lib.rollout_run(ctypes.byref(cfg.c()), ctypes.byref(pol), ctypes.c_void_p(state), t0, n_steps,
                             ctypes.byref(tr), None)


def test_error_paths_before_launch():
    L = R.lib
    cfg = _cfg()
    c = cfg.c()
    assert L.rollout_init(ctypes.byref(c), None, None, R.RL_F32, None, None) == R.RL_EINVAL
    assert L.rollout_init(ctypes.byref(c), ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), 7, None,
                          None) == R.RL_EUNSUPPORTED
    assert L.rollout_step(ctypes.byref(c), ctypes.c_void_p(0x1000), 0, 1, None, None, 0, None, None, None,
                          None) == R.RL_EINVAL
    assert L.rollout_step(ctypes.byref(c), ctypes.c_void_p(0x1000), 0, 0, ctypes.c_void_p(0x1000), None, 0, None,
                          None, None, None) == R.RL_EINVAL
    assert L.rollout_step(ctypes.byref(c), ctypes.c_void_p(0x1000), (1 << 64) - 1, 2, ctypes.c_void_p(0x1000), None,
                          0, None, None, None, None) == R.RL_EINVAL
    # policy checks
    assert _run_status(cfg, _policy_struct(dt=5)) == R.RL_EUNSUPPORTED
    assert _run_status(cfg, _policy_struct(layers=2)) == R.RL_EUNSUPPORTED
    assert _run_status(cfg, _policy_struct(dims=(192, 60, 64, 6))) == R.RL_EUNSUPPORTED
    assert _run_status(cfg, _policy_struct(dims=(192, 64, 64, 33))) == R.RL_EUNSUPPORTED
    assert _run_status(cfg, _policy_struct(null_w=True)) == R.RL_EINVAL
    assert _run_status(cfg, _policy_struct(dims=(191, 64, 64, 6))) == R.RL_ESHAPE
    assert _run_status(cfg, _policy_struct(dims=(192, 64, 64, 5))) == R.RL_ESHAPE
    assert _run_status(cfg, _policy_struct(), state=0) == R.RL_EINVAL
    assert _run_status(cfg, _policy_struct(), n_steps=0) == R.RL_EINVAL
    # a tile that cannot fit in LDS: 16x16 grid, 4 agents, 512-wide float32 layers
    big = _cfg(grid_h=16, grid_w=16, n_agents=4)
    assert _run_status(big, _policy_struct(dims=(768, 512, 512, 6))) == R.RL_EUNSUPPORTED
    assert "LDS" in L.rollout_last_error().decode()
    # population rollout
    tr = R._Traj()
    pop_run = lambda c2, n, idx=0x1000, st=0x1000: L.rollout_run_pop(
        ctypes.byref(c2.c()), ctypes.byref(_policy_struct()), n, ctypes.c_void_p(idx), ctypes.c_void_p(st), 0, 4,
        ctypes.byref(tr), None)
    assert pop_run(cfg, 0) == R.RL_EINVAL
    assert pop_run(cfg, 4097) == R.RL_EINVAL
    assert pop_run(cfg, 2, idx=0) == R.RL_EINVAL
    assert pop_run(cfg, 2, st=0) == R.RL_EINVAL
    assert pop_run(R.overcooked_config(16, cook_time=5, soup_reward=20, max_steps=30), 2) == R.RL_EUNSUPPORTED
    # actor-critic rollout and GAE
    ac = R._AcTraj()
    ac_run = lambda c2, pol2, acp=ctypes.byref(ac): L.rollout_run_ac(
        ctypes.byref(c2.c()), ctypes.byref(pol2), ctypes.c_void_p(0x1000), 0, 4, ctypes.byref(tr), acp, None)
    assert ac_run(cfg, _policy_struct(dims=(192, 64, 64, 6))) == R.RL_ESHAPE  # needs nA + 1 outputs
    assert ac_run(cfg, _policy_struct(dims=(192, 64, 64, 7)), acp=None) == R.RL_EINVAL
    assert ac_run(R.overcooked_config(16, cook_time=5, soup_reward=20, max_steps=30),
                  _policy_struct(dims=(1170, 64, 64, 7))) == R.RL_EUNSUPPORTED
    g = lambda *a: L.rl_gae(*a)
    vp = ctypes.c_void_p(0x1000)
    assert g(None, vp, vp, vp, 4, 4, 2, 0.99, 0.95, vp, None, None) == R.RL_EINVAL
    assert g(vp, vp, vp, vp, 0, 4, 2, 0.99, 0.95, vp, None, None) == R.RL_EINVAL
    assert g(vp, vp, vp, vp, 4, 4, 2, 1.5, 0.95, vp, None, None) == R.RL_EINVAL
    assert g(vp, vp, vp, vp, 4, 4, 2, 0.99, -0.1, vp, None, None) == R.RL_EINVAL
    # policy_forward and sampling
    pol = _policy_struct()
    assert L.policy_forward(ctypes.byref(pol), None, None, 10, ctypes.c_void_p(0x1000), None) == R.RL_EINVAL
    assert L.policy_forward(ctypes.byref(pol), ctypes.c_void_p(0x1000), None, 0, ctypes.c_void_p(0x1000),
                            None) == R.RL_EINVAL
    assert L.rollout_sample(ctypes.byref(c), 0, None, None, ctypes.c_void_p(0x1000), None) == R.RL_EINVAL
    assert L.rl_gumbel_noise(None, 10, ctypes.c_void_p(0x1000), None) == R.RL_EINVAL
    assert L.rl_gumbel_noise(ctypes.c_void_p(0x1000), 0, ctypes.c_void_p(0x1000), None) == R.RL_EINVAL


def test_binding_rejects_host_tensors():
    import torch
    cfg = _cfg()
    with pytest.raises(ValueError):
        R.rollout_init(cfg, torch.zeros(10, dtype=torch.int32))


def test_constant_levels_config_is_accepted():
    cfg = _cfg(grid_h=7, grid_w=7, const_levels=True, max_agent_level=1, max_food_level=2)
    assert _status(cfg) == 147
    assert cfg.c().lbf_const_levels == 1 and _cfg().c().lbf_const_levels == 0


def _s5_struct(**kw):
    v = dict(dtype=R.RL_BF16, obs_dim=192, d_model=128, d_state=128, head_width=1024, n_actions=6)
    v.update(kw)
    p = R._S5Policy(**{k: v[k] for k in ("dtype", "obs_dim", "d_model", "d_state", "head_width", "n_actions")})
    for name in ("w_enc", "b_enc", "lambda_bar", "b_bar", "c", "d"):
        setattr(p, name, v.get(name, 0x1000))
    for l in range(4):
        p.actor_w[l] = p.actor_b[l] = p.critic_w[l] = p.critic_b[l] = v.get("heads", 0x2000)
    return p


def _s5_status(cfg, pol, carry=0x3000, ws_bytes=1 << 30, workspace=0x4000, n_steps=4):
    tr, ac = R._Traj(), R._AcTraj()
    return R.lib.rollout_run_s5(ctypes.byref(cfg.c()), ctypes.byref(pol), ctypes.c_void_p(0x1000),
                                ctypes.c_void_p(carry) if carry else None, 0, n_steps, ctypes.byref(tr),
                                ctypes.byref(ac), ctypes.c_void_p(workspace) if workspace else None, ws_bytes, None)


def test_s5_checks_before_launch():
    cfg = _cfg()
    good = _s5_struct()
    need = R.lib.rl_s5_workspace_bytes(ctypes.byref(cfg.c()), ctypes.byref(good))
    E, A = 16, 2
    assert need >= 4 * E * A * 1024 * 2 + E * A * 128 * 2
    for kw, code in ((dict(dtype=R.RL_F32), R.RL_EUNSUPPORTED), (dict(d_model=96), R.RL_EUNSUPPORTED),
                     (dict(d_state=24), R.RL_EUNSUPPORTED), (dict(d_state=144), R.RL_EUNSUPPORTED), (dict(head_width=1000), R.RL_EUNSUPPORTED),
                     (dict(obs_dim=191), R.RL_ESHAPE), (dict(n_actions=5), R.RL_ESHAPE),
                     (dict(w_enc=0), R.RL_EINVAL), (dict(c=0x1004), R.RL_EINVAL), (dict(heads=0x2008), R.RL_EINVAL)):
        p = _s5_struct(**kw)
        assert _s5_status(cfg, p) == code, kw
        assert R.lib.rl_s5_workspace_bytes(ctypes.byref(cfg.c()), ctypes.byref(p)) == 0, kw
    assert _s5_status(cfg, good, carry=0) == R.RL_EINVAL
    assert _s5_status(cfg, good, ws_bytes=need - 1) == R.RL_EINVAL
    assert _s5_status(cfg, good, workspace=0x4008) == R.RL_EINVAL
    assert _s5_status(cfg, good, n_steps=0) == R.RL_EINVAL
    assert _s5_status(R.overcooked_config(16), good) == R.RL_EUNSUPPORTED
    L = R.lib
    assert L.rl_s5_discretize(0, 4, None, None, None, None, None, None) == R.RL_EINVAL
    assert L.rl_s5_discretize(4, 4, ctypes.c_void_p(0x1000), None, ctypes.c_void_p(0x1000),
                              ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), None) == R.RL_EINVAL


def test_packed_weight_queries():
    """rl_policy_packed_bytes: ceil(N/16) * ceil(K/32) KB per layer, each layer at a 256-byte boundary;
    0 for float32 policies and for a packed pointer that is not 16-byte aligned or not bf16."""
    for dims in [(658, 512, 512, 20), (1170, 256, 256, 6), (27, 16, 32, 6), (300, 48, 32, 7)]:
        p = _policy_struct(R.RL_BF16, dims)
        want = 0
        for l in range(3):
            n = -(-dims[l + 1] // 16) * -(-dims[l] // 32) * 1024
            want += n if l == 2 else -(-n // 256) * 256
        assert R.lib.rl_policy_packed_bytes(p) == want
    assert R.lib.rl_policy_packed_bytes(_policy_struct(R.RL_F32, (192, 64, 64, 6))) == 0
    p = _policy_struct(R.RL_BF16)
    p.packed = 4104  # not 16-byte aligned
    assert R.lib.rl_policy_packed_bytes(p) == 0
    assert "aligned" in R.lib.rollout_last_error().decode()
    p = _policy_struct(R.RL_F32)
    p.packed = 4096
    assert R.lib.rl_policy_packed_bytes(p) == 0
    assert "bf16" in R.lib.rollout_last_error().decode()
    q = _policy_struct(R.RL_F32)
    assert R.lib.rl_policy_pack(q, 4096, None) == R.RL_EUNSUPPORTED
    assert R.lib.rl_policy_pack(_policy_struct(R.RL_BF16), None, None) == R.RL_EINVAL



@pytest.mark.parametrize("make", [
    lambda: R.EnvConfig(n_envs=16),
    lambda: R.EnvConfig(n_envs=7, grid_h=12, grid_w=12, n_agents=3, n_food=6),
    lambda: R.overcooked_config(16),
    lambda: R.hanabi_config(16),
])
def test_binding_checks_the_state_size(make):
    """Every binding wrapper that takes a state buffer rejects one whose size is not rl_state_bytes(cfg)
    before anything is launched (the C ABI cannot see a buffer's size)."""
    import torch
    cfg = make()
    n = R.rl_state_bytes(cfg) // 4
    for bad in (torch.zeros(n - 1, dtype=torch.int32), torch.zeros(n + 4, dtype=torch.int32),
                torch.zeros(n, dtype=torch.int16)):
        with pytest.raises(ValueError, match="rl_state_bytes"):
            R.rollout_init(cfg, bad)
        with pytest.raises(ValueError, match="rl_state_bytes"):
            R.rollout_step(cfg, bad, 0, torch.zeros(1, cfg.n_envs, cfg.n_agents, dtype=torch.int32))
        with pytest.raises(ValueError, match="rl_state_bytes"):
            R._need_state(cfg, bad)
    # the right size passes the size check and then fails the device check (these are host tensors)
    with pytest.raises(ValueError, match="device tensor"):
        R.rollout_init(cfg, torch.zeros(n, dtype=torch.int32))
