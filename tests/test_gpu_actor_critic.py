"""GPU parity of the actor-critic outputs (rollout_run_ac, rl_gae) against the oracle, through the C ABI.

rollout_run_ac's trajectory is checked like rollout_run's (bit-exact env
outputs, logits and values within the dtype's tolerance, actions in lockstep
and strictly).  log pi(a) is compared with the oracle's float64 log-softmax of
the GPU's own float32 logits (strict run), so the check isolates the
log-softmax arithmetic: 1e-5 relative plus 1e-6.  GAE (float32 on the GPU,
float64 in the oracle) agrees within 1e-5 relative plus 1e-5 over up to 128 steps, for
the chunked kernel (chains cut into 16 chunks folded as affine maps, T >= 32) and the one-pass kernel.
A value head that is all zeros but its bias leaves every other output exactly
as rollout_run's (same MFMA chains for the action columns), on the generic
and on the register-resident kernel.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import actor_critic, lbf, rollout
from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import RTOL, NearTieLockstep, assert_logits_close, oracle_cfg, require_gpu, states_from_device

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _ac_weights(dims, seed):
    """An actor-critic network: dims[3] action logits plus one value output."""
    ws, bs = workloads.policy_weights((*dims[:3], dims[3] + 1), seed=seed, bias_scale=0.2)
    return ws, bs


def _run_ac(cfg, pol, T):
    E, A, D = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, 6, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"),
               value=torch.empty(T, E, A, device="cuda"), logp=torch.empty(T, E, A, device="cuda"),
               value_last=torch.empty(E, A, device="cuda"))
    R.rollout_run_ac(cfg, pol, state, 0, T, **out)
    torch.cuda.synchronize()
    return state, {k: v.cpu() for k, v in out.items()}


def _obs_np(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dims,dtype", [((192, 64, 64, 6), "f32"), ((192, 64, 64, 6), "bf16"),
                                        ((192, 128, 128, 6), "bf16")])
def test_actor_critic_rollout_parity(dims, dtype):
    require_gpu()
    cfg = R.EnvConfig(n_envs=37, seed=23, env_base=2)
    T = 60
    _note(f"rollout_run_ac {dims} {dtype}")
    ws, bs = _ac_weights(dims, seed=500)
    pol = R.Policy(ws, bs, dtype)
    state, g = _run_ac(cfg, pol, T)
    oc = oracle_cfg(cfg)
    env_ids = list(range(2, 39))
    hook = NearTieLockstep(g["actions"].numpy(), cfg.seed, env_ids, RTOL[dtype])
    ref = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, action_hook=hook, value_head=True)
    assert np.array_equal(_obs_np(g["obs"]), ref["obs"])
    assert np.array_equal(g["reward"].numpy().view(np.uint32), ref["reward"].view(np.uint32))
    assert np.array_equal(g["done"].numpy(), ref["done"])
    assert np.array_equal(g["actions"].numpy(), ref["actions"])
    assert np.array_equal(_obs_np(g["obs_last"]), ref["obs_last"])
    assert states_from_device(cfg, state) == ref["states"]
    assert_logits_close(g["logits"].numpy(), ref["logits"], RTOL[dtype])
    # values are one more output of the same layer: the same tolerance, against the layer's row scale
    lg_ref = np.concatenate([ref["logits"], ref["value"][..., None]], axis=-1)
    lg_gpu = np.concatenate([g["logits"].numpy(), g["value"].numpy()[..., None]], axis=-1)
    assert_logits_close(lg_gpu, lg_ref, RTOL[dtype])
    # V(o_last) is checked as the last output of its row, scaled like the steps' values by the row's logits
    last_ref = np.concatenate([ref["logits_last"], ref["value_last"][..., None]], axis=-1)
    last_gpu = np.concatenate([ref["logits_last"], g["value_last"].numpy()[..., None]], axis=-1)
    assert_logits_close(last_gpu, last_ref, RTOL[dtype])
    # strict: the oracle samples from the GPU's logits; log pi of the same float32 logits
    strict = rollout.rollout(lbf, oc, cfg.seed, env_ids, 0, T, ws, bs, dtype, value_head=True,
                             logits_source=lambda k, _: g["logits"][k].numpy())
    assert np.array_equal(strict["actions"], g["actions"].numpy())
    assert np.allclose(g["logp"].numpy(), strict["logp"], rtol=1e-5, atol=1e-6)
    assert (g["logp"].numpy() <= 0).all()


@pytest.mark.parametrize("dims", [(192, 48, 32, 6), (192, 64, 64, 6), (192, 128, 128, 6)])
def test_value_head_leaves_the_rollout_unchanged(dims):
    """With and without the value head each shape runs on one kernel family
    (generic for 48-32, register-resident for 64-64 and 128-128), whose action
    columns take the same MFMA chains either way."""
    require_gpu()
    cfg = R.EnvConfig(n_envs=45, seed=4)
    T = 40
    for dtype in ("f32", "bf16"):
        _note(f"value head off/on {dims} {dtype}")
        ws, bs = workloads.policy_weights(dims, seed=8, bias_scale=0.2)
        wv = [w.copy() for w in ws]
        bv = [b.copy() for b in bs]
        wv[2] = np.concatenate([ws[2], np.zeros((1, dims[2]), dtype=np.float32)])
        bv[2] = np.concatenate([bs[2], np.array([0.25], dtype=np.float32)])
        _, g = _run_ac(cfg, R.Policy(wv, bv, dtype), T)
        pol = R.Policy(ws, bs, dtype)
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
            assert torch.equal(g[k], ref[k].cpu()), (dtype, k)
        assert (g["value"] == 0.25).all() and (g["value_last"] == 0.25).all()


@pytest.mark.parametrize("T", [128, 33, 20])  # chunked chains (T >= 32) and the one-pass kernel
def test_gae_matches_the_oracle(T):
    require_gpu()
    rng = np.random.default_rng(12 + T)
    E, A = 300, 3
    reward = rng.standard_normal((T, E)).astype(np.float32)
    done = (rng.random((T, E)) < 0.05).astype(np.uint8) * rng.integers(1, 4, size=(T, E)).astype(np.uint8)
    value = rng.standard_normal((T, E, A)).astype(np.float32)
    vlast = rng.standard_normal((E, A)).astype(np.float32)
    for gamma, lam in ((0.99, 0.95), (1.0, 1.0), (0.9, 0.0), (0.0, 0.5)):
        adv, ret = R.gae(torch.from_numpy(reward).cuda(), torch.from_numpy(done).cuda(),
                         torch.from_numpy(value).cuda(), torch.from_numpy(vlast).cuda(), gamma, lam,
                         ret=torch.empty(T, E, A, device="cuda"))
        ra, rr = actor_critic.gae(reward, done, value, vlast, gamma, lam)
        assert np.allclose(adv.cpu().numpy(), ra, rtol=1e-5, atol=1e-5), (gamma, lam)
        assert np.allclose(ret.cpu().numpy(), rr, rtol=1e-5, atol=1e-5), (gamma, lam)


def test_gae_on_a_rollout():
    require_gpu()
    cfg = R.EnvConfig(n_envs=64, seed=31)
    ws, bs = _ac_weights((192, 64, 64, 6), seed=600)
    _, g = _run_ac(cfg, R.Policy(ws, bs, "f32"), 80)
    adv, ret = R.gae(g["reward"].cuda(), g["done"].cuda(), g["value"].cuda(), g["value_last"].cuda(), 0.99, 0.95,
                     ret=torch.empty(80, 64, 2, device="cuda"))
    ra, rr = actor_critic.gae(g["reward"].numpy(), g["done"].numpy(), g["value"].numpy(), g["value_last"].numpy(),
                              0.99, 0.95)
    assert g["done"].numpy().any()
    assert np.allclose(adv.cpu().numpy(), ra, rtol=1e-5, atol=1e-5)
    assert np.allclose(ret.cpu().numpy(), rr, rtol=1e-5, atol=1e-5)
