"""Fragment-major packed policy weights (rl_policy_pack) through the C ABI.

* The packed buffer equals a copy built on the host from the documented layout (tile t, K step s,
  lane l: W[16t + l % 16][32s + 8(l // 16) + j], zero outside W), byte for byte, for shapes with
  ragged rows and a partial last K step.
* Rollouts that read the packed copy (kitchen and Hanabi rollouts, and the 12x12 LBF rollout, whose
  layer 1 streams from the packed copy while without one both layers stay in registers) are
  bit-identical to the same rollouts reading W in the nn.Linear layout: observations, actions,
  logits, rewards, dones and the final state.  (Parity of the packed path against the oracle is covered by the kitchen and Hanabi
  rollout tests, whose bf16 policies are packed by default.)
"""

import sys

import numpy as np
import pytest
import torch

from paper_2609_13716_amd import rollout as R
from paper_2609_13716_amd import workloads

from parity import require_gpu

pytestmark = pytest.mark.gpu


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _host_pack(W):
    """[N, K] bf16 bits (uint16) -> the documented fragment-major uint16 array."""
    N, K = W.shape
    T, S = -(-N // 16), -(-K // 32)
    pad = np.zeros((T * 16, S * 32), np.uint16)
    pad[:N, :K] = W
    # [T, 16 rows, S, 4 chunks, 8] -> [T, S, chunk (lane // 16), row (lane % 16), 8]
    blk = pad.reshape(T, 16, S, 4, 8).transpose(0, 2, 3, 1, 4)
    return blk.reshape(-1)


@pytest.mark.parametrize("dims", [(658, 512, 512, 20), (1170, 256, 256, 6), (27, 16, 32, 6), (300, 48, 32, 7)])
def test_pack_layout(dims):
    require_gpu()
    _note(f"rl_policy_pack {dims}")
    ws, bs = workloads.policy_weights(dims, seed=5, bias_scale=0.2)
    pol = R.Policy(ws, bs, "bf16")
    torch.cuda.synchronize()
    got = pol.packed.cpu().numpy().view(np.uint16)
    off = 0
    for l in range(3):
        W = pol.W[l].cpu().view(torch.int16).numpy().view(np.uint16)
        ref = _host_pack(W)
        assert np.array_equal(got[off:off + ref.size], ref), l
        off += -(-ref.size * 2 // 256) * 256 // 2
    assert got.size * 2 == R.lib.rl_policy_packed_bytes(pol.c())


def _run(cfg, pol, T):
    E, A, D, nA = cfg.n_envs, cfg.n_agents, R.rl_obs_dim(cfg), R.rl_num_actions(cfg)
    state = R.new_state(cfg)
    R.rollout_init(cfg, state)
    out = dict(obs=torch.empty(T, E, A, D, dtype=pol.torch_dtype, device="cuda"),
               actions=torch.empty(T, E, A, dtype=torch.int32, device="cuda"),
               logits=torch.empty(T, E, A, nA, device="cuda"),
               reward=torch.empty(T, E, device="cuda"),
               done=torch.empty(T, E, dtype=torch.uint8, device="cuda"),
               obs_last=torch.empty(E, A, D, dtype=pol.torch_dtype, device="cuda"))
    R.rollout_run(cfg, pol, state, 0, T, **out)
    torch.cuda.synchronize()
    out["state"] = state
    return {k: v.cpu() for k, v in out.items()}


@pytest.mark.parametrize("env,dims", [("hanabi", (658, 512, 512, 20)), ("hanabi", (658, 64, 96, 20)),
                                      ("hanabi_mini", (278, 128, 128, 16)), ("overcooked", (1170, 256, 256, 6)),
                                      ("overcooked", (1170, 64, 48, 6)), ("lbf12", (432, 256, 256, 6))])
def test_packed_rollout_equals_unpacked(env, dims):
    require_gpu()
    _note(f"packed vs unpacked rollout {env} {dims}")
    E, T = 37, 30
    if env == "lbf12":  # (three workgroups of 16 envs, the last ragged; episodes of 50 steps cross resets)
        E, T = 37, 60
        cfg = R.EnvConfig(n_envs=E, seed=3, **workloads.WORKLOADS["lbf12_16k"]["env"])
    elif env == "hanabi":
        cfg = R.hanabi_config(E, seed=3)
    elif env == "hanabi_mini":
        cfg = R.hanabi_config(E, colours=3, ranks=3, seed=3)
    else:
        cfg = R.overcooked_config(E, seed=3)
    ws, bs = workloads.policy_weights(dims, seed=21, bias_scale=0.3)
    packed = _run(cfg, R.Policy(ws, bs, "bf16"), T)
    plain = _run(cfg, R.Policy(ws, bs, "bf16", pack=False), T)
    for k in packed:
        assert torch.equal(packed[k], plain[k]), k


@pytest.mark.parametrize("dims", [(432, 256, 256, 6), (658, 512, 512, 20), (1170, 256, 256, 6), (300, 512, 32, 20)])
def test_packed_policy_forward_equals_unpacked(dims):
    """The tiled policy forward stages its weight slices from the packed copy: same logits, bit for bit."""
    require_gpu()
    _note(f"packed vs unpacked policy_forward {dims}")
    rng = np.random.default_rng(dims[0])
    ws, bs = workloads.policy_weights(dims, seed=23, bias_scale=0.3)
    x = torch.from_numpy(rng.integers(0, 3, size=(777, dims[0])).astype(np.float32)).to("cuda", torch.bfloat16)
    a = R.policy_forward(R.Policy(ws, bs, "bf16"), x).cpu()
    b = R.policy_forward(R.Policy(ws, bs, "bf16", pack=False), x).cpu()
    assert torch.equal(a, b)


def test_packed_population_rollout_equals_unpacked():
    """Population rollouts read policy q's packed copy at q * rl_policy_packed_bytes: same trajectories."""
    require_gpu()
    _note("packed vs unpacked population rollout")
    dims = (192, 64, 32, 6)
    nets = [workloads.policy_weights(dims, seed=30 + q, bias_scale=0.3) for q in range(5)]
    E, T = 37, 30
    cfg = R.EnvConfig(n_envs=E, seed=4)
    idx = torch.from_numpy(np.random.default_rng(2).integers(0, 5, size=(E, 2)).astype(np.int32)).cuda()
    res = []
    for pk in (True, False):
        pop = R.Population([w for w, _ in nets], [b for _, b in nets], "bf16", pack=pk)
        state = R.new_state(cfg)
        R.rollout_init(cfg, state)
        out = dict(obs=torch.empty(T, E, 2, 192, dtype=torch.bfloat16, device="cuda"),
                   actions=torch.empty(T, E, 2, dtype=torch.int32, device="cuda"),
                   logits=torch.empty(T, E, 2, 6, device="cuda"),
                   reward=torch.empty(T, E, device="cuda"), done=torch.empty(T, E, dtype=torch.uint8, device="cuda"))
        R.rollout_run_pop(cfg, pop, idx, state, 0, T, **out)
        torch.cuda.synchronize()
        out["state"] = state
        res.append({k: v.cpu() for k, v in out.items()})
    for k in res[0]:
        assert torch.equal(res[0][k], res[1][k]), k
