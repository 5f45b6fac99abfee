"""Pins of the oracle MLP and its bfloat16 rounding.

* float32 mode against torch's float64 linear/tanh (an independent library).
* Closed-form special cases: zero weights give the bias; a one-hot input picks
  one weight column; with zero biases the network is odd in its input.
* bfloat16 rounding against torch's float32 -> bfloat16 cast (one rounding,
  to nearest even) and against hand-picked ties and overflow cases.
"""

import numpy as np
import pytest
import torch

from oracle import mlp


def _net(rng, dims, bias=True):
    ws, bs = [], []
    for i in range(len(dims) - 1):
        ws.append((rng.standard_normal((dims[i + 1], dims[i])) / np.sqrt(dims[i])).astype(np.float32))
        bs.append((rng.standard_normal(dims[i + 1]) * 0.1 if bias else np.zeros(dims[i + 1])).astype(np.float32))
    return ws, bs


def _torch_forward(obs, ws, bs):
    h = torch.from_numpy(np.asarray(obs, np.float64))
    for i, (w, b) in enumerate(zip(ws, bs)):
        h = torch.nn.functional.linear(h, torch.from_numpy(w.astype(np.float64)),
                                       torch.from_numpy(b.astype(np.float64)))
        if i < len(ws) - 1:
            h = torch.tanh(h)
    return h.numpy()


@pytest.mark.parametrize("dims", [(192, 64, 64, 6), (192, 128, 128, 6), (432, 256, 256, 6)])
def test_f32_matches_torch(dims):
    rng = np.random.default_rng(len(dims) + dims[1])
    ws, bs = _net(rng, dims)
    obs = rng.integers(0, 4, size=(50, dims[0])).astype(np.float32)
    got = mlp.forward(obs, ws, bs, "f32")
    ref = _torch_forward(obs, ws, bs)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_zero_weights_give_bias():
    rng = np.random.default_rng(0)
    ws, bs = _net(rng, (16, 8, 8, 5))
    ws = [np.zeros_like(w) for w in ws]
    obs = rng.standard_normal((7, 16)).astype(np.float32)
    for dt in ("f32", "bf16"):
        got = mlp.forward(obs, ws, bs, dt)
        b3 = bs[2].astype(np.float64) if dt == "f32" else mlp.round_bf16(bs[2].astype(np.float64))
        assert np.array_equal(got, np.broadcast_to(b3, got.shape))


def test_one_hot_selects_column():
    rng = np.random.default_rng(1)
    w1 = rng.standard_normal((9, 12)).astype(np.float32)
    b1 = np.zeros(9, np.float32)
    for k in range(12):
        e = np.zeros((1, 12), np.float32)
        e[0, k] = 1.0
        got = mlp.forward(e, [w1], [b1], "f32")[0]
        assert np.array_equal(got, w1[:, k].astype(np.float64))


def test_odd_symmetry_without_bias():
    rng = np.random.default_rng(2)
    ws, bs = _net(rng, (20, 10, 10, 4), bias=False)
    x = rng.standard_normal((6, 20)).astype(np.float32)
    for dt in ("f32", "bf16"):
        assert np.array_equal(mlp.forward(-x, ws, bs, dt), -mlp.forward(x, ws, bs, dt))


def test_round_bf16_matches_torch_on_f32():
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 1 << 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    special = np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 1.001953125, 1.0029296875,
                        3.4e38, -3.4e38, 1e-40, -1e-45, 1.1754944e-38, 9.18e-41], np.float32)
    x = np.concatenate([x, special])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = mlp.round_bf16(x.astype(np.float64))
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all(), x[~same][:10]


def test_round_bf16_ties_and_direct_rounding():
    # 1 + 2^-8 is exactly halfway between 1 and 1 + 2^-7: ties to even -> 1
    assert mlp.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: even is 1 + 2^-6
    assert mlp.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    # just above the tie rounds up (a float64 input is rounded once, not via float32)
    assert mlp.round_bf16(np.array([1.0 + 2.0 ** -8 + 2.0 ** -40]))[0] == 1.0 + 2.0 ** -7
    # overflow past the largest finite bfloat16 goes to inf
    assert np.isinf(mlp.round_bf16(np.array([3.5e38]))[0])
    assert np.isnan(mlp.round_bf16(np.array([np.nan]))[0])


def test_bf16_forward_near_torch_bf16_pipeline():
    rng = np.random.default_rng(4)
    ws, bs = _net(rng, (192, 128, 128, 6))
    obs = rng.integers(0, 3, size=(64, 192)).astype(np.float32)
    got = mlp.forward(obs, ws, bs, "bf16")

    def r(a):
        return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float64)
    h = r(obs)
    for i, (w, b) in enumerate(zip(ws, bs)):
        h = torch.nn.functional.linear(h, r(w), r(b))
        if i < 2:
            h = torch.tanh(h).to(torch.float32).to(torch.bfloat16).to(torch.float64)
    ref = h.numpy()
    scale = np.sqrt((ref ** 2).mean(axis=1, keepdims=True))
    assert np.all(np.abs(got - ref) <= 2e-2 * (np.abs(ref) + scale))
    # and the bf16 result differs from the f32 one (the roundings do something)
    assert not np.array_equal(got, mlp.forward(obs, ws, bs, "f32"))
