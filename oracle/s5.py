"""Recurrent S5 actor-critic, the ego agent of the paper's experiments (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline
use this module; the device path shares no code with it.

The paper's ego agents (Appendix, ego-agent architecture; Section 5 training
setup) encode observations with dense layers, run an S5 sequence model of
model dimension 128 and state size 128, and read a masked categorical policy
and a scalar value from two separate MLP heads of three 1024-unit hidden
layers each.

S5 (Smith, Warrington and Linderman, ICLR 2023) is a diagonal complex linear
state-space layer.  Continuous time: x' = Lambda x + B u, y = Re(C x) + D * u,
Lambda = diag(lambda) with Re(lambda) < 0, B complex [P, H], C complex [H, P],
D real [H].  Zero-order hold with a per-state step Delta_p = exp(log_dt_p):

    Lambda_bar = exp(Lambda Delta)
    B_bar      = Lambda^{-1} (Lambda_bar - I) B       (= int_0^Delta e^{Lambda s} ds B)

and one step of the recurrence is x_t = Lambda_bar x_{t-1} + B_bar u_t.  For
reinforcement learning the state is zeroed at the first step of every episode
(Lu et al., NeurIPS 2023, who adapt S5 to in-context RL with resets).

Readings where the paper gives only the widths:
  * encoder: one dense layer with tanh, u = tanh(W_e o + b_e), width H;
  * the S5 output y goes straight into both heads (each starts with a dense
    tanh layer); the heads are tanh MLPs with a linear output layer (nA logits,
    one value);
  * "bf16": the dense layers' weights are bfloat16 values, u, y and every head
    activation are rounded to bfloat16; the S5 parameters and the state are
    exact here (float32 on the device);
  * an episode's first step is the step whose observation comes from a fresh
    reset (the env state's step counter is 0).
"""

from dataclasses import dataclass

import numpy as np

from . import mlp


def discretize(lam_re, lam_im, log_dt, b_re, b_im):
    """Zero-order hold of the diagonal system (S5, Section 2 of Smith et al.).

    Returns (lambda_bar [P] complex128, b_bar [P, H] complex128)."""
    lam = np.asarray(lam_re, np.float64) + 1j * np.asarray(lam_im, np.float64)
    dt = np.exp(np.asarray(log_dt, np.float64))
    lbar = np.exp(lam * dt)
    b = np.asarray(b_re, np.float64) + 1j * np.asarray(b_im, np.float64)
    return lbar, ((lbar - 1.0) / lam)[:, None] * b


@dataclass
class Params:
    """Discretised S5 actor-critic.  Dense layers use the nn.Linear layout [out, in]."""
    w_enc: np.ndarray   # [H, D]
    b_enc: np.ndarray   # [H]
    lbar: np.ndarray    # [P] complex
    bbar: np.ndarray    # [P, H] complex
    c: np.ndarray       # [H, P] complex
    d: np.ndarray       # [H] real
    actor_w: list       # [F, H], [F, F], [F, F], [nA, F]
    actor_b: list
    critic_w: list      # [F, H], [F, F], [F, F], [1, F]
    critic_b: list

    @property
    def state_size(self):
        return len(self.lbar)


def encode(p, obs, dtype):
    """u = tanh(W_e o + b_e), [n, H] float64 (bfloat16 values under "bf16")."""
    u = np.tanh(mlp._prep(obs, dtype) @ mlp._prep(p.w_enc, dtype).T + mlp._prep(p.b_enc, dtype))
    return mlp.round_bf16(u) if dtype == "bf16" else u


def ssm_step(p, u, x, start):
    """One S5 step for n rows: the new complex state [n, P] and y [n, H] (unrounded).

    ``start`` [n] bool zeroes the previous state of rows that begin an episode."""
    x = np.where(np.asarray(start, bool)[:, None], 0.0, x)
    x_new = p.lbar[None, :] * x + u @ p.bbar.T
    y = (x_new @ p.c.T).real + p.d[None, :] * u
    return x_new, y


def step(p, obs, x, start, dtype):
    """Policy step: (logits [n, nA], value [n], new state [n, P]) for observations [n, D]."""
    u = encode(p, obs, dtype)
    x_new, y = ssm_step(p, u, x, start)
    if dtype == "bf16":
        y = mlp.round_bf16(y)
    return _head(y, p.actor_w, p.actor_b, dtype), _head(y, p.critic_w, p.critic_b, dtype)[:, 0], x_new


def _head(y, weights, biases, dtype):
    """A tanh MLP head on y, taken as it is (not re-rounded to the dtype)."""
    h = y
    for i, (w, b) in enumerate(zip(weights, biases)):
        h = h @ mlp._prep(w, dtype).T + mlp._prep(b, dtype)
        if i < len(weights) - 1:
            h = np.tanh(h)
            if dtype == "bf16":
                h = mlp.round_bf16(h)
    return h


def initial_state(n, p):
    return np.zeros((n, p.state_size), dtype=np.complex128)


def from_continuous(c):
    """Params from continuous-time parameters (a dict of arrays, see ``discretize``);
    dense-layer weights are taken as given."""
    lbar, bbar = discretize(c["lam_re"], c["lam_im"], c["log_dt"], c["b_re"], c["b_im"])
    f64 = lambda a: np.asarray(a, np.float64)
    return Params(f64(c["w_enc"]), f64(c["b_enc"]), lbar, bbar,
                  f64(c["c_re"]) + 1j * f64(c["c_im"]), f64(c["d"]),
                  [f64(w) for w in c["actor_w"]], [f64(b) for b in c["actor_b"]],
                  [f64(w) for w in c["critic_w"]], [f64(b) for b in c["critic_b"]])
