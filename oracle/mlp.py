"""Per-agent MLP policy forward in float64 (test infrastructure).

The policy maps an observation to action logits: x -> tanh(x W1^T + b1) ->
tanh(. W2^T + b2) -> . W3^T + b3, weights in the nn.Linear layout
W_l[fan_out, fan_in].  The paper's learners use such per-agent networks
(Section 3, decentralised policies); the layer sizes and the tanh activation
are the workload's.

Precision reading: in "f32" mode every input is taken as float32 and the
products are accumulated in float64.  In "bf16" mode the weights, biases and
observations are first rounded to bfloat16 (round to nearest, ties to even),
and so are the hidden activations before they enter the next layer; the
accumulation is again float64.  The result is the float64 logits.
"""

import numpy as np


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 value (ties to even), returned as float64.

    bfloat16 has float32's exponent range and 8 significant bits.  Values at
    or beyond the overflow threshold become +-inf; NaN stays NaN.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    finite = np.isfinite(x)
    out[~finite] = x[~finite]
    xf = x[finite]
    mant, expo = np.frexp(xf)  # xf = mant * 2**expo, 0.5 <= |mant| < 1
    # Quantum of the binade: 2**(expo - 8) for normals; subnormals share 2**-133.
    q_exp = np.maximum(expo - 8, -133)
    scaled = np.ldexp(xf, -q_exp)
    r = np.ldexp(np.rint(scaled), q_exp)  # np.rint rounds half to even
    max_bf16 = np.ldexp(np.float64(0xFF), 120)  # (2 - 2**-7) * 2**127
    r = np.where(np.abs(r) > max_bf16, np.copysign(np.inf, xf), r)
    out[finite] = r
    return out


def _prep(x, dtype):
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    return round_bf16(x) if dtype == "bf16" else x


def forward(obs, weights, biases, dtype="f32"):
    """Logits (float64, [rows, nA]) of the 3-layer tanh MLP for observations [rows, D]."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    h = _prep(obs, dtype)
    n = len(weights)
    for i, (w, b) in enumerate(zip(weights, biases)):
        w = _prep(w, dtype)
        b = _prep(b, dtype)
        h = h @ w.T + b
        if i < n - 1:
            h = np.tanh(h)
            if dtype == "bf16":
                h = round_bf16(h)
    return h
