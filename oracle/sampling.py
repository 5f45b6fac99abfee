"""Categorical action sampling by the Gumbel-max rule (test infrastructure).

Each agent draws its action from pi(a | o) given by the policy's logits
(Section 3: decentralised policies pi_i(a_i | tau_i)); the paper does not fix
the sampling procedure.  Reading used here:

* Gumbel-max: a* = argmax_a (logit_a + g_a) with g_a i.i.d. standard Gumbel.
  By the Gumbel-max theorem a* is distributed as softmax(logits).
* Noise: g(u) = -ln(-ln((u + 1/2) / 2^24)) for a 24-bit uniform integer u,
  evaluated in double precision and rounded once to float32.
* The 24-bit draws come from the action stream of the row (env, agent) at
  step t: block sub = agent * 256 + a // 8, word (a % 8) // 2 of that block,
  high 32-bit half for even a and low half for odd a, and u = half >> 8.
* Score_a = float32(logit_a + g_a) in float32 arithmetic.  A masked action or
  a NaN score counts as -inf.  Ties go to the lowest index.  If every score is
  -inf the action is 0.
"""

import math

import numpy as np

from . import philox


def gumbel_from_u24(u):
    """Standard Gumbel noise for the 24-bit uniform integer ``u``, as float32."""
    x = (float(u) + 0.5) / 16777216.0
    return np.float32(-math.log(-math.log(x)))


def gumbel_table():
    """float32 Gumbel noise for every 24-bit input (vectorised form of ``gumbel_from_u24``)."""
    u = np.arange(1 << 24, dtype=np.float64)
    x = (u + 0.5) / 16777216.0
    return (-np.log(-np.log(x))).astype(np.float32)


def action_u24(seed, env_id, t, agent, n_actions):
    """The 24-bit uniforms that drive the action choice of one row."""
    out = []
    blocks = {}
    for a in range(n_actions):
        sub = agent * 256 + a // 8
        if sub not in blocks:
            blocks[sub] = philox.block(seed, env_id, t, sub, philox.TAG_ACTION)
        w = blocks[sub][(a % 8) // 2]
        half = (w >> 32) if a % 2 == 0 else (w & philox.MASK32)
        out.append(half >> 8)
    return out


def select(logits, noise, mask=None):
    """Gumbel-max selection over float32 logits and float32 noise.

    ``mask`` (optional) is a sequence of truthy values, true = legal.
    """
    best = 0
    best_score = -math.inf
    for a in range(len(logits)):
        s = np.float32(np.float32(logits[a]) + np.float32(noise[a]))
        s = float(s)
        if (mask is not None and not mask[a]) or math.isnan(s):
            s = -math.inf
        if s > best_score:
            best_score = s
            best = a
    return best


def sample_action(seed, env_id, t, agent, logits, mask=None):
    """Sample the action of (env_id, agent) at step t from float32 logits."""
    noise = [gumbel_from_u24(u) for u in action_u24(seed, env_id, t, agent, len(logits))]
    return select(logits, noise, mask)
