"""Philox4x64-10 counter-based generator and the integer draws derived from it.

Reference: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel
Random Numbers: As Easy as 1, 2, 3", SC'11.  Philox4x64 with 10 rounds: the
state is a 4-word counter and a 2-word key; each round multiplies words 0 and
2 by fixed odd constants, keeping the 128-bit products, and mixes the high
halves with the other two words and the round key; the key is advanced by two
Weyl constants between rounds.

The paper says only that the whole rollout runs on the GPU (Section 2, the
PureJaxRL paragraph); it fixes no generator.  Reading used here: every random
decision is a pure function of (seed, env id, step t, sub-stream, tag), with

    key     = (seed, 0)
    counter = (env_id, t, sub, tag)

so that any env's draws at any step can be recomputed without replaying the
others.  One block yields four 64-bit words; each word splits into two 32-bit
halves, high half first, giving eight 32-bit draws per block.

Pinned by tests against numpy's independent ``Philox`` bit generator.
"""

MASK64 = (1 << 64) - 1
MASK32 = (1 << 32) - 1

# Round multipliers and key-schedule (Weyl) increments of Philox4x64.
_M0 = 0xD2E7470EE14C6C93
_M1 = 0xCA5A826395121157
_W0 = 0x9E3779B97F4A7C15
_W1 = 0xBB67AE8584CAA73B

# Tags separate the sub-streams a step draws from.
TAG_RESET = 1
TAG_ACTION = 2
TAG_LAYOUT = 3


def _mulhilo(a, b):
    p = a * b
    return (p >> 64) & MASK64, p & MASK64


def philox4x64_10(counter, key):
    """Return the 4 output words of Philox4x64-10 for a 4-word counter and 2-word key."""
    c0, c1, c2, c3 = (int(x) & MASK64 for x in counter)
    k0, k1 = (int(x) & MASK64 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _W0) & MASK64
            k1 = (k1 + _W1) & MASK64
        hi0, lo0 = _mulhilo(_M0, c0)
        hi1, lo1 = _mulhilo(_M1, c2)
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return [c0, c1, c2, c3]


def block(seed, env_id, t, sub, tag):
    """The four 64-bit words of the block keyed by (seed; env_id, t, sub, tag)."""
    return philox4x64_10((env_id, t, sub, tag), (seed, 0))


def u32_draws(seed, env_id, t, tag, n):
    """The first ``n`` 32-bit draws of the stream (seed; env_id, t, *, tag).

    Draw k comes from block sub = k // 8, word (k % 8) // 2, high half when k
    is even and low half when k is odd.
    """
    out = []
    sub = 0
    while len(out) < n:
        for w in block(seed, env_id, t, sub, tag):
            out.append((w >> 32) & MASK32)
            out.append(w & MASK32)
        sub += 1
    return out[:n]


def uniform_int(u32, n):
    """Map a 32-bit draw to {0, ..., n-1} by the multiply-shift rule floor(u * n / 2^32).

    (Lemire's multiply-shift without rejection; the bias is below n / 2^32.)
    """
    if n <= 0:
        raise ValueError("uniform_int needs n >= 1")
    return (int(u32) * int(n)) >> 32
