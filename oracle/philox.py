"""Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
easy as 1, 2, 3", SC'11), written from the published definition in plain
Python integers.  TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper draws uniforms (eta in Algorithm 1, the sampled token Y ~ q~ in
Sec. 3.2) without fixing a generator.  Reading used here: every draw is one
Philox4x64-10 block, keyed by the per-step rng key, whose counter names what
the draw is for, so that any implementation can reproduce it independently.

Counter layout (words c0..c3; key = (rng_key, 0)); the draw is output word 0:
  purpose DRAFT   (1): c0 = uid of the node being expanded, c1 = sequence
  purpose VERIFY  (2): c0 = 32*level + j, j = 0 for the sampled-token test,
                        j = slot of the candidate for the sequential tests
  purpose FINAL   (3): c0 = level of the final (residual or bonus) sample
Acceptance tests use the high 32 bits of the draw; categorical samples use
all 64 bits.
"""

M64 = (1 << 64) - 1

# Round multipliers and Weyl key increments of Philox4x64 (SC'11, Sec. 4).
_MUL0 = 0xD2E7470EE14C6C93
_MUL1 = 0xCA5A826395121157
_WEYL0 = 0x9E3779B97F4A7C15
_WEYL1 = 0xBB67AE8584CAA73B

DRAFT = 1
VERIFY = 2
FINAL = 3


def philox4x64_10(ctr, key):
    """Ten Philox4x64 rounds on counter ``ctr`` (4 words) under ``key`` (2
    words).  Each round multiplies words 0 and 2 by the round multipliers,
    swaps in the high halves xored with the odd words and the key, and bumps
    the key by the Weyl constants between rounds."""
    x0, x1, x2, x3 = (int(c) & M64 for c in ctr)
    k0, k1 = (int(k) & M64 for k in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _WEYL0) & M64
            k1 = (k1 + _WEYL1) & M64
        p0 = _MUL0 * x0
        p1 = _MUL1 * x2
        x0, x1, x2, x3 = ((p1 >> 64) ^ x1 ^ k0, p1 & M64,
                          (p0 >> 64) ^ x3 ^ k1, p0 & M64)
    return (x0, x1, x2, x3)


def draw_u64(rng_key, purpose, seq, index):
    """The 64-bit draw for (purpose, sequence, index) under ``rng_key``."""
    return philox4x64_10((index, seq, purpose, 0), (rng_key, 0))[0]


def draw_u32(rng_key, purpose, seq, index):
    """The 32-bit draw used by acceptance tests: the high half of the word."""
    return draw_u64(rng_key, purpose, seq, index) >> 32
