"""Philox4x32-10 counter-based generator, written from its published definition
(Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC'11, section 3.3), and the derived uniform/normal streams the oracle uses for
the method's own random draws (projection W, phases psi, Lanczos start q1,
SimHash hyperplanes R).

TEST INFRASTRUCTURE. This module is part of the CPU oracle. Only the tests, the
smoke check and the benchmark's CPU-baseline leg may import it; the product path
never does.

The paper fixes no generator; it only says its runs use seed 0 (Appendix B.2)
and that q1 is random (Algorithm 2). The reading used here: every random value
is a pure function of (seed, stream, window, element index), so that two
independent implementations can agree bit for bit.

Counter/key layout (one 128-bit block yields four 32-bit words):
    key     = (seed & 0xffffffff, seed >> 32)
    counter = (block & 0xffffffff, block >> 32, stream, window)
Uniform from two words (a, b):  u = ((a >> 5) * 2**26 + (b >> 6)) / 2**53,
in [0, 1). Block n gives u_a from words (0, 1) and u_b from words (2, 3).
Normals by Box-Muller (Box and Muller 1958): with u1 = 1 - u_a in (0, 1],
rad = sqrt(-2 ln u1), ang = 2 pi u_b, element 2n = rad cos(ang) and
element 2n+1 = rad sin(ang).
"""
import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = np.uint64(0xFFFFFFFF)

STREAM_W = 1
STREAM_PSI = 2
STREAM_Q1 = 3
STREAM_R = 4


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Ten Philox4x32 rounds on arrays of 32-bit counters (as uint64 arrays).

    Each round multiplies words 0 and 2 by the two round constants, keeps the
    high and low halves, and mixes the high halves with words 1, 3 and the round
    key; the key is bumped by the Weyl constants between rounds.
    """
    c0 = np.asarray(c0, dtype=np.uint64) & MASK32
    c1 = np.asarray(c1, dtype=np.uint64) & MASK32
    c2 = np.asarray(c2, dtype=np.uint64) & MASK32
    c3 = np.asarray(c3, dtype=np.uint64) & MASK32
    k0 = int(k0) & 0xFFFFFFFF
    k1 = int(k1) & 0xFFFFFFFF
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + W0) & 0xFFFFFFFF
            k1 = (k1 + W1) & 0xFFFFFFFF
        p0 = M0 * c0                      # < 2**64, exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1,
                          hi0 ^ c3 ^ np.uint64(k1), lo0)
    return c0, c1, c2, c3


def _blocks(seed, stream, window, nblocks):
    n = np.arange(nblocks, dtype=np.uint64)
    seed = int(seed)
    return philox4x32_10(n & MASK32, n >> np.uint64(32),
                         np.full(nblocks, stream, np.uint64),
                         np.full(nblocks, window, np.uint64),
                         seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)


def _u53(a, b):
    return ((a >> np.uint64(5)).astype(np.float64) * 67108864.0
            + (b >> np.uint64(6)).astype(np.float64)) / 9007199254740992.0


def uniforms(seed, stream, window, count):
    """count uniforms in [0,1): element n is u_a of block n."""
    w = _blocks(seed, stream, window, count)
    return _u53(w[0], w[1])


def normals(seed, stream, window, count):
    """count standard normals; block n supplies elements 2n and 2n+1."""
    nb = (count + 1) // 2
    w = _blocks(seed, stream, window, nb)
    ua = _u53(w[0], w[1])
    ub = _u53(w[2], w[3])
    rad = np.sqrt(-2.0 * np.log(1.0 - ua))
    ang = (2.0 * np.pi) * ub
    out = np.empty(2 * nb)
    out[0::2] = rad * np.cos(ang)
    out[1::2] = rad * np.sin(ang)
    return out[:count]
