"""Philox4x32-10 counter-based generator and the normal-variate stream built on it.

Oracle side (test infrastructure).  Written from the published definition of
Philox4x32 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11): a 4x32-bit counter and a 2x32-bit key; each round multiplies
counter words 0 and 2 by the two Philox multipliers, xors the high halves with
the other two counter words and the key, and the key is bumped by the two Weyl
constants between rounds; ten rounds.

The randomness that the codebook construction draws (Haar rotation, Lloyd
training samples, restart rotations, cell-repair perturbations) is defined as
a stream of standard normals produced from this generator, so that the oracle
and the library's C++ builder can reproduce the same draws from a seed without
sharing code.  The stream definition (shared as a *specification* only):

* normal ``n`` of stream ``(seed, tag)`` comes from block ``j = n // 2``,
  counter ``(j & 0xffffffff, j >> 32, tag, 0)``, key
  ``(seed & 0xffffffff, seed >> 32)``, giving words ``w0..w3``;
* ``a = (w0 << 21) | (w1 >> 11)``, ``b = (w2 << 21) | (w3 >> 11)`` (53 bits),
  ``u1 = (a + 0.5) / 2**53``, ``u2 = (b + 0.5) / 2**53``;
* Box-Muller: ``r = sqrt(-2 ln u1)``, normal ``2j`` is ``r cos(2 pi u2)``,
  normal ``2j+1`` is ``r sin(2 pi u2)``; all in float64.
"""
import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF

# stream tags used by the codebook construction
TAG_ROTATION = 1
TAG_TRAIN = 2
TAG_RESTART = 3
TAG_REPAIR = 4
TAG_HELDOUT = 5


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds on uint64 arrays holding 32-bit words.

    ``ctr`` is a tuple of four uint64 arrays (or ints), ``key`` a pair.
    Returns four uint64 arrays with 32-bit values.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & MASK32 for c in ctr)
    k0 = np.uint64(key[0] & MASK32)
    k1 = np.uint64(key[1] & MASK32)
    m0 = np.uint64(M0)
    m1 = np.uint64(M1)
    s32 = np.uint64(32)
    m32 = np.uint64(MASK32)
    for r in range(10):
        if r > 0:
            k0 = (k0 + np.uint64(W0)) & m32
            k1 = (k1 + np.uint64(W1)) & m32
        p0 = c0 * m0  # < 2**64, exact in uint64
        p1 = c2 * m1
        hi0, lo0 = p0 >> s32, p0 & m32
        hi1, lo1 = p1 >> s32, p1 & m32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
    return c0, c1, c2, c3


def normals(seed, tag, start, count, chunk=1 << 16):
    """Normals ``start .. start+count-1`` of stream ``(seed, tag)`` (float64)."""
    out = np.empty(max(count, 0), dtype=np.float64)
    for s in range(0, max(count, 0), chunk):
        c = min(chunk, count - s)
        out[s:s + c] = _normals_block(seed, tag, start + s, c)
    return out


def _normals_block(seed, tag, start, count):
    n = np.arange(start, start + count, dtype=np.uint64)
    j = n >> np.uint64(1)
    seed = int(seed)
    w0, w1, w2, w3 = philox4x32_10(
        (j & np.uint64(MASK32), j >> np.uint64(32), np.full_like(j, tag), np.zeros_like(j)),
        (seed & MASK32, (seed >> 32) & MASK32))
    a = (w0 << np.uint64(21)) | (w1 >> np.uint64(11))
    b = (w2 << np.uint64(21)) | (w3 >> np.uint64(11))
    u1 = (a.astype(np.float64) + 0.5) / 2.0 ** 53
    u2 = (b.astype(np.float64) + 0.5) / 2.0 ** 53
    r = np.sqrt(-2.0 * np.log(u1))
    odd = (n & np.uint64(1)).astype(bool)
    return np.where(odd, r * np.sin(2.0 * np.pi * u2), r * np.cos(2.0 * np.pi * u2))
