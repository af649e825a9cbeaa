"""Counter-based RNG and the Gumbel noise of the sampler (test infrastructure).

Philox4x32-10 as defined by Salmon, Moraes, Dror and Shaw, "Parallel random
numbers: as easy as 1, 2, 3" (SC'11): a 4x32-bit counter and a 2x32-bit key;
each of ten rounds multiplies counter words 0 and 2 by the round multipliers
(0xD2511F53, 0xCD9E8D57), and builds the new counter from the high halves
xor-ed with the other words and the key, and the low halves; the key is bumped
by the Weyl constants (0x9E3779B9, 0xBB67AE85) between rounds.

Sampler use (the per-token log-probabilities and sampling of the method
section, full-vocabulary temperature sampling as in the generation
hyper-parameter table):
    key     = (seed & 0xffffffff, seed >> 32)
    counter = (v >> 2, position, uid & 0xffffffff, uid >> 32)
    word    = output[v & 3]
    u       = ((word >> 9) + 0.5) * 2^-23            exact in fp32, in (0, 1)
    G       = -log(-log u)                           standard Gumbel

Published known-answer vectors are not available here, so the bit stream is
pinned by a second, independent big-integer implementation and by
distribution tests (uniformity of u, Gumbel moments, Gumbel-max frequencies
equal to softmax probabilities).
"""
import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint64(0x9E3779B9)
W1 = np.uint64(0xBB67AE85)
_LO = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10; all arguments broadcast, uint32-valued."""
    c0, c1, c2, c3 = (np.asarray(c, np.uint64) & _LO for c in (c0, c1, c2, c3))
    k0 = np.asarray(k0, np.uint64) & _LO
    k1 = np.asarray(k1, np.uint64) & _LO
    for r in range(10):
        if r:
            k0 = (k0 + W0) & _LO
            k1 = (k1 + W1) & _LO
        p0 = M0 * c0            # < 2^64: exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> _S32, p0 & _LO
        hi1, lo1 = p1 >> _S32, p1 & _LO
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def sampler_bits(vocab_ids, position, uid, seed):
    """The 32-bit word that drives the noise of token ``v`` (uint64 array)."""
    v = np.asarray(vocab_ids, np.uint64)
    uid = int(uid)
    seed = int(seed)
    out = philox4x32_10(v >> np.uint64(2), np.uint64(position & 0xFFFFFFFF),
                        np.uint64(uid & 0xFFFFFFFF), np.uint64(uid >> 32),
                        np.uint64(seed & 0xFFFFFFFF), np.uint64((seed >> 32) & 0xFFFFFFFF))
    words = np.stack(out, axis=0)
    sel = (v & np.uint64(3)).astype(np.int64)
    return np.take_along_axis(words, sel[None, :], axis=0)[0]


def uniform01(bits):
    """u = ((bits >> 9) + 0.5) * 2^-23 — exact in float32, strictly inside (0, 1)."""
    b = np.asarray(bits, np.uint64) >> np.uint64(9)
    return (b.astype(np.float64) + 0.5) * 2.0 ** -23


def gumbel_noise(vocab, position, uid, seed):
    """Standard Gumbel noise G_v = -log(-log u_v), v < vocab, in float64."""
    u = uniform01(sampler_bits(np.arange(vocab, dtype=np.uint64), position, uid, seed))
    return -np.log(-np.log(u))
