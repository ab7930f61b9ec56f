"""Philox4x32-10 counter-based RNG and the stream contract of the sampler.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Philox4x32 with 10 rounds is defined in Salmon, Moraes, Dror, Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11), Sec. 3:
  * a round maps counter (c0,c1,c2,c3) and key (k0,k1) to
        (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
    with M0 = 0xD2511F53, M1 = 0xCD9E8D57 (32x32 -> 64-bit products);
  * between rounds the key is bumped by the Weyl constants
        (0x9E3779B9, 0xBB67AE85) modulo 2^32.
Implemented with NumPy uint64 arithmetic (a 32x32-bit product fits exactly).

Stream contract (shared with the GPU implementation, which is written
independently from the same definition):
  key     = (seed & 0xffffffff, seed >> 32)
  counter = (c0, chain, round, (tag << 24) | slot)
  uniform = ((w >> 8) + 0.5) * 2^-24            -- in (0, 1), 24 bits
  normal  = Box-Muller on the word pairs (w0, w1) and (w2, w3):
            sqrt(-2 ln u_a) * (cos 2 pi u_b, sin 2 pi u_b)
For a vector of d normals, element e uses counter c0 = e >> 2, output e & 3.

Tags name the purpose of each draw so that no (tag, chain, round, slot, c0)
is ever used twice: a draft's noise is never reused by a later round.

Parity: pinned by the published known-answer vectors of Philox4x32-10
(tests/golden/philox4x32_10_kat.txt) and by distribution tests.
"""
import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint64(0x9E3779B9)
W1 = np.uint64(0xBB67AE85)
MASK32 = np.uint64(0xFFFFFFFF)
SH32 = np.uint64(32)

TAG_INIT = 1      # Y_0 ~ N(0, I)                      (Alg. 8, first line)
TAG_DRAFT = 2     # draft noise xi_i, slot = i          (Alg. 8, draft loop)
TAG_COIN = 3      # coins eta_j                          (Alg. 2 / Alg. 6)
TAG_USAMPLE = 4   # the uniform of U-sampling            (Alg. 7)
TAG_RESID = 5     # G ~ N(0, I) of the residual          (Alg. 5)
TAG_TARGET = 6    # noise of the full-accept target draw (Alg. 8)


def philox4x32_10(counter, key):
    """Philox4x32-10 block function.

    counter: uint array [..., 4] (values < 2^32); key: uint array [..., 2].
    Returns uint64 array [..., 4] holding the four 32-bit output words.
    """
    c = np.asarray(counter, dtype=np.uint64) & MASK32
    k = np.asarray(key, dtype=np.uint64) & MASK32
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0, k1 = np.broadcast_to(k[..., 0], c0.shape), np.broadcast_to(k[..., 1], c0.shape)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = M0 * c0
        p1 = M1 * c2
        hi0, lo0 = p0 >> SH32, p0 & MASK32
        hi1, lo1 = p1 >> SH32, p1 & MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1)


def seed_key(seed):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return np.array([seed & 0xFFFFFFFF, seed >> 32], dtype=np.uint64)


def words(seed, c0, chain, rnd, tag, slot):
    """Philox output words for counters (c0, chain, rnd, tag<<24|slot).

    All counter fields broadcast against each other; returns [..., 4] uint64.
    """
    c0, chain, rnd, slot = np.broadcast_arrays(
        np.asarray(c0, dtype=np.uint64), np.asarray(chain, dtype=np.uint64),
        np.asarray(rnd, dtype=np.uint64), np.asarray(slot, dtype=np.uint64))
    c3 = (np.uint64(tag) << np.uint64(24)) | slot
    ctr = np.stack([c0, chain, rnd, c3], axis=-1)
    return philox4x32_10(ctr, seed_key(seed))


def word_to_uniform(w):
    """24-bit uniform strictly inside (0, 1)."""
    w = np.asarray(w, dtype=np.uint64)
    return ((w >> np.uint64(8)).astype(np.float64) + 0.5) * (2.0 ** -24)


def words_to_normals(w):
    """Box-Muller on (w0,w1) and (w2,w3): [..., 4] words -> [..., 4] normals."""
    u = word_to_uniform(w)
    r01 = np.sqrt(-2.0 * np.log(u[..., 0]))
    r23 = np.sqrt(-2.0 * np.log(u[..., 2]))
    t01 = 2.0 * np.pi * u[..., 1]
    t23 = 2.0 * np.pi * u[..., 3]
    return np.stack([r01 * np.cos(t01), r01 * np.sin(t01),
                     r23 * np.cos(t23), r23 * np.sin(t23)], axis=-1)


def normal_vector(seed, chain, rnd, tag, slot, d):
    """d standard normals for one (chain, round, tag, slot): element e uses c0 = e>>2."""
    nblk = (d + 3) // 4
    w = words(seed, np.arange(nblk), chain, rnd, tag, slot)
    return words_to_normals(w).reshape(-1)[:d]


def uniform_at(seed, chain, rnd, tag, slot, index):
    """The uniform number `index` of a (chain, round, tag, slot) stream: word index&3 of c0=index>>2."""
    w = words(seed, int(index) >> 2, chain, rnd, tag, slot)
    return float(word_to_uniform(w[int(index) & 3]))
