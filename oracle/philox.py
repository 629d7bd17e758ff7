"""Philox4x32-10 (oracle side).  TEST INFRASTRUCTURE ONLY.

Written from the generator's published definition: Salmon, Moraes, Dror and
Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11, Section 4 (the
Philox S-box and its Weyl key schedule) with the 4x32 multipliers and key
increments given there.  The paper this repository implements does not name a
generator; it only requires unbiased stochastic rounding (Section 3.2) and
Bernoulli masks (Section 5.2).  Philox is our reading, chosen because it is a
pure function of (key, counter): the CPU and the GPU draw the same words.

Pinned by tests/test_oracle_philox.py against rocRAND's philox4x32_10 engine
(an independent library implementation, run on the host).
"""
import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)
# Multipliers and Weyl increments of Philox-4x32 (SC'11, Section 4).
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)
ROUNDS = 10


def philox4x32_10(ctr, key):
    """Apply the 10-round Philox-4x32 bijection.

    ctr : array-like (..., 4) of 32-bit counter words (c0, c1, c2, c3)
    key : pair (k0, k1) of 32-bit key words
    Returns a uint32 array (..., 4) of output words.

    One round: multiply c0 by M0 and c2 by M1 to 64-bit products; the new
    counter is (hi(c2*M1) ^ c1 ^ k0, lo(c2*M1), hi(c0*M0) ^ c3 ^ k1, lo(c0*M0)).
    Between rounds the key advances by the Weyl increments (W0, W1).
    """
    c = np.asarray(ctr, dtype=np.uint64)
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for rnd in range(ROUNDS):
        if rnd > 0:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = c0 * PHILOX_M0          # both factors < 2^32: the product is exact in uint64
        p1 = c2 * PHILOX_M1
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ k0, p1 & MASK32,
                          (p0 >> np.uint64(32)) ^ c3 ^ k1, p0 & MASK32)
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


# Streams: which random decision a word feeds (our reading; the paper names none).
STREAM_ELEM = 0      # stochastic rounding of one gradient element (shared by PSQ and PCQ)
STREAM_SAMPLE = 1    # Bernoulli keep-mask of one sample group (AGP along samples)
STREAM_CHANNEL = 2   # Bernoulli keep-mask of one channel group (AGP along channels)


def uniform_words(index, stream, seed, step, layer_id):
    """The 32-bit random word for item `index` of `stream`.

    Counter layout: (lo32(index >> 2), hi32(index >> 2) | stream << 30, layer_id, step),
    key = (lo32(seed), hi32(seed)); the word used is number (index & 3) of the
    four the bijection returns, so four consecutive items share one evaluation.
    """
    idx = np.asarray(index, dtype=np.uint64).reshape(-1)
    j = idx >> np.uint64(2)
    ctr = np.empty(idx.shape + (4,), dtype=np.uint64)
    ctr[:, 0] = j & MASK32
    ctr[:, 1] = ((j >> np.uint64(32)) & np.uint64(0x3FFFFFFF)) | (np.uint64(stream) << np.uint64(30))
    ctr[:, 2] = np.uint64(layer_id & 0xFFFFFFFF)
    ctr[:, 3] = np.uint64(step & 0xFFFFFFFF)
    seed = int(seed)
    out = philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    return out[np.arange(idx.size), (idx & np.uint64(3)).astype(np.int64)]
