"""Philox counter-based generator, written from its published definition.

TEST INFRASTRUCTURE ONLY: part of the CPU oracle. Only tests, the smoke
check and the bench's CPU-baseline leg may import it; the HIP product path
never does.

Reference: J. K. Salmon, M. A. Moraes, R. O. Dror, D. E. Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC'11 (Philox-NxW-R).  One round maps
a counter of N words and a key of N/2 words as follows (N = 4):
    (hi0, lo0) = mulhilo(M0, c0);  (hi1, lo1) = mulhilo(M1, c2)
    c' = (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)
and the key is bumped by the Weyl constants (W0, W1) between rounds.
The constants below are the ones the publication gives for W = 32 and W = 64.

The generator is written once, generic in the word size, so that the
64-bit instance can be checked against an independent implementation
(numpy's Philox bit generator, which is Philox-4x64-10) and the 32-bit
instance against published known-answer vectors.

The paper (SAKI) does not say how its coupling draws random numbers.  The
stream layout used everywhere in this project is:
    key     = (seed mod 2^32, seed >> 32)
    counter = (block j, stream id, g mod 2^32, g >> 32)
where g is the global row (position) index; the 4 output words of block j
are the uniforms for indices 4j .. 4j+3 of that stream.
"""

PHILOX_CONSTANTS = {
    32: dict(M0=0xD2511F53, M1=0xCD9E8D57, W0=0x9E3779B9, W1=0xBB67AE85),
    64: dict(M0=0xD2E7470EE14C6C93, M1=0xCA5A826395121157,
             W0=0x9E3779B97F4A7C15, W1=0xBB67AE8584CAA73B),
}

# stream ids (which purpose a uniform is drawn for)
STREAM_PROP_CHUNK = 0   # proposal race, one uniform per vocab chunk
STREAM_PROP_ELEM = 1    # proposal race, one uniform per vocab id
STREAM_ACCEPT = 2       # accept test, index 0
STREAM_RES_CHUNK = 3    # residual race, one uniform per vocab chunk
STREAM_RES_ELEM = 4     # residual race, one uniform per vocab id
STREAM_TS_CHUNK = 5     # teacher-sampled target race, one uniform per vocab chunk
STREAM_TS_ELEM = 6      # teacher-sampled target race, one uniform per vocab id
STREAM_SELECT = 7       # placement controls, index 0 of each position


def philox4(counter, key, word_bits=32, rounds=10):
    """Philox-4xW-R block function on Python ints; returns 4 output words."""
    k = PHILOX_CONSTANTS[word_bits]
    mask = (1 << word_bits) - 1
    c0, c1, c2, c3 = (int(x) & mask for x in counter)
    k0, k1 = (int(x) & mask for x in key)
    for _ in range(rounds):
        p0 = k["M0"] * c0
        p1 = k["M1"] * c2
        hi0, lo0 = p0 >> word_bits, p0 & mask
        hi1, lo1 = p1 >> word_bits, p1 & mask
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        k0 = (k0 + k["W0"]) & mask
        k1 = (k1 + k["W1"]) & mask
    return c0, c1, c2, c3


def word_to_uniform(x):
    """Map a 32-bit word to u in the open interval (0, 1).

    u = (2*(x >> 9) + 1) * 2^-24: the top 23 bits select one of 2^23 cell
    midpoints, so u is never 0 or 1 and is exact in float32 and float64.
    """
    return (2.0 * (int(x) >> 9) + 1.0) * (2.0 ** -24)


def uniform(seed, stream, g, index):
    """The uniform for (seed, stream, global row g, index) as a float."""
    j, w = divmod(int(index), 4)
    words = philox4((j, stream, g & 0xFFFFFFFF, (g >> 32) & 0xFFFFFFFF),
                    (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    return word_to_uniform(words[w])


def philox4x32_blocks(blocks, stream, g, seed, rounds=10):
    """Philox-4x32-R for many block indices j of one (stream, row, seed).

    The same round function as philox4, evaluated on numpy uint64 arrays
    (a 32x32-bit product fits in 64 bits).  Returns an array [len(blocks), 4]
    of uint32 words.
    """
    import numpy as np
    k = PHILOX_CONSTANTS[32]
    mask = np.uint64(0xFFFFFFFF)
    c0 = np.asarray(blocks, dtype=np.uint64) & mask
    n = c0.shape[0]
    c1 = np.full(n, stream & 0xFFFFFFFF, dtype=np.uint64)
    c2 = np.full(n, g & 0xFFFFFFFF, dtype=np.uint64)
    c3 = np.full(n, (g >> 32) & 0xFFFFFFFF, dtype=np.uint64)
    k0 = seed & 0xFFFFFFFF
    k1 = (seed >> 32) & 0xFFFFFFFF
    m0, m1 = np.uint64(k["M0"]), np.uint64(k["M1"])
    for _ in range(rounds):
        p0 = m0 * c0
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0)), lo1, (hi0 ^ c3 ^ np.uint64(k1)), lo0
        k0 = (k0 + k["W0"]) & 0xFFFFFFFF
        k1 = (k1 + k["W1"]) & 0xFFFFFFFF
    return np.stack([c0, c1, c2, c3], axis=1).astype(np.uint32)


def uniforms(seed, stream, g, indices):
    """Vector of uniforms (float64) for several indices of one (seed, stream, row)."""
    import numpy as np
    idx = np.asarray(list(indices) if not isinstance(indices, np.ndarray) else indices,
                     dtype=np.int64)
    if idx.size == 0:
        return np.empty(0, dtype=np.float64)
    blocks = idx // 4
    ub, inv = np.unique(blocks, return_inverse=True)
    words = philox4x32_blocks(ub, stream, g, seed)[inv, idx % 4]
    return (2.0 * (words.astype(np.float64) // 512.0) + 1.0) * (2.0 ** -24)
