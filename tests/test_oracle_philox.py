"""Pins for the oracle's Philox generator (Salmon et al., SC'11)."""
import os

import numpy as np
import pytest

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, *hexes = line.split()
            vals = [int(h, 16) for h in hexes]
            rows.append((name, vals[0:4], vals[4:6], vals[6:10]))
    return rows


@pytest.mark.parametrize("name,ctr,key,out", _kat_rows())
def test_known_answer_vectors(name, ctr, key, out):
    bits = 32 if name.startswith("philox4x32") else 64
    assert list(philox.philox4(ctr, key, word_bits=bits)) == out


def test_4x64_matches_numpy_philox():
    # numpy's Philox bit generator is Philox-4x64-10; it increments the
    # counter before each block, so its first block is counter + 1.
    for key, ctr in [((0, 0), (0, 0, 0, 0)), ((12345, 678), (5, 9, 1, 2)),
                     ((2**64 - 1, 2**63), (2**64 - 3, 7, 0, 11))]:
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.array(ctr, dtype=np.uint64))
        got = [int(x) for x in bg.random_raw(8)]
        c1 = ((ctr[0] + 1) % 2**64,) + tuple(ctr[1:])
        if ctr[0] + 1 >= 2**64:
            c1 = (0, ctr[1] + 1) + tuple(ctr[2:])
        c2 = ((c1[0] + 1) % 2**64,) + tuple(c1[1:])
        want = list(philox.philox4(c1, key, 64)) + list(philox.philox4(c2, key, 64))
        assert got == want


def test_vectorised_blocks_match_scalar():
    seed, g = 0x5A4B49 + (7 << 40), (3 << 32) + 17
    for stream in range(5):
        blocks = np.arange(0, 300, 7)
        vec = philox.philox4x32_blocks(blocks, stream, g, seed)
        for i, j in enumerate(blocks):
            want = philox.philox4((int(j), stream, g & 0xFFFFFFFF, g >> 32),
                                  (seed & 0xFFFFFFFF, seed >> 32))
            assert [int(x) for x in vec[i]] == list(want)


def test_uniform_open_interval_and_float32_exact():
    words = np.array([0, 1, 511, 512, 2**31, 2**32 - 1], dtype=np.uint64)
    for w in words:
        u = philox.word_to_uniform(int(w))
        assert 0.0 < u < 1.0
        assert float(np.float32(u)) == u
    assert philox.word_to_uniform(0) == 2.0 ** -24
    assert philox.word_to_uniform(2**32 - 1) == 1.0 - 2.0 ** -24


def test_uniformity_and_stream_independence():
    seed = 99
    u = philox.uniforms(seed, philox.STREAM_PROP_ELEM, 5, np.arange(200000))
    hist, _ = np.histogram(u, bins=50, range=(0, 1))
    expected = len(u) / 50
    chi2 = ((hist - expected) ** 2 / expected).sum()
    assert chi2 < 100.0  # 49 dof: P(chi2 > 100) < 1e-5
    v = philox.uniforms(seed, philox.STREAM_RES_ELEM, 5, np.arange(200000))
    assert abs(np.corrcoef(u, v)[0, 1]) < 0.02
    w = philox.uniforms(seed, philox.STREAM_PROP_ELEM, 6, np.arange(200000))
    assert abs(np.corrcoef(u, w)[0, 1]) < 0.02


def test_determinism():
    a = philox.uniforms(1, 2, 3, range(64))
    b = philox.uniforms(1, 2, 3, range(64))
    assert np.array_equal(a, b)
    assert not np.array_equal(a, philox.uniforms(2, 2, 3, range(64)))
