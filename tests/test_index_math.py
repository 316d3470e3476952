"""Host checks of index arithmetic the kernels rely on (no GPU).

The product kernels split flat item indices with a float reciprocal instead
of an integer division: floor(i / d) = trunc((float(i) + 0.5) * fl(1 / d))
for i + d < 2^22.  IEEE float32 arithmetic rounds the same way on the host,
so the claim is checked here exhaustively on a grid and by sampling up to
the bound.
"""
import numpy as np


def div_small(i, d):
    i = np.asarray(i, dtype=np.int64)
    d = np.asarray(d, dtype=np.int64)
    inv = np.float32(1.0) / d.astype(np.float32)
    q = (i.astype(np.float32) + np.float32(0.5)) * inv
    assert q.dtype == np.float32
    return q.astype(np.int64)  # truncation toward zero, as the device conversion


def test_div_small_exhaustive_small_range():
    i = np.arange(0, 1 << 14, dtype=np.int64)[None, :]
    d = np.arange(1, 513, dtype=np.int64)[:, None]
    np.testing.assert_array_equal(div_small(i, d), i // d)


def test_div_small_sampled_to_the_bound():
    rng = np.random.default_rng(3)
    d = rng.integers(1, 1 << 21, size=2_000_000)
    i = (rng.random(d.size) * ((1 << 22) - d)).astype(np.int64)  # i + d < 2^22
    np.testing.assert_array_equal(div_small(i, d), i // d)
    # quotients right below and at a multiple: i = q*d - 1 and q*d
    for k in (1, 2, 3, 7, 1000):
        dd = rng.integers(1, (1 << 22) // (k + 1), size=200_000)
        for i2 in (k * dd - 1, k * dd):
            ok = i2 + dd < (1 << 22)
            np.testing.assert_array_equal(div_small(i2[ok], dd[ok]), i2[ok] // dd[ok])
