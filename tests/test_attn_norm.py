"""CPU check of the attention normalisation's quotient: floor(256 num / den)
for 0 <= num <= den < 255 * 65536 taken as a float product with a reciprocal
(correctly rounded, or one unit in the last place off either way, as the
hardware reciprocal may be) and one remainder correction equals the exact
integer quotient."""
import numpy as np


def _quotient(num, den, ulp_shift):
    a = (256 * num).astype(np.uint64)
    b = den.astype(np.uint64)
    rb = (np.float32(1.0) / den.astype(np.float32)).astype(np.float32)
    if ulp_shift:
        rb = np.nextafter(rb, np.float32(np.inf) if ulp_shift > 0 else np.float32(0)).astype(np.float32)
    q = (a.astype(np.float32) * rb).astype(np.float32).astype(np.uint64)   # truncation
    r = a.astype(np.int64) - (q * b).astype(np.int64)
    q = np.where(r < 0, q - 1, np.where(r >= b.astype(np.int64), q + 1, q))
    return q


def test_float_quotient_is_exact():
    rng = np.random.default_rng(12)
    dmax = 255 * 65535
    den = np.concatenate([np.arange(1, 4097), rng.integers(1, dmax + 1, 400000),
                          np.full(4096, dmax), 255 * rng.integers(1, 65536, 100000)]).astype(np.int64)
    frac = rng.random(den.size)
    num = np.floor(frac * (den + 1)).astype(np.int64)
    num = np.minimum(num, den)
    # the extremes: empty and full value channel, and multiples that make
    # the quotient an integer
    num[:4096] = 0
    num[4096:8192] = den[4096:8192]
    k = rng.integers(0, 257, den.size)
    sel = slice(8192, 60000)
    num[sel] = np.minimum((k[sel] * den[sel]) // 256, den[sel])
    exact = (256 * num) // den
    for shift in (0, 1, -1):
        assert np.array_equal(_quotient(num, den, shift), exact)
