"""The kernels' float quotient floor(i / d) = int((float(i) + 0.5f) * (1.0f / d))
(`div_small` in csrc/common.h: tile coordinates, staging and epilogue
indices), checked exhaustively in float32 over the range the kernels use it
in (i + d < 2^21 for the grid coordinates, and far smaller elsewhere)."""
import numpy as np

LIMIT = 1 << 21


def _div_small(i: np.ndarray, d: int) -> np.ndarray:
    inv = np.float32(1.0) / np.float32(d)                    # IEEE division, as on the host
    return ((i.astype(np.float32) + np.float32(0.5)) * inv).astype(np.int64)


def test_div_small_is_exact_for_grid_divisors():
    # row blocks (gy), column tiles x row blocks (gx * gy), words of K, row-block
    # heights and segment widths of the step's products and of large grids
    divisors = sorted({1, 2, 3, 4, 5, 7, 8, 12, 16, 31, 32, 33, 48, 64, 96, 127, 128, 255, 256,
                       500, 1000, 1023, 1024, 2048, 4095, 4096, 6144, 12288, 32000, 65535, 65536,
                       96 * 4, 32 * 8, 500 * 2, 224 * 4, 48 * 128, 64 * 128, 16 * 128, 3 * 11 * 13 * 17})
    for d in divisors:
        i = np.arange(0, LIMIT - d, dtype=np.int64)
        got = _div_small(i, d)
        bad = np.nonzero(got != i // d)[0]
        assert bad.size == 0, f"d={d}: first wrong quotient at i={int(i[bad[0]])}"


def test_div_small_random_divisors():
    rng = np.random.default_rng(17)
    for d in rng.integers(1, 1 << 17, size=24):
        d = int(d)
        i = np.arange(0, LIMIT - d, 7, dtype=np.int64)
        assert np.array_equal(_div_small(i, d), i // d), d
