"""GPU parity of nmdlm_qbsm (with and without the fused IF epilogue) against
the oracle: bit-exact currents, spikes and skip statistics."""
import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

from ._gpu import assert_same, need_gpu, padding_bits_zero, run_qbsm

pytestmark = pytest.mark.gpu

SHAPES = [  # T, M, K, N, density
    (1, 1, 1, 1, 0.5),
    (4, 3, 16, 16, 0.3),
    (2, 5, 13, 9, 0.3),
    (4, 1, 63, 65, 0.2),
    (4, 2, 64, 64, 0.2),
    (4, 5, 65, 200, 0.1),
    (3, 7, 200, 63, 0.1),
    (1, 17, 100, 130, 0.05),
    (4, 40, 300, 70, 0.1),       # two row blocks
    (8, 20, 129, 190, 0.1),      # T = 8
    (4, 8, 1000, 333, 0.005),    # heavy skipping
    (4, 16, 1024, 1024, 0.1),
]


def _check(case, flags=0, theta_vec=None, blocked=False):
    I_ref = O.qbsm(case.S, case.W, case.bias)
    th = case.theta if theta_vec is None else np.asarray(theta_vec)
    s_ref, _ = O.if_neuron(I_ref, th)
    cur, spk, st, words, _ = run_qbsm(case.S, case.W, case.bias, theta=case.theta,
                                      theta_vec=theta_vec, flags=flags, blocked=blocked)
    assert_same(cur, I_ref)
    assert_same(spk, s_ref)
    assert padding_bits_zero(words, case.N)
    dense = bool(flags & 1)
    k_act = case.K if dense else O.active_rows(case.S).size
    assert st["k_total"] == case.K and st["k_active"] == k_act and st["n"] == case.N
    assert st["weight_bytes"] == k_act * case.N


def test_linear_layer_bit_exact():
    need_gpu()
    _check(synth.linear_layer_case())


@pytest.mark.parametrize("shape", SHAPES, ids=[f"T{s[0]}M{s[1]}K{s[2]}N{s[3]}" for s in SHAPES])
def test_tiny_and_ragged_shapes(shape):
    need_gpu()
    T, M, K, N, p = shape
    _check(synth.make_qbsm_case(100 + K + N, T, M, K, N, p))


NOFUSE = 1 << 20      # prep pass + list kernel
FUSED = 2 << 20       # single kernel, in-kernel list
WORDS = 3 << 20       # single kernel over 64-channel words
SCALAR = 5 << 20      # words, scalar gather-accumulate product
DMA = 4 << 20         # as WORDS, active rows gathered into LDS
BLOCKED = 6 << 20     # as WORDS, over the blocked weight copy
WIDE = 7 << 20        # as BLOCKED, four column tiles per workgroup (64-row tiles)

_FORCED = {
    "dense": 0x1, "P1": 1 << 8, "P2": 2 << 8, "P7": 7 << 8, "RT1": 1 << 16, "RT2": 2 << 16,
    "RT4": 4 << 16, "RT8": 8 << 16, "P3RT1": (3 << 8) | (1 << 16),
    "nofuse": NOFUSE, "nofuse-dense": NOFUSE | 0x1, "nofuse-P2": NOFUSE | (2 << 8),
    "nofuse-RT1": NOFUSE | (1 << 16), "nofuse-RT8": NOFUSE | (8 << 16),
    "fused": FUSED, "fused-dense": FUSED | 0x1, "fused-P2": FUSED | (2 << 8),
    "fused-RT1": FUSED | (1 << 16), "fused-RT2": FUSED | (2 << 16),
    "words": WORDS, "words-dense": WORDS | 0x1, "words-P3": WORDS | (3 << 8),
    "words-RT1": WORDS | (1 << 16), "words-RT4": WORDS | (4 << 16), "words-RT8": WORDS | (8 << 16),
    "words-P2RT2": WORDS | (2 << 8) | (2 << 16),
    "dma": DMA, "dma-dense": DMA | 0x1, "dma-P3": DMA | (3 << 8), "dma-RT1": DMA | (1 << 16),
    "dma-RT2": DMA | (2 << 16), "dma-RT4": DMA | (4 << 16), "dma-RT8": DMA | (8 << 16),
    "dma-P2RT2": DMA | (2 << 8) | (2 << 16),
    "scalar": SCALAR, "scalar-dense": SCALAR | 0x1, "scalar-P3": SCALAR | (3 << 8),
    "scalar-RT1": SCALAR | (1 << 16), "scalar-RT2": SCALAR | (2 << 16),
    "scalar-RT4": SCALAR | (4 << 16), "scalar-RT8": SCALAR | (8 << 16),
}


@pytest.mark.parametrize("flags", [SCALAR, SCALAR | (1 << 16), SCALAR | (8 << 16), SCALAR | (2 << 8)],
                         ids=["scalar", "scalar-RT1", "scalar-RT8", "scalar-P2"])
@pytest.mark.parametrize("shape", SHAPES, ids=[f"T{s[0]}M{s[1]}K{s[2]}N{s[3]}" for s in SHAPES])
def test_scalar_ragged_shapes(shape, flags):
    need_gpu()
    T, M, K, N, p = shape
    _check(synth.make_qbsm_case(100 + K + N, T, M, K, N, p), flags=flags)


@pytest.mark.parametrize("density", [0.001, 0.01, 0.05, 0.3])
def test_scalar_across_densities(density):
    # the scalar product from nearly empty to dense rows, short and long K
    need_gpu()
    for flags in (0, SCALAR):
        _check(synth.make_qbsm_case(int(1000 * density) + 7, 4, 20, 4096, 300, density), flags=flags)
        _check(synth.make_qbsm_case(int(1000 * density) + 8, 4, 1, 14336, 256, density), flags=flags)


@pytest.mark.parametrize("flags", list(_FORCED.values()), ids=list(_FORCED))
def test_forced_paths_equal(flags):
    need_gpu()
    case = synth.make_qbsm_case(5, 4, 24, 700, 300, 0.05)
    _check(case, flags=flags)


@pytest.mark.parametrize("flags", [0, NOFUSE, FUSED, WORDS, DMA, SCALAR],
                         ids=["auto", "nofuse", "fused", "words", "dma", "scalar"])
def test_degenerate_inputs(flags):
    need_gpu()
    c = synth.make_qbsm_case(9, 4, 8, 256, 128, 0.1)
    c.S[:] = False                   # no spike: K_active = 0, currents = bias
    _check(c, flags=flags)
    c.S[:] = True                    # every row active
    _check(c, flags=flags)


@pytest.mark.parametrize("flags", [0, NOFUSE, WORDS, DMA, SCALAR],
                         ids=["auto", "nofuse", "words", "dma", "scalar"])
def test_large_k_shapes(flags):
    need_gpu()
    # K beyond the in-kernel-list limit, and a long block (many row blocks)
    _check(synth.make_qbsm_case(41, 4, 4, 20000, 130, 0.02), flags=flags)
    _check(synth.make_qbsm_case(42, 4, 300, 700, 200, 0.05), flags=flags)


@pytest.mark.parametrize("flags", [0, NOFUSE, WORDS, DMA, 1], ids=["auto", "nofuse", "words", "dma", "dense"])
def test_maximum_k(flags):
    # K = NMDLM_MAX_K = 65536: the tile's staged spike rows exceed the word
    # kernel's LDS, so every requested path falls back to the list kernels
    need_gpu()
    _check(synth.make_qbsm_case(45, 4, 2, 65536, 96, 0.003), flags=flags)


@pytest.mark.parametrize("M,flags", [(3, 0), (9, 0), (9, 1 << 8), (3, 1)],
                         ids=["auto-split", "auto-split-3blocks", "P1-requested", "dense-split"])
def test_short_grid_long_k_split(M, flags):
    # at most 64 output tiles over 128 or more words of K: unrequested, K is
    # split four ways (K = 8257: a partial last word; N = 100: a ragged tile)
    need_gpu()
    _check(synth.make_qbsm_case(46, 4, M, 8257, 100, 0.02), flags=flags)


def test_words_with_more_than_64k_lds():
    need_gpu()
    # K = 14336 with two row groups: the staged spike rows need more than
    # 64 KB of LDS (the launch raises the dynamic LDS limit)
    c = synth.make_qbsm_case(44, 4, 16, 14336, 320, 0.01)
    _check(c, flags=WORDS | (2 << 16))
    _check(c)


def test_per_neuron_thresholds_and_currents_only():
    need_gpu()
    c = synth.make_qbsm_case(12, 4, 8, 300, 100, 0.2)
    tv = synth.int_uniform(synth.stream(3, 3), 128, 512, (100,))
    _check(c, theta_vec=tv)
    cur, spk, _, _, _ = run_qbsm(c.S, c.W, None, theta=None)
    assert spk is None and np.array_equal(cur, O.qbsm(c.S, c.W))


def test_workspace_reuse_across_calls():
    torch, B = need_gpu()
    c1 = synth.make_qbsm_case(21, 4, 16, 512, 256, 0.1)
    c2 = synth.make_qbsm_case(22, 4, 16, 512, 256, 0.3)
    ws = B.workspace(B.nmdlm_qbsm_workspace_size(4, 16, 512, 256))
    outs = []
    for c in (c1, c2, c1):
        s_in = B.to_dev_bits(synth.pack_bits(c.S))
        W = torch.from_numpy(c.W).cuda()
        cur = torch.empty((4, 16, 256), dtype=torch.int32, device="cuda")
        B.nmdlm_qbsm(s_in, 4, 16, 512, W, 256, 256, cur_out=cur, flags=4 << 8, ws=ws)
        torch.cuda.synchronize()
        outs.append(cur.cpu().numpy())
    assert np.array_equal(outs[0], O.qbsm(c1.S, c1.W)) and np.array_equal(outs[1], O.qbsm(c2.S, c2.W))
    assert_same(outs[2], outs[0])


def test_determinism():
    need_gpu()
    c = synth.make_qbsm_case(33, 4, 32, 2048, 2048, 0.1)
    a = run_qbsm(c.S, c.W, c.bias, theta=300)
    b = run_qbsm(c.S, c.W, c.bias, theta=300)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[3], b[3])


LARGE_BIAS_PATHS = [0, NOFUSE, FUSED, WORDS, DMA, SCALAR]


@pytest.mark.parametrize("T", [4, 8])
@pytest.mark.parametrize("path", LARGE_BIAS_PATHS, ids=["auto", "list", "fused", "words", "dma", "scalar"])
def test_membrane_beyond_int32_with_large_bias(T, path):
    """Biases near 2^30 with a threshold near 1.6e9: the membrane passes 2^31
    after two steps, so the fused IF must integrate in 64 bits as the oracle
    does (K*127 + |bias| < 2^31 keeps every current itself in int32)."""
    need_gpu()
    rng = np.random.default_rng(77 + T)
    K, N, M = 64, 130, 5
    S = rng.random((T, M, K)) < 0.3
    W = rng.integers(-127, 128, size=(K, N)).astype(np.int8)
    bias = (2 ** 30 + rng.integers(-20000, 20000, size=N)).astype(np.int32)
    bias[::7] = -bias[::7]                     # some neurons driven negative
    theta = 3 * 2 ** 29
    I_ref = O.qbsm(S, W, bias)
    s_ref, _ = O.if_neuron(I_ref, theta)
    assert s_ref.any() and not s_ref.all()
    cur, spk, _, _, _ = run_qbsm(S, W, bias, theta=theta, flags=path)
    assert_same(cur, I_ref)
    assert_same(spk, s_ref)


# ----------------------------------------------------------------------------
# blocked weight copy (nmdlm_weight_block, nmdlm_qbsm_blocked)
# ----------------------------------------------------------------------------
def _blocked_layout(W, K, N):
    """The blocked copy as the header defines it, built on the host."""
    Kw, gx = (K + 63) // 64, (N + 63) // 64
    Wp = np.zeros((Kw * 64, gx * 64), dtype=np.int8)
    Wp[:K, :N] = W[:K, :N]
    out = np.zeros((Kw, gx, 4, 64, 16), dtype=np.int8)
    for v in range(4):
        for lane in range(64):
            g, c = lane // 16, lane % 16
            # [w][j][x]: W[64w + 16g + j][64x + 4c + v]
            blk = Wp.reshape(Kw, 64, gx, 64)[:, 16 * g:16 * g + 16, :, 4 * c + v]
            out[:, :, v, lane, :] = blk.transpose(0, 2, 1)
    return out.reshape(-1)


@pytest.mark.parametrize("K,N,ldw", [(64, 64, 64), (130, 70, 80), (1, 1, 16), (200, 300, 320)])
def test_blocked_layout(K, N, ldw):
    torch, B = need_gpu()
    rng = np.random.default_rng(K * 7 + N)
    W = rng.integers(-128, 128, size=(K, ldw), dtype=np.int8)
    Wd = torch.from_numpy(W).cuda()
    Wb = B.blocked_weights(Wd, K, N, ldw)
    torch.cuda.synchronize()
    assert Wb.numel() == B.nmdlm_weight_blocked_bytes(K, N)
    assert_same(Wb.cpu().numpy(), _blocked_layout(W, K, N), "blocked copy")


@pytest.mark.parametrize("flags", [BLOCKED, BLOCKED | (1 << 16), BLOCKED | (2 << 16),
                                   BLOCKED | (8 << 16), BLOCKED | (2 << 8), BLOCKED | 0x1],
                         ids=["blocked", "blocked-RT1", "blocked-RT2", "blocked-RT8", "blocked-P2",
                              "blocked-dense"])
@pytest.mark.parametrize("shape", SHAPES, ids=[f"T{s[0]}M{s[1]}K{s[2]}N{s[3]}" for s in SHAPES])
def test_blocked_ragged_shapes(shape, flags):
    need_gpu()
    T, M, K, N, p = shape
    _check(synth.make_qbsm_case(100 + K + N, T, M, K, N, p), flags=flags, blocked=True)


@pytest.mark.parametrize("T,M,K,N,p", [
    (4, 256, 1024, 384, 0.05),      # 1024 rows: the blocked copy by default
    (4, 300, 700, 200, 0.02),       # ragged K and N, many row blocks
    (1, 1100, 130, 90, 0.3),        # T = 1
    (8, 200, 4096, 128, 0.01),      # long K, sparse words skipped
])
def test_blocked_automatic_at_many_rows(T, M, K, N, p):
    need_gpu()
    case = synth.make_qbsm_case(T * M + K, T, M, K, N, p)
    _check(case, blocked=True)
    case.S[:, :, 64:192] = False     # two words with no active row
    _check(case, blocked=True)


WIDE_SHAPES = [  # T, M, K, N, density: 64-row tiles, column groups of four tiles
    (4, 16, 64, 64, 0.2),        # one tile: three waves without a tile
    (4, 40, 300, 70, 0.1),       # two row blocks (the second ragged), ragged K
    (4, 33, 1000, 333, 0.05),    # six column tiles: one group and a ragged one
    (2, 70, 129, 520, 0.1),      # T = 2: 32-token row blocks, nine column tiles
    (1, 130, 65, 260, 0.3),      # T = 1: 64-token row blocks
    (8, 20, 4096, 200, 0.02),    # T = 8, long K, sparse words skipped
    (3, 50, 200, 1000, 0.1),     # T = 3: 21-token row blocks (one row unused)
    (4, 64, 2048, 1024, 0.1),    # sixteen column tiles, 32 words
]


@pytest.mark.parametrize("flags", [WIDE, WIDE | (4 << 16), WIDE | 0x1],
                         ids=["wide", "wide-RT4", "wide-dense"])
@pytest.mark.parametrize("shape", WIDE_SHAPES, ids=[f"T{s[0]}M{s[1]}K{s[2]}N{s[3]}" for s in WIDE_SHAPES])
def test_wide_ragged_shapes(shape, flags):
    need_gpu()
    T, M, K, N, p = shape
    _check(synth.make_qbsm_case(300 + K + N, T, M, K, N, p), flags=flags, blocked=True)


@pytest.mark.parametrize("flags", [WIDE, WIDE | (4 << 16)], ids=["wide", "wide-RT4"])
def test_wide_currents_only(flags):
    # no threshold: the currents alone, stored from the accumulators
    need_gpu()
    case = synth.make_qbsm_case(77, 2, 70, 300, 600, 0.1)
    I_ref = O.qbsm(case.S, case.W, case.bias)
    cur, spk, st, _, _ = run_qbsm(case.S, case.W, case.bias, flags=flags, blocked=True)
    assert spk is None
    assert_same(cur, I_ref)
    assert st["k_active"] == O.active_rows(case.S).size


@pytest.mark.parametrize("flags,blocked", [
    (WORDS | (4 << 16) | (2 << 8), False),     # 64-row tiles, K split two ways
    (WORDS | (4 << 16) | (3 << 8), False),     # three ways (ragged split)
    (BLOCKED | (4 << 16) | (2 << 8), True),    # the same over the blocked copy
    (DMA | (4 << 16), False),                  # the LDS-streamed kernel keeps its own tile
], ids=["rows-RT4-P2", "rows-RT4-P3", "blocked-RT4-P2", "dma-RT4"])
def test_tall_tiles_with_k_split(flags, blocked):
    # 64-row tiles reduce into an LDS tile laid over the spike rows; with a K
    # split the last arriving workgroup reads the accumulated tile from there
    need_gpu()
    _check(synth.make_qbsm_case(501, 4, 37, 1100, 333, 0.05), flags=flags, blocked=blocked)
    _check(synth.make_qbsm_case(502, 2, 70, 4100, 130, 0.02), flags=flags, blocked=blocked)


def test_wide_automatic_at_many_tiles():
    # 8192 rows x 1024 columns: 2048 output tiles of 64 x 64 (wide from 1536)
    need_gpu()
    case = synth.make_qbsm_case(4242, 4, 2048, 200, 1024, 0.1)
    _check(case, blocked=True)
    case.S[:, :, 64:128] = False     # a word with no active row
    _check(case, blocked=True)


def test_blocked_degenerate_inputs():
    need_gpu()
    c = synth.make_qbsm_case(19, 4, 300, 256, 128, 0.1)
    c.S[:] = False
    _check(c, flags=BLOCKED, blocked=True)
    _check(c, blocked=True)
    _check(c, flags=WIDE, blocked=True)
    c.S[:] = True
    _check(c, flags=BLOCKED, blocked=True)
    _check(c, blocked=True)
    _check(c, flags=WIDE, blocked=True)
