"""GPU parity of the ternary bitwise-coded conversion (Sec. III-B, Eqs.
(7)-(11)) against the oracle: bit-exact spike planes and magnitude sums from
nmdlm_ternary_encode, bit-exact reconstructed products and skip statistics
from nmdlm_qbsm_ternary."""
import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

from ._gpu import assert_same, need_gpu, pad_weights

pytestmark = pytest.mark.gpu


def _encode_gpu(a, K, T):
    torch, B = need_gpu()
    M, D = a.shape
    Dw = (D + 63) // 64
    ad = torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    sp = torch.full((T, M, Dw), -1, dtype=torch.int64, device="cuda")
    sn = torch.full((T, M, Dw), -1, dtype=torch.int64, device="cuda")
    ss = torch.zeros(M, dtype=torch.int64, device="cuda")
    B.nmdlm_ternary_encode(ad, M, D, K, T, sp, sn, ss)
    torch.cuda.synchronize()
    return sp, sn, ss


def _planes_ref(a, K, T):
    q, S = O.ternary_quantize(a, K, T)
    return O.ternary_planes(q, T), S


ENC = [(1, 1, 1, 1), (3, 63, 2, 8), (2, 65, 1, 4), (5, 300, 4, 8), (4, 4096, 2, 8), (2, 129, 3, 3),
       (3, 16384, 63, 8)]   # the largest D K accepted (< 2^20)


@pytest.mark.parametrize("M,D,K,T", ENC, ids=[f"M{e[0]}D{e[1]}K{e[2]}T{e[3]}" for e in ENC])
def test_encode_bit_exact(M, D, K, T):
    a = synth.ternary_activations(synth.stream(10 + D, M), M, D)
    a[0, : min(D, 3)] = [2 ** 31 - 1, -(2 ** 31), 7][: min(D, 3)]   # extreme magnitudes
    if M > 1 and D > 1:
        a[1] = 0                                                     # a single nonzero channel:
        a[1, D // 2] = -5                                            # |q| = D K saturates at 2^T - 1
    if M > 2:
        a[2] = 0                                                     # an all-zero token
    sp, sn, ss = _encode_gpu(a, K, T)
    s_ref, S_ref = _planes_ref(a, K, T)
    from paper_2607_24841_amd import binding as B
    assert_same(synth.unpack_bits(B.from_dev_bits(sp), D), s_ref == 1, "+1 plane")
    assert_same(synth.unpack_bits(B.from_dev_bits(sn), D), s_ref == -1, "-1 plane")
    assert_same(ss.cpu().numpy(), S_ref, "magnitude sums")
    if D % 64:   # padding bits of the last word are zero
        last = B.from_dev_bits(sp)[..., -1] | B.from_dev_bits(sn)[..., -1]
        assert np.all((last >> np.uint64(D % 64)) == 0)


def _product_gpu(sp, sn, T, M, K, W, flags=0):
    torch, B = need_gpu()
    N = W.shape[1]
    Wp, ldw = pad_weights(W)
    Wd = torch.from_numpy(Wp).cuda()
    acc = torch.full((M, N), -7, dtype=torch.int32, device="cuda")
    stats = torch.zeros(4, dtype=torch.int64, device="cuda")
    ws = B.workspace(B.nmdlm_qbsm_workspace_size(T, M, K, N))
    B.nmdlm_qbsm_ternary(sp, sn, T, M, K, Wd, N, ldw, acc, stats=stats, flags=flags, ws=ws)
    torch.cuda.synchronize()
    return acc.cpu().numpy().astype(np.int64), stats.cpu().numpy()


PROD = [(8, 4, 300, 70, 2), (8, 16, 1024, 512, 2), (4, 3, 65, 129, 1), (1, 1, 1, 1, 1),
        (8, 9, 2000, 100, 4), (8, 64, 512, 64, 2),
        (8, 2, 16384, 64, 2)]   # K = NMDLM_MAX_TERNARY_K


@pytest.mark.parametrize("T,M,K,N,Kq", PROD, ids=[f"T{p[0]}M{p[1]}K{p[2]}N{p[3]}" for p in PROD])
def test_product_bit_exact(T, M, K, N, Kq):
    c = synth.ternary_case(seed=20 + K, M=M, D=K, N=N, K=Kq, T=T)
    sp, sn, _ = _encode_gpu(c.a, c.K, c.T)
    acc, st = _product_gpu(sp, sn, T, M, K, c.W)
    s_ref, _ = _planes_ref(c.a, c.K, c.T)
    _, acc_ref = O.qbsm_ternary(s_ref, c.W)
    assert_same(acc, acc_ref, "reconstructed product")
    act = int(O.ternary_union(s_ref).sum())
    assert st[0] == K and st[1] == act and st[2] == N and st[3] == act * N


@pytest.mark.parametrize("flags", [1 << 16, 2 << 16, 4 << 16, 2 << 8, 3 << 8, 1],
                         ids=["RT1", "RT2", "RT4", "P2", "P3", "dense"])
def test_product_forced_tiles_and_splits(flags):
    c = synth.ternary_case(seed=31, M=12, D=700, N=190, K=2, T=8)
    sp, sn, _ = _encode_gpu(c.a, c.K, c.T)
    acc, st = _product_gpu(sp, sn, 8, 12, 700, c.W, flags=flags)
    s_ref, _ = _planes_ref(c.a, c.K, c.T)
    assert_same(acc, O.qbsm_ternary(s_ref, c.W)[1], "reconstructed product")
    assert st[1] == (700 if flags == 1 else int(O.ternary_union(s_ref).sum()))


def test_full_size_ffn_up():
    # the FFN up projection of the sweep's shape (4096 -> 14336), T = 8, 4 tokens
    c = synth.ternary_case()
    sp, sn, ss = _encode_gpu(c.a, c.K, c.T)
    acc, st = _product_gpu(sp, sn, c.T, c.a.shape[0], c.a.shape[1], c.W)
    s_ref, S_ref = _planes_ref(c.a, c.K, c.T)
    _, acc_ref = O.qbsm_ternary(s_ref, c.W)
    assert_same(acc, acc_ref, "reconstructed product")
    q, _ = O.ternary_quantize(c.a, c.K, c.T)
    assert np.array_equal(acc, q @ c.W.astype(np.int64))            # Eq. (11), exact
    assert st[1] == int(O.ternary_union(s_ref).sum())
    assert_same(ss.cpu().numpy(), S_ref, "magnitude sums (V_th = S / (D K))")
