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


# ---------------------------------------------------------------------------
# product + modified IF neuron (Eqs. (9)-(10)): ternary spike planes out
# ---------------------------------------------------------------------------
def _product_if_gpu(sp, sn, T, M, K, W, thr_num, thr_den, flags=0, want_v=True):
    torch, B = need_gpu()
    N = W.shape[1]
    Nw = (N + 63) // 64
    Wp, ldw = pad_weights(W)
    Wd = torch.from_numpy(Wp).cuda()
    tn = torch.from_numpy(np.asarray(thr_num, dtype=np.int64)).cuda()
    op = torch.full((T, M, Nw), -1, dtype=torch.int64, device="cuda")
    on = torch.full((T, M, Nw), -1, dtype=torch.int64, device="cuda")
    v = torch.full((M, N), 12345, dtype=torch.int64, device="cuda") if want_v else None
    stats = torch.zeros(4, dtype=torch.int64, device="cuda")
    ws = B.workspace(B.nmdlm_qbsm_workspace_size(T, M, K, N))
    B.nmdlm_qbsm_ternary_if(sp, sn, T, M, K, Wd, N, ldw, tn, thr_den, op, on, v_out=v,
                            stats=stats, flags=flags, ws=ws)
    torch.cuda.synchronize()
    return op, on, (v.cpu().numpy() if want_v else None), stats.cpu().numpy()


def _planes_to_ternary(op, on, N):
    from paper_2607_24841_amd import binding as B
    wp, wn = B.from_dev_bits(op), B.from_dev_bits(on)
    if N % 64:   # padding bits are written as zero
        assert np.all((wp[..., -1] >> np.uint64(N % 64)) == 0)
        assert np.all((wn[..., -1] >> np.uint64(N % 64)) == 0)
    p, n = synth.unpack_bits(wp, N), synth.unpack_bits(wn, N)
    assert not np.any(p & n)
    return p.astype(np.int8) - n.astype(np.int8)


MODIF = [(8, 4, 300, 70, 2), (8, 16, 1024, 512, 2), (4, 3, 65, 129, 1), (1, 1, 1, 1, 1),
         (3, 9, 2000, 100, 4), (8, 40, 512, 64, 2), (8, 2, 16384, 64, 2)]


@pytest.mark.parametrize("T,M,K,N,Kq", MODIF, ids=[f"T{p[0]}M{p[1]}K{p[2]}N{p[3]}" for p in MODIF])
def test_product_modified_if_bit_exact(T, M, K, N, Kq):
    c = synth.ternary_case(seed=40 + K, M=M, D=K, N=N, K=Kq, T=T)
    a = c.a.copy()
    if M > 2:
        a[1] = 0                                  # an all-zero token: Vth = 0, silent
    sp, sn, ss = _encode_gpu(a, c.K, c.T)
    S = ss.cpu().numpy()
    op, on, v, st = _product_if_gpu(sp, sn, T, M, K, c.W, S, K * c.K)
    s_in, S_ref = _planes_ref(a, c.K, c.T)
    assert_same(S, S_ref, "magnitude sums")
    I_ref, _ = O.qbsm_ternary(s_in, c.W)
    s_ref, V_ref = O.modified_if(I_ref, S_ref, K * c.K)
    assert_same(_planes_to_ternary(op, on, N), s_ref, "output spike planes")
    assert_same(v, V_ref, "final membrane x den")
    act = int(O.ternary_union(s_in).sum())
    assert st[0] == K and st[1] == act and st[3] == act * N
    if M > 2:
        assert not s_ref[:, 1].any()


@pytest.mark.parametrize("flags", [1 << 16, 2 << 16, 4 << 16, 2 << 8, 3 << 8, 1],
                         ids=["RT1", "RT2", "RT4", "P2", "P3", "dense"])
def test_product_modified_if_forced_tiles_and_splits(flags):
    c = synth.ternary_case(seed=33, M=12, D=700, N=190, K=2, T=8)
    sp, sn, ss = _encode_gpu(c.a, c.K, c.T)
    S = ss.cpu().numpy()
    op, on, v, _ = _product_if_gpu(sp, sn, 8, 12, 700, c.W, S, 700 * 2, flags=flags)
    s_in, S_ref = _planes_ref(c.a, c.K, c.T)
    assert_same(S, S_ref, "magnitude sums")
    s_ref, V_ref = O.modified_if(O.qbsm_ternary(s_in, c.W)[0], S_ref, 700 * 2)
    assert_same(_planes_to_ternary(op, on, 190), s_ref, "output spike planes")
    assert_same(v, V_ref, "final membrane x den")


def test_modified_if_two_layer_chain():
    """encode -> product + modified IF -> product + modified IF: the second
    layer reads the first layer's output planes directly, with the first
    layer's threshold (integer Vth = 50) reused; no GPU output feeds the oracle."""
    torch, B = need_gpu()
    c = synth.ternary_case(seed=51, M=6, D=256, N=192, K=2, T=8)
    W2 = synth.int8_uniform(synth.stream(52, 1), (192, 96))
    sp, sn, ss = _encode_gpu(c.a, c.K, c.T)
    S = ss.cpu().numpy()
    op, on, _, _ = _product_if_gpu(sp, sn, 8, 6, 256, c.W, S, 256 * 2, want_v=False)
    op2, on2, v2, _ = _product_if_gpu(op, on, 8, 6, 192, W2, np.full(6, 50), 1)
    s_in, S_ref = _planes_ref(c.a, c.K, c.T)
    assert_same(S, S_ref, "magnitude sums")
    s1, _ = O.modified_if(O.qbsm_ternary(s_in, c.W)[0], S_ref, 256 * 2)
    s2, V2 = O.modified_if(O.qbsm_ternary(s1, W2)[0], np.full(6, 50), 1)
    assert_same(_planes_to_ternary(op2, on2, 96), s2, "second layer planes")
    assert_same(v2, V2, "second layer membrane")


def test_product_modified_if_full_size_ffn_up():
    c = synth.ternary_case()
    M, D = c.a.shape
    sp, sn, ss = _encode_gpu(c.a, c.K, c.T)
    S = ss.cpu().numpy()
    op, on, v, _ = _product_if_gpu(sp, sn, c.T, M, D, c.W, S, D * c.K)
    s_in, S_ref = _planes_ref(c.a, c.K, c.T)
    assert_same(S, S_ref, "magnitude sums")
    s_ref, V_ref = O.modified_if(O.qbsm_ternary(s_in, c.W)[0], S_ref, D * c.K)
    assert_same(_planes_to_ternary(op, on, c.W.shape[1]), s_ref, "output spike planes")
    assert_same(v, V_ref, "final membrane x den")
