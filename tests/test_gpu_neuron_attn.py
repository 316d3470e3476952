"""GPU parity of nmdlm_if_neuron, nmdlm_qnl_lut and nmdlm_bbm_attn against the
oracle (bit-exact)."""
import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

from ._gpu import assert_same, need_gpu

pytestmark = pytest.mark.gpu


def _if_gpu(I, theta, theta_vec=None, resid=None, v0=None):
    torch, B = need_gpu()
    T, M, N = I.shape
    cur = torch.from_numpy(I.astype(np.int32)).cuda()
    Nw = (N + 63) // 64
    out = torch.full((T, M, Nw), -1, dtype=torch.int64, device="cuda")
    rd = B.to_dev_bits(synth.pack_bits(resid)) if resid is not None else None
    tv = torch.from_numpy(np.asarray(theta_vec, np.int32)).cuda() if theta_vec is not None else None
    vd = torch.from_numpy(v0.astype(np.int32)).cuda() if v0 is not None else None
    B.nmdlm_if_neuron(cur, T, M, N, theta=theta, theta_vec=tv, resid=rd, v_inout=vd, s_out=out)
    torch.cuda.synchronize()
    s = synth.unpack_bits(B.from_dev_bits(out), N)
    return s, (vd.cpu().numpy() if vd is not None else None)


def test_if_neuron_parity():
    rng = np.random.default_rng(0)
    I = rng.integers(-2000, 2000, size=(4, 7, 130))
    s, _ = _if_gpu(I, 300)
    assert_same(s, O.if_neuron(I, 300)[0])
    R = rng.random(I.shape) < 0.3
    s, _ = _if_gpu(I, 300, resid=R)
    assert_same(s, O.if_neuron(I, 300, resid=R)[0])
    tv = rng.integers(1, 700, size=130)
    s, _ = _if_gpu(I, 0, theta_vec=tv)
    assert_same(s, O.if_neuron(I, tv)[0])


def test_if_neuron_initial_membrane_and_hand_traces():
    rng = np.random.default_rng(1)
    I = rng.integers(-500, 900, size=(8, 3, 64))
    v0 = rng.integers(-300, 300, size=(3, 64))
    s, vend = _if_gpu(I, 256, v0=v0)
    I2 = I.copy()
    I2[0] += v0                       # starting from v0 == adding v0 to the first current
    s_ref, v_ref = O.if_neuron(I2, 256)
    assert np.array_equal(s, s_ref) and np.array_equal(vend, v_ref)
    # the hand-worked traces, one neuron each
    rows = [l for l in open(__import__("os").path.join(__import__("os").path.dirname(__file__),
                                                        "golden", "if_traces.txt"))
            if l.strip() and not l.startswith("#")]
    for line in rows:
        th, cur, spikes, vfin = [x.strip() for x in line.split("|")]
        cur = np.array([int(x) for x in cur.split()]).reshape(-1, 1, 1)
        s, v = _if_gpu(cur, int(th), v0=np.zeros((1, 1), np.int64))
        assert s[:, 0, 0].astype(int).tolist() == [int(x) for x in spikes.split()]
        assert int(v[0, 0]) == int(vfin)


def test_qnl_lut_parity():
    torch, B = need_gpu()
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.integers(-2 ** 31, 2 ** 31, size=5000),
                        np.array([-2 ** 31, 2 ** 31 - 1, -1, 0, 1, 255, 256, -129, 127, 128])])
    lut_s = synth.sorted_lut_s8(synth.stream(5, 1))
    lut_u = synth.sorted_lut_u8(synth.stream(5, 2))
    xd = torch.from_numpy(x.astype(np.int32)).cuda()
    for mode, lut in ((B.NMDLM_QNL_S8, lut_s), (B.NMDLM_QNL_U8, lut_u)):
        for shift in (0, 3, 9, 31):
            y = torch.empty(x.size, dtype=torch.uint8, device="cuda")
            B.nmdlm_qnl_lut(xd, x.size, shift, mode, torch.from_numpy(lut).cuda(), y)
            torch.cuda.synchronize()
            got = y.cpu().numpy()
            ref = O.qnl_lut(x, shift, lut, mode)
            ref_bytes = (ref & 0xFF).astype(np.uint8)
            assert np.array_equal(got, ref_bytes), (mode, shift)


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------
def _attn_case(seed, T, M, C, H, dh, p, stale=True):
    rng = np.random.default_rng(seed)
    d = H * dh
    J = C + M
    cap = (J + 63) // 64 * 64 + (64 if stale else 0)
    Q = rng.random((T, M, d)) < p
    Kc = rng.random((T, cap, d)) < p
    Vc = rng.random((T, cap, d)) < p
    if stale:                      # rows past C+M must be ignored
        Kc[:, J:] = True
        Vc[:, J:] = True
    lut = synth.sorted_lut_u8(synth.stream(seed, 7))
    return Q, Kc, Vc, lut, cap


def _vt_words(Vc):
    """Value cache [T][cap][d] bits -> device words [T][cap/64][d] (word-major)."""
    _, B = need_gpu()
    words = synth.pack_bits(Vc.transpose(0, 2, 1))            # [T][d][cap/64]
    return B.to_dev_bits(np.ascontiguousarray(words.transpose(0, 2, 1)))


def _attn_gpu(Q, Kc, Vc, lut, cap, C, H, dh, theta=None):
    torch, B = need_gpu()
    T, M, d = Q.shape
    q = B.to_dev_bits(synth.pack_bits(Q))
    k = B.to_dev_bits(synth.pack_bits(Kc))
    vt = _vt_words(Vc)
    a = torch.full((T, M, d), -5, dtype=torch.int32, device="cuda")
    s_out = torch.full((T, M, d // 64), -1, dtype=torch.int64, device="cuda") if theta else None
    B.nmdlm_bbm_attn(q, k, vt, cap, T, M, C, H, dh, torch.from_numpy(lut).cuda(), a_out=a,
                     theta_a=int(theta or 0), s_out=s_out)
    torch.cuda.synchronize()
    spikes = synth.unpack_bits(B.from_dev_bits(s_out), d) if theta else None
    return a.cpu().numpy().astype(np.int64), spikes


ATTN = [  # T, M, C, H, dh, p
    (2, 5, 37, 2, 64, 0.5),
    (1, 1, 0, 1, 128, 0.5),
    (4, 40, 100, 3, 64, 0.2),
    (4, 16, 512, 16, 64, 0.3),     # the one-block step (d=1024, 16 heads of 64)
    (4, 32, 1024, 16, 128, 0.4),   # the 12-layer model step (16 heads of 128)
    (3, 17, 63, 2, 128, 0.05),
    # grids beyond one round of the chip: 8 and 4 waves per workgroup
    (4, 192, 64, 8, 64, 0.3),
    (4, 300, 40, 8, 64, 0.25),
    (4, 520, 30, 4, 128, 0.3),
    # dh = 128, several key chunks per wave: 12 waves with five or six chunks
    # each, 8 waves with two or three
    (4, 32, 4000, 16, 128, 0.3),
    (4, 80, 1000, 16, 128, 0.3),
    # 65564 keys: the normalisation's 64-bit path (256 * num beyond 32 bits)
    (1, 4, 65560, 1, 64, 0.5),
]


@pytest.mark.parametrize("shape", ATTN, ids=[f"T{s[0]}M{s[1]}C{s[2]}H{s[3]}dh{s[4]}" for s in ATTN])
def test_attention_parity(shape):
    T, M, C, H, dh, p = shape
    Q, Kc, Vc, lut, cap = _attn_case(sum(shape[:5]), T, M, C, H, dh, p)
    a, s = _attn_gpu(Q, Kc, Vc, lut, cap, C, H, dh, theta=300)
    a_ref = O.bbm_attention(Q, Kc, Vc, C + M, H, lut)
    assert_same(a, a_ref)
    assert_same(s, O.if_neuron(a_ref, 300)[0])


def _attn_spikes_gpu(Q, Kc, Vc, lut, cap, C, H, dh, theta):
    """Spikes only (no currents out): the attention kernel with the IF fused
    in, or attention + IF when its partial sums do not fit in LDS."""
    torch, B = need_gpu()
    T, M, d = Q.shape
    q = B.to_dev_bits(synth.pack_bits(Q))
    k = B.to_dev_bits(synth.pack_bits(Kc))
    vt = _vt_words(Vc)
    s_out = torch.full((T, M, d // 64), -1, dtype=torch.int64, device="cuda")
    ws = B.workspace(B.nmdlm_bbm_attn_workspace_size(T, M, H, dh))
    B.nmdlm_bbm_attn(q, k, vt, cap, T, M, C, H, dh, torch.from_numpy(lut).cuda(),
                     theta_a=theta, s_out=s_out, ws=ws)
    torch.cuda.synchronize()
    return synth.unpack_bits(B.from_dev_bits(s_out), d)


ATTN_SPIKES = ATTN + [
    (8, 20, 70, 2, 64, 0.3),       # T = 8, fused
    (8, 9, 130, 2, 128, 0.3),      # T = 8, dh = 128: partial sums exceed LDS, two kernels
    (5, 33, 200, 1, 128, 0.2),     # T not a power of two
]


@pytest.mark.parametrize("shape", ATTN_SPIKES,
                         ids=[f"T{s[0]}M{s[1]}C{s[2]}H{s[3]}dh{s[4]}" for s in ATTN_SPIKES])
def test_attention_spikes_only_parity(shape):
    T, M, C, H, dh, p = shape
    Q, Kc, Vc, lut, cap = _attn_case(sum(shape[:5]) + 1, T, M, C, H, dh, p)
    for theta in (300, 7):
        s = _attn_spikes_gpu(Q, Kc, Vc, lut, cap, C, H, dh, theta)
        a_ref = O.bbm_attention(Q, Kc, Vc, C + M, H, lut)
        assert_same(s, O.if_neuron(a_ref, theta)[0], f"theta {theta}")


def test_attention_closed_forms_on_gpu():
    Q, Kc, Vc, _, cap = _attn_case(3, 2, 8, 50, 2, 64, 0.4, stale=False)
    const = np.full(256, 9, dtype=np.uint8)
    a, _ = _attn_gpu(Q, Kc, Vc, const, cap, 50, 2, 64)
    want = (256 * Vc[:, :58].sum(axis=1, dtype=np.int64))[:, None, :] // 58
    assert_same(a, np.broadcast_to(want, a.shape))
    ones = np.ones_like(Vc)
    a1, _ = _attn_gpu(Q, Kc, ones, synth.sorted_lut_u8(synth.stream(1, 1)), cap, 50, 2, 64)
    assert (a1 == 256).all()
