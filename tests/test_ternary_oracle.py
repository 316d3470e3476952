"""The ternary bitwise-coded conversion of the oracle (Sec. III-B, Eqs.
(7)-(11)): pinned by a hand-worked quantisation, a float64 evaluation of
Eq. (7) away from rounding ties, exhaustive decoding of Eq. (8), the exact
reconstruction of Eq. (11) against a direct product with the quantised
vector, scale invariance, saturation and the row-load rule on either plane."""
import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth


def test_hand_worked_quantisation():
    # Eq. (7) with K = 1: V_th = mean|a|.  [1, 3]: V_th = 2, a/V_th = 0.5, 1.5
    # -> 1, 2 (halves away from zero); [-5, 2]: V_th = 3.5 -> -1.43, 0.57 -> -1, 1;
    # an all-zero vector quantises to zeros; K = 3 on [2, -2, 4]: V_th = 8/9,
    # a/V_th = 2.25, -2.25, 4.5 -> 2, -2, 5
    a = np.array([[1, 3, 0], [-5, 2, 0], [0, 0, 0]])
    q, S = O.ternary_quantize(a[:, :2], 1, 8)
    assert q.tolist() == [[1, 2], [-1, 1], [0, 0]] and S.tolist() == [4, 7, 0]
    q3, _ = O.ternary_quantize(np.array([[2, -2, 4]]), 3, 8)
    assert q3.tolist() == [[2, -2, 5]]


def test_float64_definition_away_from_ties():
    rng = synth.stream(3, 1)
    for K in (1, 2, 4):
        a = synth.ternary_activations(rng, 6, 300)
        q, _ = O.ternary_quantize(a, K, 16)
        x = a.astype(np.float64) / (np.abs(a).mean(axis=1, keepdims=True) / K)
        frac = np.abs(x) - np.floor(np.abs(x))
        ok = np.abs(frac - 0.5) > 1e-9
        assert np.array_equal(q[ok], np.rint(x)[ok])


def test_bitwise_coding_round_trip_exhaustive():
    for T in (1, 3, 8):
        q = np.arange(-(2 ** T - 1), 2 ** T, dtype=np.int64)[None, :]
        s = O.ternary_planes(q, T)
        assert set(np.unique(s)) <= {-1, 0, 1}
        assert np.array_equal(sum((2 ** t) * s[t].astype(np.int64) for t in range(T)), q)
        # one sign per value: no element has both a +1 and a -1 spike
        assert not np.any((s == 1).any(axis=0) & (s == -1).any(axis=0))
    with pytest.raises(ValueError):
        O.ternary_planes(np.array([[256]]), 8)


def test_reconstruction_is_exact_inner_product():
    c = synth.ternary_case(M=3, D=200, N=70, K=2, T=8)
    q, _ = O.ternary_quantize(c.a, c.K, c.T)
    s = O.ternary_planes(q, c.T)
    I, acc = O.qbsm_ternary(s, c.W)
    assert np.array_equal(acc, q @ c.W.astype(np.int64))            # Eq. (11)
    assert np.array_equal(I[0], s[0].astype(np.int64) @ c.W.astype(np.int64))


def test_scale_invariance_and_saturation():
    c = synth.ternary_case(M=2, D=64, N=8)
    q1, _ = O.ternary_quantize(c.a, 2, 8)
    q7, _ = O.ternary_quantize(7 * c.a.astype(np.int64), 2, 8)
    assert np.array_equal(q1, q7)
    spike = np.zeros((1, 64), dtype=np.int64)
    spike[0, 5] = 1000                       # a lone large value: 64 * K levels
    qs, _ = O.ternary_quantize(spike, 8, 8)
    assert qs[0, 5] == 255 and np.count_nonzero(qs) == 1   # 512 saturates at 2^8 - 1


def test_row_load_rule_on_either_plane():
    c = synth.ternary_case(M=4, D=500, N=8)
    q, _ = O.ternary_quantize(c.a, 2, 8)
    s = O.ternary_planes(q, 8)
    assert np.array_equal(O.ternary_union(s), (q != 0).any(axis=0))
    assert 0 < O.ternary_union(s).sum() < 500       # the synthetic activations do skip rows


# ---------------------------------------------------------------------------
# the modified IF neuron (Eqs. (9)-(10)) and the reconstruction of Eq. (11)
# ---------------------------------------------------------------------------
def _traces():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "modified_if_traces.txt")
    out = []
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, I, s, v = [p.split() for p in line.split("|")]
        out.append((int(head[0]), int(head[1]), [int(x) for x in I], [int(x) for x in s], int(v[0])))
    return out


def test_modified_if_hand_traces():
    tr = _traces()
    assert len(tr) >= 12
    for num, den, I, s_want, v_want in tr:
        s, V = O.modified_if(np.array(I, dtype=np.int64)[:, None, None], [num], den)
        assert s[:, 0, 0].tolist() == s_want, (num, den, I)
        assert int(V[0, 0]) == v_want, (num, den, I)


def test_modified_if_charge_conservation():
    # den * (sum_t 2^(t-1) I_t) - num * (sum_t 2^(t-1) s_t) == den * V_final, exactly
    rng = np.random.default_rng(11)
    for T in (1, 3, 8):
        I = rng.integers(-5000, 5000, size=(T, 6, 40))
        num = rng.integers(1, 20000, size=6)
        den = 7
        s, V = O.modified_if(I, num, den)
        lhs = den * O.bitwise_value(I) - num[:, None] * O.bitwise_value(s)
        assert np.array_equal(lhs, V)
        assert set(np.unique(s)) <= {-1, 0, 1}


def test_modified_if_sign_symmetry_and_scale_invariance():
    rng = np.random.default_rng(12)
    I = rng.integers(-3000, 3000, size=(8, 5, 33))
    num = rng.integers(1, 4000, size=5)
    s, V = O.modified_if(I, num, 3)
    sn, Vn = O.modified_if(-I, num, 3)
    assert np.array_equal(sn, -s) and np.array_equal(Vn, -V)
    s7, V7 = O.modified_if(7 * I, 7 * num, 3)        # currents and threshold scaled together
    assert np.array_equal(s7, s) and np.array_equal(V7, 7 * V)


def test_modified_if_single_step_is_a_ternary_threshold():
    rng = np.random.default_rng(13)
    I = rng.integers(-300, 300, size=(1, 4, 50))
    num = np.array([1, 50, 100, 299])
    s, V = O.modified_if(I, num, 1)
    want = np.where(I[0] >= num[:, None], 1, np.where(I[0] <= -num[:, None], -1, 0))
    assert np.array_equal(s[0], want)
    assert np.array_equal(V, I[0] - want * num[:, None])


def test_eq11_reconstruction_exact_for_whole_multiple_currents():
    """With W = theta * identity the currents of a ternary-coded input are
    theta times its spikes, one sign per step; the neuron at Vth = theta then
    re-emits the input train and Eq. (11) holds with equality:
    Vth sum_t 2^(t-1) s_hat_t = w^T a_hat (here theta q)."""
    c = synth.ternary_case(M=3, D=64, N=64, K=2, T=8)
    theta = 100
    W = (theta * np.eye(64)).astype(np.int8)
    q, _ = O.ternary_quantize(c.a, c.K, c.T)
    s = O.ternary_planes(q, c.T)
    I, acc = O.qbsm_ternary(s, W)
    s_hat, V = O.modified_if(I, np.full(3, theta), 1)
    assert np.array_equal(s_hat, s) and not V.any()
    assert np.array_equal(theta * O.bitwise_value(s_hat), q @ W.astype(np.int64))
    assert np.array_equal(acc, q @ W.astype(np.int64))


def test_modified_if_zero_threshold_is_silent():
    I = np.array([[[5, -5, 0]], [[1, 2, 3]]])
    s, V = O.modified_if(I, [0], 1)
    assert not s.any()
    assert np.array_equal(V[0], [5 + 2, -5 + 4, 0 + 6])
