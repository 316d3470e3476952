"""Pins for the CPU oracle: each check compares it with something other than
itself (hand traces, brute force, closed forms, invariants, library routines
used as special cases).  CPU only."""
import itertools
import os

import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# QBSM (Sec. IV-A: Y = X W over B*T spike rows, row-load rule (ii))
# ----------------------------------------------------------------------------
def _brute_qbsm(S, W, b):
    T, M, K = S.shape
    N = W.shape[1]
    out = np.zeros((T, M, N), dtype=np.int64)
    for t in range(T):
        for m in range(M):
            for n in range(N):
                acc = int(b[n])
                for k in range(K):
                    if S[t, m, k]:
                        acc += int(W[k, n])
                out[t, m, n] = acc
    return out


def test_qbsm_brute_force_all_spike_vectors():
    # every spike vector of length K (2**K of them) as the rows of one block
    rng = np.random.default_rng(7)
    for K, N in [(1, 1), (3, 5), (8, 16), (10, 7)]:
        W = rng.integers(-127, 128, size=(K, N)).astype(np.int8)
        b = rng.integers(-64, 65, size=N).astype(np.int32)
        rows = np.array(list(itertools.product([0, 1], repeat=K)), dtype=bool)
        S = rows.reshape(1, -1, K)
        I = O.qbsm(S, W, b)
        for r, row in enumerate(rows):
            want = [int(b[n]) + sum(int(W[k, n]) for k in range(K) if row[k]) for n in range(N)]
            assert I[0, r].tolist() == want


def test_qbsm_brute_force_random_blocks():
    for seed, (T, M, K, N) in enumerate([(4, 3, 16, 16), (2, 5, 13, 9), (1, 1, 16, 1)]):
        c = synth.make_qbsm_case(seed, T, M, K, N, density=0.3)
        assert np.array_equal(O.qbsm(c.S, c.W, c.bias), _brute_qbsm(c.S, c.W, c.bias))


def test_qbsm_matches_integer_matmul_library_routine():
    c = synth.make_qbsm_case(11, 4, 8, 200, 65, density=0.2)
    want = c.S.reshape(-1, 200).astype(np.int64) @ c.W.astype(np.int64) + c.bias
    assert np.array_equal(O.qbsm(c.S, c.W, c.bias).reshape(-1, 65), want)


def test_qbsm_special_cases():
    c = synth.make_qbsm_case(3, 2, 3, 70, 33, density=0.2)
    zero = np.zeros_like(c.S)
    assert np.array_equal(O.qbsm(zero, c.W, c.bias), np.broadcast_to(c.bias, (2, 3, 33)))
    assert O.active_rows(zero).size == 0
    assert O.touched_weight_bytes(zero, 33) == 0
    ones = np.ones_like(c.S)
    colsum = c.W.astype(np.int64).sum(axis=0) + c.bias
    assert np.array_equal(O.qbsm(ones, c.W, c.bias), np.broadcast_to(colsum, (2, 3, 33)))
    one = np.zeros_like(c.S)
    one[1, 2, 17] = True
    I = O.qbsm(one, c.W, c.bias)
    assert np.array_equal(I[1, 2], c.W[17].astype(np.int64) + c.bias)
    mask = np.ones((2, 3), dtype=bool)
    mask[1, 2] = False
    assert np.array_equal(I[mask], np.broadcast_to(c.bias, (5, 33)))


def test_qbsm_linearity_and_row_permutation():
    c = synth.make_qbsm_case(5, 3, 4, 90, 21, density=0.25)
    rng = np.random.default_rng(0)
    split = rng.random(c.S.shape) < 0.5
    S1, S2 = c.S & split, c.S & ~split
    z = np.zeros(21, dtype=np.int32)
    assert np.array_equal(O.qbsm(c.S, c.W, z), O.qbsm(S1, c.W, z) + O.qbsm(S2, c.W, z))
    perm = rng.permutation(90)
    assert np.array_equal(O.qbsm(c.S[..., perm], c.W[perm], c.bias), O.qbsm(c.S, c.W, c.bias))


def test_skipped_rows_equal_dense():
    # assumption (ii): dropping the rows of silent channels changes nothing
    c = synth.make_qbsm_case(9, 4, 2, 300, 40, density=0.02)
    act = O.active_rows(c.S)
    assert 0 < act.size < 300
    skipped = O.qbsm(c.S[..., act], c.W[act], c.bias)
    assert np.array_equal(skipped, O.qbsm(c.S, c.W, c.bias))
    assert O.touched_weight_bytes(c.S, 40) == act.size * 40


def test_union_matches_any():
    c = synth.make_qbsm_case(2, 4, 8, 512, 8, density=0.01)
    u = O.block_union(c.S)
    want = [any(c.S[t, m, k] for t in range(4) for m in range(8)) for k in range(512)]
    assert u.tolist() == want
    assert O.active_rows(c.S).tolist() == [k for k in range(512) if want[k]]


def test_realized_skip_matches_eq13_expectation():
    # Eq. (13): a row is loaded with probability 1 - sigma^(B*T) for iid spikes
    for (T, M, K, p) in [(4, 8, 4096, 0.15), (4, 1, 8192, 0.05), (4, 2, 8192, 0.1)]:
        c = synth.make_qbsm_case(17, T, M, K, 1, density=p)
        q = (1 - p) ** (T * M)                    # probability a row is skipped
        skipped = K - O.active_rows(c.S).size
        sd = np.sqrt(K * q * (1 - q))
        assert abs(skipped - K * q) <= 5 * sd + 1


def test_qbsm_overflow_guard():
    S = np.ones((1, 1, 40000), dtype=bool)
    W = np.full((40000, 1), 127, dtype=np.int8)
    assert O.qbsm(S, W)[0, 0, 0] == 40000 * 127       # still in range
    S2 = np.ones((1, 1, 17_000_000), dtype=bool)
    W2 = np.full((17_000_000, 1), 127, dtype=np.int8)
    with pytest.raises(OverflowError):
        O.qbsm(S2, W2)


# ----------------------------------------------------------------------------
# IF neuron (Eqs. (3)-(4))
# ----------------------------------------------------------------------------
def _load_traces():
    out = []
    for line in open(os.path.join(GOLDEN, "if_traces.txt")):
        if line.startswith("#") or not line.strip():
            continue
        th, I, s, v = [x.strip() for x in line.split("|")]
        out.append((int(th), [int(x) for x in I.split()], [int(x) for x in s.split()], int(v)))
    return out


@pytest.mark.parametrize("th,I,s,v", _load_traces())
def test_if_hand_traces(th, I, s, v):
    spikes, V = O.if_neuron(np.array(I).reshape(-1, 1), th)
    assert spikes[:, 0].astype(int).tolist() == s
    assert int(V[0]) == v


def test_if_charge_conservation_and_floor_law():
    rng = np.random.default_rng(1)
    I = rng.integers(-2000, 2000, size=(8, 50, 60))
    th = rng.integers(1, 600, size=60)
    s, V = O.if_neuron(I, th)
    assert np.array_equal(V, I.sum(axis=0) - th * s.sum(axis=0))
    Ip = rng.integers(0, 100, size=(8, 40, 30))
    s2, V2 = O.if_neuron(Ip, 100)
    assert np.array_equal(s2.sum(axis=0), Ip.sum(axis=0) // 100)
    assert V2.min() >= 0 and V2.max() < 100


def test_if_at_most_one_spike_per_step_and_residual():
    rng = np.random.default_rng(2)
    I = rng.integers(-300, 300, size=(4, 6, 9))
    R = rng.random((4, 6, 9)) < 0.4
    s, V = O.if_neuron(I, 200, resid=R)
    s_ref, V_ref = O.if_neuron(I + 200 * R.astype(np.int64), 200)
    assert np.array_equal(s, s_ref) and np.array_equal(V, V_ref)
    # a zero branch with the residual shortcut reproduces the input spikes
    s_id, _ = O.if_neuron(np.zeros((4, 6, 9), dtype=np.int64), 200, resid=R)
    assert np.array_equal(s_id, R)
    with pytest.raises(ValueError):
        O.if_neuron(I, 0)


# ----------------------------------------------------------------------------
# QNL tables
# ----------------------------------------------------------------------------
def test_qnl_identity_table_is_saturating_shift():
    ident = (np.arange(256) & 0xFF).astype(np.uint8)     # lut[b] = b, read as int8
    x = np.arange(-70000, 70000, 37)
    for s in (0, 1, 4, 9):
        y = O.qnl_lut(x, s, ident, O.QNL_S8)
        want = [max(-128, min(127, xi >> s)) for xi in x.tolist()]
        assert y.tolist() == want


def test_qnl_exhaustive_indices():
    lut = synth.sorted_lut_s8(synth.stream(3, 9))
    for v in range(-128, 128):
        assert O.qnl_lut(np.array([v]), 0, lut, O.QNL_S8)[0] == np.int8(lut[v & 0xFF])
    # monotone in the signed input
    vals = [int(O.qnl_lut(np.array([v]), 0, lut, O.QNL_S8)[0]) for v in range(-128, 128)]
    assert vals == sorted(vals)
    u = synth.sorted_lut_u8(synth.stream(3, 10))
    xs = np.arange(-5, 300)
    assert O.qnl_lut(xs, 0, u, O.QNL_U8).tolist() == [int(u[min(255, max(0, x))]) for x in xs]


# ----------------------------------------------------------------------------
# BBM attention
# ----------------------------------------------------------------------------
def _brute_attention(Q, Kc, Vc, n_keys, H, lut):
    T, M, d = Q.shape
    dh = d // H
    out = np.zeros((T, M, d), dtype=np.int64)
    for t in range(T):
        for h in range(H):
            for i in range(M):
                ps = []
                for j in range(n_keys):
                    sc = sum(int(Q[t, i, h * dh + c]) & int(Kc[t, j, h * dh + c]) for c in range(dh))
                    ps.append(int(lut[sc]))
                den = sum(ps)
                for c in range(dh):
                    num = sum(ps[j] for j in range(n_keys) if Vc[t, j, h * dh + c])
                    out[t, i, h * dh + c] = (256 * num) // den if den else 0
    return out


def _rand_attn(seed, T=2, M=3, J=7, H=2, dh=5, p=0.5):
    rng = np.random.default_rng(seed)
    Q = rng.random((T, M, H * dh)) < p
    Kc = rng.random((T, J, H * dh)) < p
    Vc = rng.random((T, J, H * dh)) < p
    lut = synth.sorted_lut_u8(synth.stream(seed, 5))
    return Q, Kc, Vc, lut


def test_attention_brute_force():
    for seed in range(3):
        Q, Kc, Vc, lut = _rand_attn(seed)
        assert np.array_equal(O.bbm_attention(Q, Kc, Vc, 7, 2, lut),
                              _brute_attention(Q, Kc, Vc, 7, 2, lut))


def test_attention_closed_forms():
    Q, Kc, Vc, _ = _rand_attn(4, T=2, M=4, J=9, H=3, dh=6)
    const = np.full(256, 37, dtype=np.uint8)
    a = O.bbm_attention(Q, Kc, Vc, 9, 3, const)
    want = (256 * Vc.sum(axis=1, dtype=np.int64))[:, None, :] // 9
    assert np.array_equal(a, np.broadcast_to(want, a.shape))
    lut = synth.sorted_lut_u8(synth.stream(4, 5))
    assert (O.bbm_attention(Q, Kc, np.ones_like(Vc), 9, 3, lut) == 256).all()
    assert (O.bbm_attention(Q, Kc, np.zeros_like(Vc), 9, 3, lut) == 0).all()


def test_attention_key_permutation_invariance():
    Q, Kc, Vc, lut = _rand_attn(8, T=3, M=5, J=11, H=2, dh=8)
    perm = np.random.default_rng(3).permutation(11)
    a = O.bbm_attention(Q, Kc, Vc, 11, 2, lut)
    b = O.bbm_attention(Q, Kc[:, perm], Vc[:, perm], 11, 2, lut)
    assert np.array_equal(a, b)
    # keys past n_keys are ignored
    Kx = np.concatenate([Kc, np.ones_like(Kc[:, :3])], axis=1)
    Vx = np.concatenate([Vc, np.ones_like(Vc[:, :3])], axis=1)
    assert np.array_equal(O.bbm_attention(Q, Kx, Vx, 11, 2, lut), a)


# ----------------------------------------------------------------------------
# head, confidence, unmasking
# ----------------------------------------------------------------------------
def test_head_logits_exact_single_multiply():
    rng = np.random.default_rng(5)
    Y = rng.random((4, 3, 70)) < 0.4
    W = rng.integers(-127, 128, size=(70, 11)).astype(np.int8)
    scale = (rng.uniform(0.5, 1.5, 11) * 2 ** -10).astype(np.float32)
    lg = O.head_logits(Y, W, scale)
    for m in range(3):
        for v in range(11):
            acc = sum(int(W[c, v]) for t in range(4) for c in range(70) if Y[t, m, c])
            assert lg[m, v] == np.float32(np.float32(acc) * scale[v])
    assert lg.dtype == np.float32


def test_confidence_matches_softmax_and_ties():
    from scipy.special import softmax
    rng = np.random.default_rng(6)
    lg = (rng.normal(size=(5, 40)) * 3).astype(np.float32)
    pred, conf = O.confidence(lg)
    sm = softmax(lg.astype(np.float64), axis=1)
    assert np.array_equal(pred, sm.argmax(axis=1))
    assert np.allclose(conf, sm.max(axis=1), rtol=1e-12)
    tie = np.zeros((1, 6), dtype=np.float32)
    tie[0, 2] = tie[0, 4] = 1.0
    p, c = O.confidence(tie)
    assert p[0] == 2
    assert np.isclose(c[0], np.e / (2 * np.e + 4))


def test_unmask_rules():
    tokens = np.array([5, 0, 0, 0, 0, 9], dtype=np.int32)
    masked = np.array([False, True, True, True, True, False])
    pred = np.array([1, 2, 3, 4, 5, 6], dtype=np.int32)
    conf = np.array([0.99, 0.5, 0.7, 0.7, 0.1, 0.99])
    t2, m2, ch = O.unmask(tokens, masked, pred, conf, 2)
    assert ch.tolist() == [2, 3]                       # ties -> lower position
    assert t2.tolist() == [5, 0, 3, 4, 0, 9]           # unmasked tokens untouched
    assert m2.tolist() == [False, True, False, False, True, False]
    t3, m3, ch3 = O.unmask(t2, m2, pred, conf, 5)      # fewer left than k
    assert ch3.tolist() == [1, 4] and not m3.any()


# ----------------------------------------------------------------------------
# layer / block step / generation invariants on a tiny model
# ----------------------------------------------------------------------------
def _tiny_model(seed=21, n_layers=2):
    return synth.make_mdlm(seed, n_layers, d=128, H=2, F=256, V=50, T=4, max_pos=64)


def test_block_input_definition():
    m = _tiny_model()
    emb = O.unpack_model_emb(m)
    toks = np.array([3, m.mask_id, 7])
    X = O.block_input(toks, np.array([10, 11, 12]), emb, m.pos_ch)
    for i, (tok, pos) in enumerate(zip(toks, [10, 11, 12])):
        for t in range(4):
            want = emb[tok, t].copy()
            want[m.pos_ch[pos, t]] = True
            assert np.array_equal(X[t, i], want)


def test_layer_zero_branch_identity_and_cache_write():
    L = synth.make_layer(3, 0, 128, 256, 2)
    T, M, C = 4, 5, 6
    X = np.random.default_rng(1).random((T, M, 128)) < 0.2
    kc, vc = O.new_caches(1, T, C + M, 128)
    tr = O.layer_forward(X, L, kc[0], vc[0], C)
    assert np.array_equal(kc[0][:, C:C + M], tr.K) and np.array_equal(vc[0][:, C:C + M], tr.V)
    assert not kc[0][:, :C].any()
    # with all projection weights zero every branch current is zero, so the
    # residual shortcuts pass the input straight through: X1 = X and Y = X1
    import copy
    Z = copy.copy(L)
    Z.W_o = np.zeros_like(L.W_o)
    Z.W_dn = np.zeros_like(L.W_dn)
    kc2, vc2 = O.new_caches(1, T, C + M, 128)
    tr2 = O.layer_forward(X, Z, kc2[0], vc2[0], C)
    assert np.array_equal(tr2.X1, X) and np.array_equal(tr2.Y, X)
    # zeroing only W_dn: Y must equal X1 (the down residual is X1, not X)
    Z2 = copy.copy(L)
    Z2.W_dn = np.zeros_like(L.W_dn)
    kc3, vc3 = O.new_caches(1, T, C + M, 128)
    tr3 = O.layer_forward(X, Z2, kc3[0], vc3[0], C)
    assert not np.array_equal(tr3.X1, X)
    assert np.array_equal(tr3.Y, tr3.X1)


def test_generation_invariants():
    m = _tiny_model()
    prompt = synth.random_tokens(4, 12, m.V)
    out, log = O.generate(m, prompt, n_blocks=2, B=8, steps=4, k_unmask=2)
    assert out.shape == (16,)
    assert ((out >= 0) & (out < m.V)).all()
    for blk in range(2):
        chosen = np.concatenate(log[blk * 4:(blk + 1) * 4])
        assert sorted(chosen.tolist()) == list(range(8))   # each position once, none re-masked
        assert all(len(c) == 2 for c in log[blk * 4:(blk + 1) * 4])
    out2, _ = O.generate(m, prompt, n_blocks=2, B=8, steps=4, k_unmask=2)
    assert np.array_equal(out, out2)


def test_generation_resume_from_block_snapshot():
    m = _tiny_model(seed=22)
    prompt = synth.random_tokens(5, 10, m.V)
    emb = O.unpack_model_emb(m)
    full, _ = O.generate(m, prompt, n_blocks=2, B=4, steps=2, k_unmask=2, emb01=emb)
    # generate block 0, snapshot caches, then continue block 1 from the snapshot
    kc, vc = O.new_caches(m.n_layers, m.T, 18, m.d)
    O.prefill(O.block_input(prompt, np.arange(10), emb, m.pos_ch), m.layers, kc, vc)
    tokens, masked = np.zeros(4, np.int32), np.ones(4, bool)
    for _ in range(2):
        r = O.block_step(m, emb, tokens, masked, 10, 10, kc, vc, 2)
        tokens, masked = r.tokens, r.masked
    snap_k = [k.copy() for k in kc]
    snap_v = [v.copy() for v in vc]
    tokens2, masked2 = np.zeros(4, np.int32), np.ones(4, bool)
    for _ in range(2):
        r = O.block_step(m, emb, tokens2, masked2, 14, 14, snap_k, snap_v, 2)
        tokens2, masked2 = r.tokens, r.masked
    assert np.array_equal(np.concatenate([tokens, tokens2]), full)


def test_tie_equivalent_selection_checker():
    """The full-size GPU tests accept a different set of unmasked positions
    only across exact confidence ties at the boundary; check that rule on
    hand-made cases (and that it rejects everything else)."""
    from tests.test_gpu_full_size import _chosen_ok, _tokens_after
    conf = [0.9, 0.5, 0.7, 0.7, 0.1]
    assert _chosen_ok([0, 2], [0, 2], conf)
    assert _chosen_ok([0, 3], [0, 2], conf)                 # 2 and 3 tie at the boundary
    assert not _chosen_ok([0, 1], [0, 2], conf)             # 1 is less confident than 2, 3
    assert not _chosen_ok([2, 0], [0, 2], conf)             # order must follow confidence
    assert not _chosen_ok([0, 0], [0, 2], conf)
    assert not _chosen_ok([0, 2], [0, 2, 3], conf)
    assert not _chosen_ok([0, 4], [0, 2], conf, masked0=[1, 1, 1, 1, 1])
    assert _tokens_after([2, 0], [5, 6, 7, 8, 9], [0, 0, 0, 0, 0], [1, 1, 1, 1, 1]) == \
        ([5, 0, 7, 0, 0], [0, 1, 0, 1, 1])
