"""GPU parity at full size: the FFN sweep, the 12-layer block step and the 24-layer generation.

The FFN sweep is checked element by element against the oracle
computed in the test.  The 12- and 24-layer models compare against stored values
written by tests/golden/make_golden.py (oracle only): exact digests of the
logits, last-layer spikes and every cache, and the unmasking decisions."""
import hashlib
import json
import os

import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

from ._gpu import assert_same, need_gpu, run_qbsm

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sha(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


# ----------------------------------------------------------------------------
# FFN weight-traffic sweep (16 points x 2 products)
# ----------------------------------------------------------------------------
@pytest.fixture(scope="module")
def ffn():
    need_gpu()
    return synth.ffn_sweep_weights()


@pytest.mark.parametrize("iB", range(4), ids=[f"B{b}" for b in synth.FFN_SWEEP_BLOCKS])
def test_ffn_sweep_points(ffn, iB):
    for iR in range(4):
        pt = synth.ffn_sweep_point(iB, iR)
        for name, X, W, th in (("up", pt.X_up, ffn.W_up, ffn.theta_up),
                               ("dn", pt.X_dn, ffn.W_dn, ffn.theta_dn)):
            I_ref = O.qbsm(X, W)
            cur, spk, st, _, _ = run_qbsm(X, W, None, theta=th)
            tag = f"B={pt.B} rho={pt.density} {name}"
            assert_same(cur, I_ref, tag + " currents")
            assert_same(spk, O.if_neuron(I_ref, th)[0], tag + " spikes")
            act = O.active_rows(X).size
            assert st["k_active"] == act and st["weight_bytes"] == act * W.shape[1], tag


def test_ffn_chained(ffn):
    # X_dn = IF output of the up product, as in a real FFN
    for iB, iR in ((1, 0), (3, 3)):
        pt = synth.ffn_sweep_point(iB, iR)
        _, h, _, _, _ = run_qbsm(pt.X_up, ffn.W_up, None, theta=ffn.theta_up, want_cur=False)
        h_ref = O.if_neuron(O.qbsm(pt.X_up, ffn.W_up), ffn.theta_up)[0]
        assert_same(h, h_ref, "hidden spikes")
        _, y, st, _, _ = run_qbsm(h, ffn.W_dn, None, theta=ffn.theta_dn, want_cur=False)
        assert_same(y, O.if_neuron(O.qbsm(h_ref, ffn.W_dn), ffn.theta_dn)[0], "output spikes")
        assert st["k_active"] == O.active_rows(h_ref).size


# ----------------------------------------------------------------------------
# 12- and 24-layer MDLM against stored oracle values
# ----------------------------------------------------------------------------
def _load(name):
    path = os.path.join(GOLDEN, name)
    if not os.path.exists(path):
        pytest.fail(f"missing stored values {path}: run tests/golden/make_golden.py")
    with open(path) as f:
        return json.load(f)


def _chosen_ok(got, want, conf, masked0=None, tol=1e-9):
    """The selection is the stored one, or differs from it only where
    confidences tie (within tol): the same number of positions, all
    distinct and masked before the step, in order of non-increasing
    confidence, and none of them less confident than a masked position left
    out (ties allowed)."""
    got, want = [int(g) for g in got], [int(w) for w in want]
    if got == want:
        return True
    if len(got) != len(want) or len(set(got)) != len(got):
        return False
    cand = [p for p in range(len(conf)) if masked0 is None or masked0[p]]
    if not set(got) <= set(cand):
        return False
    close = lambda a, b: abs(a - b) <= tol * max(abs(a), abs(b))
    c = [conf[p] for p in got]
    if any(c[i + 1] > c[i] and not close(c[i + 1], c[i]) for i in range(len(c) - 1)):
        return False
    left = [conf[p] for p in cand if p not in got]
    return all(x <= min(c) or close(x, min(c)) for x in left)


def _tokens_after(chosen, pred, tokens0, masked0):
    """Tokens and masked flags after revealing `chosen` (Sec. III-A: a chosen
    position takes its prediction; nothing else changes)."""
    tok = np.array(tokens0, dtype=np.int64)
    msk = np.array(masked0, dtype=np.int64)
    for p in chosen:
        if p >= 0:
            tok[p] = pred[p]
            msk[p] = 0
    return tok.tolist(), msk.tolist()


@pytest.mark.parametrize("flags,blocked", [(0, False), (0x4, False), (4 << 20, False), (0, True),
                                           (6 << 20, True)],
                         ids=["default", "attn-fused", "dma", "blocked-copies", "blocked-forced"])
def test_mdlm12_step_matches_stored_oracle(flags, blocked):
    torch, B = need_gpu()
    ref = _load("mdlm12_block_step.json")
    case = synth.mdlm12_step_case()
    m = case.model
    C, M, k = case.C, case.B, case.k_unmask
    dm = B.DeviceModel.from_mdlm(m, C + M, blocked=blocked)
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, C, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, M, 0)))
    ctx = torch.from_numpy(case.ctx_tokens.astype(np.int32)).cuda()
    B.nmdlm_block_step(dm, B.step_io(C, 0, flags=B.NMDLM_NO_HEAD | flags, tokens=ctx,
                                     masked=torch.zeros(C, dtype=torch.uint8, device="cuda")), ws)
    tok = torch.zeros(M, dtype=torch.int32, device="cuda")
    msk = torch.ones(M, dtype=torch.uint8, device="cuda")
    logits = torch.empty((M, m.V), dtype=torch.float32, device="cuda")
    pred = torch.empty(M, dtype=torch.int32, device="cuda")
    conf = torch.empty(M, dtype=torch.float64, device="cuda")
    chosen = torch.empty(k, dtype=torch.int32, device="cuda")
    y = torch.empty((m.T, M, m.d // 64), dtype=torch.int64, device="cuda")
    stats = torch.zeros((4 * m.n_layers + 1, 4), dtype=torch.int64, device="cuda")
    B.nmdlm_block_step(dm, B.step_io(M, C, pos0=C, flags=flags, tokens=tok, masked=msk,
                                     k_unmask=k, y_out=y,
                                     logits=logits, pred=pred, conf=conf, unmasked_pos=chosen,
                                     stats=stats), ws)
    torch.cuda.synchronize()
    st = stats.cpu().numpy()
    assert st[:-1, 1].reshape(m.n_layers, 4).tolist() == ref["k_active"]
    assert int(st[-1, 1]) == ref["head_k_active"]
    assert B.from_dev_bits(y).tobytes() and _sha(B.from_dev_bits(y)) == ref["y_sha256"]
    lg = logits.cpu().numpy()
    for i, j, v in ref["logits_sample"]:
        assert lg[i, j] == np.float32(v), (i, j)
    assert _sha(lg) == ref["logits_sha256"]
    assert pred.cpu().numpy().tolist() == ref["pred"]
    assert np.allclose(conf.cpu().numpy(), ref["conf"], rtol=1e-12, atol=0)
    got = chosen.cpu().numpy().tolist()
    assert _chosen_ok(got, ref["chosen"], ref["conf"], masked0=[1] * M)
    # tokens and flags always: those of the stored step, or of a tie-equivalent choice
    want_tok, want_msk = _tokens_after(got, ref["pred"], [0] * M, [1] * M)
    if got == ref["chosen"]:
        assert (want_tok, want_msk) == (ref["tokens"], ref["masked"])
    assert tok.cpu().numpy().tolist() == want_tok
    assert msk.cpu().numpy().tolist() == want_msk
    J = C + M
    for l, layer in enumerate(dm.layers):
        kd = _sha(B.from_dev_bits(layer.k_cache)[:, :J])
        words = np.ascontiguousarray(B.from_dev_bits(layer.vt_cache).transpose(0, 2, 1))  # [T][d][cap/64]
        vt = synth.unpack_bits(words, dm.cache_cap)
        vd = _sha(synth.pack_bits(vt.transpose(0, 2, 1)[:, :J]))
        assert kd == ref["k_cache_sha256"][l], f"K cache layer {l}"
        assert vd == ref["v_cache_sha256"][l], f"V cache layer {l}"


def test_mdlm24_generation_matches_stored_oracle():
    need_gpu()
    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd.generate import generate
    ref = _load("mdlm24_generation.json")
    case = synth.mdlm24_generation_case()
    m = case.model
    dm = B.DeviceModel.from_mdlm(m, len(case.prompt) + case.n_blocks * case.B)
    ids, log = generate(dm, case.prompt, case.n_blocks, case.B, case.steps, case.k_unmask)
    assert ids.tolist() == ref["ids"]
    assert [c.tolist() for c in log] == ref["chosen"]


def _packed_caches(layer, cap, d, J):
    """(K, V) of a device layer as packed spike rows [T][J][d/64] (the layout
    the stored digests use)."""
    from paper_2607_24841_amd import binding as B
    k = B.from_dev_bits(layer.k_cache)[:, :J]
    words = np.ascontiguousarray(B.from_dev_bits(layer.vt_cache).transpose(0, 2, 1))  # [T][d][cap/64]
    vt = synth.unpack_bits(words, cap)
    return np.ascontiguousarray(k), synth.pack_bits(vt.transpose(0, 2, 1)[:, :J])


def test_e2d2_full_shape_matches_stored_oracle():
    """The paper's own shape (28 encoder + 4 decoder layers, d=512, F=1536,
    T=8, 64-id prompt, 4 blocks of 4 tokens, one token per step) against the
    stored oracle generation: ids, every step's choice, the caches of every
    decoder layer and of the last encoder layer."""
    torch, B = need_gpu()
    from paper_2607_24841_amd.e2d2 import E2D2
    with open(os.path.join(GOLDEN, "e2d2_generation.json")) as f:
        ref = json.load(f)
    case = synth.e2d2_case()
    m = case.model
    P = len(case.prompt)
    J = P + case.n_blocks * case.B
    dm = B.DeviceModel.from_mdlm(m, J)
    g = E2D2(dm, case.n_enc, P, case.n_blocks, case.B)
    g.ctx[:P].copy_(torch.from_numpy(np.asarray(case.prompt, dtype=np.int32)))
    log = []
    C = g.generate(P, case.n_blocks, case.steps, case.k_unmask, log)
    torch.cuda.synchronize()
    assert g.ctx[P:C].cpu().numpy().tolist() == ref["ids"]
    assert [c.cpu().numpy().tolist() for c in log] == ref["chosen"]
    for l in range(m.n_layers - case.n_enc):
        k, v = _packed_caches(dm.layers[case.n_enc + l], dm.cache_cap, m.d, J)
        assert _sha(k) == ref["dec_k_cache_sha256"][l], f"decoder layer {l} keys"
        assert _sha(v) == ref["dec_v_cache_sha256"][l], f"decoder layer {l} values"
    k, v = _packed_caches(dm.layers[case.n_enc - 1], dm.cache_cap, m.d, J)
    assert _sha(k) == ref["last_enc_k_cache_sha256"] and _sha(v) == ref["last_enc_v_cache_sha256"]


# ----------------------------------------------------------------------------
# full-size head on diverse inputs: ordering, not ties
# ----------------------------------------------------------------------------
@pytest.fixture(scope="module")
def head_case():
    # the 12-layer model's head shape (d=2048, V=32000, T=4) with no layers,
    # fed with per-token Bernoulli(0.05) spikes: the masked positions predict
    # many different ids, with distinct confidences
    m = synth.make_mdlm(synth.SEEDS["mdlm12"] + 50, 0, max_pos=64)
    T, M, k = m.T, 32, 8
    X = synth.bernoulli(synth.stream(synth.SEEDS["mdlm12"] + 50, 9), 0.05, (T, M, m.d))
    tok0 = synth.random_tokens(synth.SEEDS["mdlm12"] + 51, M, m.V).astype(np.int32)
    msk0 = np.ones(M, dtype=bool)
    msk0[::4] = False                                 # 24 masked positions
    logits = O.head_logits(X, m.W_head, m.scale)
    pred, conf = O.confidence(logits)
    tok_ref, msk_ref, chosen = O.unmask(tok0, msk0, pred, conf, k)
    return m, X, tok0, msk0, k, logits, pred, conf, tok_ref, msk_ref, chosen


def test_full_size_head_case_is_not_tied(head_case):
    m, X, tok0, msk0, k, logits, pred, conf, tok_ref, msk_ref, chosen = head_case
    cm = np.sort(conf[msk0])[::-1]
    assert len(set(pred[msk0].tolist())) >= 16        # many different predictions
    assert len(np.unique(cm)) == cm.size              # no two masked confidences equal
    assert cm[k - 1] > cm[k]                          # the top-k boundary is not a tie
    assert len(chosen) == k and not msk_ref[chosen].any()


@pytest.mark.parametrize("blocked", [False, True], ids=["rows", "blocked-copy"])
def test_full_size_head_matches_oracle(head_case, blocked):
    torch, B = need_gpu()
    m, X, tok0, msk0, k, logits_ref, pred_ref, conf_ref, tok_ref, msk_ref, chosen_ref = head_case
    T, M = X.shape[0], X.shape[1]
    dm = B.DeviceModel.from_mdlm(m, 64, blocked=blocked)
    ws = B.workspace(B.nmdlm_block_step_workspace_size(dm, M, 0))
    tok = torch.from_numpy(tok0).cuda()
    msk = torch.from_numpy(msk0.astype(np.uint8)).cuda()
    logits = torch.empty((M, m.V), dtype=torch.float32, device="cuda")
    pred = torch.empty(M, dtype=torch.int32, device="cuda")
    conf = torch.empty(M, dtype=torch.float64, device="cuda")
    chosen = torch.full((k,), -7, dtype=torch.int32, device="cuda")
    B.nmdlm_block_step(dm, B.step_io(M, 0, x_in=B.to_dev_bits(synth.pack_bits(X)), tokens=tok,
                                     masked=msk, k_unmask=k, logits=logits, pred=pred, conf=conf,
                                     unmasked_pos=chosen), ws)
    torch.cuda.synchronize()
    assert_same(logits.cpu().numpy(), logits_ref, "logits")
    assert_same(pred.cpu().numpy(), pred_ref, "pred")
    assert np.allclose(conf.cpu().numpy(), conf_ref, rtol=1e-12, atol=0)
    assert np.array_equal(chosen.cpu().numpy(), np.asarray(chosen_ref))
    assert np.array_equal(tok.cpu().numpy(), tok_ref)
    assert np.array_equal(msk.cpu().numpy().astype(bool), msk_ref)
