"""The encoder-decoder generation of the oracle (Sec. III-A, Eqs. (5)-(6)):
with no encoder layer, one decoder layer and one block it is the plain
block-diffusion generation (the context keys/values of a one-layer decoder
over the raw context are its prefill); invariants of the unmasking."""
import dataclasses

import numpy as np

from oracle import nmdlm_oracle as O
from workloads import synth


def _model(seed, n_layers, T=8):
    return synth.make_mdlm(seed, n_layers, d=128, H=2, F=256, V=64, T=T, max_pos=64)


def test_no_encoder_one_block_is_plain_generation():
    m = _model(41, 1)
    prompt = synth.random_tokens(5, 14, m.V)
    ids, log = O.e2d2_generate(m, 0, prompt, n_blocks=1, B=4, steps=4, k_unmask=1)
    ref, ref_log = O.generate(m, prompt, n_blocks=1, B=4, steps=4, k_unmask=1)
    assert np.array_equal(ids, ref)
    assert all(np.array_equal(a, b) for a, b in zip(log, ref_log))


def test_unmask_invariants_and_determinism():
    m = _model(42, 3)
    prompt = synth.random_tokens(6, 10, m.V)
    ids, log = O.e2d2_generate(m, 2, prompt, n_blocks=2, B=4, steps=4, k_unmask=1)
    assert ids.shape == (8,) and np.all((ids >= 0) & (ids < m.V))
    assert len(log) == 8 and all(len(c) == 1 for c in log)
    for b in range(2):   # one new position per step, every position once per block
        assert sorted(int(c[0]) for c in log[4 * b:4 * b + 4]) == [0, 1, 2, 3]
    ids2, _ = O.e2d2_generate(m, 2, prompt, n_blocks=2, B=4, steps=4, k_unmask=1)
    assert np.array_equal(ids, ids2)


def test_decoder_reads_the_encoder_output():
    # the same decoder with a different encoder generally predicts differently
    m = _model(43, 3)
    other = synth.make_layer(999, 0, m.d, m.F, m.H)
    m2 = dataclasses.replace(m, layers=[other] + m.layers[1:])
    prompt = synth.random_tokens(7, 12, m.V)
    a, _ = O.e2d2_generate(m, 1, prompt, n_blocks=1, B=4, steps=2, k_unmask=2)
    b, _ = O.e2d2_generate(m2, 1, prompt, n_blocks=1, B=4, steps=2, k_unmask=2)
    c, _ = O.e2d2_generate(m, 1, prompt, n_blocks=1, B=4, steps=2, k_unmask=2)
    assert np.array_equal(a, c) and not np.array_equal(a, b)


def _hand_model():
    """Two layers, d = F = 64, one head, T = 4, built so that the encoder
    output h is known in closed form and the decoder's key/value projections
    copy their input:
      encoder: all projections zero except the down weights (column c: +2 for
        even c, -8 for odd c), activation table 127 everywhere, thresholds 128.
        Q = K = V = 0 so the attention output and A are 0, X1 = IF(128 X) = X;
        the up neurons get 127 every step and fire at steps 1, 2, 3 (V = 127,
        254 - 128, ...), so the down current is 0 at step 0 and 64 * (+2) = +128
        (even c) or 64 * (-8) = -512 (odd c) after; with the residual 128 X1 the
        output is h[0] = X[0], and for steps 1..3 every even channel fires and no
        odd one does (its membrane only falls).
      decoder: W_k = W_v = 100 I with thresholds 100, so K = V = the layer input."""
    m = synth.make_mdlm(61, 2, d=64, H=1, F=64, V=8, T=4, max_pos=32)
    th = {n: 128 for n in synth.THETA_NAMES}
    W_dn = np.where(np.arange(64)[None, :] % 2 == 0, 2, -8).repeat(64, axis=0).astype(np.int8)
    enc = synth.LayerParams(64, 64, 1, 64, np.zeros((64, 192), np.int8), np.zeros((64, 64), np.int8),
                            np.zeros((64, 64), np.int8), W_dn, th,
                            np.full(256, 1, np.uint8), np.full(256, 127, np.uint8), 0)
    dec0 = m.layers[1]
    Wqkv = dec0.W_qkv.copy()
    Wqkv[:, 64:128] = 100 * np.eye(64, dtype=np.int8)
    Wqkv[:, 128:192] = 100 * np.eye(64, dtype=np.int8)
    thd = dict(dec0.theta, k=100, v=100)
    dec = dataclasses.replace(dec0, W_qkv=Wqkv, theta=thd)
    return dataclasses.replace(m, layers=[enc, dec])


def test_decoder_context_keys_values_are_projections_of_the_encoder_output():
    m = _hand_model()
    emb01 = synth.unpack_bits(m.emb, m.d)                       # [V+1][T][d]
    prompt = np.array([3, 0, 7, 5, 1, 1, 6, 2], dtype=np.int32)
    st = O.e2d2_new_state(m, 1, 16)
    O.e2d2_encode(m, 1, prompt, 0, st, emb01)
    blk = np.array([4, 2, 2, 0], dtype=np.int32)
    O.e2d2_encode(m, 1, blk, 8, st, emb01)
    toks = np.concatenate([prompt, blk])
    X = np.zeros((m.T, 12, m.d), dtype=bool)                    # raw block input, by hand
    for j, tok in enumerate(toks):
        for t in range(m.T):
            X[t, j] = emb01[tok, t]
            X[t, j, m.pos_ch[j, t]] = True
    h = np.zeros_like(X)
    h[0] = X[0]
    h[1:, :, 0::2] = True                                       # the closed form above
    assert not np.array_equal(h[1:], X[1:])                     # h is not the raw input
    assert np.array_equal(st.kc_dec[0][:, :12], h)
    assert np.array_equal(st.vc_dec[0][:, :12], h)
    assert not st.kc_enc[0][:, :12].any() and not st.vc_enc[0][:, :12].any()
