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
