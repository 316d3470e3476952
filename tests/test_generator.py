"""Seeded input generator: reproducibility, bit layout and the stated
distributions (CPU only)."""
import numpy as np

from workloads import synth


def test_pack_unpack_roundtrip_and_layout():
    rng = np.random.default_rng(0)
    for k in (1, 63, 64, 65, 200):
        bits = rng.random((3, 2, k)) < 0.5
        w = synth.pack_bits(bits)
        assert w.dtype == np.uint64 and w.shape == (3, 2, (k + 63) // 64)
        assert np.array_equal(synth.unpack_bits(w, k), bits)
    one = np.zeros(130, dtype=bool)
    one[0] = one[64 + 5] = one[129] = True
    w = synth.pack_bits(one)
    assert w.tolist() == [1, 1 << 5, 1 << 1]          # bit j of word w = channel 64w+j


def test_seeds_reproduce_and_differ():
    a = synth.linear_layer_case()
    b = synth.linear_layer_case()
    assert np.array_equal(a.S, b.S) and np.array_equal(a.W, b.W) and np.array_equal(a.bias, b.bias)
    c = synth.linear_layer_case(seed=7)
    assert not np.array_equal(a.W, c.W)


def test_linear_layer_distributions():
    c = synth.linear_layer_case()
    assert c.S.shape == (4, 8, 512) and c.W.shape == (512, 512) and c.theta == 256
    n = c.S.size
    assert abs(c.S.mean() - 0.15) < 5 * np.sqrt(0.15 * 0.85 / n)
    assert c.W.min() >= -127 and c.W.max() <= 127 and c.W.dtype == np.int8
    assert c.bias.min() >= -64 and c.bias.max() <= 64 and c.bias.dtype == np.int32


def test_rate_scaling_hits_target_mean():
    rng = synth.stream(1, 2)
    for rho in (0.02, 0.05, 0.1, 0.3):
        r = synth.scale_rates_to_mean(rng.beta(0.5, 8, size=5000), rho)
        assert abs(r.mean() - rho) < 1e-9 and r.max() <= 1.0 and r.min() >= 0


def test_layer_params_ranges():
    L = synth.make_layer(5, 0, 128, 256, 2)
    assert L.W_qkv.shape == (128, 384) and L.W_dn.shape == (256, 128)
    assert all(128 <= v <= 512 for v in L.theta.values()) and len(L.theta) == 7
    assert L.lut_att.min() >= 1 and np.all(np.diff(L.lut_att.astype(int)) >= 0)
    signed = L.lut_act.view(np.int8)[(np.arange(-128, 128) & 0xFF)]
    assert np.all(np.diff(signed.astype(int)) >= 0)
    assert L.s_up == 1


def test_mdlm_tables():
    m = synth.make_mdlm(3, 1, d=128, H=2, F=256, V=40, T=4, max_pos=32)
    assert m.emb.shape == (41, 4, 2) and m.pos_ch.shape == (32, 4)
    assert m.pos_ch.min() >= 0 and m.pos_ch.max() < 128
    assert m.scale.dtype == np.float32 and (m.scale >= 0.5 * 2 ** -10).all() and (m.scale < 1.5 * 2 ** -10).all()
