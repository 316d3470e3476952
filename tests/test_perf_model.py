"""The paper's analytic performance model (Sec. IV, Eqs. (12)-(16), Table I):
pinned by the printed Table I, the special cases the paper names (AR-LLM,
MDLM), a Monte Carlo count of spikes and loaded rows, and closed forms."""
import math
import os

import numpy as np
import pytest

from paper_2607_24841_amd import perf_model as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_platforms.txt")


def _table1():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, lops, ldata, eops, edata = [x.strip() for x in line.split("|")]
        rows[name] = (float(lops) * 1e12, float(ldata) * 1e12, float(eops) * 1e-12, float(edata) * 1e-12)
    return rows


def test_table1_platforms():
    t = _table1()
    for plat in (P.OCMS, P.ICMS):
        assert (plat.L_ops, plat.L_data, plat.E_ops, plat.E_data) == pytest.approx(t[plat.name])
    # Sec. V-B: the in-chip system has a compute-to-bandwidth ratio below 1 OP/b
    assert P.ICMS.ridge < 1.0 < P.OCMS.ridge


def test_special_cases_named_by_the_paper():
    D, T, b = 512, 8, 16
    # AR-LLM: B = 1, sigma = 0 -> every weight loaded for every token
    assert P.n_data(1, T, D, D, 0.0, b) == D * D * b
    assert P.n_ops(T, D, D, 0.0) == 2 * T * D * D
    # MDLM: sigma = 0, B tokens share one load of the weights
    for B in (2, 4, 32):
        assert P.n_data(B, T, D, D, 0.0, b) == pytest.approx(D * D * b / B)
    # all-silent input: no operations and no loads
    assert P.n_ops(T, D, D, 1.0) == 0.0 and P.n_data(4, T, D, D, 1.0, b) == 0.0


@pytest.mark.parametrize("B,T,sigma", [(1, 4, 0.9), (4, 4, 0.95), (16, 2, 0.97)])
def test_monte_carlo_counts(B, T, sigma):
    # i.i.d. spikes: count operations (2 per spike per output) and loaded
    # rows (rows with any spike in the block) and compare with Eqs. (12)-(13)
    rng = np.random.default_rng(1234 + B)
    d_in, d_out, b, reps = 256, 96, 8, 400
    ops, bits = [], []
    for _ in range(reps):
        X = rng.random((B * T, d_in)) >= sigma          # spike with prob 1 - sigma
        ops.append(2.0 * X.sum() * d_out / B)           # per token
        bits.append(X.any(axis=0).sum() * d_out * b / B)
    e_ops, e_bits = P.n_ops(T, d_in, d_out, sigma), P.n_data(B, T, d_in, d_out, sigma, b)
    # within 5 standard errors of the sample mean
    assert abs(np.mean(ops) - e_ops) <= 5 * np.std(ops) / math.sqrt(reps) + 1e-9
    assert abs(np.mean(bits) - e_bits) <= 5 * np.std(bits) / math.sqrt(reps) + 1e-9


def test_sparsity_erosion_with_block_size():
    # Sec. IV-B: the effective data-loading sparsity sigma^(BT) falls with B, so
    # the bits per block rise towards the dense load while the bits per token fall
    D, T, b, s = 512, 8, 16, 0.95
    per_block = [P.n_data(B, T, D, D, s, b) * B for B in (1, 2, 4, 8, 16)]
    per_token = [P.n_data(B, T, D, D, s, b) for B in (1, 2, 4, 8, 16)]
    assert all(x < y for x, y in zip(per_block, per_block[1:])) and per_block[-1] < D * D * b
    assert all(x > y for x, y in zip(per_token, per_token[1:]))


def test_regime_crossover_closed_form():
    # sigma = 0: ops/bit = 2 T B / b_W; compute-bound exactly when that reaches the ridge
    D, T, b = 512, 8, 16
    for plat in (P.OCMS, P.ICMS, P.MI355X):
        b_star = plat.ridge * b / (2 * T)
        for B in (1, 2, 4, 8, 16, 32, 64, 128):
            tl, regime = P.token_latency(P.n_ops(T, D, D, 0.0), P.n_data(B, T, D, D, 0.0, b), plat)
            assert regime == ("compute" if B >= b_star else "memory")
            assert tl == pytest.approx(max(2 * T * D * D / plat.L_ops, D * D * b / B / plat.L_data))
    # the OCMS system turns compute-bound at B = 37.5; the in-chip one at B < 1
    assert P.OCMS.ridge * b / (2 * T) == pytest.approx(37.5)


def test_throughput_trend_of_section_v():
    # Sec. V-C: on the off-chip system throughput keeps rising with B (memory-
    # bound); on the in-chip system it rises while memory-bound and saturates
    # once the layer turns compute-bound (here from B = 4)
    D, T, b = 512, 8, 16
    oc = P.throughput_curve(D, T, 0.8, b, (1, 2, 4, 8, 16), P.OCMS)
    ic = P.throughput_curve(D, T, 0.8, b, (1, 2, 4, 8, 16), P.ICMS)
    assert all(x[1] < y[1] for x, y in zip(oc, oc[1:])) and all(r == "memory" for _, _, r in oc)
    assert all(x[1] <= y[1] * (1 + 1e-12) for x, y in zip(ic, ic[1:]))
    assert [r for _, _, r in ic] == ["memory", "memory", "compute", "compute", "compute"]
    assert ic[2][1] == pytest.approx(ic[4][1])


def test_e2e_throughput_and_energy():
    enc = [2e-6, 3e-6]
    dec = [[1e-6, 1e-6], [0.5e-6, 0.5e-6]]          # two denoising steps
    assert P.e2e_throughput(enc, dec) == pytest.approx(1.0 / 8e-6)
    loads = [(1e9, 1e6), (2e9, 4e6)]
    assert P.energy_per_token(loads, P.OCMS) == pytest.approx(3e9 * 0.05e-12 + 5e6 * 10e-12)
    with pytest.raises(ValueError):
        P.energy_per_token(loads, P.MI355X)


def test_sigma_from_union_inverts_eq13():
    for s in (0.0, 0.5, 0.9, 0.99):
        for B, T in ((1, 4), (16, 4), (32, 8)):
            u = 1.0 - s ** (B * T)
            if 0.0 < 1.0 - u < 1.0:        # the union is not rounded to all rows
                assert P.sigma_from_union(u, B, T) == pytest.approx(s, rel=1e-6)
    assert P.sigma_from_union(1.0, 16, 4) == 0.0 and P.sigma_from_union(0.0, 16, 4) == 1.0


def test_layer_report_uses_measured_union():
    r = P.layer_report("x", B=16, T=4, d_in=1024, d_out=1024, union_frac=0.5, b_w=8, measured_us=3.0)
    assert r["n_data_bits_per_token"] == pytest.approx(1024 * 1024 * 0.5 * 8 / 16)
    tl, _ = P.token_latency(r["n_ops_per_token"], r["n_data_bits_per_token"], P.MI355X)
    assert r["MI355X"]["us_per_block"] == pytest.approx(tl * 16 * 1e6)
    rep = P.block_report([r, r], measured_step_us=10.0)
    assert rep["MI355X_us_per_block"] == pytest.approx(2 * r["MI355X"]["us_per_block"])
    assert rep["measured_products_us_per_block"] == 6.0
