"""Host-side checks of bench.py's contract (no GPU): more than one GPU is
refused with a message, the workloads parse, and the product-source digest
that guards the stored HBM traffic figure is the one of the sources."""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.parametrize("w", ["block", "ffn-sweep", "mdlm12-step", "mdlm24-generate",
                               "e2d2-generate", "ternary-ffn", "block-batch", "tp-shard"])
def test_workloads_parse(w, monkeypatch):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", w, "--flags", "0x10000"])
    a = bench.parse()
    assert a.workload == w and a.flags == 0x10000 and a.gpus == 1


def test_traffic_digest_covers_the_product_sources():
    h = hashlib.sha256()
    for rel in bench.PRODUCT_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    assert bench.product_sources_sha256() == h.hexdigest()
    # a stored figure is reported only for the sources it was measured on
    for w, rec in bench.TRAFFIC.items():
        want = rec["bytes_per_launch"] if rec["sources_sha256"] == h.hexdigest() else None
        assert bench.product_traffic(w) == want
    assert bench.product_traffic("no such workload") is None


def test_default_workload_is_the_twelve_layer_step(monkeypatch):
    monkeypatch.setattr(sys, "argv", ["bench.py"])
    a = bench.parse()
    assert a.workload == "mdlm12-step" and a.gpus == 1 and a.steps > 0 and a.warmup >= 0


def test_product_bytes_is_the_row_load_rule():
    # K_active * N weight bytes + packed spikes in and out (T*M rows)
    assert bench.product_bytes(1024, 100, 512, 4, 16) == 100 * 512 + 4 * 16 * 16 * 8 + 4 * 16 * 8 * 8


def test_batched_prefill_fits_the_step_row_limit():
    # the block-batch mode prefills every sequence's context in one call:
    # T * n * C must stay within a step's 2^19 rows (and so must the block)
    from workloads import synth
    c = synth.block_case()
    n = max(bench.BATCH_SEQS)
    assert c.T * n * c.C <= 1 << 19 and c.T * n * c.M <= 1 << 19
    assert c.M % (16 // c.T) == 0          # batched steps need M a multiple of 16/T


@pytest.mark.parametrize("k_active", [0, 1, 37, 2048])
def test_shard_inputs_have_the_requested_union(k_active):
    import numpy as np
    S = bench._spikes_with_union(np.random.default_rng(k_active), 4, 32, 2048, k_active, 0.3)
    assert S.shape == (4, 32, 2048) and int(S.any(axis=(0, 1)).sum()) == k_active


@pytest.mark.parametrize("g", [1, 2, 4, 8, 16])
def test_shard_dims_are_whole_tiles(g):
    # the 12-layer model: d=2048, 16 heads, FFN 8192, vocabulary 32000
    c = bench.shard_dims(2048, 16, 8192, 32000, g)
    assert c["qkv"] == 3 * c["o"] and c["o"] * g == 2048 and c["up"] * g == 8192
    assert all(v % 64 == 0 for v in c.values())
    assert 32000 <= c["head"] * g < 32000 + 64 * g


def test_shard_dims_refuse_uneven_splits():
    assert bench.shard_dims(2048, 16, 8192, 32000, 3) is None
    assert bench.shard_dims(2048, 16, 8192, 32000, 32) is None   # heads
    assert bench.shard_dims(2048, 16, 8192, 32000, 0) is None
