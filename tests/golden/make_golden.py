"""Write the stored expected values of the full-size MDLM cases.

Usage:  python tests/golden/make_golden.py mdlm12|mdlm24|e2d2

Calls only the oracle (oracle/) and the seeded generator (workloads/); the
HIP library is never imported here.  Outputs are JSON files next to this
script.  Large tensors are stored as SHA-256 digests of a fixed byte layout
(described in each file) plus small samples, so a GPU run is compared bit
for bit without shipping the tensors.
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import nmdlm_oracle as O  # noqa: E402
from workloads import synth  # noqa: E402


def sha(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def cache_digests(kc, vc, J):
    """Packed spike rows [T][J][d/64] (uint64 little endian) of each cache."""
    return ([sha(synth.pack_bits(k[:, :J])) for k in kc],
            [sha(synth.pack_bits(v[:, :J])) for v in vc])


def mdlm12():
    t0 = time.time()
    case = synth.mdlm12_step_case()
    m = case.model
    emb = O.unpack_model_emb(m)
    C, M = case.C, case.B
    kc, vc = O.new_caches(m.n_layers, m.T, C + M, m.d)
    O.prefill(O.block_input(case.ctx_tokens, np.arange(C), emb, m.pos_ch), m.layers, kc, vc)
    tokens = np.zeros(M, dtype=np.int32)
    masked = np.ones(M, dtype=bool)
    r = O.block_step(m, emb, tokens, masked, C, C, kc, vc, case.k_unmask)
    kd, vd = cache_digests(kc, vc, C + M)
    rng = np.random.default_rng(4)
    sample = [(int(i), int(j)) for i, j in zip(rng.integers(0, M, 256), rng.integers(0, m.V, 256))]
    unions = [[int(tr.unions[k].sum()) for k in ("qkv", "o", "up", "dn")] for tr in r.traces]
    out = {
        "case": "12-layer MDLM, one block step: d=2048, 16 heads x 128, FFN 8192, V=32000, T=4, "
                "1024 context tokens (prefill), block of 32 masked tokens, top-8 unmasking",
        "seed": synth.SEEDS["mdlm12"],
        "layout": "logits: float32 [M][V]; y: packed last-layer spikes uint64 [T][M][d/64]; "
                  "caches: packed spike rows uint64 [T][C+M][d/64] per layer",
        "tokens": r.tokens.tolist(),
        "masked": r.masked.astype(int).tolist(),
        "chosen": r.chosen.tolist(),
        "pred": r.pred.tolist(),
        "conf": [float(x) for x in r.conf],
        "logits_sha256": sha(r.logits.astype(np.float32)),
        "logits_sample": [[i, j, float(r.logits[i, j])] for i, j in sample],
        "y_sha256": sha(synth.pack_bits(r.Y)),
        "k_cache_sha256": kd,
        "v_cache_sha256": vd,
        "k_active": unions,
        "head_k_active": int(O.block_union(r.Y).sum()),
        "seconds": round(time.time() - t0, 1),
    }
    with open(os.path.join(HERE, "mdlm12_block_step.json"), "w") as f:
        json.dump(out, f, indent=1)


def mdlm24():
    t0 = time.time()
    case = synth.mdlm24_generation_case()
    m = case.model
    ids, log = O.generate(m, case.prompt, case.n_blocks, case.B, case.steps, case.k_unmask)
    out = {
        "case": "24-layer MDLM generation: d=2048, 16 heads x 128, FFN 8192, V=32000, T=4, "
                "2048-token prompt, 8 blocks of 32 tokens, 8 steps per block, 4 tokens per step",
        "seed": synth.SEEDS["mdlm24"],
        "ids": ids.tolist(),
        "chosen": [c.tolist() for c in log],
        "seconds": round(time.time() - t0, 1),
    }
    with open(os.path.join(HERE, "mdlm24_generation.json"), "w") as f:
        json.dump(out, f, indent=1)


def e2d2():
    t0 = time.time()
    case = synth.e2d2_case()
    m = case.model
    P = len(case.prompt)
    ids, log, st = O.e2d2_generate(m, case.n_enc, case.prompt, case.n_blocks, case.B,
                                   case.steps, case.k_unmask, return_state=True)
    J = P + case.n_blocks * case.B
    kd, vd = cache_digests(st.kc_dec, st.vc_dec, J)
    ke, ve = cache_digests(st.kc_enc[-1:], st.vc_enc[-1:], J)
    out = {
        "case": "encoder-decoder MDLM in the paper's shape: 28 encoder + 4 decoder layers, d=512, "
                "8 heads x 64, FFN 1536, V=32000, T=8; prompt 64 ids, 4 blocks of 4 tokens, "
                "4 denoising steps per block, 1 token unmasked per step",
        "seed": synth.SEEDS["e2d2"],
        "layout": "caches: packed spike rows uint64 [T][J][d/64], J = prompt + generated tokens",
        "ids": ids.tolist(),
        "chosen": [c.tolist() for c in log],
        "dec_k_cache_sha256": kd,
        "dec_v_cache_sha256": vd,
        "last_enc_k_cache_sha256": ke[0],
        "last_enc_v_cache_sha256": ve[0],
        "seconds": round(time.time() - t0, 1),
    }
    with open(os.path.join(HERE, "e2d2_generation.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    which = sys.argv[1] if len(sys.argv) > 1 else "mdlm12"
    {"mdlm12": mdlm12, "mdlm24": mdlm24, "e2d2": e2d2}[which]()
