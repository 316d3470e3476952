#!/usr/bin/env python3
"""Benchmark of the N-MDLM block-denoising step on one MI355X.

Workload (default, --workload mdlm12-step): a 12-layer spiking MDLM
(d=2048, 16 heads of 128, FFN 8192, vocab 32000 with an int8 head
dequantised to fp32 logits, T=4) at one block-denoising step: 32 masked
tokens over 1024 context tokens, head, confidence and top-8 unmasking.  The
context prefill runs once, untimed.  Weights are seeded int8 uniforms
(workloads/synth.py); 640 MB of weights per step, more than the 256 MB
last-level cache, so every step streams its weights from HBM.  The model
also holds the blocked copies of its weights (--weights blocked, the
default): each wave of a product reads them when its words' union is dense;
--weights rows keeps the row-major weights only.

A "step" is one nmdlm_block_step (block input, per layer the QKV product,
attention, O, up and down products with their neurons, then the head,
confidence and unmasking), preceded by two small copies that reset the
block to fully masked so that every step is the same workload.  One step is
captured as a HIP graph before the timed region; the timed region replays it
--steps times after --warmup replays.

Prints one JSON line: block-denoise tokens/s, the weight-skip fraction, the
touched-weight bandwidth of the whole step, the roofline of the product
kernel (every product launch of one step timed with HIP events stamped by
its own dispatch), and the CPU oracle's rate on a bounded sample.

Other workloads (--workload):
  block            one spiking transformer block (d=1024, 16 heads of 64, FFN 4096, T=4) at
     one denoising step, 16 masked tokens over 512 context tokens, inputs
     Bernoulli(0.10); 32 rotating layer copies (403 MB) so that weights stream
     from HBM; with the paper's analytic model beside the measured products.
  ffn-sweep        FFN weight-traffic sweep, d=4096 -> 14336 -> 4096, T=4, B in {1,4,16,64},
     mean input density in {.02,.05,.10,.30}: skipped-row fraction, touched
     bytes and GB/s of the up and down products at every point (4 rotating
     weight copies, 470 MB, so that weights stream from HBM).
  mdlm24-generate  24-layer MDLM generation: prompt of 2048 ids, 8 blocks of 32 tokens,
     8 steps per block, 4 tokens unmasked per step.
  e2d2-generate    the paper's own shape: encoder-decoder MDLM with 28 encoder and 4
     decoder layers, d=512, FFN 1536, T=8; 64-id prompt, 4 blocks of 4 tokens, one
     token unmasked per step (block-causal encoder, each token encoded once).
  ternary-ffn      the paper's ternary bitwise coding (T=8) through the FFN
     4096 -> 14336 -> 4096: encode, up product, encode, down product, for B in
     {1, 4, 16} tokens and K in {1, 2, 4} quantisation levels.
  block-batch      the block step over n_seq in {1, 2, 4, 8, 16, 32, 64, 128}
     sequences at once (each with its own 512-token context and 16-token block): every product
     reads a weight row once for the whole batch; tokens/s, union fractions and
     touched bytes per point, beside the analytic model at the measured unions.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E, published


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--copies", type=int, default=32, help="rotating layer copies (>= 256 MB total)")
    p.add_argument("--eager", action="store_true", help="issue kernels directly, no HIP graph")
    p.add_argument("--weights", choices=("rows", "blocked"), default="blocked",
                   help="rows: row-major weights only; blocked: also the blocked copies, read by "
                        "products over dense unions")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="host seconds of oracle steps for cpu_baseline")
    p.add_argument("--seed", type=int, default=1002)
    p.add_argument("--flags", type=lambda x: int(x, 0), default=0,
                   help="extra block-step flags (path overrides; results do not change)")
    p.add_argument("--workload", default="mdlm12-step",
                   choices=("mdlm12-step", "block", "ffn-sweep", "mdlm24-generate",
                            "e2d2-generate", "ternary-ffn", "block-batch", "tp-shard"),
                   help="mdlm12-step: the 12-layer MDLM at one block step (default)")
    p.add_argument("--tp", type=int, default=8,
                   help="tp-shard: GPUs the 12-layer step's columns and heads are split over")
    p.add_argument("--reps", type=int, default=20,
                   help="timed repetitions (ffn-sweep, mdlm12-step)")
    return p.parse_args()


# HBM bytes per launch of the product kernel, per workload, from two rocprofv3
# --pmc passes (FETCH_SIZE, then WRITE_SIZE) over `bench.py --eager`, each
# scaled by what the counter reads for a 64 MiB device copy (FETCH_SIZE x 2.0,
# WRITE_SIZE x 1.0); the summaries with their commands are under profiles/.
# A value holds only for the product-kernel sources with the recorded digest:
# any change to them reports null until the counters are taken again.
TRAFFIC = {
    "block": {"sources_sha256": "fc86da0ff2f80f4b93457c5fe8375e7be50dccbc03ec8dba1b5897440c3dd954",
              "bytes_per_launch": 2773553.6},
    "mdlm12": {"sources_sha256": "fc86da0ff2f80f4b93457c5fe8375e7be50dccbc03ec8dba1b5897440c3dd954",
               "bytes_per_launch": 14211689.4},
}
PRODUCT_SOURCES = ("paper_2607_24841_amd/csrc/qbsm.hip", "paper_2607_24841_amd/csrc/common.h")


def product_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for rel in PRODUCT_SOURCES:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def product_traffic(workload: str):
    rec = TRAFFIC.get(workload)
    if rec and rec["sources_sha256"] and rec["sources_sha256"] == product_sources_sha256():
        return rec["bytes_per_launch"]
    return None


def stream_copy_gbps(torch, nbytes=2 << 30, reps=10):
    """A measured streaming rate of the device's HBM: the median of a
    device-to-device copy of nbytes, counting the bytes read and written, in
    GB/s."""
    import numpy as np
    x = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        y.copy_(x)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    del x, y
    return 2 * nbytes / (float(np.median(ts)) * 1e-3) / 1e9


def product_bytes(k_total, k_active, n, T, M):
    """Algorithmic bytes of one product launch: active weight rows, packed
    input spikes, packed output spikes."""
    kw = (k_total + 63) // 64
    nw = (n + 63) // 64
    return k_active * n + T * M * kw * 8 + T * M * nw * 8


def cpu_baseline(case, seconds: float):
    """The oracle (as it stands) on the host: untimed prefill, then as many
    block steps as fit in `seconds` (at least 2)."""
    import numpy as np
    from oracle import nmdlm_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    L = case.layer
    kc, vc = O.new_caches(1, case.T, case.C + case.M, L.d)
    O.prefill(case.X_ctx, [L], kc, vc)
    n = 0
    t0 = time.perf_counter()
    while True:
        O.layer_forward(case.X_blk, L, kc[0], vc[0], case.C)
        n += 1
        dt = time.perf_counter() - t0
        if (dt >= seconds and n >= 2) or n >= 1000:
            break
    return {"value": case.M * n / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n} oracle block steps of the same workload (16 tokens each) after an "
                      f"untimed oracle prefill of the 512 context tokens; {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the step over "
              f"several GPUs is not built.", file=sys.stderr)
        sys.exit(2)
    {"block": bench_block, "ffn-sweep": bench_ffn_sweep, "mdlm12-step": bench_mdlm12_step,
     "mdlm24-generate": bench_mdlm24_generate,
     "e2d2-generate": bench_e2d2_generate, "ternary-ffn": bench_ternary_ffn,
     "block-batch": bench_block_batch, "tp-shard": bench_tp_shard}[args.workload](args)


def _graph(fn):
    """Capture fn() (library calls on torch's current stream) into a HIP graph,
    after one warm run on the capture stream."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _time_eager(fn, reps):
    """Median over reps of fn() issued directly, in ms (torch events)."""
    import numpy as np
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def _time_graph(g, reps):
    """Median over reps of one replay, in ms (torch events on the replay stream)."""
    import numpy as np
    import torch
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def bench_ffn_sweep(args):
    """FFN weight-traffic sweep: both projections driven by synthetic spikes."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd import perf_model
    from workloads import synth

    B.load()
    ffn = synth.ffn_sweep_weights()
    d, F = ffn.W_up.shape
    T = 4
    n_copies = 4                       # 4 x (58.7 + 58.7) MB > 256 MB last-level cache
    W_up = [torch.from_numpy(ffn.W_up).cuda() for _ in range(n_copies)]
    W_dn = [torch.from_numpy(ffn.W_dn).cuda() for _ in range(n_copies)]
    blocked = args.weights == "blocked"
    # blocked operand-order copies beside the row-major weights (each wave of
    # a product reads the copy or the rows by its union)
    Wb_up = [B.blocked_weights(w, d, F, F) for w in W_up] if blocked else None
    Wb_dn = [B.blocked_weights(w, F, d, d) for w in W_dn] if blocked else None
    th_up, th_dn = int(ffn.theta_up), int(ffn.theta_dn)
    points = []
    for iB in range(len(synth.FFN_SWEEP_BLOCKS)):
        for iR in range(len(synth.FFN_SWEEP_DENSITIES)):
            pt = synth.ffn_sweep_point(iB, iR)
            Bk = pt.B
            xu = B.to_dev_bits(synth.pack_bits(pt.X_up))
            xd = B.to_dev_bits(synth.pack_bits(pt.X_dn))
            su = torch.empty((T, Bk, (F + 63) // 64), dtype=torch.int64, device="cuda")
            sd = torch.empty((T, Bk, (d + 63) // 64), dtype=torch.int64, device="cuda")
            st = torch.zeros((2, 4), dtype=torch.int64, device="cuda")
            ws = B.workspace(max(B.nmdlm_qbsm_workspace_size(T, Bk, d, F),
                                 B.nmdlm_qbsm_workspace_size(T, Bk, F, d)))

            def up(c):
                if blocked:
                    B.nmdlm_qbsm_blocked(xu, T, Bk, d, W_up[c], Wb_up[c], F, F, theta=th_up,
                                         s_out=su, stats=st[0], flags=args.flags, ws=ws)
                else:
                    B.nmdlm_qbsm(xu, T, Bk, d, W_up[c], F, F, theta=th_up, s_out=su, stats=st[0],
                                 flags=args.flags, ws=ws)

            def dn(c):
                if blocked:
                    B.nmdlm_qbsm_blocked(xd, T, Bk, F, W_dn[c], Wb_dn[c], d, d, theta=th_dn,
                                         s_out=sd, stats=st[1], flags=args.flags, ws=ws)
                else:
                    B.nmdlm_qbsm(xd, T, Bk, F, W_dn[c], d, d, theta=th_dn, s_out=sd, stats=st[1],
                                 flags=args.flags, ws=ws)

            if args.eager:           # one dispatch per launch (for counter passes)
                t_up = _time_eager(lambda: [up(c) for c in range(n_copies)], args.reps) / n_copies
                t_dn = _time_eager(lambda: [dn(c) for c in range(n_copies)], args.reps) / n_copies
            else:
                g_up = _graph(lambda: [up(c) for c in range(n_copies)])
                g_dn = _graph(lambda: [dn(c) for c in range(n_copies)])
                t_up = _time_graph(g_up, args.reps) / n_copies
                t_dn = _time_graph(g_dn, args.reps) / n_copies
                del g_up, g_dn
            k = st.cpu().numpy()
            rec = {"B": Bk, "density": pt.density}
            for nm, row, t, X in (("up", k[0], t_up, pt.X_up), ("dn", k[1], t_dn, pt.X_dn)):
                touched = int(row[1] * row[2])
                # the paper's Eqs. (12)-(14) at MI355X peaks from the measured
                # union and input sparsity
                mod = perf_model.layer_report(nm, Bk, T, int(row[0]), int(row[2]),
                                              float(row[1]) / float(row[0]), b_w=8,
                                              sigma=1.0 - float(np.mean(X)))
                rec[nm] = {"us": t * 1e3, "k_active": int(row[1]), "k_total": int(row[0]),
                           "skip": 1.0 - row[1] / row[0], "touched_bytes": touched,
                           "GBps": touched / (t * 1e-3) / 1e9,
                           "model_us_MI355X": mod["MI355X"]["us_per_block"],
                           "model_regime_MI355X": mod["MI355X"]["regime"]}
            rec["tokens_per_s"] = Bk / ((t_up + t_dn) * 1e-3)
            points.append(rec)
    # time against the active-row fraction per block size and product: a
    # least-squares line t = t0 + slope * (K_active / K) over the densities
    lin = []
    for Bk in sorted({p["B"] for p in points}):
        for nm in ("up", "dn"):
            xs = np.array([p[nm]["k_active"] / p[nm]["k_total"] for p in points if p["B"] == Bk])
            ys = np.array([p[nm]["us"] for p in points if p["B"] == Bk])
            slope, t0 = np.polyfit(xs, ys, 1)
            fit = t0 + slope * xs
            ss = float(((ys - ys.mean()) ** 2).sum())
            r2 = 1.0 - float(((ys - fit) ** 2).sum()) / ss if ss > 0 else 1.0
            lin.append({"B": Bk, "product": nm, "active_frac": [round(float(x), 4) for x in xs],
                        "us": [round(float(y), 2) for y in ys], "t0_us": float(t0),
                        "slope_us_per_active_frac": float(slope), "r2": r2,
                        "scaling_share_at_max": float(slope * xs.max() / ys.max())})
    head = [p for p in points if p["B"] == 64 and p["density"] == 0.30][0]
    best = max((p[m]["GBps"], p, m) for p in points for m in ("up", "dn"))
    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": head["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.reps,
        "warmup": 1, "ms_per_step": (head["up"]["us"] + head["dn"]["us"]) / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "FFN weight-traffic sweep d=4096->14336->4096, T=4, "
                               "Beta(0.5,8) per-neuron rates; value at B=64, density 0.30",
                   "weight_copies_rotated": n_copies, "weights": args.weights,
                   "issue": "eager" if args.eager else "hip_graph"},
        "weight_skip_fraction": 1.0 - (head["up"]["touched_bytes"] + head["dn"]["touched_bytes"])
        / (head["up"]["k_total"] * F + head["dn"]["k_total"] * d),
        "roofline": {"kernel": "k_qbsm (int8 MFMA spike product with fused IF epilogue)",
                     "bound": "hbm", "achieved": best[0], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": best[0] / HBM_PEAK_GBPS, "traffic": None,
                     "at": f"B={best[1]['B']} density={best[1]['density']} {best[2]}"},
        "sweep": points,
        "time_vs_active_fraction": lin,
    }
    print(json.dumps(out), flush=True)


def _mdlm_step_io(B, torch, m, C, M, k, flags, ev=None):
    tok = torch.zeros(M, dtype=torch.int32, device="cuda")
    msk = torch.ones(M, dtype=torch.uint8, device="cuda")
    bufs = dict(
        tok=tok, msk=msk, tok0=tok.clone(), msk0=msk.clone(),
        logits=torch.empty((M, m.V), dtype=torch.float32, device="cuda"),
        pred=torch.empty(M, dtype=torch.int32, device="cuda"),
        conf=torch.empty(M, dtype=torch.float64, device="cuda"),
        chosen=torch.empty(k, dtype=torch.int32, device="cuda"),
        stats=torch.zeros((4 * m.n_layers + 1, 4), dtype=torch.int64, device="cuda"))
    io = B.step_io(M, C, pos0=C, flags=flags, tokens=tok, masked=msk, k_unmask=k,
                   logits=bufs["logits"], pred=bufs["pred"], conf=bufs["conf"],
                   unmasked_pos=bufs["chosen"], stats=bufs["stats"],
                   prof_events=ev)
    return io, bufs


def cpu_info():
    """Host CPU model and logical core count (for the oracle's timing)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count() or 1


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        return os.cpu_count() or 1


def cpu_baseline_mdlm12(case, seconds: float, one_thread_layers: int = 2):
    """The oracle (as it stands) on the host for the 12-layer step: the same
    step (block input, 12 layers, head, confidence, top-8 unmasking of 32
    masked tokens over 1024 context rows) timed in full for about `seconds`.
    The context keys/values the step attends to come from a seeded
    Bernoulli(0.3) fill of the caches instead of the oracle's prefill (about
    4 minutes of host time): the oracle's work does not depend on the cache
    values, only on their shapes.  A 1-thread rate is taken on a sample of
    `one_thread_layers` layers plus the head, scaled to the 12 layers."""
    import numpy as np
    from oracle import nmdlm_oracle as O
    m = case.model
    C, M, k = case.C, case.B, case.k_unmask
    emb = O.unpack_model_emb(m)
    kc, vc = O.new_caches(m.n_layers, m.T, C + M, m.d)
    rng = np.random.default_rng(20261202)
    for l in range(m.n_layers):
        kc[l][:, :C] = rng.random((m.T, C, m.d)) < 0.3
        vc[l][:, :C] = rng.random((m.T, C, m.d)) < 0.3
    tokens = np.zeros(M, dtype=np.int32)
    masked = np.ones(M, dtype=bool)
    n = 0
    t0 = time.perf_counter()
    while True:
        O.block_step(m, emb, tokens, masked, C, C, kc, vc, k)
        n += 1
        dt = time.perf_counter() - t0
        if dt >= seconds or n >= 100:
            break
    threads = blas_threads()
    # 1 thread: a sample of layers and the head, scaled to the whole stack
    one = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            X = O.block_input(np.full(M, m.mask_id, dtype=np.int32), np.arange(C, C + M), emb,
                              m.pos_ch)
            t1 = time.perf_counter()
            for l in range(one_thread_layers):
                X = O.layer_forward(X, m.layers[l], kc[l], vc[l], C).Y
            t_layers = time.perf_counter() - t1
            t1 = time.perf_counter()
            logits = O.head_logits(X, m.W_head, m.scale)
            pred, conf = O.confidence(logits)
            O.unmask(tokens, masked, pred, conf, k)
            t_head = time.perf_counter() - t1
        t_step1 = t_layers * m.n_layers / one_thread_layers + t_head
        one = {"value": M / t_step1, "unit": "tokens/s", "cores": 1,
               "sample": f"{one_thread_layers} oracle layers ({t_layers:.1f} s) + head, "
                         f"confidence and unmasking ({t_head:.1f} s) at 1 thread, the layers "
                         f"scaled to {m.n_layers}"}
    except Exception as e:  # threadpoolctl missing: no 1-thread figure
        one = {"error": repr(e)}
    model_name, nproc = cpu_info()
    return {"value": M * n / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} full oracle block steps of the 12-layer workload (32 block tokens "
                      f"each) in {dt:.1f} s; context keys/values from a seeded Bernoulli(0.3) "
                      f"cache fill instead of the oracle prefill",
            "cpu_model": model_name, "nproc": nproc, "one_thread": one}


def bench_mdlm12_step(args):
    """12-layer MDLM, one block step with head, confidence and unmasking
    (the default workload)."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from workloads import synth

    B.load()
    case = synth.mdlm12_step_case()
    m = case.model
    C, M, k = case.C, case.B, case.k_unmask
    dm = B.DeviceModel.from_mdlm(m, C + M, blocked=args.weights == "blocked")
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, C, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, M, 0)))
    ctx = torch.from_numpy(case.ctx_tokens.astype(np.int32)).cuda()
    # context prefill (Eq. (5)), untimed
    B.nmdlm_block_step(dm, B.step_io(C, 0, flags=B.NMDLM_NO_HEAD, tokens=ctx,
                                     masked=torch.zeros(C, dtype=torch.uint8, device="cuda")), ws)
    io, b = _mdlm_step_io(B, torch, m, C, M, k, args.flags)

    def step():
        # every step starts from the fully masked block (two small copies),
        # so that each timed step is the same workload
        b["tok"].copy_(b["tok0"])
        b["msk"].copy_(b["msk0"])
        B.nmdlm_block_step(dm, io, ws)

    # --- everything the timed region replays is captured before it -----------
    g = None if args.eager else _graph(step)

    def run(n):
        for _ in range(n):
            if g is None:
                step()
            else:
                g.replay()

    run(args.warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = 1e3 * dt / args.steps
    # per-step distribution after the timed region (HIP events around single steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    per = []
    for _ in range(20):
        e0.record()
        run(1)
        e1.record()
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1))
    pct = {"p10": float(np.percentile(per, 10)), "p50": float(np.percentile(per, 50)),
           "p90": float(np.percentile(per, 90)), "samples": len(per)}
    st = b["stats"].cpu().numpy()
    touched = int((st[:, 1] * st[:, 2]).sum())
    dense = int((st[:, 0] * st[:, 2]).sum())

    # --- product kernel timed per launch: the library stamps a HIP event pair
    #     with the start and end of every product kernel (from its dispatch).
    #     Events cannot be graph nodes here, so one step is issued directly
    #     behind a spin kernel: the queue fills while it spins and the kernels
    #     then run back to back, as in the timed region.
    n_prod = 4 * m.n_layers + 1
    ev = B.HipEvents(2 * n_prod)
    pio, pb = _mdlm_step_io(B, torch, m, C, M, k, args.flags, ev=ev.arr)
    B.nmdlm_block_step(dm, pio, ws)          # warm the event path
    torch.cuda.synchronize()
    pb["tok"].copy_(pb["tok0"])
    pb["msk"].copy_(pb["msk0"])
    torch.cuda._sleep(50_000_000)
    B.nmdlm_block_step(dm, pio, ws)
    torch.cuda.synchronize()
    dur = [ev.elapsed_ms(2 * p, 2 * p + 1) for p in range(n_prod)]
    pst = pb["stats"].cpu().numpy()
    nbytes = [product_bytes(int(r[0]), int(r[1]), int(r[2]), m.T, M) for r in pst]
    ev.close()
    achieved = sum(nbytes) / (sum(dur) * 1e-3) / 1e9
    kinds = {}
    for p in range(n_prod):
        nm = "head" if p == n_prod - 1 else ("qkv", "o", "up", "down")[p % 4]
        kd = kinds.setdefault(nm, {"launches": 0, "us": 0.0, "bytes": 0})
        kd["launches"] += 1
        kd["us"] += 1e3 * dur[p]
        kd["bytes"] += nbytes[p]
    per_kind = {nm: {"launches": v["launches"], "avg_us": v["us"] / v["launches"],
                     "avg_bytes": v["bytes"] / v["launches"],
                     "GBps": v["bytes"] / (v["us"] * 1e-6) / 1e9} for nm, v in kinds.items()}
    traffic = product_traffic("mdlm12")
    stream = stream_copy_gbps(torch)
    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": M / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": "12-layer spiking MDLM, one block step: d=2048, 16 heads x 128, "
                               "FFN 8192, vocab 32000 (int8 head, fp32 logits), T=4, 32 masked "
                               "tokens over 1024 context tokens (prefilled, untimed), head + "
                               "confidence + top-8 unmasking",
                   "block_tokens": M, "context_tokens": C, "layers": m.n_layers,
                   "issue": "eager" if args.eager else "hip_graph (one step per replay)",
                   "weights": args.weights},
        "step_ms_percentiles": pct,
        "timing_check": {"ms_per_step_over_replay_p50": ms_per_step / pct["p50"]},
        "unmasked_tokens_per_s": k / (ms_per_step * 1e-3),
        "weight_skip_fraction": 1.0 - touched / dense,
        "touched_weight_bytes_per_step": touched,
        "touched_weight_GBps": touched / (ms_per_step * 1e-3) / 1e9,
        "roofline": {"kernel": "k_qbsm_words (int8 MFMA spike product with fused epilogue; all "
                               "49 product launches of the step)",
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "stream_copy_GBps": stream, "frac_of_stream_copy": achieved / stream,
                     "avg_launch_ms": float(np.mean(dur)), "launches_timed": len(dur),
                     "algorithmic_bytes_per_launch": float(np.mean(nbytes)),
                     "per_product": per_kind,
                     "timing_issue": "direct issue behind a spin kernel (queue full)"},
        "per_layer_k_active": st[:-1, 1].reshape(m.n_layers, 4).tolist(),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_mdlm12(case, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def _spikes_with_union(rng, T, M, K, k_active, fill):
    """Spikes bool [T][M][K] whose block union is exactly k_active input
    neurons: each chosen neuron spikes at one random (t, m) and with
    probability `fill` at the others."""
    import numpy as np
    S = np.zeros((T, M, K), dtype=bool)
    rows = rng.choice(K, k_active, replace=False)
    S[:, :, rows] = rng.random((T, M, k_active)) < fill
    S[rng.integers(0, T, k_active), rng.integers(0, M, k_active), rows] = True
    return S


def shard_dims(d, H, F, V, g):
    """Output columns of one GPU's products when the step is split over g
    GPUs by columns (attention by heads): QKV, O, up, down and the head's
    vocabulary slice, each a whole number of 64-column tiles (the vocabulary
    padded up to one).  None when g does not divide the heads and tiles."""
    if g < 1 or H % g or d % (64 * g) or F % (64 * g):
        return None
    return {"qkv": 3 * d // g, "o": d // g, "up": F // g, "down": d // g,
            "head": (V + 64 * g - 1) // (64 * g) * 64}


def bench_tp_shard(args):
    """One GPU's share of the 12-layer block step split over --tp GPUs by
    output columns (every product) and by heads (attention): the shard-shape
    kernels of all layers and the head's vocabulary slice, chained in one HIP
    graph.  The collectives between them (four spike all-gathers per layer
    and the confidence combine) are not run on one GPU; their count and
    payloads are reported.  Union sizes come from one full step of the
    12-layer model, inputs with exactly those unions from a seeded generator."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from workloads import synth

    B.load()
    g = args.tp
    case = synth.mdlm12_step_case()
    m = case.model
    C, M, k = case.C, case.B, case.k_unmask
    T, d, H, F, V = m.T, m.d, m.H, m.F, m.V
    cols = shard_dims(d, H, F, V, g)
    if cols is None:
        print(f"tp-shard: {g} does not divide the heads ({H}) and 64-column tiles", file=sys.stderr)
        sys.exit(2)
    # union sizes of every product: one full step (prefill untimed)
    dm = B.DeviceModel.from_mdlm(m, C + M, blocked=True)
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, C, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, M, 0)))
    ctx = torch.from_numpy(case.ctx_tokens.astype(np.int32)).cuda()
    B.nmdlm_block_step(dm, B.step_io(C, 0, flags=B.NMDLM_NO_HEAD, tokens=ctx,
                                     masked=torch.zeros(C, dtype=torch.uint8, device="cuda")), ws)
    io, b = _mdlm_step_io(B, torch, m, C, M, k, 0)
    B.nmdlm_block_step(dm, io, ws)
    torch.cuda.synchronize()
    kact = b["stats"].cpu().numpy()[:, 1].astype(int)
    del dm, ws, io, b, ctx
    torch.cuda.empty_cache()

    rng = np.random.default_rng(args.seed)
    dh, Hs, ds = d // H, H // g, d // g
    cap = (C + M + 63) // 64 * 64
    dims = (("qkv", d, cols["qkv"]), ("o", d, cols["o"]), ("up", d, cols["up"]),
            ("down", F, cols["down"]))
    lut = torch.from_numpy(synth.sorted_lut_u8(synth.stream(args.seed, 7))).cuda()
    calls = []      # (kind, zero-argument launcher)
    keep = []       # device buffers the launchers use

    def product(kind, K, N, ka):
        W = torch.randint(-127, 128, (K, N), dtype=torch.int8, device="cuda")
        Wb = B.blocked_weights(W, K, N, N)
        s_in = B.to_dev_bits(synth.pack_bits(_spikes_with_union(rng, T, M, K, ka, 0.3)))
        out = torch.empty((T, M, (N + 63) // 64), dtype=torch.int64, device="cuda")
        pws = B.workspace(B.nmdlm_qbsm_workspace_size(T, M, K, N))
        keep.extend((W, Wb, s_in, out, pws))
        calls.append((kind, lambda: B.nmdlm_qbsm_blocked(s_in, T, M, K, W, Wb, N, N, theta=300,
                                                          s_out=out, ws=pws)))

    for l in range(m.n_layers):
        for p, (nm, K, N) in enumerate(dims):
            product(nm, K, N, int(kact[4 * l + p]))
            if nm == "qkv":      # this GPU's heads over the full context
                q = B.to_dev_bits(synth.pack_bits(rng.random((T, M, ds)) < 0.45))
                kc = B.to_dev_bits(synth.pack_bits(rng.random((T, cap, ds)) < 0.45))
                vw = synth.pack_bits(rng.random((T, ds, cap)) < 0.45)          # [T][ds][cap/64]
                vt = B.to_dev_bits(np.ascontiguousarray(vw.transpose(0, 2, 1)))
                a = torch.empty((T, M, ds), dtype=torch.int32, device="cuda")
                sa = torch.empty((T, M, ds // 64), dtype=torch.int64, device="cuda")
                keep.extend((q, kc, vt, a, sa))
                calls.append(("attn", lambda q=q, kc=kc, vt=vt, a=a, sa=sa: B.nmdlm_bbm_attn(
                    q, kc, vt, cap, T, M, C, Hs, dh, lut, a_out=a, theta_a=300, s_out=sa)))
    Vs = cols["head"]
    product("head", d, Vs, int(kact[-1]))

    def run_all():
        for _, fn in calls:
            fn()
    gr = _graph(run_all)
    ms = _time_graph(gr, args.reps)
    # each kind alone: its calls back to back in a graph of their own, the
    # head's repeated 12 times so that the graph launch is amortised alike
    per_kind = {}
    for kind in ("qkv", "attn", "o", "up", "down", "head"):
        fns = [fn for kd, fn in calls if kd == kind]
        fns = fns * max(1, m.n_layers // len(fns))
        gk = _graph(lambda fns=fns: [fn() for fn in fns])
        per_kind[kind] = {"calls_per_step": len(fns) if kind != "head" else 1,
                          "us_per_call": 1e3 * _time_graph(gk, args.reps) / len(fns)}
        del gk
    gather_bytes = [T * M * d // 8, T * M * d // 8, T * M * F // 8, T * M * d // 8]
    out = {
        "metric": "per-GPU kernel time of a tensor-parallel shard of the block step",
        "value": ms, "unit": "ms", "n_gpus": 1, "steps": args.reps, "warmup": 1,
        "ms_per_step": ms, "higher_is_better": False, "scaling": "strong", "vs_baseline": None,
        "dtype": "int8", "data": "synthetic",
        "config": {"workload": f"the 12-layer block step (d=2048, 16 heads x 128, FFN 8192, vocab "
                               f"32000, T=4, 32 block tokens over 1024 context tokens) as one of "
                               f"{g} GPUs: every product over {1}/{g} of its output columns, "
                               f"attention over {Hs} heads, the head over {Vs} vocabulary "
                               f"entries (product with IF output standing in for the logits "
                               f"epilogue); collectives not run",
                   "tp": g, "issue": "hip_graph", "weights": "blocked"},
        "per_kind": per_kind,
        "collectives_per_step": {"spike_all_gathers": 4 * m.n_layers,
                                 "all_gather_bytes_per_layer": gather_bytes,
                                 "confidence_combines": 1},
        "one_gpu_union_sizes": kact.tolist(),
    }
    print(json.dumps(out), flush=True)


def bench_mdlm24_generate(args):
    """24-layer MDLM block-diffusion generation (prefill timed apart)."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd.generate import Generator
    from workloads import synth

    B.load()
    case = synth.mdlm24_generation_case()
    m = case.model
    P = len(case.prompt)
    dm = B.DeviceModel.from_mdlm(m, P + case.n_blocks * case.B, blocked=args.weights == "blocked")
    gen = Generator(dm, P, case.B)
    ids = torch.from_numpy(np.asarray(case.prompt, dtype=np.int32)).cuda()
    # warm run (fills the caches, loads code), then the timed one
    gen.run(ids, case.n_blocks, case.steps, case.k_unmask)
    torch.cuda.synchronize()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    C = gen.prefill(ids)
    e[1].record()
    for _ in range(case.n_blocks):
        gen.run_block(C, case.steps, case.k_unmask)
        C += case.B
    e[2].record()
    torch.cuda.synchronize()
    t_pre, t_gen = e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])
    n_tok = case.n_blocks * case.B
    n_steps = case.n_blocks * case.steps
    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": n_steps * case.B / (t_gen * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": n_steps, "warmup": n_steps, "ms_per_step": t_gen / n_steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "24-layer spiking MDLM generation: prompt 2048 ids, 8 blocks x 32 "
                               "tokens, 8 denoising steps per block, 4 unmasked per step",
                   "weights": args.weights},
        "generated_tokens_per_s": n_tok / (t_gen * 1e-3),
        "generated_tokens_per_s_with_prefill": n_tok / ((t_pre + t_gen) * 1e-3),
        "prefill_ms": t_pre, "generation_ms": t_gen, "issue": "eager",
    }
    print(json.dumps(out), flush=True)


def bench_ternary_ffn(args):
    """Ternary bitwise-coded FFN (Sec. III-B): integer activations [B][4096]
    -> encode (T=8) -> up product 4096->14336 -> encode its output -> down
    product 14336->4096, for B in {1, 4, 16} and K in {1, 2, 4} quantisation
    levels; 4 rotating weight copies (470 MB) so that weights stream from HBM."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from workloads import synth

    B.load()
    ffn = synth.ffn_sweep_weights()
    d, F = ffn.W_up.shape
    T = 8
    n_copies = 4
    W_up = [torch.from_numpy(ffn.W_up).cuda() for _ in range(n_copies)]
    W_dn = [torch.from_numpy(ffn.W_dn).cuda() for _ in range(n_copies)]
    points = []
    for Bk in (1, 4, 16):
        for Kq in (1, 2, 4):
            a = torch.from_numpy(synth.ternary_activations(synth.stream(1007, 40 + Bk, Kq), Bk, d)).cuda()
            dw, Fw = d // 64, F // 64
            up_p = torch.empty((T, Bk, dw), dtype=torch.int64, device="cuda")
            up_n = torch.empty_like(up_p)
            dn_p = torch.empty((T, Bk, Fw), dtype=torch.int64, device="cuda")
            dn_n = torch.empty_like(dn_p)
            h = torch.empty((Bk, F), dtype=torch.int32, device="cuda")
            y = torch.empty((Bk, d), dtype=torch.int32, device="cuda")
            st = torch.zeros((2, 4), dtype=torch.int64, device="cuda")
            ws = B.workspace(max(B.nmdlm_qbsm_workspace_size(T, Bk, d, F),
                                 B.nmdlm_qbsm_workspace_size(T, Bk, F, d)))

            def chain(c):
                B.nmdlm_ternary_encode(a, Bk, d, Kq, T, up_p, up_n)
                B.nmdlm_qbsm_ternary(up_p, up_n, T, Bk, d, W_up[c], F, F, h, stats=st[0], ws=ws)
                B.nmdlm_ternary_encode(h, Bk, F, Kq, T, dn_p, dn_n)
                B.nmdlm_qbsm_ternary(dn_p, dn_n, T, Bk, F, W_dn[c], d, d, y, stats=st[1], ws=ws)

            def up(c):
                B.nmdlm_qbsm_ternary(up_p, up_n, T, Bk, d, W_up[c], F, F, h, ws=ws)

            def dn(c):
                B.nmdlm_qbsm_ternary(dn_p, dn_n, T, Bk, F, W_dn[c], d, d, y, ws=ws)

            g_chain = _graph(lambda: [chain(c) for c in range(n_copies)])
            t_chain = _time_graph(g_chain, args.reps) / n_copies
            g_up = _graph(lambda: [up(c) for c in range(n_copies)])
            g_dn = _graph(lambda: [dn(c) for c in range(n_copies)])
            t_up = _time_graph(g_up, args.reps) / n_copies
            t_dn = _time_graph(g_dn, args.reps) / n_copies
            k = st.cpu().numpy()
            rec = {"B": Bk, "K": Kq, "T": T, "chain_us": t_chain * 1e3,
                   "tokens_per_s": Bk / (t_chain * 1e-3)}
            for nm, row, t in (("up", k[0], t_up), ("dn", k[1], t_dn)):
                touched = int(row[1] * row[2])
                rec[nm] = {"us": t * 1e3, "skip": 1.0 - row[1] / row[0], "touched_bytes": touched,
                           "GBps": touched / (t * 1e-3) / 1e9}
            points.append(rec)
            del g_chain, g_up, g_dn
    head = [p for p in points if p["B"] == 16 and p["K"] == 2][0]
    best = max((p[m]["GBps"], p, m) for p in points for m in ("up", "dn"))
    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": head["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.reps,
        "warmup": 1, "ms_per_step": head["chain_us"] / 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": "ternary bitwise-coded FFN d=4096->14336->4096, T=8, integer "
                               "activations with Beta(0.5,6) channel scales; value at B=16, K=2",
                   "weight_copies_rotated": n_copies},
        "roofline": {"kernel": "k_qbsm (ternary word product, 2^(t-1)-weighted reconstruction)",
                     "bound": "hbm", "achieved": best[0], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": best[0] / HBM_PEAK_GBPS, "traffic": None,
                     "at": f"B={best[1]['B']} K={best[1]['K']} {best[2]}"},
        "points": points,
    }
    print(json.dumps(out), flush=True)


def bench_e2d2_generate(args):
    """The paper's own model shape (Sec. V-A): encoder-decoder block diffusion
    with 28 encoder and 4 decoder layers, D=512, D_hid=1536, T=8, a 64-token
    prompt, 4 blocks of 4 tokens, one token revealed per step (S=B).  The
    whole generation (prompt encode aside) is captured as one HIP graph."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd.e2d2 import E2D2
    from workloads import synth

    B.load()
    case = synth.e2d2_case()
    m = case.model
    P, nb, Bk = len(case.prompt), case.n_blocks, case.B
    dm = B.DeviceModel.from_mdlm(m, P + nb * Bk, blocked=args.weights == "blocked")
    g = E2D2(dm, case.n_enc, P, nb, Bk)
    g.ctx[:P].copy_(torch.from_numpy(np.asarray(case.prompt, dtype=np.int32)))

    def blocks():
        C = P
        for _ in range(nb):
            g.denoise(C, case.steps, case.k_unmask)
            g.encode(C, Bk)
            C += Bk

    g.encode(0, P)                       # prompt (untimed here, timed below)
    blocks()                             # warm run
    torch.cuda.synchronize()
    ref = g.ctx.clone()
    graph = _graph(blocks)
    t_blocks = _time_graph(graph, args.reps)
    if not torch.equal(g.ctx, ref):
        raise RuntimeError("graph replays of the generation differ from the eager run")
    # phases (eager, HIP events on the stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    ev[0].record()
    g.encode(0, P)
    ev[1].record()
    g.denoise(P, case.steps, case.k_unmask)
    ev[2].record()
    g.encode(P, Bk)
    ev[3].record()
    torch.cuda.synchronize()
    t_prompt, t_den, t_enc = (ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]),
                              ev[2].elapsed_time(ev[3]))
    n_tok = nb * Bk
    n_steps = nb * case.steps
    d, F, V = m.d, m.F, m.V
    layer_bytes = 3 * d * d + d * d + 2 * d * F
    # the paper's Eq. (15) for this shape with every weight row loaded
    # (sigma = 0, an upper bound on the modelled time): encoder layers once
    # per token, decoder layers and head once per token and denoising step
    from paper_2607_24841_amd import perf_model as PM
    T = m.T
    prods = ((d, 3 * d), (d, d), (d, F), (F, d))

    def tl(di, do):
        return PM.token_latency(PM.n_ops(T, di, do, 0.0), PM.n_data(Bk, T, di, do, 0.0, 8),
                                PM.MI355X)[0]
    enc_tl = [tl(di, do) for _ in range(case.n_enc) for di, do in prods]
    dec_tl = [[tl(di, do) for _ in range(m.n_layers - case.n_enc) for di, do in prods] + [tl(d, V)]
              for _ in range(case.steps)]
    model_tt = PM.e2e_throughput(enc_tl, dec_tl)
    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": n_tok / (t_blocks * 1e-3), "unit": "generated tokens/s (encoder included)",
        "n_gpus": 1, "steps": n_steps, "warmup": n_steps, "ms_per_step": t_den / case.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "encoder-decoder spiking MDLM in the paper's shape: 28 encoder + 4 "
                               "decoder layers, d=512, 8 heads x 64, FFN 1536, T=8, vocab 32000; "
                               "prompt 64 ids, 4 blocks x 4 tokens, 4 steps per block, 1 token "
                               "unmasked per step",
                   "issue": "hip_graph (generation), eager (phases)"},
        "blocks_ms": t_blocks, "prompt_encode_ms": t_prompt,
        "decoder_step_us": 1e3 * t_den / case.steps,
        "block_encode_us": 1e3 * t_enc,
        "paper_model_MI355X_sigma0_tokens_per_s": model_tt,
        "weights_bytes": {"encoder": case.n_enc * layer_bytes,
                          "decoder": (m.n_layers - case.n_enc) * layer_bytes, "head": d * V},
    }
    print(json.dumps(out), flush=True)


def product_input_sparsity(B, torch, dl, L, case, xb, y_step):
    """Fraction of zero input spikes of the step's four products (the paper's
    sigma, measured per linear layer): the step is replayed, untimed, through
    the single-call C ABI (products with currents out, attention with spikes
    out, IF neurons, activation table) after the step itself has written this
    block's keys and values into the caches; its output must equal the step's."""
    import numpy as np
    T, M, C_ctx = case.T, case.M, case.C
    d, F, H = L.d, L.F, L.H
    dw, Fw = d // 64, (F + 63) // 64
    th = L.theta
    i64 = dict(dtype=torch.int64, device="cuda")
    i32 = dict(dtype=torch.int32, device="cuda")
    ws = B.workspace(max(B.nmdlm_qbsm_workspace_size(T, M, d, 3 * d),
                         B.nmdlm_qbsm_workspace_size(T, M, d, F),
                         B.nmdlm_qbsm_workspace_size(T, M, F, d),
                         B.nmdlm_bbm_attn_workspace_size(T, M, H, d // H)))
    Q = torch.empty((T, M, dw), **i64)
    B.nmdlm_qbsm(xb, T, M, d, dl.w_qkv, d, 3 * d, theta=th["q"], s_out=Q, ws=ws)
    A = torch.empty((T, M, dw), **i64)
    B.nmdlm_bbm_attn(Q, dl.k_cache, dl.vt_cache, dl.k_cache.shape[1], T, M, C_ctx, H, d // H,
                     dl.lut_att, theta_a=th["a"], s_out=A, ws=ws)
    cur = torch.empty((T, M, max(d, F)), **i32)
    X1 = torch.empty((T, M, dw), **i64)
    c_o = cur[..., :d].contiguous()
    B.nmdlm_qbsm(A, T, M, d, dl.w_o, d, d, cur_out=c_o, ws=ws)
    B.nmdlm_if_neuron(c_o, T, M, d, theta=th["o"], resid=xb, s_out=X1)
    c_up = torch.empty((T, M, F), **i32)
    B.nmdlm_qbsm(X1, T, M, d, dl.w_up, F, F, cur_out=c_up, ws=ws)
    g8 = torch.empty((T, M, F), dtype=torch.uint8, device="cuda")
    B.nmdlm_qnl_lut(c_up, T * M * F, L.s_up, B.NMDLM_QNL_S8, dl.lut_act, g8)
    Hs = torch.empty((T, M, Fw), **i64)
    B.nmdlm_if_neuron(g8.view(torch.int8).to(torch.int32), T, M, F, theta=th["up"], s_out=Hs)
    c_dn = torch.empty((T, M, d), **i32)
    B.nmdlm_qbsm(Hs, T, M, F, dl.w_dn, d, d, cur_out=c_dn, ws=ws)
    Y = torch.empty((T, M, dw), **i64)
    B.nmdlm_if_neuron(c_dn, T, M, d, theta=th["dn"], resid=X1, s_out=Y)
    torch.cuda.synchronize()
    if not torch.equal(Y, y_step):
        raise RuntimeError("single-call replay of the block step differs from the step")

    def zero_frac(t, k):
        ones = int(np.unpackbits(t.cpu().numpy().view(np.uint8)).sum())
        return 1.0 - ones / float(T * M * k)

    return [zero_frac(xb, d), zero_frac(A, d), zero_frac(X1, d), zero_frac(Hs, F)]


def bench_block(args):
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from workloads import synth

    B.load()
    dev = "cuda"
    import ctypes as C
    case = synth.block_case(seed=args.seed)
    L = case.layer
    T, C_ctx, M, d, H, F = case.T, case.C, case.M, L.d, L.H, L.F

    # --- device state (untimed): layer copies, prefilled caches ----------------
    dms = [B.DeviceModel([L], T, C_ctx + M, d, H, F, blocked=args.weights == "blocked")
           for _ in range(args.copies)]
    nb = max(B.nmdlm_block_step_workspace_size(dms[0], C_ctx, B.NMDLM_NO_HEAD),
             B.nmdlm_block_step_workspace_size(dms[0], M, B.NMDLM_NO_HEAD))
    ws = B.workspace(nb)
    xc = B.to_dev_bits(synth.pack_bits(case.X_ctx))
    for dm in dms:
        B.nmdlm_block_step(dm, B.step_io(C_ctx, 0, flags=B.NMDLM_NO_HEAD, x_in=xc), ws)
    xb = B.to_dev_bits(synth.pack_bits(case.X_blk))
    y = torch.zeros((T, M, d // 64), dtype=torch.int64, device=dev)
    stats = torch.zeros((4, 4), dtype=torch.int64, device=dev)
    io = B.step_io(M, C_ctx, flags=B.NMDLM_NO_HEAD | args.flags, x_in=xb, y_out=y, stats=stats)
    torch.cuda.synchronize()

    def eager_steps(i0, n):
        for i in range(i0, i0 + n):
            B.nmdlm_block_step(dms[i % args.copies], io, ws)

    graphs = {}

    def graph_for(n):
        if n not in graphs:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                eager_steps(0, n)          # warm the path on the capture stream
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                eager_steps(0, n)
            torch.cuda.synchronize()
            graphs[n] = g
        return graphs[n]

    def run(n):
        if args.eager:
            eager_steps(0, n)
            return
        full, rest = divmod(n, args.copies)
        if full:
            g = graph_for(args.copies)
            for _ in range(full):
                g.replay()
        if rest:
            graph_for(rest).replay()

    # --- warmup + timed region: every graph the timed region replays is
    #     captured before it (runs of args.copies steps and the remainder)
    if not args.eager:
        for n in (args.copies, args.steps % args.copies, args.warmup % args.copies):
            if n:
                graph_for(n)
    run(args.warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = 1e3 * dt / args.steps
    # distribution over graph replays (each a run of args.copies steps),
    # after the timed region
    pct = None
    if not args.eager:
        g = graph_for(args.copies)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        per = []
        for _ in range(20):
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            per.append(1e3 * e0.elapsed_time(e1) / args.copies)
        pct = {"p10": float(np.percentile(per, 10)), "p50": float(np.percentile(per, 50)),
               "p90": float(np.percentile(per, 90)), "replays": len(per),
               "steps_per_replay": args.copies}

    st = stats.cpu().numpy()
    k_total, k_active, n_col = st[:, 0], st[:, 1], st[:, 2]
    w_touched = int((k_active * n_col).sum())
    w_dense = int((k_total * n_col).sum())
    skip = 1.0 - w_touched / w_dense

    # --- product kernel timed per launch: the library stamps a HIP event
    #     pair with the start and end of every product kernel (from its
    #     dispatch).  Events cannot be graph nodes here, so the same steps are
    #     issued directly behind a spin kernel: the queue fills while it spins
    #     and the kernels then run back to back, as in the timed region
    n_ev = 2 * 4
    ev = B.HipEvents(n_ev * args.copies)
    ptr_size = C.sizeof(C.c_void_p)
    sub = [(C.c_void_p * n_ev).from_address(C.addressof(ev.arr) + i * n_ev * ptr_size)
           for i in range(args.copies)]
    pios = [B.step_io(M, C_ctx, flags=B.NMDLM_NO_HEAD | args.flags, x_in=xb, y_out=y,
                      stats=stats, prof_events=sub[i]) for i in range(args.copies)]
    for i in range(args.copies):                 # warm the event path
        B.nmdlm_block_step(dms[i], pios[i], ws)
    torch.cuda.synchronize()
    torch.cuda._sleep(50_000_000)
    for i in range(args.copies):
        B.nmdlm_block_step(dms[i], pios[i], ws)
    torch.cuda.synchronize()
    timing_issue = "direct issue behind a spin kernel (queue full)"
    dur = []
    nbytes = []
    for i in range(args.copies):
        for p in range(4):
            dur.append(ev.elapsed_ms(i * n_ev + 2 * p, i * n_ev + 2 * p + 1))
            nbytes.append(product_bytes(int(k_total[p]), int(k_active[p]), int(n_col[p]), T, M))
    ev.close()
    avg_ms = float(np.mean(dur))
    achieved = sum(nbytes) / (sum(dur) * 1e-3) / 1e9
    traffic = product_traffic("block")
    # the paper's analytic model (Eqs. (12)-(14)) of the step's four products,
    # from their measured union fractions, beside their measured kernel times
    from paper_2607_24841_amd import perf_model
    dims = (("qkv", d, 3 * d), ("o", d, d), ("up", d, F), ("down", F, d))
    sig = product_input_sparsity(B, torch, dms[0].layers[0], L, case, xb, y)
    reports = [perf_model.layer_report(nm, M, T, di, do, float(k_active[p]) / float(k_total[p]),
                                       b_w=8, measured_us=1e3 * float(np.mean(dur[p::4])),
                                       sigma=sig[p])
               for p, (nm, di, do) in enumerate(dims)]
    paper_model = perf_model.block_report(reports, measured_step_us=1e3 * ms_per_step)
    stream = stream_copy_gbps(torch)

    out = {
        "metric": "block-denoise tokens/s; weight-skip fraction; achieved HBM GB/s on touched bytes",
        "value": M / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {
            "workload": "one spiking transformer block at a single denoising step: d=1024, "
                        "16 heads x 64, FFN 4096, T=4, block of 16 masked tokens over 512 "
                        "context tokens, input spike rate 0.10, int8 weights",
            "block_tokens": M, "context_tokens": C_ctx, "timesteps": T,
            "layer_copies_rotated": args.copies, "issue": "eager" if args.eager else "hip_graph",
            "weights": args.weights,
        },
        "step_us_percentiles": pct,
        "weight_skip_fraction": skip,
        "touched_weight_bytes_per_step": w_touched,
        "touched_weight_GBps": w_touched / (ms_per_step * 1e-3) / 1e9,
        "roofline": {
            "kernel": "k_qbsm (int8 MFMA spike product with fused IF epilogue)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "stream_copy_GBps": stream,
            "frac_of_stream_copy": achieved / stream,
            "avg_launch_ms": avg_ms,
            "launches_timed": len(dur),
            "timing_issue": timing_issue,
        },
        "paper_model": paper_model,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    print(json.dumps(out), flush=True)


BATCH_SEQS = (1, 2, 4, 8, 16, 32, 64, 128)


def bench_block_batch(args):
    """The one-block step over several sequences per call (each sequence its
    own seeded context and block inputs, one shared layer)."""
    import numpy as np
    import torch

    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd import perf_model
    from workloads import synth

    B.load()
    nmax = max(BATCH_SEQS)
    base = synth.block_case(seed=args.seed)
    L = base.layer
    T, C_ctx, M, d, H, F = base.T, base.C, base.M, L.d, L.H, L.F
    inputs = [synth.block_inputs(args.seed + 1000 * s, C_ctx, M, d, T) for s in range(nmax)]
    dms = [B.DeviceModel([L], T, C_ctx + M, d, H, F, max_seq=nmax, blocked=args.weights == "blocked")
           for _ in range(args.copies)]
    nb = max(B.nmdlm_block_step_workspace_size(dms[0], nmax * C_ctx, B.NMDLM_NO_HEAD),
             B.nmdlm_block_step_workspace_size(dms[0], nmax * M, B.NMDLM_NO_HEAD))
    ws = B.workspace(nb)
    xc = B.to_dev_bits(synth.pack_bits(np.concatenate([x for x, _ in inputs], axis=1)))
    B.nmdlm_block_step(dms[0], B.step_io(C_ctx, 0, flags=B.NMDLM_NO_HEAD, x_in=xc, n_seq=nmax), ws)
    for dm in dms[1:]:                     # identical layers: copy the prefilled caches
        dm.layers[0].k_seq.copy_(dms[0].layers[0].k_seq)
        dm.layers[0].vt_seq.copy_(dms[0].layers[0].vt_seq)
    del xc
    xb_all = np.concatenate([x for _, x in inputs], axis=1)        # [T][nmax M][d]
    torch.cuda.synchronize()
    dims = (("qkv", d, 3 * d), ("o", d, d), ("up", d, F), ("down", F, d))
    points = []
    for n in BATCH_SEQS:
        xb = B.to_dev_bits(synth.pack_bits(np.ascontiguousarray(xb_all[:, :n * M])))
        y = torch.zeros((T, n * M, d // 64), dtype=torch.int64, device="cuda")
        stats = torch.zeros((4, 4), dtype=torch.int64, device="cuda")
        io = B.step_io(M, C_ctx, flags=B.NMDLM_NO_HEAD | args.flags, x_in=xb, y_out=y,
                       stats=stats, n_seq=n)

        def steps():
            for dm in dms:
                B.nmdlm_block_step(dm, io, ws)
        g = _graph(steps)
        ms = _time_graph(g, args.reps) / len(dms)
        del g
        st = stats.cpu().numpy()
        k_total, k_active, n_col = st[:, 0], st[:, 1], st[:, 2]
        touched = int((k_active * n_col).sum())
        reps = [perf_model.layer_report(nm, n * M, T, di, do, float(k_active[p]) / float(k_total[p]),
                                        b_w=8)
                for p, (nm, di, do) in enumerate(dims)]
        model = perf_model.block_report(reps)
        points.append({
            "n_seq": n, "tokens_per_step": n * M, "ms_per_step": ms,
            "tokens_per_s": n * M / (ms * 1e-3),
            "union_frac": {nm: float(k_active[p]) / float(k_total[p])
                           for p, (nm, _, _) in enumerate(dims)},
            "touched_weight_bytes_per_step": touched,
            "touched_weight_bytes_per_token": touched / (n * M),
            "touched_weight_GBps": touched / (ms * 1e-3) / 1e9,
            "model_us_per_step_MI355X": model["MI355X_us_per_block"],
        })
        print(json.dumps({"progress": "block-batch", **points[-1]}), file=sys.stderr, flush=True)
    best = points[-1]
    out = {
        "metric": "batched block-denoise tokens/s",
        "value": best["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.reps * len(dms),
        "warmup": 1,
        "ms_per_step": best["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {
            "workload": f"one spiking transformer block at a single denoising step over {nmax} "
                        "sequences at once: d=1024, 16 heads x 64, FFN 4096, T=4, per sequence a "
                        "block of 16 masked tokens over 512 context tokens, input spike rate "
                        "0.10, int8 weights",
            "layer_copies_rotated": len(dms), "issue": "hip_graph", "weights": args.weights,
        },
        "points": points,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
