"""GPU parity of block steps over several sequences at once: every sequence
of a batched nmdlm_block_step must equal an independent oracle run of that
sequence alone (outputs, K/V caches, head, confidence, unmasking,
generation); the weight-skip statistics are those of the batch's union."""
import numpy as np
import pytest

from oracle import nmdlm_oracle as O
from workloads import synth

from ._gpu import assert_same, need_gpu

pytestmark = pytest.mark.gpu


def _seq_caches_to_host(dm, s, d, J):
    from paper_2607_24841_amd import binding as B
    ks, vs = [], []
    for l in dm.layers:
        ks.append(synth.unpack_bits(B.from_dev_bits(l.k_seq[s]), d)[:, :J])
        words = np.ascontiguousarray(B.from_dev_bits(l.vt_seq[s]).transpose(0, 2, 1))
        vs.append(synth.unpack_bits(words, dm.cache_cap).transpose(0, 2, 1)[:, :J])
    return ks, vs


def _cases(n, C, M, d, H, F, seed, T=4):
    """n sequences sharing one layer's weights, each with its own context and
    block inputs (seeded per sequence)."""
    base = synth.block_case(seed=seed, C=C, M=M, d=d, H=H, F=F, T=T)
    out = []
    for s in range(n):
        xc, xb = synth.block_inputs(seed + 100 * (s + 1), C, M, d, base.T)
        out.append(synth.BlockCase(base.T, C, M, base.layer, xc, xb))
    return out


@pytest.mark.parametrize("n,C,M,d,H,F,flags,T", [
    (3, 60, 8, 128, 2, 256, 0, 4),          # block positions 60..67 cross a value-cache word
    (2, 64, 16, 256, 4, 512, 0, 4),         # whole-byte value-cache stores
    (4, 40, 12, 128, 2, 256, 2 << 16, 4),   # forced 2-row tiles: 8-token row blocks straddle the
                                            # 12-token sequences (QKV falls back to 4-token blocks)
    (5, 32, 4, 128, 2, 256, 1, 4),          # dense product
    (4, 512, 16, 1024, 16, 4096, 0, 4),     # full-size layer, four sequences
    (16, 64, 4, 1024, 16, 4096, 0, 4),      # 16 sequences: attention beyond one round of the chip
    (3, 62, 6, 128, 2, 256, 0, 8),          # T = 8: 2-token row blocks, positions cross a word
    (3, 35, 5, 128, 2, 256, 0, 3),          # T = 3: 5-token row blocks (16 // 3)
    (2, 48, 16, 256, 2, 512, 0, 4),         # heads of 128 channels
    (3, 60, 8, 128, 2, 256, 0x4, 4),        # the fused-attention flag (single-sequence) is ignored
    (128, 40, 16, 128, 2, 256, 0, 4),       # 128 sequences: attention at 4 waves per workgroup
], ids=["straddle", "bytes", "rt2-ragged", "dense", "full-4seq", "16seq", "T8", "T3", "dh128",
        "attn-fused-flag", "128seq"])
def test_batched_block_step_matches_independent_sequences(n, C, M, d, H, F, flags, T):
    _batched_matches_independent(n, C, M, d, H, F, flags, T)


@pytest.mark.parametrize("n,C,M,d,H,F,flags,T", [
    (4, 512, 16, 1024, 16, 4096, 0, 4),     # full-size layer, four sequences
    (128, 40, 16, 128, 2, 256, 0, 4),       # 128 sequences: 8192 rows per product
    (3, 62, 6, 128, 2, 256, 6 << 20, 8),    # every word from the copies, T = 8
    (128, 40, 16, 128, 2, 256, (7 << 20) | (4 << 16), 4),  # wide tiles, 8192 rows
    (8, 64, 32, 192, 3, 320, (7 << 20) | (4 << 16), 2),    # wide tiles, T = 2 (32-token blocks)
], ids=["full-4seq", "128seq", "T8-forced", "128seq-wide", "T2-wide"])
def test_batched_step_with_blocked_weights(n, C, M, d, H, F, flags, T):
    _batched_matches_independent(n, C, M, d, H, F, flags, T, blocked=True)


def _batched_matches_independent(n, C, M, d, H, F, flags, T, blocked=False):
    torch, B = need_gpu()
    cases = _cases(n, C, M, d, H, F, seed=71, T=T)
    L, T = cases[0].layer, cases[0].T
    dm = B.DeviceModel([L], T, C + M, d, H, F, max_seq=n, blocked=blocked)
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, n * C, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, n * M, B.NMDLM_NO_HEAD)))
    # batched prefill of the n contexts, then the batched block step
    xc = np.concatenate([c.X_ctx for c in cases], axis=1)            # [T][n C][d]
    B.nmdlm_block_step(dm, B.step_io(C, 0, flags=B.NMDLM_NO_HEAD | flags, n_seq=n,
                                     x_in=B.to_dev_bits(synth.pack_bits(xc))), ws)
    xb = np.concatenate([c.X_blk for c in cases], axis=1)            # [T][n M][d]
    y = torch.zeros((T, n * M, d // 64), dtype=torch.int64, device="cuda")
    stats = torch.zeros((4, 4), dtype=torch.int64, device="cuda")
    B.nmdlm_block_step(dm, B.step_io(M, C, flags=B.NMDLM_NO_HEAD | flags, n_seq=n, y_out=y,
                                     stats=stats, x_in=B.to_dev_bits(synth.pack_bits(xb))), ws)
    torch.cuda.synchronize()
    Y = synth.unpack_bits(B.from_dev_bits(y), d)
    st = stats.cpu().numpy()
    unions = {}
    for s, c in enumerate(cases):
        kc, vc = O.new_caches(1, T, C + M, d)
        O.prefill(c.X_ctx, [L], kc, vc)
        tr = O.layer_forward(c.X_blk, L, kc[0], vc[0], C)
        assert_same(Y[:, s * M:(s + 1) * M], tr.Y, f"Y of sequence {s}")
        ks, vs = _seq_caches_to_host(dm, s, d, C + M)
        assert_same(ks[0], kc[0], f"K cache of sequence {s}")
        assert_same(vs[0], vc[0], f"V cache of sequence {s}")
        for key, u in tr.unions.items():
            unions[key] = u if key not in unions else (unions[key] | u)
    for i, key in enumerate(("qkv", "o", "up", "dn")):
        K = unions[key].size
        assert st[i, 0] == K
        assert st[i, 1] == (K if flags & 1 else int(unions[key].sum())), key


def test_batched_mdlm_step_with_head():
    torch, B = need_gpu()
    m = synth.make_mdlm(33, 2, d=128, H=2, F=256, V=64, T=4, max_pos=64)
    emb = O.unpack_model_emb(m)
    n, P, M, k = 3, 12, 8, 3
    prompts = [synth.random_tokens(40 + s, P, m.V) for s in range(n)]
    tok0 = synth.random_tokens(60, n * M, m.V).astype(np.int32).reshape(n, M)
    msk0 = synth.bernoulli(synth.stream(61, 0), 0.7, (n, M))
    msk0[2, :] = True                      # one sequence fully masked
    msk0[1, :] = False
    msk0[1, 3] = True                      # one with a single masked token (< k)
    tok0[msk0] = 0
    refs = []
    for s in range(n):
        kc, vc = O.new_caches(m.n_layers, m.T, P + M, m.d)
        O.prefill(O.block_input(prompts[s], np.arange(P), emb, m.pos_ch), m.layers, kc, vc)
        refs.append(O.block_step(m, emb, tok0[s], msk0[s], P, P, kc, vc, k))
    dm = B.DeviceModel.from_mdlm(m, P + M, max_seq=n)
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, n * P, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, n * M, 0)))
    pr = torch.from_numpy(np.concatenate(prompts).astype(np.int32)).cuda()
    B.nmdlm_block_step(dm, B.step_io(P, 0, flags=B.NMDLM_NO_HEAD, tokens=pr, n_seq=n,
                                     masked=torch.zeros(n * P, dtype=torch.uint8, device="cuda")), ws)
    tok = torch.from_numpy(tok0.reshape(-1)).cuda()
    msk = torch.from_numpy(msk0.reshape(-1).astype(np.uint8)).cuda()
    logits = torch.empty((n * M, m.V), dtype=torch.float32, device="cuda")
    pred = torch.empty(n * M, dtype=torch.int32, device="cuda")
    conf = torch.empty(n * M, dtype=torch.float64, device="cuda")
    chosen = torch.empty(n * k, dtype=torch.int32, device="cuda")
    B.nmdlm_block_step(dm, B.step_io(M, P, pos0=P, tokens=tok, masked=msk, k_unmask=k, n_seq=n,
                                     logits=logits, pred=pred, conf=conf, unmasked_pos=chosen), ws)
    torch.cuda.synchronize()
    lg, pd, cf = logits.cpu().numpy(), pred.cpu().numpy(), conf.cpu().numpy()
    ch, tk = chosen.cpu().numpy().reshape(n, k), tok.cpu().numpy().reshape(n, M)
    mk = msk.cpu().numpy().reshape(n, M).astype(bool)
    for s, ref in enumerate(refs):
        r = slice(s * M, (s + 1) * M)
        assert_same(lg[r], ref.logits, f"logits of sequence {s}")
        assert_same(pd[r], ref.pred, f"pred of sequence {s}")
        assert np.allclose(cf[r], ref.conf, rtol=1e-12, atol=0)
        nc = len(ref.chosen)              # fewer masked than k: the rest are -1
        assert np.array_equal(ch[s][:nc], ref.chosen) and (ch[s][nc:] == -1).all(), s
        assert np.array_equal(tk[s], ref.tokens), s
        assert np.array_equal(mk[s], ref.masked), s


def test_batched_generation_matches_oracle():
    need_gpu()
    from paper_2607_24841_amd import binding as B
    from paper_2607_24841_amd.generate import generate_batch
    m = synth.make_mdlm(34, 2, d=128, H=2, F=256, V=64, T=4, max_pos=64)
    n, P = 4, 20
    prompts = np.stack([synth.random_tokens(50 + s, P, m.V) for s in range(n)])
    dm = B.DeviceModel.from_mdlm(m, P + 24, max_seq=n)
    ids, log = generate_batch(dm, prompts, n_blocks=3, block=8, steps=4, k_unmask=2)
    for s in range(n):
        ids_ref, log_ref = O.generate(m, prompts[s], n_blocks=3, B=8, steps=4, k_unmask=2)
        assert_same(ids[s], ids_ref, f"ids of sequence {s}")
        assert all(np.array_equal(a[s], b) for a, b in zip(log, log_ref)), s


def test_batched_step_graph_replays_match_eager():
    # the batched step captured in a HIP graph: every replay equals the eager
    # step (with eager work and synchronisations between the replays)
    torch, B = need_gpu()
    n, C, M, d, H, F = 3, 60, 8, 128, 2, 256
    cases = _cases(n, C, M, d, H, F, seed=91)
    L, T = cases[0].layer, cases[0].T
    dm = B.DeviceModel([L], T, C + M, d, H, F, max_seq=n)
    ws = B.workspace(max(B.nmdlm_block_step_workspace_size(dm, n * C, B.NMDLM_NO_HEAD),
                         B.nmdlm_block_step_workspace_size(dm, n * M, B.NMDLM_NO_HEAD)))
    xc = np.concatenate([c.X_ctx for c in cases], axis=1)
    B.nmdlm_block_step(dm, B.step_io(C, 0, flags=B.NMDLM_NO_HEAD, n_seq=n,
                                     x_in=B.to_dev_bits(synth.pack_bits(xc))), ws)
    xb = B.to_dev_bits(synth.pack_bits(np.concatenate([c.X_blk for c in cases], axis=1)))
    y = torch.zeros((T, n * M, d // 64), dtype=torch.int64, device="cuda")
    io = B.step_io(M, C, flags=B.NMDLM_NO_HEAD, n_seq=n, x_in=xb, y_out=y)
    B.nmdlm_block_step(dm, io, ws)
    torch.cuda.synchronize()
    eager = y.clone()
    Y = synth.unpack_bits(B.from_dev_bits(eager), d)
    for s, c in enumerate(cases):
        kc, vc = O.new_caches(1, T, C + M, d)
        O.prefill(c.X_ctx, [L], kc, vc)
        assert_same(Y[:, s * M:(s + 1) * M], O.layer_forward(c.X_blk, L, kc[0], vc[0], C).Y,
                    f"eager Y of sequence {s}")
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        B.nmdlm_block_step(dm, io, ws)
    torch.cuda.current_stream().wait_stream(st)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        B.nmdlm_block_step(dm, io, ws)
    for r in range(4):
        y.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, eager), f"replay {r} differs from the eager step"
