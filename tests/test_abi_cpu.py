"""The C ABI on the host: the library loads, exports every function the
header declares, sizes workspaces and rejects bad arguments before any HIP
call (so these run without a GPU)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nmdlm.h")

torch = pytest.importorskip("torch")
from paper_2607_24841_amd import binding as B  # noqa: E402


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(nmdlm_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libnmdlm.so not built")
    return B.load()


def test_exports_every_declared_function(lib):
    names = _declared()
    assert set(B.EXPORTS) <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.nmdlm_abi_version() == 5
    assert lib.nmdlm_status_string(0) == b"ok"
    assert lib.nmdlm_status_string(3).startswith(b"workspace")


def test_single_hip_runtime(lib):
    assert len(B._hip_runtimes_mapped()) <= 1


def test_workspace_sizes(lib):
    s1 = lib.nmdlm_qbsm_workspace_size(4, 8, 512, 512)
    s2 = lib.nmdlm_qbsm_workspace_size(4, 64, 14336, 4096)
    assert 0 < s1 < s2 and s1 % 256 == 0
    assert lib.nmdlm_qbsm_workspace_size(0, 8, 512, 512) == 0
    assert lib.nmdlm_qbsm_workspace_size(4, 8, 70000, 512) == 0
    assert lib.nmdlm_bbm_attn_workspace_size(4, 16, 16, 64) == 4 * 16 * 1024 * 4


FAKE = 1 << 40   # never dereferenced: every call below fails validation first


def _qbsm(lib, **kw):
    a = dict(s_in=FAKE, T=4, M=8, K=512, W=FAKE, N=512, ldw=512, bias=None, cur=FAKE,
             theta=256, theta_vec=None, s_out=None, stats=None, flags=0, ws=FAKE, ws_bytes=1 << 30,
             stream=None)
    a.update(kw)
    return lib.nmdlm_qbsm(a["s_in"], a["T"], a["M"], a["K"], a["W"], a["N"], a["ldw"], a["bias"],
                          a["cur"], a["theta"], a["theta_vec"], a["s_out"], a["stats"], a["flags"],
                          a["ws"], a["ws_bytes"], a["stream"])


def test_qbsm_argument_errors(lib):
    assert _qbsm(lib, s_in=None) == B.NMDLM_ERR_INVALID_ARG
    assert _qbsm(lib, T=0) == B.NMDLM_ERR_INVALID_ARG
    assert _qbsm(lib, M=-1) == B.NMDLM_ERR_INVALID_ARG
    assert _qbsm(lib, M=0) == B.NMDLM_ERR_INVALID_ARG            # an empty block is rejected
    assert _qbsm(lib, T=9) == B.NMDLM_ERR_UNSUPPORTED
    assert _qbsm(lib, K=70000) == B.NMDLM_ERR_UNSUPPORTED
    assert _qbsm(lib, ldw=500) == B.NMDLM_ERR_INVALID_ARG          # < N
    assert _qbsm(lib, ldw=520) == B.NMDLM_ERR_INVALID_ARG          # not a multiple of 16
    assert _qbsm(lib, W=FAKE + 4) == B.NMDLM_ERR_INVALID_ARG       # misaligned weights
    assert _qbsm(lib, cur=None) == B.NMDLM_ERR_INVALID_ARG         # no output
    assert _qbsm(lib, cur=None, s_out=FAKE, theta=0) == B.NMDLM_ERR_INVALID_ARG
    assert _qbsm(lib, ws=None) == B.NMDLM_ERR_WORKSPACE
    assert _qbsm(lib, ws_bytes=16) == B.NMDLM_ERR_WORKSPACE
    assert _qbsm(lib, ws=FAKE + 8) == B.NMDLM_ERR_WORKSPACE        # misaligned workspace
    assert _qbsm(lib, K=40000, N=60000, ldw=60000) == B.NMDLM_ERR_INVALID_ARG  # K*ldw >= 2^31


def test_other_argument_errors(lib):
    assert lib.nmdlm_if_neuron(None, 4, 1, 1, 256, None, None, None, FAKE, None) == 1
    assert lib.nmdlm_if_neuron(FAKE, 4, 1, 1, 0, None, None, None, FAKE, None) == 1
    assert lib.nmdlm_qnl_lut(FAKE, 10, 32, 0, FAKE, FAKE, None) == 1
    assert lib.nmdlm_qnl_lut(FAKE, 10, 3, 7, FAKE, FAKE, None) == 1
    assert lib.nmdlm_qnl_lut(FAKE, -1, 3, 0, FAKE, FAKE, None) == 1
    assert lib.nmdlm_qnl_lut(None, 0, 3, 0, FAKE, None, None) == 0   # empty input: nothing to do
    a = lambda **k: lib.nmdlm_bbm_attn(FAKE, FAKE, FAKE, k.get("cap", 576), 4, k.get("M", 16),
                                       k.get("C", 512), 16, k.get("dh", 64), FAKE, FAKE, 256, None,
                                       None, 0, None)
    assert a(dh=96) == B.NMDLM_ERR_UNSUPPORTED
    assert a(cap=512) == B.NMDLM_ERR_INVALID_ARG                   # C + M > cap
    assert a(cap=600) == B.NMDLM_ERR_INVALID_ARG                   # cap not a multiple of 64
    assert lib.nmdlm_bbm_attn(FAKE, FAKE, FAKE, 576, 4, 16, 512, 16, 64, FAKE, None, 256, None,
                              None, 0, None) == 1                  # no output requested
    assert a(M=(1 << 17) + 1) == B.NMDLM_ERR_UNSUPPORTED           # T*M beyond 2^19
    big = (1 << 23) + 64                                            # keys beyond NMDLM_MAX_KEYS
    assert a(C=(1 << 23) - 15, cap=big) == B.NMDLM_ERR_UNSUPPORTED
    assert a(C=0, cap=64 * (2 ** 31)) == B.NMDLM_ERR_UNSUPPORTED   # cap/64 beyond INT_MAX
    assert lib.nmdlm_bbm_attn(FAKE, FAKE, FAKE, 576, 4, 16, 512, 1025, 64, FAKE, FAKE, 256,
                              None, None, 0, None) == B.NMDLM_ERR_UNSUPPORTED   # d > 65536
    # IF grid beyond 2^32 threads, and T beyond 8192
    assert lib.nmdlm_if_neuron(FAKE, 4, 1 << 20, 64 * 65, 256, None, None, None, FAKE,
                               None) == B.NMDLM_ERR_UNSUPPORTED
    assert lib.nmdlm_if_neuron(FAKE, 8193, 1, 1, 256, None, None, None, FAKE,
                               None) == B.NMDLM_ERR_UNSUPPORTED
    assert lib.nmdlm_workspace_clear(FAKE, 17, None) == 1


def test_block_step_argument_errors(lib):
    L = B.Layer(FAKE, FAKE, FAKE, FAKE, 200, 200, 200, 200, 200, 200, 200, 4, FAKE, FAKE, FAKE, FAKE)
    layers = (B.Layer * 1)(L)
    m = B.Model(1, 1024, 16, 4096, 32000, 4, 576, 0, layers, None, None, None, None)
    io = B.step_io(16, 512, flags=B.NMDLM_NO_HEAD, x_in=FAKE)
    ws_need = lib.nmdlm_block_step_workspace_size(C.byref(m), 16, B.NMDLM_NO_HEAD)
    assert ws_need > 0
    call = lambda mm, ii, ws=FAKE, nb=ws_need: lib.nmdlm_block_step(C.byref(mm), C.byref(ii), ws, nb, None)
    assert lib.nmdlm_block_step(None, C.byref(io), FAKE, ws_need, None) == 1
    assert call(m, io, nb=ws_need - 256) == B.NMDLM_ERR_WORKSPACE
    bad = B.step_io(16, 600, flags=B.NMDLM_NO_HEAD, x_in=FAKE)      # C + M > cache_cap
    assert call(m, bad) == 1
    # more attention keys than NMDLM_MAX_KEYS, with a cache that holds them
    mk = B.Model(1, 1024, 16, 4096, 32000, 4, (1 << 23) + 64, 0, layers, None, None, None, None)
    nbk = lib.nmdlm_block_step_workspace_size(C.byref(mk), 16, B.NMDLM_NO_HEAD)
    many = B.step_io(16, (1 << 23) - 15, flags=B.NMDLM_NO_HEAD, x_in=FAKE)
    assert lib.nmdlm_block_step(C.byref(mk), C.byref(many), FAKE, nbk, None) == B.NMDLM_ERR_UNSUPPORTED
    L2 = B.Layer(FAKE, FAKE, FAKE, FAKE, 200, 0, 200, 200, 200, 200, 200, 4, FAKE, FAKE, FAKE, FAKE)
    m2 = B.Model(1, 1024, 16, 4096, 32000, 4, 576, 0, (B.Layer * 1)(L2), None, None, None, None)
    assert call(m2, io) == 1                                        # threshold 0
    m3 = B.Model(1, 1024, 12, 4096, 32000, 4, 576, 0, layers, None, None, None, None)
    assert call(m3, io) == B.NMDLM_ERR_UNSUPPORTED                  # d/H not a multiple of 64
    head_io = B.step_io(16, 512, flags=0, x_in=FAKE)                # head without weights
    assert call(m, head_io) == 1
    no_in = B.step_io(16, 512, flags=B.NMDLM_NO_HEAD)               # no input and no tables
    assert call(m, no_in) == 1
    # a step with the head takes at most NMDLM_MAX_HEAD_M block tokens
    mh = B.Model(1, 1024, 16, 4096, 32000, 4, 8192, 0, layers, None, None, FAKE, FAKE)
    big = B.step_io(4097, 0, flags=0, x_in=FAKE, tokens=FAKE, masked=FAKE, k_unmask=4)
    nb = lib.nmdlm_block_step_workspace_size(C.byref(mh), 4097, 0)
    assert nb > 0 and call(mh, big, nb=nb) == B.NMDLM_ERR_UNSUPPORTED
    # blocked weight copies must be 16-byte aligned
    Lb = B.Layer(FAKE, FAKE, FAKE, FAKE, 200, 200, 200, 200, 200, 200, 200, 4, FAKE, FAKE, FAKE,
                 FAKE, FAKE, FAKE + 8, None, None)
    mb = B.Model(1, 1024, 16, 4096, 32000, 4, 576, 0, (B.Layer * 1)(Lb), None, None, None, None)
    assert call(mb, io) == B.NMDLM_ERR_INVALID_ARG
    mhb = B.Model(1, 1024, 16, 4096, 32000, 4, 8192, 0, layers, None, None, FAKE, FAKE, 1, FAKE + 4)
    head16 = B.step_io(16, 512, flags=0, x_in=FAKE, tokens=FAKE, masked=FAKE, k_unmask=4)
    assert call(mhb, head16) == B.NMDLM_ERR_INVALID_ARG
    # path 6 forced: every layer (and the head) needs its blocked copies
    forced = B.step_io(16, 512, flags=B.NMDLM_NO_HEAD | B.NMDLM_PATH_BLOCKED, x_in=FAKE)
    assert call(m, forced) == B.NMDLM_ERR_INVALID_ARG
    Lc = B.Layer(FAKE, FAKE, FAKE, FAKE, 200, 200, 200, 200, 200, 200, 200, 4, FAKE, FAKE, FAKE,
                 FAKE, FAKE, FAKE, FAKE, FAKE)
    mc = B.Model(1, 1024, 16, 4096, 32000, 4, 8192, 0, (B.Layer * 1)(Lc), None, None, FAKE, FAKE)
    forced_head = B.step_io(16, 512, flags=B.NMDLM_PATH_BLOCKED, x_in=FAKE, tokens=FAKE,
                            masked=FAKE, k_unmask=4)
    assert call(mc, forced_head) == B.NMDLM_ERR_INVALID_ARG       # head copy missing
    # path 7 (wide tiles over the copies) needs them the same way
    wide = B.step_io(16, 512, flags=B.NMDLM_NO_HEAD | B.NMDLM_PATH_WIDE, x_in=FAKE)
    assert call(m, wide) == B.NMDLM_ERR_INVALID_ARG
    wide_head = B.step_io(16, 512, flags=B.NMDLM_PATH_WIDE, x_in=FAKE, tokens=FAKE,
                          masked=FAKE, k_unmask=4)
    assert call(mc, wide_head) == B.NMDLM_ERR_INVALID_ARG


def test_batched_step_argument_errors(lib):
    L = B.Layer(FAKE, FAKE, FAKE, FAKE, 200, 200, 200, 200, 200, 200, 200, 4, FAKE, FAKE, FAKE, FAKE)
    layers = (B.Layer * 1)(L)
    m1 = B.Model(1, 1024, 16, 4096, 32000, 4, 576, 0, layers, None, None, None, None)   # max_seq 0
    m4 = B.Model(1, 1024, 16, 4096, 32000, 4, 576, 0, layers, None, None, None, None, 4)
    nb = lib.nmdlm_block_step_workspace_size(C.byref(m4), 4 * 16, B.NMDLM_NO_HEAD)
    assert nb > lib.nmdlm_block_step_workspace_size(C.byref(m4), 16, B.NMDLM_NO_HEAD)
    call = lambda mm, ii: lib.nmdlm_block_step(C.byref(mm), C.byref(ii), FAKE, nb, None)
    io = lambda M, n: B.step_io(M, 512, flags=B.NMDLM_NO_HEAD, x_in=FAKE, n_seq=n)
    assert call(m1, io(16, 2)) == B.NMDLM_ERR_INVALID_ARG          # caches hold one sequence
    assert call(m4, io(16, 5)) == B.NMDLM_ERR_INVALID_ARG          # more than max_seq
    assert call(m4, io(16, -1)) == B.NMDLM_ERR_INVALID_ARG
    assert call(m4, io(6, 2)) == B.NMDLM_ERR_UNSUPPORTED           # T = 4: M a multiple of 4
    m4.max_seq = -1
    assert call(m4, io(16, 1)) == B.NMDLM_ERR_INVALID_ARG
    m4.max_seq = 4
    small = lib.nmdlm_block_step_workspace_size(C.byref(m4), 16, B.NMDLM_NO_HEAD)
    assert lib.nmdlm_block_step(C.byref(m4), C.byref(io(16, 4)), FAKE, small, None) == B.NMDLM_ERR_WORKSPACE


def test_ternary_argument_errors(lib):
    def enc(**kw):
        a = dict(a=FAKE, M=4, D=512, K=2, T=8, sp=FAKE, sn=FAKE, ss=None)
        a.update(kw)
        return lib.nmdlm_ternary_encode(a["a"], a["M"], a["D"], a["K"], a["T"], a["sp"], a["sn"],
                                        a["ss"], None)
    assert enc(a=None) == B.NMDLM_ERR_INVALID_ARG
    assert enc(sn=None) == B.NMDLM_ERR_INVALID_ARG
    assert enc(K=0) == B.NMDLM_ERR_INVALID_ARG
    assert enc(T=9) == B.NMDLM_ERR_UNSUPPORTED
    assert enc(D=4096, K=256) == B.NMDLM_ERR_UNSUPPORTED          # D K >= 2^20

    def prod(**kw):
        a = dict(sp=FAKE, sn=FAKE, T=8, M=4, K=4096, W=FAKE, N=512, ldw=512, acc=FAKE, ws=FAKE,
                 ws_bytes=1 << 30)
        a.update(kw)
        return lib.nmdlm_qbsm_ternary(a["sp"], a["sn"], a["T"], a["M"], a["K"], a["W"], a["N"],
                                      a["ldw"], a["acc"], None, 0, a["ws"], a["ws_bytes"], None)
    assert prod(sn=None) == B.NMDLM_ERR_INVALID_ARG
    assert prod(acc=None) == B.NMDLM_ERR_INVALID_ARG
    assert prod(K=20000) == B.NMDLM_ERR_UNSUPPORTED                # beyond the staged planes
    assert prod(ldw=500) == B.NMDLM_ERR_INVALID_ARG
    assert prod(ws=None) == B.NMDLM_ERR_WORKSPACE

    def prod_if(**kw):
        a = dict(sp=FAKE, sn=FAKE, T=8, M=4, K=4096, W=FAKE, N=512, ldw=512, num=FAKE, den=8192,
                 op=FAKE, on=FAKE, ws=FAKE, ws_bytes=1 << 30)
        a.update(kw)
        return lib.nmdlm_qbsm_ternary_if(a["sp"], a["sn"], a["T"], a["M"], a["K"], a["W"], a["N"],
                                         a["ldw"], a["num"], a["den"], a["op"], a["on"], None,
                                         None, 0, a["ws"], a["ws_bytes"], None)
    assert prod_if(num=None) == B.NMDLM_ERR_INVALID_ARG
    assert prod_if(on=None) == B.NMDLM_ERR_INVALID_ARG
    assert prod_if(den=0) == B.NMDLM_ERR_INVALID_ARG
    assert prod_if(den=(1 << 24) + 1) == B.NMDLM_ERR_UNSUPPORTED
    assert prod_if(K=20000) == B.NMDLM_ERR_UNSUPPORTED
    assert prod_if(T=9) == B.NMDLM_ERR_UNSUPPORTED
    assert prod_if(ws_bytes=16) == B.NMDLM_ERR_WORKSPACE


def test_binding_constants_match_the_header():
    text = open(HEADER).read()
    for name in ("NMDLM_FORCE_DENSE", "NMDLM_NO_HEAD", "NMDLM_ATTN_FUSED", "NMDLM_SPLIT_SHIFT",
                 "NMDLM_ROWTILE_SHIFT", "NMDLM_MAX_HEAD_M", "NMDLM_MAX_T", "NMDLM_MAX_K",
                 "NMDLM_MAX_KEYS", "NMDLM_STATUS_TOKEN_CLAMPED", "NMDLM_MAX_THR_DEN",
                 "NMDLM_NOALLOC_SCRATCH_BYTES", "NMDLM_BLOCKED_MIN_ROWS"):
        m = re.search(r"#define\s+%s\s+([0-9xXa-fA-F]+)u?" % name, text)
        assert m, name
        if hasattr(B, name):
            assert getattr(B, name) == int(m.group(1).rstrip("u"), 0), name


def test_blocked_weight_sizes_and_errors(lib):
    # 4096 bytes per (64-row word, 64-column tile), ragged K and N rounded up
    assert lib.nmdlm_weight_blocked_bytes(64, 64) == 4096
    assert lib.nmdlm_weight_blocked_bytes(700, 300) == 11 * 5 * 4096
    assert lib.nmdlm_weight_blocked_bytes(0, 64) == 0
    assert lib.nmdlm_weight_blocked_bytes(70000, 64) == 0
    # validation before any HIP call
    assert lib.nmdlm_weight_block(FAKE, 0, 64, 64, FAKE, None) == B.NMDLM_ERR_INVALID_ARG
    assert lib.nmdlm_weight_block(FAKE, 64, 64, 64, None, None) == B.NMDLM_ERR_INVALID_ARG
    assert lib.nmdlm_weight_block(FAKE, 64, 64, 64, FAKE + 8, None) == B.NMDLM_ERR_INVALID_ARG
    assert lib.nmdlm_weight_block(FAKE, 64, 64, 60, FAKE, None) == B.NMDLM_ERR_INVALID_ARG
    assert lib.nmdlm_weight_block(FAKE, 70000, 64, 64, FAKE, None) == B.NMDLM_ERR_UNSUPPORTED

    def blk(Wb=FAKE, K=512, N=512, ldw=512, ws_bytes=1 << 30):
        return lib.nmdlm_qbsm_blocked(FAKE, 4, 8, K, FAKE, Wb, N, ldw, None, FAKE, 256, None, None,
                                      None, 0, FAKE, ws_bytes, None)
    assert blk(Wb=None) == B.NMDLM_ERR_INVALID_ARG
    assert blk(Wb=FAKE + 4) == B.NMDLM_ERR_INVALID_ARG
    assert blk(K=65536, N=40000, ldw=40000) == B.NMDLM_ERR_UNSUPPORTED  # copy beyond 2^31 bytes
    assert blk(ldw=500) == B.NMDLM_ERR_INVALID_ARG
    assert blk(ws_bytes=16) == B.NMDLM_ERR_WORKSPACE
