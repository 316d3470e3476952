"""ctypes binding of libnmdlm: argument marshalling only.

Every function here passes torch tensor device pointers and the current torch
stream to the C ABI declared in ``include/nmdlm.h``; all arithmetic runs in
the library's HIP kernels.  torch is imported before the library is loaded so
that the library binds to the HIP runtime already in the process (both carry
the soname libamdhip64.so.7); the loader refuses to continue if two HIP
runtimes end up mapped.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libnmdlm.so")

NMDLM_OK = 0
NMDLM_ERR_INVALID_ARG = 1
NMDLM_ERR_UNSUPPORTED = 2
NMDLM_ERR_WORKSPACE = 3
NMDLM_ERR_HIP = 4
NMDLM_FORCE_DENSE = 0x1
NMDLM_NO_HEAD = 0x2
NMDLM_SPLIT_SHIFT = 8
NMDLM_ROWTILE_SHIFT = 16
NMDLM_ATTN_FUSED = 0x4
NMDLM_MAX_HEAD_M = 4096   # block tokens of a step that runs the head
NMDLM_MAX_KEYS = 1 << 23   # attention keys C+M per sequence
NMDLM_STATUS_TOKEN_CLAMPED = 0x1
NMDLM_NOALLOC_SCRATCH_BYTES = 16 << 20   # static scratch of nmdlm_qbsm_noalloc per GPU
NMDLM_MAX_THR_DEN = 1 << 24
NMDLM_PATH_SHIFT = 20
NMDLM_NO_FUSE = 1 << NMDLM_PATH_SHIFT      # separate pass building the active-row list
NMDLM_PATH_FUSED = 2 << NMDLM_PATH_SHIFT   # single kernel, in-kernel list
NMDLM_PATH_WORDS = 3 << NMDLM_PATH_SHIFT   # single kernel over 64-channel words
NMDLM_PATH_DMA = 4 << NMDLM_PATH_SHIFT     # as words, active rows gathered into LDS
NMDLM_PATH_SCALAR = 5 << NMDLM_PATH_SHIFT  # as words, scalar gather-accumulate product
NMDLM_PATH_BLOCKED = 6 << NMDLM_PATH_SHIFT  # as words, over the blocked weight copy
NMDLM_PATH_WIDE = 7 << NMDLM_PATH_SHIFT     # as blocked, four column tiles per workgroup
NMDLM_BLOCKED_MIN_ROWS = 32
NMDLM_QNL_S8 = 0
NMDLM_QNL_U8 = 1

EXPORTS = (
    "nmdlm_qbsm", "nmdlm_qbsm_workspace_size", "nmdlm_if_neuron", "nmdlm_qnl_lut",
    "nmdlm_bbm_attn", "nmdlm_bbm_attn_workspace_size", "nmdlm_block_step",
    "nmdlm_block_step_workspace_size", "nmdlm_workspace_clear", "nmdlm_status_string",
    "nmdlm_abi_version", "nmdlm_ternary_encode", "nmdlm_qbsm_ternary", "nmdlm_qbsm_ternary_if",
    "nmdlm_qbsm_blocked", "nmdlm_weight_blocked_bytes", "nmdlm_weight_block",
)


class NmdlmError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: status {status}")


class QbsmStats(C.Structure):
    _fields_ = [("k_total", C.c_int64), ("k_active", C.c_int64), ("n", C.c_int64),
                ("weight_bytes", C.c_int64)]


class Layer(C.Structure):
    _fields_ = [
        ("w_qkv", C.c_void_p), ("w_o", C.c_void_p), ("w_up", C.c_void_p), ("w_dn", C.c_void_p),
        ("theta_q", C.c_int32), ("theta_k", C.c_int32), ("theta_v", C.c_int32),
        ("theta_a", C.c_int32), ("theta_o", C.c_int32), ("theta_up", C.c_int32),
        ("theta_dn", C.c_int32), ("s_up", C.c_int32),
        ("lut_att", C.c_void_p), ("lut_act", C.c_void_p),
        ("k_cache", C.c_void_p), ("vt_cache", C.c_void_p),
        ("w_qkv_b", C.c_void_p), ("w_o_b", C.c_void_p), ("w_up_b", C.c_void_p),
        ("w_dn_b", C.c_void_p),
    ]


class Model(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int), ("d", C.c_int), ("H", C.c_int), ("F", C.c_int), ("V", C.c_int),
        ("T", C.c_int), ("cache_cap", C.c_int64), ("max_pos", C.c_int),
        ("layers", C.POINTER(Layer)), ("emb", C.c_void_p), ("pos_ch", C.c_void_p),
        ("w_head", C.c_void_p), ("head_scale", C.c_void_p), ("max_seq", C.c_int),
        ("w_head_b", C.c_void_p),
    ]


class StepIO(C.Structure):
    _fields_ = [
        ("M", C.c_int), ("C", C.c_int), ("pos0", C.c_int), ("flags", C.c_uint),
        ("x_in", C.c_void_p), ("tokens", C.c_void_p), ("masked", C.c_void_p),
        ("k_unmask", C.c_int), ("y_out", C.c_void_p), ("logits", C.c_void_p),
        ("pred", C.c_void_p), ("conf", C.c_void_p), ("unmasked_pos", C.c_void_p),
        ("stats", C.c_void_p), ("prof_events", C.POINTER(C.c_void_p)), ("n_prof_events", C.c_int),
        ("n_seq", C.c_int), ("status", C.c_void_p),
    ]


_lib = None


def _hip_runtimes_mapped() -> set:
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


def load(path: str = LIB_PATH):
    """Load libnmdlm.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2607_24841_amd.build`")
    lib = C.CDLL(path)
    vp, i32, i64, sz, u = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_uint
    lib.nmdlm_qbsm.argtypes = [vp, C.c_int, C.c_int, C.c_int, vp, C.c_int, i64, vp, vp, i32, vp,
                               vp, vp, u, vp, sz, vp]
    lib.nmdlm_qbsm_noalloc.argtypes = [vp, C.c_int, C.c_int, C.c_int, vp, C.c_int, i64, vp, vp,
                                       i32, vp, vp, vp, u, vp]
    lib.nmdlm_qbsm_blocked.argtypes = [vp, C.c_int, C.c_int, C.c_int, vp, vp, C.c_int, i64, vp,
                                       vp, i32, vp, vp, vp, u, vp, sz, vp]
    lib.nmdlm_weight_blocked_bytes.argtypes = [C.c_int, C.c_int]
    lib.nmdlm_weight_blocked_bytes.restype = sz
    lib.nmdlm_weight_block.argtypes = [vp, C.c_int, C.c_int, i64, vp, vp]
    lib.nmdlm_qbsm_workspace_size.argtypes = [C.c_int] * 4
    lib.nmdlm_qbsm_workspace_size.restype = sz
    lib.nmdlm_if_neuron.argtypes = [vp, C.c_int, C.c_int, C.c_int, i32, vp, vp, vp, vp, vp]
    lib.nmdlm_ternary_encode.argtypes = [vp, C.c_int, C.c_int, C.c_int, C.c_int, vp, vp, vp, vp]
    lib.nmdlm_qbsm_ternary.argtypes = [vp, vp, C.c_int, C.c_int, C.c_int, vp, C.c_int, i64, vp, vp,
                                       u, vp, sz, vp]
    lib.nmdlm_qbsm_ternary_if.argtypes = [vp, vp, C.c_int, C.c_int, C.c_int, vp, C.c_int, i64,
                                          vp, i64, vp, vp, vp, vp, u, vp, sz, vp]
    lib.nmdlm_qnl_lut.argtypes = [vp, i64, C.c_int, C.c_int, vp, vp, vp]
    lib.nmdlm_bbm_attn.argtypes = [vp, vp, vp, i64, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                   vp, vp, i32, vp, vp, sz, vp]
    lib.nmdlm_bbm_attn_workspace_size.argtypes = [C.c_int] * 4
    lib.nmdlm_bbm_attn_workspace_size.restype = sz
    lib.nmdlm_block_step.argtypes = [C.POINTER(Model), C.POINTER(StepIO), vp, sz, vp]
    lib.nmdlm_block_step_workspace_size.argtypes = [C.POINTER(Model), C.c_int, u]
    lib.nmdlm_block_step_workspace_size.restype = sz
    lib.nmdlm_workspace_clear.argtypes = [vp, sz, vp]
    lib.nmdlm_status_string.argtypes = [C.c_int]
    lib.nmdlm_status_string.restype = C.c_char_p
    lib.nmdlm_abi_version.restype = C.c_int
    for fn in ("nmdlm_qbsm", "nmdlm_qbsm_noalloc", "nmdlm_if_neuron", "nmdlm_qnl_lut", "nmdlm_bbm_attn",
               "nmdlm_block_step", "nmdlm_workspace_clear", "nmdlm_ternary_encode",
               "nmdlm_qbsm_ternary", "nmdlm_qbsm_ternary_if"):
        getattr(lib, fn).restype = C.c_int
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes mapped in this process: {sorted(runtimes)}")
    _lib = lib
    return lib


# ----------------------------------------------------------------------------
# marshalling helpers
# ----------------------------------------------------------------------------
def ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def stream_handle(stream=None) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def check(status: int, what: str) -> None:
    if status != NMDLM_OK:
        msg = load().nmdlm_status_string(status).decode()
        raise NmdlmError(status, f"{what} failed ({msg})")


def to_dev_bits(words: np.ndarray, device="cuda") -> torch.Tensor:
    """uint64 numpy spike words -> int64 device tensor with the same bits."""
    return torch.from_numpy(np.ascontiguousarray(words).view(np.int64)).to(device)


def from_dev_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint64)


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """Zero-filled workspace (the counter/accumulator regions must start at 0)."""
    return torch.zeros(max(256, int(nbytes)), dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------
# the five calls (same names as the C ABI)
# ----------------------------------------------------------------------------
def nmdlm_qbsm(s_in, T, M, K, W, N, ldw, bias=None, cur_out=None, theta=0, theta_vec=None,
               s_out=None, stats=None, flags=0, ws=None, stream=None) -> None:
    lib = load()
    st = lib.nmdlm_qbsm(ptr(s_in), T, M, K, ptr(W), N, ldw, ptr(bias), ptr(cur_out), theta,
                        ptr(theta_vec), ptr(s_out), ptr(stats), flags, ptr(ws),
                        0 if ws is None else ws.numel() * ws.element_size(), stream_handle(stream))
    check(st, "nmdlm_qbsm")


def nmdlm_qbsm_blocked(s_in, T, M, K, W, Wb, N, ldw, bias=None, cur_out=None, theta=0,
                       theta_vec=None, s_out=None, stats=None, flags=0, ws=None,
                       stream=None) -> None:
    """nmdlm_qbsm with the blocked copy Wb of W (see nmdlm_weight_block)."""
    st = load().nmdlm_qbsm_blocked(ptr(s_in), T, M, K, ptr(W), ptr(Wb), N, ldw, ptr(bias),
                                   ptr(cur_out), theta, ptr(theta_vec), ptr(s_out), ptr(stats),
                                   flags, ptr(ws),
                                   0 if ws is None else ws.numel() * ws.element_size(),
                                   stream_handle(stream))
    check(st, "nmdlm_qbsm_blocked")


def nmdlm_weight_blocked_bytes(K, N) -> int:
    return load().nmdlm_weight_blocked_bytes(K, N)


def nmdlm_weight_block(W, K, N, ldw, Wb, stream=None) -> None:
    check(load().nmdlm_weight_block(ptr(W), K, N, ldw, ptr(Wb), stream_handle(stream)),
          "nmdlm_weight_block")


def blocked_weights(W, K, N, ldw, stream=None):
    """A device uint8 tensor holding the blocked copy of the int8 weights W."""
    import torch
    Wb = torch.empty(nmdlm_weight_blocked_bytes(K, N), dtype=torch.int8, device=W.device)
    nmdlm_weight_block(W, K, N, ldw, Wb, stream)
    return Wb


def nmdlm_qbsm_noalloc(s_in, T, M, K, W, N, ldw, bias=None, cur_out=None, theta=0,
                       theta_vec=None, s_out=None, stats=None, flags=0, stream=None) -> None:
    """nmdlm_qbsm with the library's static per-GPU scratch (no workspace)."""
    st = load().nmdlm_qbsm_noalloc(ptr(s_in), T, M, K, ptr(W), N, ldw, ptr(bias), ptr(cur_out),
                                   theta, ptr(theta_vec), ptr(s_out), ptr(stats), flags,
                                   stream_handle(stream))
    check(st, "nmdlm_qbsm_noalloc")


def nmdlm_qbsm_workspace_size(T, M, K, N) -> int:
    return load().nmdlm_qbsm_workspace_size(T, M, K, N)


def nmdlm_ternary_encode(a, M, D, K, T, s_pos, s_neg, s_sum=None, stream=None) -> None:
    st = load().nmdlm_ternary_encode(ptr(a), M, D, K, T, ptr(s_pos), ptr(s_neg), ptr(s_sum),
                                     stream_handle(stream))
    check(st, "nmdlm_ternary_encode")


def nmdlm_qbsm_ternary(s_pos, s_neg, T, M, K, W, N, ldw, acc_out, stats=None, flags=0, ws=None,
                       stream=None) -> None:
    st = load().nmdlm_qbsm_ternary(ptr(s_pos), ptr(s_neg), T, M, K, ptr(W), N, ldw, ptr(acc_out),
                                   ptr(stats), flags, ptr(ws),
                                   0 if ws is None else ws.numel() * ws.element_size(),
                                   stream_handle(stream))
    check(st, "nmdlm_qbsm_ternary")


def nmdlm_qbsm_ternary_if(s_pos, s_neg, T, M, K, W, N, ldw, thr_num, thr_den, out_pos, out_neg,
                          v_out=None, stats=None, flags=0, ws=None, stream=None) -> None:
    st = load().nmdlm_qbsm_ternary_if(ptr(s_pos), ptr(s_neg), T, M, K, ptr(W), N, ldw,
                                      ptr(thr_num), int(thr_den), ptr(out_pos), ptr(out_neg),
                                      ptr(v_out), ptr(stats), flags, ptr(ws),
                                      0 if ws is None else ws.numel() * ws.element_size(),
                                      stream_handle(stream))
    check(st, "nmdlm_qbsm_ternary_if")


def nmdlm_if_neuron(cur, T, M, N, theta=0, theta_vec=None, resid=None, v_inout=None, s_out=None,
                    stream=None) -> None:
    st = load().nmdlm_if_neuron(ptr(cur), T, M, N, theta, ptr(theta_vec), ptr(resid),
                                ptr(v_inout), ptr(s_out), stream_handle(stream))
    check(st, "nmdlm_if_neuron")


def nmdlm_qnl_lut(x, n, shift, mode, lut, y, stream=None) -> None:
    st = load().nmdlm_qnl_lut(ptr(x), n, shift, mode, ptr(lut), ptr(y), stream_handle(stream))
    check(st, "nmdlm_qnl_lut")


def nmdlm_bbm_attn(q, k_cache, vt_cache, cache_cap, T, M, C_, H, dh, lut_att, a_out=None,
                   theta_a=0, s_out=None, ws=None, stream=None) -> None:
    st = load().nmdlm_bbm_attn(ptr(q), ptr(k_cache), ptr(vt_cache), cache_cap, T, M, C_, H, dh,
                               ptr(lut_att), ptr(a_out), theta_a, ptr(s_out), ptr(ws),
                               0 if ws is None else ws.numel() * ws.element_size(),
                               stream_handle(stream))
    check(st, "nmdlm_bbm_attn")


def nmdlm_bbm_attn_workspace_size(T, M, H, dh) -> int:
    return load().nmdlm_bbm_attn_workspace_size(T, M, H, dh)


def nmdlm_block_step(model: "DeviceModel", io: StepIO, ws: torch.Tensor, stream=None) -> None:
    st = load().nmdlm_block_step(C.byref(model.c), C.byref(io), ptr(ws),
                                 ws.numel() * ws.element_size(), stream_handle(stream))
    check(st, "nmdlm_block_step")


def nmdlm_block_step_workspace_size(model: "DeviceModel", M: int, flags: int = 0) -> int:
    return load().nmdlm_block_step_workspace_size(C.byref(model.c), M, flags)


def nmdlm_workspace_clear(ws: torch.Tensor, stream=None) -> None:
    check(load().nmdlm_workspace_clear(ptr(ws), ws.numel() * ws.element_size(),
                                       stream_handle(stream)), "nmdlm_workspace_clear")


# ----------------------------------------------------------------------------
# device-resident model (uploads host arrays and fills the C structs)
# ----------------------------------------------------------------------------
def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to(device)


class DeviceLayer:
    """One layer's weights and tables on the GPU, with K/V caches for
    max_seq sequences: k_seq [max_seq][T][cap][d/64], vt_seq
    [max_seq][T][cap/64][d]; k_cache / vt_cache are sequence 0's."""

    def __init__(self, L, T: int, cache_cap: int, device="cuda", max_seq: int = 1,
                 blocked: bool = False):
        d = L.d
        self.w_qkv = _dev(L.W_qkv, device)
        self.w_o = _dev(L.W_o, device)
        self.w_up = _dev(L.W_up, device)
        self.w_dn = _dev(L.W_dn, device)
        # blocked copies (nmdlm_weight_block) for products over dense unions
        self.blk = {}
        if blocked:
            for name in ("w_qkv", "w_o", "w_up", "w_dn"):
                w = getattr(self, name)
                K, N = w.shape
                self.blk[name] = blocked_weights(w, K, N, N)
        self.lut_att = _dev(L.lut_att, device)
        self.lut_act = _dev(L.lut_act, device)
        self.k_seq = torch.zeros((max_seq, T, cache_cap, d // 64), dtype=torch.int64, device=device)
        self.vt_seq = torch.zeros((max_seq, T, cache_cap // 64, d), dtype=torch.int64, device=device)
        self.k_cache, self.vt_cache = self.k_seq[0], self.vt_seq[0]  # word-major values
        th = L.theta
        self.c = Layer(ptr(self.w_qkv), ptr(self.w_o), ptr(self.w_up), ptr(self.w_dn),
                       th["q"], th["k"], th["v"], th["a"], th["o"], th["up"], th["dn"], L.s_up,
                       ptr(self.lut_att), ptr(self.lut_act), ptr(self.k_cache), ptr(self.vt_cache),
                       *[ptr(self.blk.get(n)) for n in ("w_qkv", "w_o", "w_up", "w_dn")])


class DeviceModel:
    """A stack of layers (and optionally token tables and a head) on the GPU."""

    def __init__(self, layers, T: int, cache_cap: int, d: int, H: int, F: int, V: int = 1,
                 emb=None, pos_ch=None, W_head=None, scale=None, device="cuda", max_seq: int = 1,
                 blocked: bool = False):
        """blocked: also hold blocked copies of every weight (twice the weight
        bytes), which products over dense unions read."""
        cache_cap = (cache_cap + 63) // 64 * 64
        self.T, self.d, self.H, self.F, self.V, self.cache_cap = T, d, H, F, V, cache_cap
        self.max_seq = max(1, int(max_seq))
        self.layers = [DeviceLayer(L, T, cache_cap, device, self.max_seq, blocked) for L in layers]
        self._c_layers = (Layer * max(1, len(self.layers)))(*[l.c for l in self.layers])
        self.emb = _dev(emb, device) if emb is not None else None
        self.pos_ch = _dev(pos_ch.astype(np.int32), device) if pos_ch is not None else None
        self.w_head = _dev(W_head, device) if W_head is not None else None
        self.scale = _dev(scale.astype(np.float32), device) if scale is not None else None
        self.max_pos = 0 if pos_ch is None else int(pos_ch.shape[0])
        self.w_head_b = None
        if blocked and self.w_head is not None:
            self.w_head_b = blocked_weights(self.w_head, d, V, V)
        self.c = Model(len(self.layers), d, H, F, V, T, cache_cap, self.max_pos, self._c_layers,
                       ptr(self.emb), ptr(self.pos_ch), ptr(self.w_head), ptr(self.scale),
                       self.max_seq, ptr(self.w_head_b))

    @classmethod
    def from_mdlm(cls, m, cache_cap: int, device="cuda", max_seq: int = 1, blocked: bool = False):
        return cls(m.layers, m.T, cache_cap, m.d, m.H, m.F, m.V, emb=m.emb, pos_ch=m.pos_ch,
                   W_head=m.W_head, scale=m.scale, device=device, max_seq=max_seq,
                   blocked=blocked)

    def reset_caches(self):
        for l in self.layers:
            l.k_seq.zero_()
            l.vt_seq.zero_()

    def view(self, first: int, count: int, head: bool) -> "ModelView":
        """Layers [first, first+count) of this model (their weights and caches
        are shared, not copied), with the token tables, and the head if asked."""
        return ModelView(self, self.layers[first:first + count], head)


class ModelView:
    """A model struct over a slice of another model's layers."""

    def __init__(self, parent: DeviceModel, layers, head: bool):
        self.parent = parent                      # keeps the device tensors alive
        self.layers = list(layers)
        self.T, self.d, self.H, self.F = parent.T, parent.d, parent.H, parent.F
        self.V, self.cache_cap, self.max_seq = parent.V, parent.cache_cap, parent.max_seq
        self._c_layers = (Layer * max(1, len(self.layers)))(*[l.c for l in self.layers])
        p = parent.c
        self.c = Model(len(self.layers), p.d, p.H, p.F, p.V, p.T, p.cache_cap, p.max_pos,
                       self._c_layers, p.emb, p.pos_ch, p.w_head if head else None,
                       p.head_scale if head else None, p.max_seq,
                       p.w_head_b if head else None)


def step_io(M, C_, pos0=0, flags=0, x_in=None, tokens=None, masked=None, k_unmask=0, y_out=None,
            logits=None, pred=None, conf=None, unmasked_pos=None, stats=None,
            prof_events=None, n_seq: int = 1, status=None) -> StepIO:
    """prof_events: optional ctypes array of hipEvent_t handles (see HipEvents).
    n_seq: sequences in the step; M is per sequence, token buffers hold the
    sequences one after the other.  status: optional device int32 word that
    the step ORs NMDLM_STATUS_* bits into."""
    ev = prof_events if prof_events is not None else None
    return StepIO(M, C_, pos0, flags, ptr(x_in), ptr(tokens), ptr(masked), k_unmask, ptr(y_out),
                  ptr(logits), ptr(pred), ptr(conf), ptr(unmasked_pos), ptr(stats),
                  ev, 0 if ev is None else len(ev), n_seq, ptr(status))


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime already loaded by torch,
    for timing kernels that the library launches on a stream."""

    def __init__(self, n: int):
        self.hip = C.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]
        self.arr = (C.c_void_p * n)()
        for i in range(n):
            h = C.c_void_p()
            if self.hip.hipEventCreate(C.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.arr[i] = h

    def __len__(self):
        return len(self.arr)

    def elapsed_ms(self, i: int, j: int) -> float:
        self.hip.hipEventSynchronize(self.arr[j])
        out = C.c_float()
        if self.hip.hipEventElapsedTime(C.byref(out), self.arr[i], self.arr[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(out.value)

    def close(self):
        for h in self.arr:
            self.hip.hipEventDestroy(h)
