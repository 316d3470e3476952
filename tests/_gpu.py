"""Helpers shared by the GPU tests: run the C ABI through the binding and
bring results back as numpy arrays."""
import numpy as np
import pytest

from workloads import synth


def need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24841_amd import binding as B
    B.load()          # raises (fails the test) if the library is not built
    return torch, B


def pad_weights(W: np.ndarray) -> tuple[np.ndarray, int]:
    K, N = W.shape
    ldw = (N + 15) // 16 * 16
    Wp = np.zeros((K, ldw), dtype=np.int8)
    Wp[:, :N] = W
    return Wp, ldw


def run_qbsm(S, W, bias=None, theta=None, theta_vec=None, flags=0, want_cur=True, blocked=False):
    """Run nmdlm_qbsm (nmdlm_qbsm_blocked with a blocked copy of the weights
    when blocked); returns (currents int64 or None, spikes bool or None, stats
    dict, raw spike words)."""
    torch, B = need_gpu()
    T, M, K = S.shape
    N = W.shape[1]
    Wp, ldw = pad_weights(W)
    dev = "cuda"
    s_in = B.to_dev_bits(synth.pack_bits(S), dev)
    Wd = torch.from_numpy(Wp).to(dev)
    bd = torch.from_numpy(np.asarray(bias, dtype=np.int32)).to(dev) if bias is not None else None
    tv = torch.from_numpy(np.asarray(theta_vec, dtype=np.int32)).to(dev) if theta_vec is not None else None
    cur = torch.full((T, M, N), -7, dtype=torch.int32, device=dev) if want_cur else None
    Nw = (N + 63) // 64
    spk = None
    if theta is not None or theta_vec is not None:
        spk = torch.full((T, M, Nw), -1, dtype=torch.int64, device=dev)
    stats = torch.zeros(4, dtype=torch.int64, device=dev)
    ws = B.workspace(B.nmdlm_qbsm_workspace_size(T, M, K, N), dev)
    if blocked:
        Wb = B.blocked_weights(Wd, K, N, ldw)
        B.nmdlm_qbsm_blocked(s_in, T, M, K, Wd, Wb, N, ldw, bias=bd, cur_out=cur,
                             theta=int(theta or 0), theta_vec=tv, s_out=spk, stats=stats,
                             flags=flags, ws=ws)
    else:
        B.nmdlm_qbsm(s_in, T, M, K, Wd, N, ldw, bias=bd, cur_out=cur, theta=int(theta or 0),
                     theta_vec=tv, s_out=spk, stats=stats, flags=flags, ws=ws)
    torch.cuda.synchronize()
    st = stats.cpu().numpy()
    out_cur = cur.cpu().numpy().astype(np.int64) if cur is not None else None
    words = B.from_dev_bits(spk) if spk is not None else None
    out_spk = synth.unpack_bits(words, N) if words is not None else None
    # the workspace's accumulator region must be left at zero
    return out_cur, out_spk, dict(k_total=st[0], k_active=st[1], n=st[2], weight_bytes=st[3]), words, ws


def padding_bits_zero(words: np.ndarray, N: int) -> bool:
    if N % 64 == 0:
        return True
    last = words[..., -1]
    return bool(np.all((last >> np.uint64(N % 64)) == 0))


def assert_same(got, want, what="array"):
    """Element-wise equality with a short report of the first differences."""
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, f"{what}: shape {got.shape} != {want.shape}"
    bad = np.argwhere(got != want)
    if bad.size:
        first = [tuple(int(v) for v in b) for b in bad[:5]]
        vals = [(got[tuple(b)].item(), want[tuple(b)].item()) for b in bad[:5]]
        raise AssertionError(f"{what}: {len(bad)} of {got.size} differ; first at {first}: "
                             f"(got, want) = {vals}")
