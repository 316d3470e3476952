"""nmdlm_qbsm_noalloc (static per-GPU scratch, no workspace argument) against
nmdlm_qbsm with a caller workspace: the same integers on two calls in a row,
the second with a smaller input, on the default path, a forced K split
(accumulators in the scratch) and the list path (active-row list in the
scratch); and the size limit."""
import numpy as np
import pytest

from workloads import synth

from ._gpu import assert_same, need_gpu, pad_weights

pytestmark = pytest.mark.gpu


def _both(S, W, bias, theta, flags):
    torch, B = need_gpu()
    T, M, K = S.shape
    N = W.shape[1]
    Wp, ldw = pad_weights(W)
    s_in = B.to_dev_bits(synth.pack_bits(S))
    Wd = torch.from_numpy(Wp).cuda()
    bd = torch.from_numpy(bias.astype(np.int32)).cuda()
    Nw = (N + 63) // 64
    out = []
    for noalloc in (False, True):
        cur = torch.full((T, M, N), -7, dtype=torch.int32, device="cuda")
        spk = torch.full((T, M, Nw), -1, dtype=torch.int64, device="cuda")
        st = torch.zeros(4, dtype=torch.int64, device="cuda")
        if noalloc:
            B.nmdlm_qbsm_noalloc(s_in, T, M, K, Wd, N, ldw, bias=bd, cur_out=cur, theta=theta,
                                 s_out=spk, stats=st, flags=flags)
        else:
            ws = B.workspace(B.nmdlm_qbsm_workspace_size(T, M, K, N))
            B.nmdlm_qbsm(s_in, T, M, K, Wd, N, ldw, bias=bd, cur_out=cur, theta=theta,
                         s_out=spk, stats=st, flags=flags, ws=ws)
        torch.cuda.synchronize()
        out.append((cur.cpu().numpy(), B.from_dev_bits(spk), st.cpu().numpy()))
    return out


@pytest.mark.parametrize("flags", [0, 4 << 8, 1 << 20], ids=["auto", "split4", "list"])
def test_noalloc_matches_workspace_call_twice(flags):
    need_gpu()
    for i, (T, M, K, N) in enumerate(((4, 40, 1100, 700), (4, 9, 300, 130))):
        c = synth.make_qbsm_case(900 + i, T, M, K, N, 0.1)
        (c0, s0, t0), (c1, s1, t1) = _both(c.S, c.W, c.bias, c.theta, flags)
        assert_same(c1, c0, "currents")
        assert_same(s1, s0, "spike words")
        assert_same(t1, t0, "stats")


def test_noalloc_rejects_products_beyond_its_scratch():
    torch, B = need_gpu()
    lib = B.load()
    # workspace of 4 x 4096 rows x 65536 inputs exceeds NMDLM_NOALLOC_SCRATCH_BYTES
    assert lib.nmdlm_qbsm_workspace_size(4, 4096, 65536, 64) > B.NMDLM_NOALLOC_SCRATCH_BYTES
    fake = 1 << 40
    assert lib.nmdlm_qbsm_noalloc(fake, 4, 4096, 65536, fake, 64, 64, None, fake, 256, None,
                                  None, None, 0, None) == B.NMDLM_ERR_UNSUPPORTED
