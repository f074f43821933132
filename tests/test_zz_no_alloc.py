"""kvq_decode_attention_noalloc (the decode entry point that allocates
nothing: its workspace is the library's own per-GPU scratch array) against
kvq_decode_attention with a caller workspace, through the C ABI: bitwise
equal outputs on two calls in a row, the second with a smaller input, both
within 2e-3 of the oracle on sampled heads; and a call that would need more
than the array's size is refused before anything is launched."""
import numpy as np
import pytest

from helpers import ATTN_TOL, Case, log, row_rel_err
from workloads import Workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def W(name, batch, hq, lens, bk, bv, R=0):
    return Workload(name, batch, hq, 8, 128, tuple(lens), (bk,) * batch, (bv,) * batch, 32, 32, R, cfg_id=95)


def _both(c):
    from paper_2607_16248_amd import kvq
    w = c.w
    ref = torch.empty((w.batch, w.num_q_heads, 128), dtype=torch.float32, device="cuda")
    got = torch.full_like(ref, float("nan"))
    kvq.kvq_decode_attention(c.cache.handle, c.qd, ref, c.cache.workspace())
    kvq.kvq_decode_attention_noalloc(c.cache.handle, c.qd, got)
    torch.cuda.synchronize()
    return ref.cpu().numpy(), got.cpu().numpy()


def test_noalloc_matches_the_workspace_entry_point():
    for w, heads in ((W("noalloc_big", 2, 32, (20000, 9000), 1, 1), [0, 6]),
                     (W("noalloc_small", 1, 40, (700,), 2, 2, R=40), [1, 7])):
        log(f"[noalloc] {w.name}")
        c = Case(w, heads=heads)
        c.append_all()
        ref, got = _both(c)
        assert (ref.view(np.uint32) == got.view(np.uint32)).all(), w.name
        gq = w.num_q_heads // 8
        rows = [h * gq + j for h in heads for j in range(gq)]
        for s in range(w.batch):
            o = c.oracle_out(s, heads=heads)
            assert row_rel_err(got[s][rows], o[rows]).max() <= ATTN_TOL, (w.name, s)


def test_noalloc_refuses_more_than_its_array():
    from paper_2607_16248_amd import KvqError, kvq
    big = W("noalloc_refused", 8, 64, (16384,) * 8, 1, 1)
    cb = Case(big, heads=[0])
    cb.append_all()
    kvq.kvq_set_split_tokens(cb.cache.handle, 64)  # 8 sequences x 256 splits x 64 heads x 528 B = 69 MB > 16 MiB
    o2 = torch.zeros((8, 64, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(KvqError) as e:
        kvq.kvq_decode_attention_noalloc(cb.cache.handle, cb.qd, o2)
    assert e.value.status == kvq.ERR_CAPACITY and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (o2 == 0).all()   # nothing ran
    kvq.kvq_set_split_tokens(cb.cache.handle, 0)   # the library's own plan fits the array
    kvq.kvq_decode_attention_noalloc(cb.cache.handle, cb.qd, o2)
    ref = cb.decode()
    assert (ref.view(np.uint32) == o2.cpu().numpy().view(np.uint32)).all()
