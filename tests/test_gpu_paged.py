"""GPU parity of paged caches (page_tokens > 0: the packed data of every
page_tokens tokens live in pool pages found through a block table) against
the oracle and against the same inputs in a contiguous cache.

- canonical export bytes identical to the oracle's image, also after
  appends that interleave the sequences (their pages alternate in the
  pool) and after a sequence is released and its slot refilled (reused
  pages);
- decode outputs bit-identical to the contiguous cache's (same split plan,
  same arithmetic) and within 2e-3 of the fp64 oracle;
- chunk attention and kvq_dequant over paged caches;
- the matrix kernels (1/2-bit, 4 and 8 bits) and the vector kernel
  (canonical layout) both read through the table;
- a shared pool smaller than batch x capacity: an append that needs more
  pages fails up front, and succeeds after a release.
"""
import numpy as np
import pytest

import oracle
from helpers import ATTN_TOL, Case, log, row_rel_err
from workloads import Workload, gen_kv, gen_q, gen_q_chunk

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def W(name, batch, hq, hkv, lens, bk, bv, gk=32, gv=32, R=0, dist="normal", cfg=93):
    if isinstance(lens, int):
        lens = (lens,) * batch
    return Workload(name, batch, hq, hkv, 128, tuple(lens), (bk,) * batch, (bv,) * batch, gk, gv, R,
                    key_dist=dist, cfg_id=cfg)


def _bytes_match(c, w):
    for s in range(w.batch):
        for h in range(w.num_kv_heads):
            got, ref = c.cache.export(s, h), c.oracle_image(s, h)
            assert got.size == ref.size and (got == ref).all(), (s, h, np.flatnonzero(got != ref)[:5])


CASES = [
    (W("k1v1_gq4", 3, 32, 8, (1000, 517, 2100), 1, 1), 64, [100, 37, 300, 1, 64, 700, 900]),
    (W("k2v2_gq5_R128", 2, 40, 8, (900, 1400), 2, 2, R=128, dist="student_t3"), 128, [257, 1000, 300]),
    (W("k8v8_gq4_g64", 2, 32, 8, (700, 1111), 8, 8, gk=64), 256, [333, 333, 333, 333]),
    (W("k4v4_gq8", 2, 64, 8, (640, 800), 4, 4), 64, [80, 720]),
    (W("k1v4_gq4_vector", 2, 32, 8, (950, 260), 1, 4), 64, [31, 500, 500]),
    (W("k2v2_gq2_g64", 2, 16, 8, (700, 333), 2, 2, gk=64, R=40), 128, [1, 2, 3, 700]),
    (W("k2v4_gq2_vector", 2, 16, 8, (700, 333), 2, 4, R=40), 128, [1, 2, 3, 700]),
]


@pytest.mark.parametrize("w,P,chunks", CASES, ids=[f"{w.name}_P{P}" for w, P, _ in CASES])
def test_paged_matches_contiguous_and_oracle(w, P, chunks):
    log(f"[paged] {w.name} P={P}: append {chunks}")
    paged = Case(w, page_tokens=P)
    flat = Case(w)
    paged.append_all(chunks)          # chunked appends interleave the sequences' pages
    flat.append_all()
    paged.cache.check()
    _bytes_match(paged, w)
    a, b = paged.decode(), flat.decode()
    assert (a.view(np.uint32) == b.view(np.uint32)).all()
    worst = 0.0
    for s in range(w.batch):
        err = row_rel_err(a[s], paged.oracle_out(s))
        worst = max(worst, float(err.max()))
        assert err.max() <= ATTN_TOL
    log(f"[paged] {w.name} P={P}: max row-relative error {worst:.3e}")
    # dequantization reads the same pages
    for s in range(w.batch):
        L = w.lens[s]
        Kd, Vd = paged.cache.dequant(s, 0, L)
        Kf, Vf = flat.cache.dequant(s, 0, L)
        assert torch.equal(Kd, Kf) and torch.equal(Vd, Vf), s


def _append_rows(c, rows):
    """Append rows[s] (fp16 [n][Hkv][d]) to every sequence s."""
    n = [len(r) for r in rows]
    Kb = np.zeros((len(rows), max(n), 8, 128), np.float16)
    Vb = np.zeros_like(Kb)
    for s, r in enumerate(rows):
        Kb[s, :n[s]], Vb[s, :n[s]] = r[0], r[1]
    c.cache.append(torch.from_numpy(Kb).cuda(), torch.from_numpy(Vb).cuda(), n)


class _Rows(list):
    def __len__(self):
        return len(self[0])


def test_release_reuses_pages_and_pool_capacity():
    w = W("pool", 2, 32, 8, (1300, 1300), 1, 1)
    c = Case(w, page_tokens=128, num_pages=16)   # 10 pages per full sequence, 16 shared
    _append_rows(c, [_Rows([c.K[s][:600], c.V[s][:600]]) for s in range(2)])  # 576 packed: 5 pages each
    torch.cuda.synchronize()
    assert c.cache.free_pages() == 6
    from paper_2607_16248_amd import KvqError
    with pytest.raises(KvqError):                 # both to 1300 tokens: 10 more pages > 6
        _append_rows(c, [_Rows([c.K[s][600:], c.V[s][600:]]) for s in range(2)])
    assert c.cache.seq_len(0) == 600 and c.cache.free_pages() == 6
    # release sequence 0 and give it 640 tokens of sequence 1's draw; sequence 1 grows to 1300
    c.cache.release(0)
    assert c.cache.seq_len(0) == 0 and c.cache.free_pages() == 11
    K1, V1 = c.K[1], c.V[1]
    Kb = np.zeros((2, 700, 8, 128), np.float16)
    Vb = np.zeros_like(Kb)
    Kb[0, :640], Vb[0, :640] = K1[:640], V1[:640]
    Kb[1], Vb[1] = K1[600:1300], V1[600:1300]
    c.cache.append(torch.from_numpy(Kb).cuda(), torch.from_numpy(Vb).cuda(), [640, 700])
    torch.cuda.synchronize()
    c.cache.check()
    assert c.cache.seq_len(0) == 640 and c.cache.seq_len(1) == 1300 and c.cache.free_pages() == 1
    for s, L in ((0, 640), (1, 1300)):
        for h in (0, 7):
            ref = oracle.build_head(K1[:L, h, :], V1[:L, h, :], 1, 1, 32, 32, 0)
            assert (c.cache.export(s, h) == ref).all(), (s, h)
    out = c.decode()
    ref0 = oracle.decode_seq(c.q[0], K1[:640], V1[:640], 1, 1, 32, 32, 0)
    assert row_rel_err(out[0], ref0).max() <= ATTN_TOL
    assert row_rel_err(out[1], c.oracle_out(1)).max() <= ATTN_TOL


@pytest.mark.parametrize("n_q", [24, 7])   # three 32-row groups; one with a spare query (odd n_q)
def test_chunk_attention_over_pages(n_q):
    from paper_2607_16248_amd import kvq
    w = W("chunk_paged", 2, 32, 8, (1200, 777), 1, 1)
    c = Case(w, page_tokens=64)
    c.append_all([100, 1100])
    q = np.stack([gen_q_chunk(w, n_q, 0, s) for s in range(w.batch)])
    out = torch.empty((2, n_q, 32, 128), dtype=torch.float32, device="cuda")
    ws = torch.empty(kvq.kvq_chunk_workspace_bytes(c.cache.handle, n_q), dtype=torch.uint8, device="cuda")
    kvq.kvq_chunk_attention(c.cache.handle, torch.from_numpy(q).cuda(), n_q, out, ws)
    got = out.cpu().numpy()
    for s in range(2):
        ref = oracle.chunk_seq(q[s], c.K[s], c.V[s], 1, 1, 32, 32, 0)
        assert row_rel_err(got[s], ref).max() <= ATTN_TOL, s


def test_append_decode_steps_on_pages():
    """Token-by-token kvq_append_decode over a paged and a contiguous cache:
    70 steps cross two key-group flushes (pages taken mid-stream); outputs
    bit-identical at every step, bytes equal to the oracle at the end."""
    from paper_2607_16248_amd import kvq
    w = W("steps_paged", 2, 32, 8, (400, 400), 1, 1)
    paged, flat = Case(w, page_tokens=64), Case(w)
    for c in (paged, flat):
        K = np.stack([c.K[s][:300] for s in range(2)])
        V = np.stack([c.V[s][:300] for s in range(2)])
        c.cache.append(torch.from_numpy(K).cuda(), torch.from_numpy(V).cuda(), [300, 300])
    q = torch.from_numpy(np.stack(paged.q)).cuda()
    for t in range(300, 370):
        outs = []
        for c in (paged, flat):
            Kn = torch.from_numpy(np.stack([c.K[s][t:t + 1] for s in range(2)])).cuda()
            Vn = torch.from_numpy(np.stack([c.V[s][t:t + 1] for s in range(2)])).cuda()
            o = torch.empty((2, 32, 128), dtype=torch.float32, device="cuda")
            kvq.kvq_append_decode(c.cache.handle, Kn, Vn, [1, 1], q, o, c.cache.workspace())
            outs.append(o)
        torch.cuda.synchronize()
        assert torch.equal(outs[0], outs[1]), t
    paged.cache.check()
    for s in range(2):
        for h in (0, 3):
            ref = oracle.build_head(paged.K[s][:370, h, :], paged.V[s][:370, h, :], 1, 1, 32, 32, 0)
            assert (paged.cache.export(s, h) == ref).all(), (s, h)


@pytest.mark.parametrize("bk,bv,hq", [(1, 1, 32), (2, 2, 40), (4, 4, 32)])
def test_split_spanning_more_than_64_pages(bk, bv, hq):
    """One split per head over 32-token pages: a split of 5000 tokens spans
    157 pages, so every block past the split's first 64 pages takes its page
    from the block table itself (the matrix kernel keeps only the first 64
    page offsets in lanes).  Decode and chunk outputs bit-identical to a
    contiguous cache with the same split, and within 2e-3 of the oracle."""
    from paper_2607_16248_amd import kvq
    w = W(f"long_split_k{bk}v{bv}", 2, hq, 8, (5000, 4200), bk, bv)
    paged, flat = Case(w, page_tokens=32), Case(w)
    paged.append_all([1000, 4000])
    flat.append_all()
    paged.cache.check()
    for c in (paged, flat):
        kvq.kvq_set_split_tokens(c.cache.handle, 5024)
    a, b = paged.decode(), flat.decode()
    assert (a.view(np.uint32) == b.view(np.uint32)).all()
    for s in range(2):
        ref = paged.oracle_out(s, heads=[0, 5])
        gq = hq // 8
        rows = list(range(0, gq)) + list(range(5 * gq, 6 * gq))
        assert row_rel_err(a[s][rows], ref[rows]).max() <= ATTN_TOL, s
    n_q = 8
    q = torch.from_numpy(np.stack([gen_q_chunk(w, n_q, 0, s) for s in range(2)])).cuda()
    outs = []
    for c in (paged, flat):
        o = torch.empty((2, n_q, hq, 128), dtype=torch.float32, device="cuda")
        ws = torch.empty(kvq.kvq_chunk_workspace_bytes(c.cache.handle, n_q), dtype=torch.uint8, device="cuda")
        kvq.kvq_chunk_attention(c.cache.handle, q, n_q, o, ws)
        outs.append(o)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


def test_pool_larger_than_4_GiB():
    """A paged pool of 9.7 GB (K8V8, 4096-token pages of 9.4 MB): sequence 0
    fills 464 pages (4.4 GB), so every page of sequence 1 starts beyond
    4 GiB of the pool.  The matrix kernel addresses each page through a
    resource of its own: outputs bit-identical to a contiguous cache (the
    vector kernel would round differently), and sequence 1 within 2e-3 of
    the oracle."""
    from paper_2607_16248_amd import kvq
    L0, L1, cap, P = 464 * 4096, 6000, 1 << 21, 4096
    w = W("pool_over_4GiB", 2, 32, 8, (L0, L1), 8, 8, cfg=95)
    K1, V1 = gen_kv(w, 0, 1)                       # host draw of sequence 1 only
    q = np.stack([gen_q(w, 0, s) for s in range(2)])
    caches = [kvq.KVCache(2, 32, 8, cap, [8, 8], [8, 8], key_group=32, value_group=32, device="cuda",
                          page_tokens=P),
              kvq.KVCache(2, 32, 8, cap, [8, 8], [8, 8], key_group=32, value_group=32, device="cuda")]
    assert caches[0].arena.numel() > (9 << 30)
    g = torch.Generator(device="cuda").manual_seed(4242)
    step = 131072
    for t0 in range(0, L0, step):                  # sequence 0: device draws, same rows into both caches
        n = min(step, L0 - t0)
        K = torch.randn((1, n, 8, 128), generator=g, device="cuda").half()
        V = torch.randn((1, n, 8, 128), generator=g, device="cuda").half()
        Kb = torch.cat([K, torch.zeros_like(K)]), torch.cat([V, torch.zeros_like(V)])
        for c in caches:
            c.append(Kb[0], Kb[1], [n, 0])
        del K, V, Kb
    Kb = torch.from_numpy(K1[None]).cuda()
    Vb = torch.from_numpy(V1[None]).cuda()
    zk = torch.zeros_like(Kb)
    for c in caches:
        c.append(torch.cat([zk, Kb]), torch.cat([zk, Vb]), [0, L1])
    torch.cuda.synchronize()
    for c in caches:
        c.check()
    qd = torch.from_numpy(q).cuda()
    a = caches[0].decode(qd).cpu().numpy()
    b = caches[1].decode(qd).cpu().numpy()
    assert (a.view(np.uint32) == b.view(np.uint32)).all()
    for h in (0, 7):
        assert (caches[0].export(1, h) == oracle.build_head(K1[:, h], V1[:, h], 8, 8, 32, 32, 0)).all(), h
    ref = oracle.decode_seq(q[1], K1, V1, 8, 8, 32, 32, 0)
    err = row_rel_err(a[1], ref).max()
    log(f"[paged] pool of {caches[0].arena.numel() / 2**30:.1f} GiB, sequence 1 beyond 4 GiB: "
        f"max row-relative error {err:.3e}")
    assert err <= ATTN_TOL
    del caches
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
