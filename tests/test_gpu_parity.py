"""GPU parity: the HIP library against the CPU oracle, through the C ABI.

- packed codes, scales, zeros and fp16 tail: byte-identical to the oracle's
  canonical image (kvq_export), after one-shot and piecewise appends;
- kvq_dequant: bit-identical to the oracle's exact value rounded to fp32;
- decode attention: row-normwise relative error <= 2e-3 against the fp64
  oracle on the same (byte-identical) cache;
- properties: split-count independence, bitwise determinism, empty and
  single-token sequences, ragged batches with mixed bit widths, the device
  error flag.
"""
import numpy as np
import pytest

import oracle
from helpers import ATTN_TOL, Case, log, row_rel_err
from workloads import Workload, workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def W(name, batch, hq, hkv, lens, bk, bv, gk=32, gv=32, R=0, dist="normal", cfg=90):
    if isinstance(lens, int):
        lens = (lens,) * batch
    if isinstance(bk, int):
        bk = (bk,) * batch
    if isinstance(bv, int):
        bv = (bv,) * batch
    return Workload(name, batch, hq, hkv, 128, tuple(lens), tuple(bk), tuple(bv), gk, gv, R,
                    key_dist=dist, cfg_id=cfg)


SMALL = [
    W("k2v2_g32_L1000", 1, 32, 8, 1000, 2, 2),
    W("k1v1_g32_L2048", 1, 32, 8, 2048, 1, 1),
    W("k4v4_g32_L1111", 1, 32, 8, 1111, 4, 4),
    W("k8v8_g32_L777", 1, 32, 8, 777, 8, 8),
    W("k2v1_g32_L999", 1, 32, 8, 999, 2, 1),
    W("k1v2_g32_L999", 1, 32, 8, 999, 1, 2),
    W("k4v8_g64_gv8_L1300", 1, 16, 4, 1300, 4, 8, gk=64, gv=8),
    W("k1v4_g128_gv128_L1500", 1, 8, 8, 1500, 1, 4, gk=128, gv=128),
    W("gq5_k2v2_R128_t3", 2, 40, 8, (1000, 517), 2, 2, R=128, dist="student_t3"),
    W("gq2_k1v1_R40", 1, 16, 8, 333, 1, 1, R=40),
    W("gq8_k8v8_gv16", 1, 64, 8, 600, 8, 8, gv=16),
    W("ragged_mixed", 4, 32, 8, (900, 64, 31, 1500), (2, 2, 4, 4), (2, 2, 4, 4), gk=64),
    W("window_bigger_than_L", 1, 32, 8, 100, 1, 1, R=300),
    W("k1v1_g128_L1100", 1, 32, 8, 1100, 1, 1, gk=128),
    W("mixed_asym_g64_gv64", 4, 32, 8, (700, 1300, 520, 64), (1, 2, 1, 2), (2, 1, 1, 2), gk=64, gv=64),
    W("gq5_k4v4_R128_t3", 2, 40, 8, (1000, 517), 4, 4, R=128, dist="student_t3"),
    W("gq5_k8v8_R128_t3", 2, 40, 8, (1200, 300), 8, 8, R=128, dist="student_t3"),
    W("gq8_k4v4_g128", 1, 64, 8, 1500, 4, 4, gk=128),
    W("k8v8_g64_gv64_L2000", 1, 32, 8, 2000, 8, 8, gk=64, gv=64),
    # 4- and 8-bit keys and values of different widths on the matrix cores
    W("k4v8_gq4_L1300", 1, 32, 8, 1300, 4, 8),
    W("k8v4_gq5_g64_R40", 2, 40, 8, (900, 1100), 8, 4, gk=64, R=40),
    W("gq8_k4v8_gv64", 1, 64, 8, 700, 4, 8, gv=64),
    # five and eight heads at 1-4 bits (one value accumulator per tile) with
    # value groups of 64 and 128 channels
    W("gq5_k1v1_gv64_R40", 2, 40, 8, (1100, 600), 1, 1, gv=64, R=40),
    W("gq5_k2v2_gv128_g128", 1, 40, 8, 1300, 2, 2, gk=128, gv=128),
    W("gq8_k2v2_gv64", 1, 64, 8, 900, 2, 2, gv=64),
    W("gq8_k4v4_gv128_g64", 1, 64, 8, 800, 4, 4, gk=64, gv=128),
    # one or two query heads per kv head on the matrix cores (key groups of
    # 32, 64 and 128 tokens)
    W("gq1_k2v1_L700", 1, 8, 8, 700, 2, 1),
    W("gq2_k1v2_R40_t3", 2, 16, 8, (900, 333), 1, 2, R=40, dist="student_t3"),
    W("gq1_k4v8_L600", 1, 8, 8, 600, 4, 8),
    W("gq1_k1v1_g64_L1100", 1, 8, 8, 1100, 1, 1, gk=64),
    W("gq2_k2v2_g128_R40", 2, 16, 8, (1500, 700), 2, 2, gk=128, R=40),
    W("gq2_k8v4_g64_L900", 1, 16, 8, 900, 8, 4, gk=64),
]


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_bytes_and_attention_match_oracle(w):
    log(f"[parity] {w.name}: append")
    c = Case(w)
    c.append_all()
    c.cache.check()
    for s in range(w.batch):
        for h in range(w.num_kv_heads):
            got = c.cache.export(s, h)
            ref = c.oracle_image(s, h)
            assert got.size == ref.size, (s, h)
            bad = np.flatnonzero(got != ref)
            assert bad.size == 0, f"seq {s} head {h}: {bad.size} bytes differ, first at {bad[:5]}"
    log(f"[parity] {w.name}: decode")
    out = c.decode()
    worst = 0.0
    for s in range(w.batch):
        ref = c.oracle_out(s)
        err = row_rel_err(out[s], ref)
        worst = max(worst, float(err.max()))
        assert err.max() <= ATTN_TOL, (s, err.max())
    log(f"[parity] {w.name}: max row-relative error {worst:.3e}")


@pytest.mark.parametrize("chunks", [
    [1] * 70,                        # token by token across two key-group flushes
    [5, 31, 32, 33, 64, 1, 100],     # ragged chunks crossing group edges
    [300],                           # prefill larger than ring + window
])
def test_piecewise_appends_give_the_same_bytes(chunks):
    L = sum(chunks)
    w = W(f"pieces_{L}", 2, 32, 8, (L, max(1, L - 7)), 2, 2, R=40)
    c = Case(w)
    log(f"[append] chunks {chunks[:8]}...")
    c.append_all(chunks)
    c.cache.check()
    for s in range(2):
        for h in (0, 5):
            assert (c.cache.export(s, h) == c.oracle_image(s, h)).all(), (s, h)
    out = c.decode()
    for s in range(2):
        assert row_rel_err(out[s], c.oracle_out(s)).max() <= ATTN_TOL


def test_dequant_is_bit_exact():
    w = W("dq", 2, 32, 8, (700, 450), (1, 4), (2, 8), gk=64, gv=16, R=50)
    c = Case(w)
    c.append_all()
    for s in range(2):
        L = w.lens[s]
        Kd, Vd = c.cache.dequant(s, 0, L)
        Kd, Vd = Kd.cpu().numpy(), Vd.cpu().numpy()
        for h in range(w.num_kv_heads):
            Kh, Vh = oracle.dequant_head(c.oracle_image(s, h), L, 128, w.bits_k[s], w.bits_v[s],
                                         w.key_group, w.value_group, w.window)
            assert (Kd[:, h].view(np.uint32) == Kh.astype(np.float32).view(np.uint32)).all(), (s, h)
            assert (Vd[:, h].view(np.uint32) == Vh.astype(np.float32).view(np.uint32)).all(), (s, h)
        # a sub-range starting mid-group
        Kd2, _ = c.cache.dequant(s, 37, 100)
        assert (Kd2.cpu().numpy() == Kd[37:137]).all()


def test_split_independence_and_determinism():
    w = W("splits", 1, 32, 8, 4100, 2, 2, R=3)
    c = Case(w)
    c.append_all()
    ref = c.oracle_out(0)
    outs = {}
    # 129, 65, 33, 17, 5 and 2 records per head: the merge loads 17, 17, 8,
    # 4, 4 and 4 records per round trip
    for st in (32, 64, 128, 256, 1024, 4096, 0):
        kvq_set = __import__("paper_2607_16248_amd").kvq_set_split_tokens
        kvq_set(c.cache.handle, st)
        a = c.decode()
        b = c.decode()
        assert (a.view(np.uint32) == b.view(np.uint32)).all(), st     # bitwise reproducible
        assert row_rel_err(a[0], ref).max() <= ATTN_TOL, st
        outs[st] = a
    for st, a in outs.items():
        assert row_rel_err(a[0], outs[128][0].astype(np.float64)).max() <= ATTN_TOL


@pytest.mark.parametrize("bits", [1, 2])
def test_short_sequence_split_plan(bits):
    # 8192 packed tokens of 8 kv heads: the plan takes two blocks per wave
    # (256-token splits, 32 per head) instead of one; the same outputs as
    # 128-token splits within the tolerance, and the oracle's
    w = W(f"short8k_k{bits}", 1, 32, 8, 8192 + 37, bits, bits, R=37)
    c = Case(w)
    c.append_all()
    a = c.decode()
    kvq_set = __import__("paper_2607_16248_amd").kvq_set_split_tokens
    kvq_set(c.cache.handle, 128)
    b = c.decode()
    ref = c.oracle_out(0)
    for out in (a, b):
        assert row_rel_err(out[0], ref).max() <= ATTN_TOL
    log(f"[parity] {w.name}: default plan {row_rel_err(a[0], ref).max():.3e}, 128-token splits "
        f"{row_rel_err(b[0], ref).max():.3e}")


@pytest.mark.parametrize("L,st,n", [(4096, 128, 32), (4224, 128, 33), (4096, 64, 64), (4160, 64, 65), (4608, 64, 72),
                                     (4352, 32, 136), (4384, 32, 137)])
def test_merge_at_its_load_counts(L, st, n):
    # 32, 33, 64, 65, 72 and 136 records per head (round trips of 4, 5, 8, 9,
    # 9 and 17 loads per thread) and 137 (two rounds of 17)
    w = W(f"merge_n{n}", 1, 32, 8, L, 1, 1)
    c = Case(w)
    c.append_all()
    kvq_set = __import__("paper_2607_16248_amd").kvq_set_split_tokens
    kvq_set(c.cache.handle, st)
    assert -(-L // st) == n
    a = c.decode()
    b = c.decode()
    assert (a.view(np.uint32) == b.view(np.uint32)).all()
    err = row_rel_err(a[0], c.oracle_out(0)).max()
    log(f"[parity] {n} records per head: max row-relative error {err:.3e}")
    assert err <= ATTN_TOL


@pytest.mark.parametrize("gk,bk,bv", [(32, 1, 1), (64, 2, 1), (128, 1, 2), (32, 8, 8), (64, 4, 4)])
def test_long_splits(gk, bk, bv):
    # One split per head: every wave of the matrix kernel takes more than
    # 48 blocks, so the per-wave zero-point table is refilled (and each fill
    # covers more than 16 key groups); a 3-token fp16 tail rides along.
    w = W(f"long_split_g{gk}_k{bk}v{bv}", 1, 32, 8, 6400 + 3 * gk + 3, bk, bv, gk=gk)
    c = Case(w)
    c.append_all()
    kvq_set = __import__("paper_2607_16248_amd").kvq_set_split_tokens
    kvq_set(c.cache.handle, (w.lens[0] // gk + 1) * gk)
    out = c.decode()
    err = row_rel_err(out[0], c.oracle_out(0)).max()
    log(f"[parity] {w.name}: max row-relative error {err:.3e}")
    assert err <= ATTN_TOL


def test_empty_and_single_token_sequences():
    w = W("tiny", 3, 32, 8, (0, 1, 40), 1, 1)
    c = Case(w)
    c.append_all()
    out = c.decode()
    assert (out[0] == 0).all()                          # no tokens: zeros
    gq = 4
    for h in range(32):                                 # one fp16 token: its value row, exactly
        assert (out[1, h] == c.V[1][0, h // gq].astype(np.float32)).all()
    assert row_rel_err(out[2], c.oracle_out(2)).max() <= ATTN_TOL


def test_range_flag_is_sticky_until_reset():
    from paper_2607_16248_amd import KvqError
    from paper_2607_16248_amd.kvq import ERR_RANGE
    cache = __import__("paper_2607_16248_amd").KVCache(1, 8, 8, 64, [1], [1])
    K = torch.zeros((1, 32, 8, 128), dtype=torch.float16, device="cuda")
    K[0, 0, 3, 7] = 65504.0
    K[0, 1, 3, 7] = -65504.0                            # range 131008 > largest fp16 at one bit
    V = torch.zeros_like(K)
    cache.append(K, V)
    with pytest.raises(KvqError) as e:
        cache.check()
    assert e.value.status == ERR_RANGE
    cache.reset()
    cache.check()
    assert cache.seq_len(0) == 0


# ------------------------------------------------ full-size workloads (sampled)

def _sampled_parity(w, samples, layer=0):
    heads = sorted({h for _, h in samples})
    log(f"[full] {w.name}: generate heads {heads}")
    c = Case(w, layer=layer, heads=heads)
    log(f"[full] {w.name}: append")
    c.append_all()
    c.cache.check()
    log(f"[full] {w.name}: decode")
    out = c.decode()
    gq = w.group_q
    for s, h in samples:
        assert (c.cache.export(s, h) == c.oracle_image(s, h)).all(), (s, h)
        ref = c.oracle_out(s, heads=[h])
        err = row_rel_err(out[s, h * gq:(h + 1) * gq], ref[h * gq:(h + 1) * gq])
        log(f"[full] {w.name}: seq {s} head {h} max row-relative error {err.max():.3e}")
        assert err.max() <= ATTN_TOL


def test_full_workload_0_all_heads():
    w = workload(0)
    _sampled_parity(w, [(0, h) for h in range(8)])


def test_full_workload_1_all_heads():
    w = workload(1)
    _sampled_parity(w, [(0, h) for h in range(8)])


def test_full_workload_2_one_layer():
    w = workload(2)
    _sampled_parity(w, [(0, 0), (0, 5)], layer=7)


def test_full_workload_3_sampled():
    w = workload(3)
    _sampled_parity(w, [(2, 1), (13, 6)])


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_full_workload_4_sampled(bits):
    w = workload(4, bits)
    _sampled_parity(w, [(0, 3), (3, 6)])


FUSED = [
    W("fused_k1v1_matrix", 2, 32, 8, (300, 45), 1, 1),
    W("fused_gq5_k2v2_R128", 2, 40, 8, (200, 31), 2, 2, R=128, dist="student_t3"),
    W("fused_mixed_g64", 3, 32, 8, (130, 64, 0), (1, 2, 4), (1, 2, 4), gk=64),
]


@pytest.mark.parametrize("w", FUSED, ids=[w.name for w in FUSED])
def test_append_decode_matches_separate_calls(w):
    """kvq_append_decode gives the bytes, lengths and outputs of kvq_append
    followed by kvq_decode_attention, bit for bit, across key-group flushes."""
    import torch
    steps = 40
    a = Case(w, max_tokens=max(w.lens) + 2 * steps + 2)
    b = Case(w, max_tokens=max(w.lens) + 2 * steps + 2)
    a.append_all()
    b.append_all()
    rng = np.random.default_rng(7)
    for st in range(steps):
        n_new = [int(x) for x in rng.integers(0, 3, size=w.batch)]
        if st % 5 == 0:
            n_new = [1] * w.batch
        nmax = max(max(n_new), 1)
        Kn = torch.from_numpy(rng.standard_normal((w.batch, nmax, w.num_kv_heads, 128)).astype(np.float16)).cuda()
        Vn = torch.from_numpy(rng.standard_normal((w.batch, nmax, w.num_kv_heads, 128)).astype(np.float16)).cuda()
        out_a = a.cache.append_decode(Kn, Vn, a.qd, n_new=n_new)
        b.cache.append(Kn, Vn, n_new)
        out_b = b.cache.decode(b.qd)
        torch.cuda.synchronize()
        assert [a.cache.seq_len(s) for s in range(w.batch)] == [b.cache.seq_len(s) for s in range(w.batch)]
        assert torch.equal(out_a, out_b), (w.name, st, n_new)
    a.cache.check()
    for s in range(w.batch):
        for h in range(w.num_kv_heads):
            assert np.array_equal(a.cache.export(s, h), b.cache.export(s, h)), (w.name, s, h)
    log(f"[fused] {w.name}: {steps} steps bit-identical to separate append + decode")


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
@pytest.mark.parametrize("scale", [1e-1, 1e-3, 1e-5])
def test_small_value_scales(bits, scale):
    # values drawn N(0, scale^2): their fp16 scales (range / (2^b - 1)) reach
    # the fp16 subnormal range; the weight shift sized by the head's bound on
    # the value scales keeps p * s_v normal
    w = W(f"vscale_{scale:g}_k{bits}", 1, 32, 8, 3000, bits, bits, R=5, cfg=96)
    c = Case(w)
    c.V = [(v.astype(np.float32) * scale).astype(np.float16) for v in c.V]
    c.append_all()
    out = c.decode()
    err = row_rel_err(out[0], c.oracle_out(0)).max()
    log(f"[parity] value scale {scale:g}, K{bits}V{bits}: max row-relative error {err:.3e}")
    assert err <= ATTN_TOL


@pytest.mark.parametrize("how", ["reset", "release"])
def test_value_bound_starts_fresh(how):
    # A sequence packed with values of scale ~1e4 (a value-scale bound near
    # 2^15: no weight shift), then emptied and refilled with values of scale
    # ~1e-5: the refill must start a fresh bound, since with the stale one the
    # shift stays 0 and p * s_v of the small values (value scales ~1e-4) is
    # below the fp16 normal range.
    w = W("vbound_fresh_k1", 1, 32, 8, 3000, 1, 1, R=5, cfg=96)
    kw = {"page_tokens": 256, "num_pages": 16} if how == "release" else {}
    c = Case(w, **kw)
    V0 = c.V
    c.V = [(v.astype(np.float32) * 3000.0).astype(np.float16) for v in V0]
    c.append_all()
    if how == "reset":
        c.cache.reset()
    else:
        c.cache.release(0)
    c.V = [(v.astype(np.float32) * 1e-5).astype(np.float16) for v in V0]
    c.append_all()
    out = c.decode()
    err = row_rel_err(out[0], c.oracle_out(0)).max()
    log(f"[parity] value bound after {how}: max row-relative error {err:.3e}")
    assert err <= ATTN_TOL
