"""Host-side tests of the C-ABI library (no GPU needed).

The library loads, exports every function include/*.h declares, sizes its
arena as documented, and rejects bad arguments before touching any device
memory, leaving the cache unchanged.
"""
import os
import re

import pytest

from paper_2607_16248_amd import kvq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE_ARENA = 1 << 30   # a 256-aligned address that is never dereferenced on these paths


def declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b((?:kvq|dgap)_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = kvq.lib()
    names = declared_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(kvq.EXPORTED)
    assert "gfx950" in kvq.kvq_version()


def align(x, a=256):
    return (x + a - 1) // a * a


def expected_bytes(batch, hkv, max_tokens, gk, gv, R, bits_k, bits_v):
    """Arena size from the documented region list, written out independently."""
    cq = max(0, max_tokens - R) // gk * gk
    W = R + gk
    total = 256
    for bk, bv in zip(bits_k, bits_v):
        per_head = (align(cq * 16 * bk) + align(cq // gk * 512) + align(cq * 16 * bv)
                    + align(cq * (128 // gv) * 4) + 2 * align(W * 256) + align(4))  # + value-scale bound
        total += hkv * per_head
    return total


@pytest.mark.parametrize("args", [
    (1, 32, 8, 4096, 32, 32, 0, [2], [2]),
    (1, 32, 8, 131072, 32, 32, 0, [1], [1]),
    (16, 32, 8, 32768, 64, 32, 0, [2] * 8 + [4] * 8, [2] * 8 + [4] * 8),
    (4, 40, 8, 131072, 32, 32, 128, [8] * 4, [8] * 4),
    (3, 8, 8, 100, 128, 8, 300, [1, 2, 4], [8, 4, 1]),
])
def test_cache_bytes(args):
    b, hq, hkv, L, gk, gv, R, bk, bv = args
    d = kvq.make_desc(b, hq, hkv, 128, L, gk, gv, R, bk, bv)
    assert kvq.kvq_cache_bytes(d) == expected_bytes(b, hkv, L, gk, gv, R, bk, bv)


BAD = [
    (dict(batch=0), kvq.ERR_ARG),
    (dict(num_kv_heads=0), kvq.ERR_ARG),
    (dict(num_q_heads=12), kvq.ERR_ARG),          # not a multiple of 8
    (dict(num_q_heads=24), kvq.ERR_UNSUPPORTED),  # 3 query heads per kv head
    (dict(head_dim=64), kvq.ERR_UNSUPPORTED),
    (dict(head_dim=0), kvq.ERR_ARG),
    (dict(max_tokens=0), kvq.ERR_ARG),
    (dict(key_group=16), kvq.ERR_ARG),
    (dict(key_group=48), kvq.ERR_ARG),
    (dict(value_group=24), kvq.ERR_ARG),
    (dict(fp16_window=-1), kvq.ERR_ARG),
    (dict(bits_k=[3]), kvq.ERR_ARG),
    (dict(bits_v=[0]), kvq.ERR_ARG),
]


def desc(**kw):
    p = dict(batch=1, num_q_heads=32, num_kv_heads=8, head_dim=128, max_tokens=4096, key_group=32,
             value_group=32, fp16_window=0, bits_k=[2], bits_v=[2])
    p.update(kw)
    return kvq.make_desc(**p)


@pytest.mark.parametrize("kw,status", BAD)
def test_invalid_descriptors(kw, status):
    d = desc(**kw)
    assert kvq.kvq_cache_bytes(d) == 0
    with pytest.raises(kvq.KvqError) as e:
        kvq.kvq_cache_init(d, FAKE_ARENA, 1 << 40)
    assert e.value.status == status
    assert kvq.kvq_last_error() != ""


def test_init_checks_arena():
    d = desc()
    n = kvq.kvq_cache_bytes(d)
    with pytest.raises(kvq.KvqError) as e:
        kvq.kvq_cache_init(d, FAKE_ARENA, n - 1)
    assert e.value.status == kvq.ERR_CAPACITY
    with pytest.raises(kvq.KvqError) as e:
        kvq.kvq_cache_init(d, FAKE_ARENA + 16, n)
    assert e.value.status == kvq.ERR_ARG
    with pytest.raises(kvq.KvqError) as e:
        kvq.kvq_cache_init(d, None, n)
    assert e.value.status == kvq.ERR_ARG
    h = kvq.kvq_cache_init(d, FAKE_ARENA, n)
    assert kvq.kvq_last_error() == ""
    kvq.kvq_cache_destroy(h)


def test_append_errors_leave_cache_unchanged():
    d = desc(batch=2, bits_k=[1, 4], bits_v=[1, 4], max_tokens=100)
    h = kvq.kvq_cache_init(d, FAKE_ARENA, kvq.kvq_cache_bytes(d))
    try:
        for n_new, n_max, status in [([101, 0], 200, kvq.ERR_CAPACITY), ([5, -1], 10, kvq.ERR_ARG),
                                     ([11, 0], 10, kvq.ERR_ARG), ([0, 0], -1, kvq.ERR_ARG)]:
            with pytest.raises(kvq.KvqError) as e:
                kvq.kvq_append(h, FAKE_ARENA, FAKE_ARENA, n_new, n_max=n_max)
            assert e.value.status == status
            assert kvq.kvq_seq_len(h, 0) == 0 and kvq.kvq_seq_len(h, 1) == 0
        # nothing to append: a no-op that launches nothing
        kvq.kvq_append(h, None, None, [0, 0], n_max=0)
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_append(h, None, None, [1, 0], n_max=1)
        assert e.value.status == kvq.ERR_ARG
        assert kvq.kvq_seq_len(h, 2) == -1 and kvq.kvq_seq_len(h, -1) == -1
    finally:
        kvq.kvq_cache_destroy(h)


def test_append_decode_errors_leave_cache_unchanged():
    """Every check of the fused append + decode precedes any launch."""
    d = desc(batch=2, bits_k=[1, 4], bits_v=[1, 4], max_tokens=100)
    h = kvq.kvq_cache_init(d, FAKE_ARENA, kvq.kvq_cache_bytes(d))
    F = FAKE_ARENA
    try:
        cases = [
            (dict(K=F, V=F, n_new=[101, 0], n_max=200), kvq.ERR_CAPACITY),
            (dict(K=F, V=F, n_new=[11, 0], n_max=10), kvq.ERR_ARG),
            (dict(K=F, V=F, n_new=[1, 0], n_max=1, q=None), kvq.ERR_ARG),
            (dict(K=None, V=F, n_new=[1, 0], n_max=1), kvq.ERR_ARG),
            (dict(K=F + 2, V=F, n_new=[1, 0], n_max=1), kvq.ERR_ARG),
            (dict(K=F, V=F, n_new=[5, 3], n_max=5, ws_bytes=16), kvq.ERR_CAPACITY),
            (dict(K=F, V=F, n_new=[5, 3], n_max=5, ws=F + 8, ws_bytes=1 << 20), kvq.ERR_ARG),
        ]
        for kw, status in cases:
            args = dict(q=F, out=F, ws=F, ws_bytes=1 << 20)
            args.update(kw)
            with pytest.raises(kvq.KvqError) as e:
                kvq.kvq_append_decode(h, args["K"], args["V"], args["n_new"], args["q"], args["out"], args["ws"],
                                      ws_bytes=args["ws_bytes"], n_max=args["n_max"])
            assert e.value.status == status, kw
            assert kvq.kvq_seq_len(h, 0) == 0 and kvq.kvq_seq_len(h, 1) == 0, kw
    finally:
        kvq.kvq_cache_destroy(h)


def test_split_setting_and_workspace_bound():
    d = desc(max_tokens=131072, bits_k=[1], bits_v=[1])
    h = kvq.kvq_cache_init(d, FAKE_ARENA, kvq.kvq_cache_bytes(d))
    try:
        rec = 132 * 4
        # automatic: at most 512 packed splits (and >= 4 key groups each) + one tail split
        assert kvq.kvq_workspace_bytes(h) == 32 * (min(512, 131072 // 128) + 1) * rec
        kvq.kvq_set_split_tokens(h, 1024)
        assert kvq.kvq_workspace_bytes(h) == 32 * (128 + 1) * rec
        for bad in (-32, 33, 100, 128):
            with pytest.raises(kvq.KvqError) as e:
                kvq.kvq_set_split_tokens(h, bad)
            assert e.value.status == kvq.ERR_ARG
        kvq.kvq_set_split_tokens(h, 0)
        # an empty cache exports nothing
        assert kvq.kvq_export_bytes(h, 0, 0) == 0
        assert kvq.kvq_export_bytes(h, 0, 8) == 0 and kvq.kvq_export_bytes(h, 1, 0) == 0
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_dequant(h, 0, 0, 1, FAKE_ARENA, FAKE_ARENA)
        assert e.value.status == kvq.ERR_ARG
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_decode_attention(h, None, None, None)
        assert e.value.status == kvq.ERR_ARG
    finally:
        kvq.kvq_cache_destroy(h)


@pytest.mark.parametrize("kw,status", [
    (dict(page_tokens=48), "ARG"),                         # not a power of two
    (dict(page_tokens=16), "ARG"),                         # below key_group
    (dict(page_tokens=-64), "ARG"),
    (dict(num_pages=4), "ARG"),                            # a pool without pages
    (dict(page_tokens=64, num_pages=-1), "ARG"),
    (dict(page_tokens=64, batch=2, bits_k=[1, 2], bits_v=[1, 2]), "UNSUPPORTED"),
])
def test_paged_descriptor_errors(kw, status):
    d = desc(**kw)
    assert kvq.kvq_cache_bytes(d) == 0
    with pytest.raises(kvq.KvqError) as e:
        kvq.kvq_cache_init(d, FAKE_ARENA, 1 << 30)
    assert e.value.status == getattr(kvq, "ERR_" + status)


def test_paged_pool_size_and_capacity_errors():
    # K1V1, 8 kv heads, pages of 256 tokens: 4 KiB of codes, 4 KiB of key
    # scales, 4 KiB of value codes and 4 KiB of value scales per head
    base = desc(max_tokens=4096, bits_k=[1], bits_v=[1], page_tokens=256, num_pages=3)
    more = desc(max_tokens=4096, bits_k=[1], bits_v=[1], page_tokens=256, num_pages=4)
    assert kvq.kvq_cache_bytes(more) - kvq.kvq_cache_bytes(base) == 8 * 4 * 4096
    full = desc(max_tokens=4096, bits_k=[1], bits_v=[1], page_tokens=256)
    assert kvq.kvq_cache_bytes(full) - kvq.kvq_cache_bytes(base) == 13 * 8 * 4 * 4096   # 16 pages by default
    h = kvq.kvq_cache_init(base, FAKE_ARENA, kvq.kvq_cache_bytes(base))
    try:
        assert kvq.kvq_free_pages(h) == 3
        # 1000 tokens pack 992 (31 key groups): 4 pages, one more than the pool
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_append(h, FAKE_ARENA, FAKE_ARENA, [1000], n_max=1000)
        assert e.value.status == kvq.ERR_CAPACITY and "pages" in kvq.kvq_last_error()
        assert kvq.kvq_seq_len(h, 0) == 0 and kvq.kvq_free_pages(h) == 3
        kvq.kvq_seq_release(h, 0)
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_seq_release(h, 1)
        assert e.value.status == kvq.ERR_ARG
    finally:
        kvq.kvq_cache_destroy(h)
    c = kvq.kvq_cache_init(desc(), FAKE_ARENA, kvq.kvq_cache_bytes(desc()))
    assert kvq.kvq_free_pages(c) == -1
    kvq.kvq_cache_destroy(c)


def test_chunk_attention_sizes_and_argument_errors():
    """Every check of kvq_chunk_attention precedes any launch."""
    d = desc(max_tokens=4096, bits_k=[1], bits_v=[1])
    h = kvq.kvq_cache_init(d, FAKE_ARENA, kvq.kvq_cache_bytes(d))
    F = FAKE_ARENA
    try:
        one = kvq.kvq_workspace_bytes(h)
        assert kvq.kvq_chunk_workspace_bytes(h, 1) == one
        assert kvq.kvq_chunk_workspace_bytes(h, 16) == 16 * one
        assert kvq.kvq_chunk_workspace_bytes(h, 1024) == 1024 * one
        assert kvq.kvq_chunk_workspace_bytes(h, 0) == 0 and kvq.kvq_chunk_workspace_bytes(h, 1025) == 0
        for n_q, q, out in [(0, F, F), (1025, F, F), (1, None, F), (1, F, None)]:
            with pytest.raises(kvq.KvqError) as e:
                kvq.kvq_chunk_attention(h, q, n_q, out, F, ws_bytes=1 << 30)
            assert e.value.status == kvq.ERR_ARG, (n_q, q, out)
        # an empty sequence holds fewer tokens than any chunk
        with pytest.raises(kvq.KvqError) as e:
            kvq.kvq_chunk_attention(h, F, 1, F, F, ws_bytes=1 << 30)
        assert e.value.status == kvq.ERR_ARG and "fewer than" in kvq.kvq_last_error()
    finally:
        kvq.kvq_cache_destroy(h)


def test_dgap_sizes_and_argument_errors():
    """dgap_restore checks every argument before it launches anything."""
    # workspace: chunk statistics (256-byte aligned) + one 8-byte key per window slot per chunk
    assert kvq.dgap_workspace_bytes(1, 152064, 128) == align(75 * 16) + 75 * 128 * 8
    assert kvq.dgap_workspace_bytes(4, 128256, 64) == align(4 * 63 * 16) + 4 * 63 * 64 * 8
    assert kvq.dgap_workspace_bytes(1, 100, 4) == 0            # k below 8
    assert kvq.dgap_workspace_bytes(1, 100, 200) == 0          # vocab below k
    assert kvq.dgap_workspace_bytes(1, 1 << 20, 256) == 0      # 512 chunks x 256 > 32768 candidates
    assert kvq.dgap_info_floats(128) == 16 + 256
    F = FAKE_ARENA

    def params(**kw):
        d = dict(vocab=32768, k=32, tau=0.6)
        d.update(kw)
        p = kvq.DgapParams(d["vocab"], d["k"], kw.get("hd", 32), kw.get("hc", 32), d["tau"], 0.0, 0.0, 0,
                           F, F, F, F, F, kw.get("cw2", F))
        return p

    ws_ok = kvq.dgap_workspace_bytes(1, 32768, 32)
    cases = [
        (params(k=4), ws_ok, F, kvq.ERR_ARG),
        (params(k=300), ws_ok, F, kvq.ERR_ARG),
        (params(vocab=16, k=32), ws_ok, F, kvq.ERR_ARG),
        (params(hd=0), ws_ok, F, kvq.ERR_ARG),
        (params(hc=65), ws_ok, F, kvq.ERR_ARG),
        (params(cw2=None), ws_ok, F, kvq.ERR_ARG),
        (params(tau=float("nan")), ws_ok, F, kvq.ERR_ARG),
        (params(vocab=(1 << 24) + 1, k=8), 1 << 30, F, kvq.ERR_UNSUPPORTED),
        (params(), ws_ok - 8, F, kvq.ERR_CAPACITY),
        (params(), ws_ok, F + 8, kvq.ERR_ARG),
    ]
    for p, wsb, wsp, status in cases:
        with pytest.raises(kvq.KvqError) as e:
            kvq.dgap_restore(p, F, 1, wsp, ws_bytes=wsb, stream=0)
        assert e.value.status == status, (p.k, p.vocab, wsb, status)
    with pytest.raises(kvq.KvqError) as e:
        kvq.dgap_restore(params(), F, 0, F, ws_bytes=ws_ok, stream=0)
    assert e.value.status == kvq.ERR_ARG
