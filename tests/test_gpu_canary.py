"""Guard bands around every buffer the library writes on the GPU.

The cache arena, the decode and chunk workspaces, the outputs, the export
and dequantization buffers each sit between two 64 KiB bands filled with a
known byte; after every call (appends, fused append + decode, decode, its
two phases, chunk queries, dequantization, export, release, reset) the bands
must be unchanged.  Matrix-core and vector kernels, contiguous and paged
caches, fp16 windows.
"""
import numpy as np
import pytest

from workloads import Workload, gen_kv, gen_q, gen_q_chunk

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GUARD = 1 << 16
PATTERN = 0xA5


class Guarded:
    """A device buffer of n bytes between two guard bands."""

    def __init__(self, n):
        self.buf = torch.full((int(n) + 2 * GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
        self.n = int(n)
        self.t = self.buf[GUARD:GUARD + self.n]
        self.t.zero_()

    def view(self, dtype, shape):
        return self.t.view(dtype).view(shape)

    def intact(self):
        return bool((self.buf[:GUARD] == PATTERN).all()) and bool((self.buf[GUARD + self.n:] == PATTERN).all())


CASES = [
    ("k1v1_gq4", 2, 32, 8, (1500, 900), 1, 1, 32, 32, 0, 0),
    ("k2v2_gq5_R128", 2, 40, 8, (1100, 700), 2, 2, 32, 32, 128, 0),
    ("k8v8_gq8_gk64", 1, 64, 8, (1300,), 8, 8, 64, 32, 0, 0),
    ("k1v4_gq2_vector", 2, 16, 8, (800, 1200), 1, 4, 32, 16, 40, 0),
    ("k1v1_gq4_paged", 3, 32, 8, (1000, 600, 1400), 1, 1, 32, 32, 0, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_no_write_outside_buffers(case):
    from paper_2607_16248_amd import kvq
    name, B, hq, hkv, lens, bk, bv, gk, gv, R, P = case
    w = Workload(name, B, hq, hkv, 128, lens, (bk,) * B, (bv,) * B, gk, gv, R, cfg_id=97)
    cap = max(lens) + 64
    desc = kvq.make_desc(B, hq, hkv, 128, cap, gk, gv, R, [bk] * B, [bv] * B, P, 0)
    arena = Guarded(kvq.kvq_cache_bytes(desc))
    h = kvq.kvq_cache_init(desc, arena.t.data_ptr(), arena.n)
    bufs = [arena]

    def check(what):
        torch.cuda.synchronize()
        for b in bufs:
            assert b.intact(), what

    KV = [gen_kv(w, 0, s) for s in range(B)]
    q = torch.from_numpy(np.stack([gen_q(w, 0, s) for s in range(B)])).cuda()
    pos = [0] * B
    for n in (100, 333, 1, 700, 2000):          # ragged appends
        n_new = [min(n, lens[s] - 40 - pos[s]) for s in range(B)]
        n_new = [max(0, x) for x in n_new]
        nm = max(max(n_new), 1)
        Kb = np.zeros((B, nm, hkv, 128), np.float16)
        Vb = np.zeros_like(Kb)
        for s in range(B):
            Kb[s, :n_new[s]] = KV[s][0][pos[s]:pos[s] + n_new[s]]
            Vb[s, :n_new[s]] = KV[s][1][pos[s]:pos[s] + n_new[s]]
        kin, vin = Guarded(Kb.nbytes), Guarded(Vb.nbytes)
        kin.t.copy_(torch.from_numpy(Kb.view(np.uint8).ravel()))
        vin.t.copy_(torch.from_numpy(Vb.view(np.uint8).ravel()))
        kvq.kvq_append(h, kin.t.data_ptr(), vin.t.data_ptr(), n_new, n_max=nm)
        check(f"append {n_new}")
        pos = [p + x for p, x in zip(pos, n_new)]
    ws = Guarded(kvq.kvq_workspace_bytes(h))
    out = Guarded(B * hq * 128 * 4)
    bufs += [ws, out]
    o = out.view(torch.float32, (B, hq, 128))
    for t in range(40):                         # fused append + decode, token by token
        Kn = np.stack([KV[s][0][pos[s]:pos[s] + 1] for s in range(B)])
        Vn = np.stack([KV[s][1][pos[s]:pos[s] + 1] for s in range(B)])
        kvq.kvq_append_decode(h, torch.from_numpy(Kn).cuda(), torch.from_numpy(Vn).cuda(), [1] * B, q, o,
                              ws.t, ws_bytes=ws.n, n_max=1)
        pos = [p + 1 for p in pos]
        if t % 13 == 0:
            check(f"append_decode step {t}")
    check("append_decode")
    kvq.kvq_decode_attention(h, q, o, ws.t, ws.n)
    check("decode")
    kvq.kvq_decode_partials(h, q, ws.t, ws.n)
    kvq.kvq_decode_merge(h, ws.t, o)
    check("partials + merge")
    for n_q in (16, 5):
        cws = Guarded(kvq.kvq_chunk_workspace_bytes(h, n_q))
        cout = Guarded(B * n_q * hq * 128 * 4)
        bufs += [cws, cout]
        qc = torch.from_numpy(np.stack([gen_q_chunk(w, n_q, 0, s) for s in range(B)])).cuda()
        kvq.kvq_chunk_attention(h, qc, n_q, cout.view(torch.float32, (B, n_q, hq, 128)), cws.t, cws.n)
        check(f"chunk {n_q}")
    for s in range(B):
        L = kvq.kvq_seq_len(h, s)
        Kd, Vd = Guarded(L * hkv * 128 * 4), Guarded(L * hkv * 128 * 4)
        bufs += [Kd, Vd]
        kvq.kvq_dequant(h, s, 0, L, Kd.t, Vd.t)
        check(f"dequant {s}")
        for hh in (0, hkv - 1):
            n = kvq.kvq_export_bytes(h, s, hh)
            dst = Guarded(n)
            bufs.append(dst)
            kvq.kvq_export(h, s, hh, dst.t, n)
            check(f"export {s} {hh}")
    kvq.kvq_check(h)
    kvq.kvq_seq_release(h, 0)
    check("release")
    kvq.kvq_cache_reset(h)
    check("reset")
    kvq.kvq_cache_destroy(h)
