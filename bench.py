#!/usr/bin/env python3
"""Decode-attention benchmark over the packed low-bit KV cache on one MI355X.

Default workload (the headline): Llama-3.1-8B-shaped layers (32 query heads,
8 kv heads, head dim 128), batch 1, 131072 cached tokens, K1V1 with groups of
32, 32 layers with independent seeded caches.  One step = for every layer,
append one token and decode one token (kvq_append_decode).  Inputs are
synthetic and resident in HBM before timing; the 32 caches (2 GiB) rotate
through HBM, well beyond the 256 MB last-level cache.

Prints ONE JSON line.  value = packed-KV bytes the decode kernels must read
per step (codes + fp16 scales/zeros + fp16 tail, all layers) / step time.
Besides the timed steps the line carries:
- "roofline": the split kernel alone (events mean and per-launch median),
  against the 8 TB/s peak and against the streaming-read rate measured on
  the same box ("read_ceiling");
- "parity": two (layer, kv head) units of the timed caches rebuilt on the
  host and checked against the oracle (bytes identical, outputs within 2e-3);
- "step_graph": the whole step captured in one HIP graph and replayed;
- "workloads": split-kernel timings of the other workloads (0, 1, 3 and 4
  at every width; --no-workloads skips them);
- "dgap": DGAP's logit-side step on one logit row of the model vocabulary
  (--no-dgap skips it);
- "chunk": the last 4 / 16 / 64 tokens attending causally over the same
  caches (kvq_chunk_attention; --no-chunk skips it);
- "paged": the split kernel over 8 layers held in 256-token pages against the
  same layers held contiguously (--no-paged skips it);
- "cpu_baseline": the oracle on one full layer on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_FP16_PEAK_TFLOPS = 2500.0  # dense fp16 / bf16 matrix cores
METRIC = "decode-attn effective KV GB/s (% of HBM peak) + µs/layer, K1V1 @128K ctx"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def packed_bytes(L: int, w, bk: int, bv: int) -> int:
    """Bytes decode attention must read for one sequence of L tokens (all kv heads)."""
    past = L - w.window
    Lq = 0 if past <= 0 else past // w.key_group * w.key_group
    per_tok = 16 * bk + 16 * bv + 2 * w.head_dim * 2 // w.key_group + (w.head_dim // w.value_group) * 4
    return w.num_kv_heads * (Lq * per_tok + (L - Lq) * w.head_dim * 2 * 2)


def matrix_path(w) -> bool:
    """Whether the library decodes this workload on the matrix cores."""
    bk, bv = w.bits_k[0], w.bits_v[0]
    bits = (bk in (1, 2) and bv in (1, 2)) or (bk == bv and bk in (4, 8))
    return w.group_q in (4, 5, 8) and bits and w.value_group >= 32


def source_digest() -> str:
    h = hashlib.sha256()
    for f in ("csrc/decode.hip", "csrc/decode_mfma.hip", "csrc/chunk_mfma.hip", "csrc/mfma_common.h",
              "csrc/decode_common.h", "csrc/kvq_internal.h", "csrc/kvq_layout.h", "build.py"):
        with open(os.path.join(ROOT, "paper_2607_16248_amd", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic(name: str):
    """HBM bytes per launch from a committed counter summary, if it matches the kernel source."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != source_digest():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_info():
    """Cores this process may run on and the CPU model of the host it runs on."""
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def cpu_baseline(w):
    """The oracle on one full layer of the workload: quantize (prefill append),
    fp64 dequantization and fp64 attention, each timed separately.  The
    kv heads are independent calls into the plain C oracle, run concurrently
    on the host cores (the C code releases no state between calls; ctypes
    drops the interpreter lock); the attention itself is OpenMP over query
    heads."""
    import concurrent.futures as cf

    import numpy as np

    import oracle
    from workloads import gen_kv, gen_q

    cores, model = host_info()
    threads = oracle.num_threads()
    L = w.lens[0]
    bk, bv = w.bits_k[0], w.bits_v[0]
    heads = list(range(w.num_kv_heads))
    K, V = gen_kv(w, 0, 0)
    q = gen_q(w)
    Kh = [np.ascontiguousarray(K[:, h]) for h in heads]
    Vh = [np.ascontiguousarray(V[:, h]) for h in heads]
    del K, V
    pool = cf.ThreadPoolExecutor(max_workers=max(1, min(threads, len(heads))))
    t0 = time.perf_counter()
    imgs = list(pool.map(lambda h: oracle.build_head(Kh[h], Vh[h], bk, bv, w.key_group, w.value_group, w.window),
                         heads))
    t_quant = time.perf_counter() - t0
    t0 = time.perf_counter()
    deq = list(pool.map(lambda h: oracle.dequant_head(imgs[h], L, w.head_dim, bk, bv, w.key_group,
                                                      w.value_group, w.window), heads))
    t_deq = time.perf_counter() - t0
    Kd = np.stack([d[0] for d in deq])
    Vd = np.stack([d[1] for d in deq])
    del deq
    t0 = time.perf_counter()
    oracle.attention(q, Kd, Vd)
    t_att = time.perf_counter() - t0
    pool.shutdown()
    nbytes = packed_bytes(L, w, bk, bv)
    dt = t_deq + t_att
    return {
        "value": round(nbytes / dt / 1e9, 4),
        "unit": "GB/s",
        # the most threads the sample keeps busy at once (the attention phase)
        "cores": max(threads, max(1, min(threads, len(heads)))),
        "kind": "oracle",
        "sample": (f"one full {L}-token K{bk}V{bv} layer ({w.num_kv_heads} kv heads, {w.num_q_heads} query heads): "
                   f"fp64 dequantization ({len(heads)} independent per-head calls on "
                   f"{max(1, min(threads, len(heads)))} threads) + fp64 attention (OpenMP over query heads, "
                   f"{threads} threads); value = packed bytes of the layer / (dequantization + attention)"),
        "host_cores": cores,
        "cpu_model": model,
        "omp_threads": threads,
        "quantize_us_per_layer": round(t_quant * 1e6, 1),
        "dequant_us_per_layer": round(t_deq * 1e6, 1),
        "attention_us_per_layer": round(t_att * 1e6, 1),
        "bytes_per_layer": nbytes,
    }


def parity_units(w, caches, outs, qs, app, n_appended, units, dev):
    """Same-run parity of the timed caches: for each sampled (layer, kv head)
    the prefill drawn on the device is copied to the host, the appended
    tokens are added, and the oracle (fp64, test infrastructure) rebuilds the
    canonical image and attends.  Export bytes must be identical; the
    decode outputs of the timed step must be within 2e-3 row-normwise."""
    import numpy as np
    import torch

    import oracle
    from workloads import gen_kv_device

    res = []
    L0 = w.lens[0]
    gq = w.group_q
    for layer, h in units:
        K, V = gen_kv_device(w, layer, 0, L0, dev, torch)
        Kh = K[:, h].cpu().numpy()
        Vh = V[:, h].cpu().numpy()
        del K, V
        if n_appended:
            Ka = np.concatenate([app[st][layer][0][0, :, h].cpu().numpy() for st in range(n_appended)])
            Va = np.concatenate([app[st][layer][1][0, :, h].cpu().numpy() for st in range(n_appended)])
            Kh = np.concatenate([Kh, Ka])
            Vh = np.concatenate([Vh, Va])
        img = oracle.build_head(Kh, Vh, w.bits_k[0], w.bits_v[0], w.key_group, w.value_group, w.window)
        got = caches[layer].export(0, h)
        bytes_ok = bool(got.shape == img.shape and (got == img).all())
        Kd, Vd = oracle.dequant_head(img, Kh.shape[0], w.head_dim, w.bits_k[0], w.bits_v[0], w.key_group,
                                     w.value_group, w.window)
        q = qs[layer][0, h * gq:(h + 1) * gq].cpu().numpy()
        ref = oracle.attention(q, Kd[None], Vd[None])
        o = outs[layer][0, h * gq:(h + 1) * gq].cpu().numpy().astype(np.float64)
        err = float((np.abs(o - ref).max(1) / np.abs(ref).max(1)).max())
        res.append({"layer": layer, "kv_head": h, "tokens": int(Kh.shape[0]), "bytes_identical": bytes_ok,
                    "max_row_rel_err": err, "within_2e-3": err <= 2e-3})
    return res


def read_ceiling(dev, stream, gib: int = 4, iters: int = 8):
    """Measured streaming-read rate: the library's plain 16-byte read kernel
    over a 4 GiB device buffer (beyond the 256 MB last-level cache)."""
    import torch

    from paper_2607_16248_amd import kvq

    n = gib << 30
    buf = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    sink = torch.empty(kvq.kvq_read_probe_sink_bytes(), dtype=torch.uint8, device=dev)
    for _ in range(2):
        kvq.kvq_read_probe(buf, n, sink, stream=stream)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(iters):
        kvq.kvq_read_probe(buf, n, sink, stream=stream)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / iters
    del buf, sink
    return {"gbs": round(n / (us * 1e-6) / 1e9, 1), "bytes": n, "us": round(us, 2),
            "kernel": "read_probe_kernel (16-byte grid-stride loads)"}


def workload_leg(idx: int, bits, dev, stream, iters: int = 64, rotate_bytes: int = 512 << 20, max_copies: int = 192):
    """Split kernel (and split + merge) of one workload, back to back over
    rotating layer caches, HIP events on the launch stream."""
    import numpy as np
    import torch

    from paper_2607_16248_amd import kvq
    from workloads import gen_kv_device, gen_q, workload

    w = workload(idx, bits)
    per = sum(packed_bytes(L, w, bk, bv) for L, bk, bv in zip(w.lens, w.bits_k, w.bits_v))
    copies = max(1, min(max_copies, -(-rotate_bytes // per)))
    caches, qs = [], []
    for l in range(copies):
        c = kvq.KVCache(w.batch, w.num_q_heads, w.num_kv_heads, max(w.lens), list(w.bits_k), list(w.bits_v),
                        key_group=w.key_group, value_group=w.value_group, fp16_window=w.window, device=dev)
        nmax = max(w.lens)
        Kb = torch.zeros((w.batch, nmax, w.num_kv_heads, w.head_dim), dtype=torch.float16, device=dev)
        Vb = torch.zeros_like(Kb)
        for s_ in range(w.batch):
            K, V = gen_kv_device(w, l, s_, w.lens[s_], dev, torch)
            Kb[s_, :w.lens[s_]] = K
            Vb[s_, :w.lens[s_]] = V
            del K, V
        c.append(Kb, Vb, list(w.lens))
        del Kb, Vb
        c.check()
        caches.append(c)
        qs.append(torch.from_numpy(np.stack([gen_q(w, l, s_) for s_ in range(w.batch)])).to(dev))
    hs = [c.handle for c in caches]
    wsb = max(kvq.kvq_workspace_bytes(h) for h in hs)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    out = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)

    def timed(fn):
        for i in range(8):
            fn(i)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(iters):
            fn(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / iters

    split = timed(lambda i: kvq.kvq_decode_partials(hs[i % copies], qs[i % copies], ws, wsb, stream=stream))
    dec = timed(lambda i: kvq.kvq_decode_attention(hs[i % copies], qs[i % copies], out, ws, wsb, stream=stream))
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(32)]
    for i, (a, b) in enumerate(pairs):
        a.record()
        kvq.kvq_decode_partials(hs[i % copies], qs[i % copies], ws, wsb, stream=stream)
        b.record()
    torch.cuda.synchronize()
    med = sorted(a.elapsed_time(b) * 1e3 for a, b in pairs)[len(pairs) // 2]
    kernels = sorted({(bk, bv) for bk, bv in zip(w.bits_k, w.bits_v)})
    out_d = {
        "workload": w.name,
        "bits": [f"K{a}V{b}" for a, b in kernels],
        "kernel": ["matrix" if matrix_path(w) else "vector"],
        "bytes_per_launch": per,
        "rotating_copies": copies,
        "split_us": round(split, 3),
        "split_us_median": round(med, 3),
        "decode_us": round(dec, 3),
        "achieved_gbs": round(per / (split * 1e-6) / 1e9, 1),
        "frac": round(per / (split * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "frac_median": round(per / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
    }
    del caches, qs, ws, out
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out_d


# DGAP window sizes K_b per KbVb precision (a reading: the paper calibrates
# them from traces; lower bits, larger windows) and the vocabulary of each
# workload's model.
DGAP_K = {1: 128, 2: 64, 4: 32, 8: 16}
DGAP_VOCAB = {0: ("llama3_8b", 128256), 1: ("llama3_8b", 128256), 2: ("llama3_8b", 128256),
              3: ("mistral_7b", 32768), 4: ("qwen2_5_14b", 152064)}


def dgap_leg(workload_idx: int, bits: int, iters: int):
    """DGAP's logit-side step after each decode step: one batch-1 logit row of
    the workload's vocabulary, timed back to back with HIP events on the
    launch stream, once with a detector that always corrects and once with one
    that never does."""
    import torch

    from dgap_inputs import gen_logits, gen_weights
    from paper_2607_16248_amd import kvq

    dev = torch.device("cuda:0")
    model, V = DGAP_VOCAB[workload_idx]
    k = DGAP_K[bits]
    stream = torch.cuda.current_stream().cuda_stream
    z0 = gen_logits(V, 1, seed=0)
    out = {"model_vocab": model, "vocab": V, "k": k, "tau": 0.6, "batch": 1}
    for name, bias in (("corrected", 20.0), ("bypass", -20.0)):
        w = gen_weights(0, det_bias=bias)
        t = {n: torch.from_numpy(getattr(w, n)).to(dev) for n in ("w1", "b1", "w2", "c1", "cb1", "c2")}
        p = kvq.dgap_params(V, k, 0.6, t["w1"], t["b1"], t["w2"], w.b2, t["c1"], t["cb1"], t["c2"], w.cb2)
        z = torch.from_numpy(z0).to(dev)
        ws = torch.empty(kvq.dgap_workspace_bytes(1, V, k), dtype=torch.uint8, device=dev)
        for _ in range(8):
            kvq.dgap_restore(p, z, 1, ws, stream=stream)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(iters):
            kvq.dgap_restore(p, z, 1, ws, stream=stream)
        b.record()
        torch.cuda.synchronize()
        out[f"us_{name}"] = round(a.elapsed_time(b) * 1e3 / iters, 3)
    # bytes one call must move: the row (read once) and the chunk partials
    nchunk = -(-V // 2048)
    out["bytes_per_call"] = V * 4 + nchunk * (16 + 8 * k) * 2 + 2 * k * 4
    out["gbs_corrected"] = round(out["bytes_per_call"] / (out["us_corrected"] * 1e-6) / 1e9, 2)
    out["bound"] = "latency (two dependent launches; the row is 0.5-0.6 MB)"
    return out


CHUNK_SIZES = (4, 5, 16, 64)


def chunk_row_groups(n_q: int, gq: int):
    """Rows per group and groups per kv head as the library plans chunk
    queries on 1- and 2-bit caches with value groups of 32: of 32 or 16 rows
    (the chunk kernel, floor(rows / gq) queries each) and 8, 5 or 4 (the
    decode kernel, whole sets of heads), the one with the fewest estimated
    microseconds, ceil(n_q / queries) passes at 38, 30, 21, 19 or 18."""
    cost = {32: 38, 16: 30, 8: 21, 5: 19, 4: 18}
    best = None
    for r in (32, 16, 8, 5, 4):
        if (r < 16 and r % gq) or r // gq == 0:
            continue
        n = -(-n_q // (r // gq))
        if best is None or n * cost[r] < best[0]:
            best = (n * cost[r], r, n)
    return best[1], best[2]


def chunk_leg(handles, w, launch_bytes: int, stream, iters: int):
    """Chunk queries over the same layer caches: the last n_q tokens of the
    sequence attend causally (chunked prefill, speculative verification),
    timed with HIP events on the launch stream over the rotating layers."""
    import torch

    from paper_2607_16248_amd import kvq

    dev = torch.device("cuda:0")
    layers = len(handles)
    out = {"n_q": list(CHUNK_SIZES), "us_per_layer": [], "query_tokens_per_s_per_layer": [],
           "cache_gbs_one_pass": [], "useful_tflops": [], "row_groups_per_kv_head": [], "rows_per_group": []}
    L = min(kvq.kvq_seq_len(handles[0], s) for s in range(w.batch))
    for n_q in CHUNK_SIZES:
        g = torch.Generator(device=dev).manual_seed(n_q)
        q = torch.randn((w.batch, n_q, w.num_q_heads, w.head_dim), generator=g, device=dev).half()
        o = torch.empty((w.batch, n_q, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)
        need = max(kvq.kvq_chunk_workspace_bytes(h, n_q) for h in handles)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        for i in range(8):
            kvq.kvq_chunk_attention(handles[i % layers], q, n_q, o, ws, need, stream=stream)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(iters):
            kvq.kvq_chunk_attention(handles[i % layers], q, n_q, o, ws, need, stream=stream)
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / iters
        # QK and PV: 2 * 2 * d flops per (query, head, visible token)
        flops = 4 * w.head_dim * w.num_q_heads * w.batch * sum(L - n_q + 1 + i for i in range(n_q))
        rows, groups = chunk_row_groups(n_q, w.group_q)
        out["us_per_layer"].append(round(us, 3))
        out["query_tokens_per_s_per_layer"].append(round(n_q * w.batch / (us * 1e-6), 1))
        out["cache_gbs_one_pass"].append(round(launch_bytes / (us * 1e-6) / 1e9, 2))
        out["useful_tflops"].append(round(flops / (us * 1e-6) / 1e12, 2))
        out["row_groups_per_kv_head"].append(groups)
        out["rows_per_group"].append(rows)
        del q, o, ws
    out["note"] = ("each row group of up to 32 (query, head) rows is one pass over the kv head's cache "
                   "(the chunk kernel: two row halves of 16 share each unpacked code operand); a last group "
                   "with fewer queries repeats the last one in its spare rows (n_q = 5: one 32-row group, the "
                   "verification step of 4 drafted tokens); the useful flops count each visible (query, head, "
                   "token) once")
    # the matrix-core roofline of the contraction (fp16 operands, fp32 accumulation)
    out["roofline"] = {"bound": "mfma", "peak": MFMA_FP16_PEAK_TFLOPS, "unit": "TFLOP/s",
                       "frac": [round(t / MFMA_FP16_PEAK_TFLOPS, 4) for t in out["useful_tflops"]]}
    return out


PAGE_TOKENS = 256


def paged_leg(w, qs, dev, stream, iters: int, nlayers: int = 8):
    """The split kernel over paged caches (pages of PAGE_TOKENS tokens from a
    shared pool, block table per sequence) against contiguous caches holding
    the same seeded tokens: nlayers of each, rotating, HIP events on the
    launch stream; and the decode outputs of the two compared bit for bit.
    The two sets are allocated layer by layer in turn, so that both meet the
    same state of device memory."""
    import torch

    from paper_2607_16248_amd import kvq
    from workloads import gen_kv_device

    sets = {"contiguous": [], "paged": []}
    for l in range(nlayers):
        for name, P in (("contiguous", 0), ("paged", PAGE_TOKENS)):
            c = kvq.KVCache(w.batch, w.num_q_heads, w.num_kv_heads, max(w.lens), list(w.bits_k), list(w.bits_v),
                            key_group=w.key_group, value_group=w.value_group, fp16_window=w.window, device=dev,
                            page_tokens=P)
            Kb = torch.zeros((w.batch, max(w.lens), w.num_kv_heads, w.head_dim), dtype=torch.float16, device=dev)
            Vb = torch.zeros_like(Kb)
            for s in range(w.batch):
                K, V = gen_kv_device(w, l, s, w.lens[s], dev, torch)
                Kb[s, :w.lens[s]] = K
                Vb[s, :w.lens[s]] = V
                del K, V
            c.append(Kb, Vb, list(w.lens))
            del Kb, Vb
            sets[name].append(c)
    torch.cuda.synchronize()
    out = {"page_tokens": PAGE_TOKENS, "layers": nlayers}
    outs = {}
    for name, cs in sets.items():
        ws_bytes = max(kvq.kvq_workspace_bytes(c.handle) for c in cs)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        for i in range(8):
            kvq.kvq_decode_partials(cs[i % nlayers].handle, qs[i % nlayers], ws, ws_bytes, stream=stream)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(iters):
            kvq.kvq_decode_partials(cs[i % nlayers].handle, qs[i % nlayers], ws, ws_bytes, stream=stream)
        b.record()
        torch.cuda.synchronize()
        out[f"split_us_{name}"] = round(a.elapsed_time(b) * 1e3 / iters, 3)
        o = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)
        cs[0].decode(qs[0], o)
        torch.cuda.synchronize()
        outs[name] = o
    out["outputs_bit_identical"] = bool(torch.equal(outs["contiguous"], outs["paged"]))
    nbytes = sum(packed_bytes(L, w, bk, bv) for L, bk, bv in zip(w.lens, w.bits_k, w.bits_v))
    out["roofline_paged"] = {"bound": "hbm", "achieved": round(nbytes / (out["split_us_paged"] * 1e-6) / 1e9, 2),
                             "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(nbytes / (out["split_us_paged"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    return out


def dgap_cpu_baseline(workload_idx: int, bits: int) -> float:
    """Part of the CPU-baseline leg: the DGAP oracle (fp64, one thread) on the
    same row, microseconds per corrected step."""
    from dgap_inputs import gen_logits, gen_weights
    from oracle import dgap as odgap

    _, V = DGAP_VOCAB[workload_idx]
    z0 = gen_logits(V, 1, seed=0)[0]
    w = gen_weights(0, det_bias=20.0)
    reps = 5
    t0 = time.perf_counter()
    for _ in range(reps):
        odgap.restore(z0, DGAP_K[bits], w)
    return round((time.perf_counter() - t0) * 1e6 / reps, 1)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=2, help="0-4; 2 is the headline")
    ap.add_argument("--bits", type=int, default=None, help="bit width for workload 4")
    ap.add_argument("--kernel-iters", type=int, default=256)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the split-kernel timings of the other workloads (0, 1, 3, 4 at every width)")
    ap.add_argument("--no-parity", action="store_true", help="skip the same-run oracle check of the timed caches")
    ap.add_argument("--no-dgap", action="store_true", help="skip the DGAP logit-side leg")
    ap.add_argument("--no-chunk", action="store_true", help="skip the chunk-query leg")
    ap.add_argument("--no-paged", action="store_true", help="skip the paged-cache leg")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="end with 4 plain device copies of 256 MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU path is not "
              f"part of this library", file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_16248_amd import kvq
    from workloads import gen_append, gen_kv_device, gen_q, workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = workload(args.workload, args.bits)
    steps, warm = args.steps, args.warmup
    appending = args.workload == 2
    layers = w.layers if w.layers > 1 else max(1, min(64, -(-(1 << 30) // max(1, sum(
        packed_bytes(L, w, bk, bv) for L, bk, bv in zip(w.lens, w.bits_k, w.bits_v))))))
    append_rounds = 4  # extra appends per layer timed on their own after the steps
    extra = (steps + warm + 3 + append_rounds) if appending else 0
    cap = max(w.lens) + extra

    log(f"[bench] workload {w.name}: {layers} layer caches, capacity {cap}")
    caches, qs, outs = [], [], []
    for l in range(layers):
        c = kvq.KVCache(w.batch, w.num_q_heads, w.num_kv_heads, cap, list(w.bits_k), list(w.bits_v),
                        key_group=w.key_group, value_group=w.value_group, fp16_window=w.window, device=dev)
        nmax = max(w.lens)
        Kb = torch.zeros((w.batch, nmax, w.num_kv_heads, w.head_dim), dtype=torch.float16, device=dev)
        Vb = torch.zeros_like(Kb)
        for s in range(w.batch):
            K, V = gen_kv_device(w, l, s, w.lens[s], dev, torch)
            Kb[s, :w.lens[s]] = K
            Vb[s, :w.lens[s]] = V
            del K, V
        c.append(Kb, Vb, list(w.lens))
        del Kb, Vb
        qs.append(torch.from_numpy(np.stack([gen_q(w, l, s) for s in range(w.batch)])).to(dev))
        outs.append(torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev))
        caches.append(c)
    torch.cuda.synchronize()
    for c in caches:
        c.check()
    ws_bytes = max(kvq.kvq_workspace_bytes(c.handle) for c in caches)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)

    # appended tokens for every step, generated up front and resident on the device
    app = []
    if appending:
        for st in range(steps + warm + 2 + append_rounds):
            row = []
            for l in range(layers):
                Kn, Vn = gen_append(w, l, 0, st)
                row.append((torch.from_numpy(Kn[None]).to(dev), torch.from_numpy(Vn[None]).to(dev)))
            app.append(row)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream().cuda_stream
    one = [1] * w.batch
    handles = [c.handle for c in caches]

    # one decode step: every layer appends its token and attends (one call;
    # the token is stored by the decode launch unless a key group fills)
    def step(st):
        for l in range(layers):
            if appending:
                kvq.kvq_append_decode(handles[l], app[st][l][0], app[st][l][1], one, qs[l], outs[l], ws,
                                      ws_bytes=ws_bytes, n_max=1, stream=stream)
            else:
                kvq.kvq_decode_attention(handles[l], qs[l], outs[l], ws, ws_bytes, stream=stream)

    # bring the GPU to its working clocks before the warmup steps (about
    # 100 ms of decode launches over the rotating layers; outputs discarded)
    t_w = time.perf_counter()
    i_w = 0
    while time.perf_counter() - t_w < 0.1:
        for _ in range(64):
            kvq.kvq_decode_partials(handles[i_w % layers], qs[i_w % layers], ws, ws_bytes, stream=stream)
            i_w += 1
        torch.cuda.synchronize()
    log(f"[bench] warmup {warm} steps")
    for st in range(warm):
        step(st)
    torch.cuda.synchronize()

    lens_before = [[kvq.kvq_seq_len(h, s) for s in range(w.batch)] for h in handles]
    moved = 0
    for st in range(steps):
        for l in range(layers):
            for s in range(w.batch):
                L = lens_before[l][s] + ((st + 1) if appending else 0)
                moved += packed_bytes(L, w, w.bits_k[s], w.bits_v[s])

    log(f"[bench] timing {steps} steps")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for st in range(steps):
        step(warm + st)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = ev0.elapsed_time(ev1) / steps
    for c in caches:
        c.check()

    # dominant kernel alone: split kernels of kvq_decode_partials, back to back
    # over the rotating layer caches, timed with events on the launch stream
    def timed(fn, iters):
        for i in range(max(8, iters // 2)):
            fn(i)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(iters):
            fn(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / iters  # microseconds

    it = args.kernel_iters
    split_us = timed(lambda i: kvq.kvq_decode_partials(handles[i % layers], qs[i % layers], ws, ws_bytes,
                                                       stream=stream), it)
    merge_us = timed(lambda i: kvq.kvq_decode_merge(handles[i % layers], ws, outs[i % layers], stream=stream), it)
    decode_us = timed(lambda i: kvq.kvq_decode_attention(handles[i % layers], qs[i % layers], outs[i % layers],
                                                         ws, ws_bytes, stream=stream), it)
    # per-launch spread of the split kernel: one event pair per launch
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(64)]
    for i, (a, b) in enumerate(pairs):
        a.record()
        kvq.kvq_decode_partials(handles[i % layers], qs[i % layers], ws, ws_bytes, stream=stream)
        b.record()
    torch.cuda.synchronize()
    per_launch = sorted(a.elapsed_time(b) * 1e3 for a, b in pairs)
    split_med = per_launch[len(per_launch) // 2]
    split_p95 = per_launch[int(0.95 * (len(per_launch) - 1))]

    # decode of every layer replayed from one captured graph (lengths are fixed
    # between appends, so the launches of a decode are the same every replay);
    # every replay must reproduce the eager outputs bit for bit
    graph_us = None
    graph_exact = None
    try:
        for l in range(layers):
            kvq.kvq_decode_attention(handles[l], qs[l], outs[l], ws, ws_bytes, stream=stream)
        torch.cuda.synchronize()
        eager = [o.clone() for o in outs]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            gs = torch.cuda.current_stream().cuda_stream
            for l in range(layers):
                kvq.kvq_decode_attention(handles[l], qs[l], outs[l], ws, ws_bytes, stream=gs)
        graph_exact = True
        for _ in range(3):
            for o in outs:
                o.zero_()
            g.replay()
            torch.cuda.synchronize()
            graph_exact &= all(torch.equal(o, e) for o, e in zip(outs, eager))
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = max(4, it // layers)
        a.record()
        for _ in range(reps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        graph_us = a.elapsed_time(b) * 1e3 / (reps * layers)
        del g
    except RuntimeError as e:  # capture unsupported: report and go on
        log(f"[bench] graph replay skipped: {e}")

    # parity of the timed caches against the oracle, before the step graph
    # appends to them: two sampled (layer, kv head) units, bytes and the
    # outputs of the last timed step (the kernel timings above write only the
    # outputs of decode calls over the same state, which are identical)
    parity = None
    if not args.no_parity:
        log("[bench] same-run parity of two sampled (layer, kv head) units against the oracle")
        n_app = (warm + steps) if appending else 0
        parity = parity_units(w, caches, outs, qs, app, n_app, [(0, 3), (layers - 1, 6 % w.num_kv_heads)], dev)

    # one whole decode step (every layer: append one token, attend) captured in
    # one graph and replayed; the capture advances the host lengths by one
    # token, every replay stores that token again and attends over the same
    # lengths, so each replay is the same step.  The replay outputs must equal
    # an eager decode over the same cache state bit for bit.
    step_graph = None
    if appending:
        try:
            gstep = warm + steps + append_rounds
            torch.cuda.synchronize()
            g2 = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g2):
                gs = torch.cuda.current_stream().cuda_stream
                for l in range(layers):
                    kvq.kvq_append_decode(handles[l], app[gstep][l][0], app[gstep][l][1], one, qs[l], outs[l], ws,
                                          ws_bytes=ws_bytes, n_max=1, stream=gs)
            g2.replay()
            torch.cuda.synchronize()
            replayed = [o.clone() for o in outs]
            reps = 16
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                g2.replay()
            b.record()
            torch.cuda.synchronize()
            step_us = a.elapsed_time(b) * 1e3 / reps
            same = all(torch.equal(o, r) for o, r in zip(outs, replayed))
            for l in range(layers):
                kvq.kvq_decode_attention(handles[l], qs[l], outs[l], ws, ws_bytes, stream=stream)
            torch.cuda.synchronize()
            same &= all(torch.equal(o, r) for o, r in zip(outs, replayed))
            Lg = [kvq.kvq_seq_len(h, 0) for h in handles]
            gbytes = sum(packed_bytes(L, w, w.bits_k[0], w.bits_v[0]) for L in Lg)
            step_graph = {"us_per_step": round(step_us, 2), "us_per_layer": round(step_us / layers, 3),
                          "gbs": round(gbytes / (step_us * 1e-6) / 1e9, 1), "replays": reps,
                          "outputs_equal_eager": bool(same)}
            del g2
        except RuntimeError as e:  # capture unsupported: report and go on
            log(f"[bench] step graph skipped: {e}")

    # appends on their own: append_rounds more tokens per layer (copies into
    # the fp16 ring; a key group flushes once every key_group tokens)
    append_us = None
    if appending:
        base = warm + steps
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(append_rounds):
            for l in range(layers):
                kvq.kvq_append(handles[l], app[base + r][l][0], app[base + r][l][1], one, n_max=1, stream=stream)
        b.record()
        torch.cuda.synchronize()
        append_us = a.elapsed_time(b) * 1e3 / (append_rounds * layers)
        for c in caches:
            c.check()

    L_now = [kvq.kvq_seq_len(handles[0], s) for s in range(w.batch)]
    launch_bytes = sum(packed_bytes(L, w, bk, bv) for L, bk, bv in zip(L_now, w.bits_k, w.bits_v))
    achieved = launch_bytes / (split_us * 1e-6) / 1e9

    value = moved / (step_ms * steps * 1e-3) / 1e9
    us_per_layer = step_ms * 1e3 / layers
    traffic_name = f"decode_split_{w.name}_traffic.txt"
    traffic = read_traffic(traffic_name)

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 matrix-core products, f32 accumulation" if matrix_path(w) else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "layers": layers,
            "batch": w.batch,
            "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim,
            "context": list(w.lens) if w.batch <= 4 else f"{min(w.lens)}..{max(w.lens)}",
            "bits": [f"K{a}V{b}" for a, b in sorted(set(zip(w.bits_k, w.bits_v)))],
            "key_group": w.key_group,
            "value_group": w.value_group,
            "fp16_window": w.window,
            "append_per_step": appending,
            "parallelism": "single GPU, split-K over tokens",
        },
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "us_per_layer": round(us_per_layer, 3),
        "decode_us_per_layer": round(decode_us, 3),
        "split_kernel_us": round(split_us, 3),
        "split_kernel_us_median": round(split_med, 3),
        "split_kernel_us_p95": round(split_p95, 3),
        "merge_kernel_us": round(merge_us, 3),
        "decode_graph_us_per_layer": None if graph_us is None else round(graph_us, 3),
        "decode_graph_exact": graph_exact,
        "append_us": None if append_us is None else round(append_us, 3),
        "bytes_per_layer": launch_bytes,
        "wall_s_timed": round(wall, 4),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "achieved_median": round(launch_bytes / (split_med * 1e-6) / 1e9, 2),
            "frac_median": round(launch_bytes / (split_med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "timing": ("achieved/frac: mean over back-to-back launches (events around the batch); "
                       "*_median: median of per-launch event pairs"),
            "traffic": traffic,
            "kernel": (f"decode_mfma_kernel<{w.bits_k[0]},{w.bits_v[0]},{w.key_group // 32},{w.group_q},false,false>" if matrix_path(w) else
                       f"decode_split_kernel<{w.bits_k[0]},{w.bits_v[0]},{w.group_q}>"),
            "bytes_per_launch": launch_bytes,
            "kernel_source_sha256_16": source_digest(),
        },
    }
    result["parity"] = parity
    result["step_graph"] = step_graph
    log("[bench] streaming-read ceiling")
    rc = read_ceiling(dev, stream)
    result["roofline"]["measured_read_ceiling_gbs"] = rc["gbs"]
    result["roofline"]["frac_of_measured_ceiling"] = round(achieved / rc["gbs"], 4)
    result["read_ceiling"] = rc
    if args.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.uint8, device=dev).fill_(3)
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_paged:
        log("[bench] paged caches")
        result["paged"] = paged_leg(w, qs, dev, stream, 64)
    if not args.no_chunk:
        log("[bench] chunk queries")
        result["chunk"] = chunk_leg(handles, w, launch_bytes, stream, max(2 * layers, 32))
    if not args.no_dgap:
        log("[bench] DGAP logit-side step")
        result["dgap"] = dgap_leg(args.workload, w.bits_k[0], 200)
    if not args.no_workloads and args.workload == 2:
        del caches, app
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        wl = []
        for idx, bits in ((0, None), (1, None), (3, None), (4, 1), (4, 2), (4, 4), (4, 8)):
            log(f"[bench] workload {idx}" + (f" K{bits}V{bits}" if bits else ""))
            wl.append(workload_leg(idx, bits, dev, stream))
        result["workloads"] = wl
    if not args.no_cpu_baseline:
        log("[bench] CPU baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(w)
        if not args.no_dgap:
            result["cpu_baseline"]["dgap_oracle_us_per_step"] = dgap_cpu_baseline(args.workload, w.bits_k[0])
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
