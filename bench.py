#!/usr/bin/env python3
"""Decode-attention benchmark over the packed low-bit KV cache on one MI355X.

Default workload (the headline): Llama-3.1-8B-shaped layers (32 query heads,
8 kv heads, head dim 128), batch 1, 131072 cached tokens, K1V1 with groups of
32, 32 layers with independent seeded caches.  One step = for every layer,
append one token (kvq_append) then decode one token (kvq_decode_attention).
Inputs are synthetic and resident in HBM before timing; the 32 caches
(2 GiB) rotate through HBM, well beyond the 256 MB last-level cache.

Prints ONE JSON line.  value = packed-KV bytes the decode kernels must read
per step (codes + fp16 scales/zeros + fp16 tail, all layers) / step time.
The line also carries "dgap": DGAP's logit-side step (features, detector,
top-K window, corrector, merge) on one logit row of the workload's model
vocabulary, timed on its own (--no-dgap skips it), and "chunk": the last
4 / 16 / 64 tokens attending causally over the same caches
(kvq_chunk_attention; --no-chunk skips it), and "paged": the split kernel
over 8 layers held in 256-token pages against the same layers held
contiguously (--no-paged skips it).
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
    for f in ("csrc/decode.hip", "csrc/decode_mfma.hip", "csrc/decode_common.h", "csrc/kvq_internal.h",
              "csrc/kvq_layout.h", "build.py"):
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


def cpu_baseline(w, kv_heads: int):
    """The oracle (fp64 dequantization + attention) on a bounded sample of one layer."""
    import numpy as np

    import oracle
    from workloads import gen_kv, gen_q

    heads = list(range(kv_heads))
    L = w.lens[0]
    bk, bv = w.bits_k[0], w.bits_v[0]
    K, V = gen_kv(w, 0, 0, heads=heads)
    q = gen_q(w)
    imgs = [oracle.build_head(K[:, h], V[:, h], bk, bv, w.key_group, w.value_group, w.window) for h in heads]
    del K, V
    gq = w.group_q
    t0 = time.perf_counter()
    Kh = np.empty((kv_heads, L, w.head_dim))
    Vh = np.empty_like(Kh)
    for i, img in enumerate(imgs):
        Kh[i], Vh[i] = oracle.dequant_head(img, L, w.head_dim, bk, bv, w.key_group, w.value_group, w.window)
    oracle.attention(q[:kv_heads * gq], Kh, Vh)
    dt = time.perf_counter() - t0
    nbytes = packed_bytes(L, w, bk, bv) * kv_heads // w.num_kv_heads
    threads = oracle.num_threads()
    return {
        "value": round(nbytes / dt / 1e9, 4),
        "unit": "GB/s",
        "cores": min(threads, kv_heads * gq),
        "kind": "oracle",
        "sample": (f"{kv_heads} of {w.num_kv_heads} kv heads ({kv_heads * gq} query heads) of one "
                   f"{L}-token K{bk}V{bv} layer: fp64 dequantization (one thread per call) + fp64 "
                   f"attention (OpenMP over query heads, {min(threads, kv_heads * gq)} threads); "
                   f"{dt:.2f} s for {nbytes / 1e6:.1f} MB of packed KV; "
                   f"{dt * 1e6 * w.num_kv_heads / kv_heads:.0f} us per full layer"),
    }


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


CHUNK_SIZES = (4, 16, 64)


def chunk_leg(handles, w, launch_bytes: int, stream, iters: int):
    """Chunk queries over the same layer caches: the last n_q tokens of the
    sequence attend causally (chunked prefill, speculative verification),
    timed with HIP events on the launch stream over the rotating layers."""
    import torch

    from paper_2607_16248_amd import kvq

    dev = torch.device("cuda:0")
    layers = len(handles)
    out = {"n_q": list(CHUNK_SIZES), "us_per_layer": [], "query_tokens_per_s_per_layer": [],
           "cache_gbs_one_pass": [], "useful_tflops": [], "row_groups_per_kv_head": []}
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
        gq = w.group_q
        rows = 8 if (gq == 4 and n_q % 2 == 0) or gq == 8 else gq
        out["us_per_layer"].append(round(us, 3))
        out["query_tokens_per_s_per_layer"].append(round(n_q * w.batch / (us * 1e-6), 1))
        out["cache_gbs_one_pass"].append(round(launch_bytes / (us * 1e-6) / 1e9, 2))
        out["useful_tflops"].append(round(flops / (us * 1e-6) / 1e12, 2))
        out["row_groups_per_kv_head"].append(n_q * gq // rows)
        del q, o, ws
    out["note"] = ("each row group of up to 8 (query, head) rows is one pass over the kv head's cache; "
                   "the useful flops count each visible (query, head, token) once")
    # the matrix-core roofline of the contraction (fp16 operands, fp32 accumulation)
    out["roofline"] = {"bound": "mfma", "peak": MFMA_FP16_PEAK_TFLOPS, "unit": "TFLOP/s",
                       "frac": [round(t / MFMA_FP16_PEAK_TFLOPS, 4) for t in out["useful_tflops"]]}
    return out


PAGE_TOKENS = 256


def paged_leg(w, qs, dev, stream, iters: int, nlayers: int = 8):
    """The split kernel over paged caches (pages of PAGE_TOKENS tokens from a
    shared pool, block table per sequence) against contiguous caches holding
    the same seeded tokens: nlayers of each, rotating, HIP events on the
    launch stream; and the decode outputs of the two compared bit for bit."""
    import torch

    from paper_2607_16248_amd import kvq
    from workloads import gen_kv_device

    sets = {}
    for name, P in (("contiguous", 0), ("paged", PAGE_TOKENS)):
        cs = []
        for l in range(nlayers):
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
            cs.append(c)
        sets[name] = cs
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
    ap.add_argument("--cpu-heads", type=int, default=4, help="kv heads in the CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    extra = (steps + warm + 2 + append_rounds) if appending else 0
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
        for st in range(steps + warm + 1 + append_rounds):
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
        for i in range(8):
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
        "dtype": "fp32 (1-bit codes, fp16 scales)" if w.bits_k[0] == 1 else "fp32",
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
            "traffic": traffic,
            "kernel": (f"decode_mfma_kernel<{w.bits_k[0]},{w.bits_v[0]},{w.key_group // 32},{w.group_q},false,false>" if matrix_path(w) else
                       f"decode_split_kernel<{w.bits_k[0]},{w.bits_v[0]},{w.group_q}>"),
            "bytes_per_launch": launch_bytes,
            "kernel_source_sha256_16": source_digest(),
        },
    }
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
    if not args.no_cpu_baseline:
        log("[bench] CPU baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(w, min(args.cpu_heads, w.num_kv_heads))
        if not args.no_dgap:
            result["cpu_baseline"]["dgap_oracle_us_per_step"] = dgap_cpu_baseline(args.workload, w.bits_k[0])
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
