"""Seeded synthetic inputs for the packed low-bit KV-cache decode path.

This module draws random numbers and nothing else: it holds none of the
quantization or attention arithmetic, so both the CPU oracle and the HIP
path can consume its outputs without sharing any of the method.

The paper evaluates on real long-context benchmarks with Llama-3.1-8B,
Mistral-7B and Qwen2.5-14B (Experimental Setup, "Models and benchmarks");
none of those weights or datasets are used here.  The generators below stand
in for them with the same head shapes and context lengths (8K-128K,
Efficiency Analysis tables) and with the value structure that matters for a
per-channel key quantizer: a few outlier key channels per head.

Every draw comes from ``numpy.random.default_rng([MAGIC, cfg, layer, seq,
tensor, *extra])`` so any single (layer, seq, kv head) unit can be rebuilt on
its own, on the host, without generating the rest of the workload.

Tensor ids: 0 = q, 1 = K, 2 = V, 3 = outlier channel choice, 4 = context
lengths, 5 = appended K, 6 = appended V, 7 = chunk queries (with n_q).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

MAGIC = 0x4B5651  # "KVQ"

T_Q, T_K, T_V, T_OUTLIER, T_LENS, T_APPEND_K, T_APPEND_V, T_Q_CHUNK = range(8)

# Inputs are kept at |x| <= this bound so that a 1-bit group's range
# (max - min) can never exceed the largest finite fp16 scale; only the
# Student-t workload ever reaches it (probability ~1e-9 per element).
CLIP = 32752.0


@dataclass(frozen=True)
class Workload:
    """Shape and quantizer settings of one synthetic workload."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    lens: Tuple[int, ...]          # context length per sequence
    bits_k: Tuple[int, ...]        # key bits per sequence
    bits_v: Tuple[int, ...]        # value bits per sequence
    key_group: int                 # tokens per key group (per channel)
    value_group: int               # channels per value group (per token)
    window: int                    # recent tokens kept in fp16
    layers: int = 1
    key_dist: str = "normal"       # "normal" or "student_t3"
    outliers: int = 4              # outlier key channels per kv head
    outlier_scale: float = 10.0
    cfg_id: int = 0
    note: str = ""

    @property
    def group_q(self) -> int:
        return self.num_q_heads // self.num_kv_heads


def _rng(cfg: int, layer: int, seq: int, tensor: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng([MAGIC, cfg, layer, seq, tensor, *extra])


def ragged_lens(cfg: int, batch: int, lo: int, hi: int) -> Tuple[int, ...]:
    """Context lengths drawn uniformly from [lo, hi] (inclusive), seeded."""
    r = _rng(cfg, 0, 0, T_LENS)
    return tuple(int(x) for x in r.integers(lo, hi + 1, size=batch))


def workload(idx: int, bits: Optional[int] = None) -> Workload:
    """The five synthetic workloads, by index.

    0: one Llama-3.1-8B-shaped layer, 4K context, K2V2, groups of 32.
    1: one Llama-3.1-8B-shaped layer, 32K context, K1V1, groups of 32.
    2: Llama-3.1-8B shapes at 128K context, K1V1, 32 layers + 1-token appends.
    3: Mistral-7B shapes, batch 16, ragged 8K-32K, K2V2 / K4V4 halves,
       key groups of 64 tokens, value groups of 32 channels.
    4: Qwen2.5-14B shapes (40 q heads / 8 kv heads), batch 4, 128K, a 128-token
       fp16 window, Student-t(3) keys; ``bits`` picks K1V1/K2V2/K4V4/K8V8.
    """
    if idx == 0:
        return Workload("llama8b_L4096_K2V2_G32", 1, 32, 8, 128, (4096,), (2,), (2,),
                        32, 32, 0, cfg_id=0)
    if idx == 1:
        return Workload("llama8b_L32768_K1V1_G32", 1, 32, 8, 128, (32768,), (1,), (1,),
                        32, 32, 0, cfg_id=1)
    if idx == 2:
        return Workload("llama8b_L131072_K1V1_G32_32layers", 1, 32, 8, 128, (131072,), (1,), (1,),
                        32, 32, 0, layers=32, cfg_id=2)
    if idx == 3:
        lens = ragged_lens(3, 16, 8192, 32768)
        return Workload("mistral7b_B16_ragged8K-32K_K2V2+K4V4_Gk64_Gv32", 16, 32, 8, 128, lens,
                        (2,) * 8 + (4,) * 8, (2,) * 8 + (4,) * 8, 64, 32, 0, cfg_id=3)
    if idx == 4:
        b = 1 if bits is None else int(bits)
        return Workload(f"qwen14b_B4_L131072_K{b}V{b}_G32_R128", 4, 40, 8, 128, (131072,) * 4,
                        (b,) * 4, (b,) * 4, 32, 32, 128, key_dist="student_t3", cfg_id=4)
    raise ValueError(f"unknown workload {idx}")


def outlier_channels(w: Workload, layer: int, seq: int) -> np.ndarray:
    """[Hkv][outliers] distinct channel indices per kv head."""
    r = _rng(w.cfg_id, layer, seq, T_OUTLIER)
    return np.stack([r.choice(w.head_dim, w.outliers, replace=False)
                     for _ in range(w.num_kv_heads)]) if w.outliers else \
        np.zeros((w.num_kv_heads, 0), dtype=np.int64)


def _keys(w: Workload, r: np.random.Generator, shape, outl: np.ndarray) -> np.ndarray:
    if w.key_dist == "normal":
        x = r.standard_normal(shape, dtype=np.float32)
    elif w.key_dist == "student_t3":
        x = r.standard_t(3, size=shape).astype(np.float32)
    else:
        raise ValueError(w.key_dist)
    for h in range(shape[1]):
        x[:, h, outl[h]] *= w.outlier_scale
    return np.clip(x, -CLIP, CLIP).astype(np.float16)


def gen_q(w: Workload, layer: int = 0, seq: int = 0) -> np.ndarray:
    """q for one sequence: fp16 [Hq][d], ~N(0,1)."""
    r = _rng(w.cfg_id, layer, seq, T_Q)
    return r.standard_normal((w.num_q_heads, w.head_dim), dtype=np.float32).astype(np.float16)


def gen_q_chunk(w: Workload, n_q: int, layer: int = 0, seq: int = 0) -> np.ndarray:
    """Queries of the last n_q positions of one sequence: fp16 [n_q][Hq][d], ~N(0,1)."""
    r = _rng(w.cfg_id, layer, seq, T_Q_CHUNK, n_q)
    return r.standard_normal((n_q, w.num_q_heads, w.head_dim), dtype=np.float32).astype(np.float16)


def gen_kv(w: Workload, layer: int, seq: int, n: Optional[int] = None,
           heads: Optional[List[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Prefill K and V for one sequence: fp16 [n][Hkv][d] each.

    ``heads`` restricts the draw to some kv heads (others are left zero) while
    keeping their values identical to a full draw: each head has its own stream.
    """
    n = w.lens[seq] if n is None else n
    outl = outlier_channels(w, layer, seq)
    K = np.zeros((n, w.num_kv_heads, w.head_dim), dtype=np.float16)
    V = np.zeros_like(K)
    for h in (range(w.num_kv_heads) if heads is None else heads):
        rk = _rng(w.cfg_id, layer, seq, T_K, h)
        rv = _rng(w.cfg_id, layer, seq, T_V, h)
        K[:, h:h + 1, :] = _keys(w, rk, (n, 1, w.head_dim), outl[h:h + 1])
        V[:, h, :] = rv.standard_normal((n, w.head_dim), dtype=np.float32).astype(np.float16)
    return K, V


def gen_append(w: Workload, layer: int, seq: int, step: int, n: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """Tokens appended at decode step ``step``: fp16 [n][Hkv][d] each.

    They reuse the layer's outlier channels, like the prefill keys.
    """
    outl = outlier_channels(w, layer, seq)
    rk = _rng(w.cfg_id, layer, seq, T_APPEND_K, step)
    rv = _rng(w.cfg_id, layer, seq, T_APPEND_V, step)
    K = _keys(w, rk, (n, w.num_kv_heads, w.head_dim), outl)
    V = rv.standard_normal((n, w.num_kv_heads, w.head_dim), dtype=np.float32).astype(np.float16)
    return K, V


def gen_kv_device(w: Workload, layer: int, seq: int, n: int, device, torch):
    """Bulk prefill K and V on a device, for timing runs only.

    Uses torch's seeded device generator (same distributions, different
    stream from :func:`gen_kv`); used where drawing gigabytes on the host
    would dominate a benchmark's set-up time.
    """
    g = torch.Generator(device=device)
    g.manual_seed(int(np.random.SeedSequence([MAGIC, w.cfg_id, layer, seq]).generate_state(1)[0]))
    shape = (n, w.num_kv_heads, w.head_dim)
    if w.key_dist == "normal":
        K = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    else:
        # Student-t(3) = N / sqrt(chi2_3 / 3)
        z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        c = torch.randn((3,) + shape, generator=g, device=device, dtype=torch.float32).pow_(2).sum(0)
        K = z / torch.sqrt(c / 3.0)
    outl = torch.as_tensor(outlier_channels(w, layer, seq), device=device)
    for h in range(w.num_kv_heads):
        K[:, h, outl[h]] *= w.outlier_scale
    K = K.clamp_(-CLIP, CLIP).to(torch.float16)
    V = torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.float16)
    return K, V
