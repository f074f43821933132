"""Shared set-up for the GPU parity tests: build a cache through the C ABI
from seeded inputs, and compare its bytes and outputs with the oracle."""
from __future__ import annotations

import sys
from typing import List, Optional, Sequence

import numpy as np

import oracle
from paper_2607_16248_amd import kvq
from workloads import Workload, gen_kv, gen_q

# Row-normwise relative error bound of decode attention against the fp64
# oracle on the same dequantized cache.
ATTN_TOL = 2e-3


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """max_c |got - ref| / max_c |ref| for every leading index."""
    num = np.abs(got.astype(np.float64) - ref).max(-1)
    den = np.abs(ref).max(-1)
    return num / np.maximum(den, 1e-300)


class Case:
    """Seeded inputs for a batch plus a cache holding them."""

    def __init__(self, w: Workload, layer: int = 0, heads: Optional[List[int]] = None,
                 device: str = "cuda", max_tokens: Optional[int] = None, **cache_kw):
        import torch
        self.w = w
        self.heads = heads
        self.K, self.V, self.q = [], [], []
        for s in range(w.batch):
            K, V = gen_kv(w, layer, s, heads=heads)
            self.K.append(K)
            self.V.append(V)
            self.q.append(gen_q(w, layer, s))
        self.cache = kvq.KVCache(w.batch, w.num_q_heads, w.num_kv_heads,
                                 max_tokens or max(max(w.lens), 1), list(w.bits_k), list(w.bits_v),
                                 key_group=w.key_group, value_group=w.value_group,
                                 fp16_window=w.window, device=device, **cache_kw)
        self.qd = torch.from_numpy(np.stack(self.q)).to(device)

    def append_all(self, chunks: Optional[Sequence[int]] = None):
        """Append every sequence's tokens, in one call or in the given chunk sizes."""
        import torch
        w = self.w
        pos = [0] * w.batch
        steps = [max(w.lens)] if chunks is None else list(chunks)
        for n in steps:
            n_new = [min(n, w.lens[s] - pos[s]) for s in range(w.batch)]
            nmax = max(max(n_new), 1)
            Kb = np.zeros((w.batch, nmax, w.num_kv_heads, w.head_dim), dtype=np.float16)
            Vb = np.zeros_like(Kb)
            for s in range(w.batch):
                Kb[s, :n_new[s]] = self.K[s][pos[s]:pos[s] + n_new[s]]
                Vb[s, :n_new[s]] = self.V[s][pos[s]:pos[s] + n_new[s]]
            self.cache.append(torch.from_numpy(Kb).cuda(), torch.from_numpy(Vb).cuda(), n_new)
            pos = [p + n for p, n in zip(pos, n_new)]
        torch.cuda.synchronize()
        assert pos == list(w.lens)

    def oracle_image(self, s: int, h: int) -> np.ndarray:
        w = self.w
        return oracle.build_head(self.K[s][:, h, :], self.V[s][:, h, :], w.bits_k[s], w.bits_v[s],
                                 w.key_group, w.value_group, w.window)

    def oracle_out(self, s: int, heads: Optional[List[int]] = None) -> np.ndarray:
        w = self.w
        return oracle.decode_seq(self.q[s], self.K[s], self.V[s], w.bits_k[s], w.bits_v[s],
                                 w.key_group, w.value_group, w.window, heads=heads)

    def decode(self) -> np.ndarray:
        import torch
        out = self.cache.decode(self.qd)
        torch.cuda.synchronize()
        return out.cpu().numpy()
