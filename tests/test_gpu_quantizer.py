"""The GPU's quantize-on-append kernel on crafted groups (quant_edges.py):
key and value groups whose scale is every positive finite fp16 value that
fp16 inputs reach, approached exactly, from just above the value below, from
just below and at the midpoint, with elements on exact rounding ties
(min + (k + 1/2) s).  The packed bytes (codes, scales, zeros) must equal the
oracle's canonical image, on the matrix-core layout (4 query heads per kv
head) after one prefill and on the canonical layout (1 query head per kv
head) after appends of 45 tokens at a time, which pack groups from the fp16
ring."""
import functools

import numpy as np
import pytest

import oracle
from helpers import log
from quant_edges import crafted_kv

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _inputs(bits):
    return crafted_kv(bits)


@pytest.mark.parametrize("bits,gq,chunk", [(1, 4, 0), (2, 4, 0), (4, 4, 0), (8, 4, 0), (2, 1, 45), (8, 1, 45),
                                           (1, 1, 45)])
def test_crafted_scales_and_ties_pack_like_the_oracle(bits, gq, chunk):
    from paper_2607_16248_amd import KVCache

    K, V, cases = _inputs(bits)
    L, hkv, d = K.shape
    log(f"[quant] K{bits}V{bits} gq {gq}: {len(cases)} crafted groups over {L} tokens, chunk {chunk or L}")
    cache = KVCache(1, gq * hkv, hkv, L, [bits], [bits], key_group=32, value_group=32, fp16_window=0)
    Kd, Vd = torch.from_numpy(K[None]).cuda(), torch.from_numpy(V[None]).cuda()
    step = chunk or L
    for p in range(0, L, step):
        n = min(step, L - p)
        cache.append(Kd[:, p:p + n].contiguous(), Vd[:, p:p + n].contiguous(), [n])
    torch.cuda.synchronize()
    cache.check()  # no scale beyond the fp16 range: the device flag stays clear
    for h in range(hkv):
        got = cache.export(0, h)
        ref = oracle.build_head(np.ascontiguousarray(K[:, h]), np.ascontiguousarray(V[:, h]), bits, bits, 32, 32, 0)
        bad = np.flatnonzero(got != ref)
        assert got.size == ref.size and bad.size == 0, f"head {h}: {bad.size} bytes differ, first at {bad[:5]}"
