"""The crafted quantizer groups of quant_edges.py, checked on the CPU: the
oracle gives each group the scale pattern it was built for, and every
positive finite fp16 pattern that fp16 inputs can reach is hit exactly,
from just above the pattern below it, from just below, and at the midpoint.
(The same groups go through the GPU's append kernel in test_gpu_quantizer.py.)"""
import numpy as np
import pytest

import oracle
from quant_edges import POS16, crafted_kv, scale_pairs, tie_pairs


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_crafted_groups_get_their_scale(bits):
    q = (1 << bits) - 1
    cases = scale_pairs(bits) + tie_pairs(bits)
    rng = np.random.default_rng(bits)
    from quant_edges import group_values
    for i, (mn, mx, p, kind) in enumerate(cases):
        if kind in ("exact", "tie") or i % 7 == 0:   # every exact case, a sample of the rest
            x = group_values(mn, mx, p, 32, rng)
            s, z, codes = oracle.quantize_group(x, bits)
            assert s == p, (mn, mx, p, kind, s)
            assert oracle.half_value(z) == mn
    exact = {p for _, _, p, k in cases if k == "exact"}
    # every pattern whose exact range fits inside the fp16 maximum is hit
    fits = {i + 1 for i, v in enumerate(POS16) if q * v <= 65504.0}
    assert fits <= exact
    if bits == 1:
        assert len(exact) == 0x7BFF
    # (at one bit s* is the range itself, a multiple of 2^-24, so below 2^-13,
    # where fp16 values are 2^-24 apart, nothing lies strictly between two)
    for kind in ("above", "below", "mid"):
        hit = {p for _, _, p, k in cases if k == kind}
        assert len(hit) >= 0.9 * len(exact), kind


def test_crafted_cache_layout():
    K, V, cases = crafted_kv(8)
    assert K.shape == V.shape and K.shape[0] % 32 == 0
    assert np.isfinite(K.astype(np.float64)).all() and np.isfinite(V.astype(np.float64)).all()
