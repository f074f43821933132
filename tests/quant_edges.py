"""Crafted quantizer inputs: groups whose scale lands on, or just beside,
every positive finite fp16 value.

The scale of a group is the smallest fp16 value s with s >= s*, where
s* = (max - min) / (2^b - 1) (asymmetric min-max quantization with the scale
rounded up; the library's reading of the paper's b-bit key/value storage).
For a bit width b and an fp16 pattern p (value v_p) this module builds fp16
pairs (min, max) whose range makes s*:
  - exactly v_p,
  - just above v_(p-1) (the pair of p-1 with its minimum moved one fp16 step
    down),
  - just below v_p (the pair of p with its minimum moved one step up),
  - the midpoint of v_(p-1) and v_p,
and fills each group of 32 elements with values between them, among them
the points min + (k + 1/2) v_p that fp16 can hold (exact rounding ties).
The intended pattern is a label only: the tests check it against the oracle
and compare the GPU's packed bytes with the oracle's image.  Pairs that fp16
inputs cannot reach (ranges beyond 2 * 65504) are left out.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

POS16 = np.arange(1, 0x7C00, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
F16_MAX = 65504.0


def _is_f16(x: float) -> bool:
    return bool(np.isfinite(x)) and abs(x) <= F16_MAX and float(np.float16(x)) == x


def _step(x: float, up: bool) -> float:
    """The next fp16 value above or below x (inf past the largest)."""
    with np.errstate(over="ignore"):
        return float(np.nextafter(np.float16(x), np.float16(np.inf if up else -np.inf)))


def _top_values() -> np.ndarray:
    return POS16[POS16 >= 16384.0]


def pair_for_range(D: float):
    """fp16 (mn, mx) with mx - mn == D exactly, or None."""
    if D <= 0:
        return None
    if D <= F16_MAX:
        mx = float(POS16[np.searchsorted(POS16, D)])  # smallest fp16 >= D
        mn = mx - D
        if _is_f16(mn):
            return (mn, mx)
    # ranges past the fp16 maximum (or a remainder fp16 cannot hold): a
    # negative minimum; search the maxima of the top binades
    cand = _top_values()
    cand = cand[cand - D >= -F16_MAX]
    mns = cand - D
    ok = (np.abs(mns) <= F16_MAX) & (mns.astype(np.float16).astype(np.float64) == mns)
    if ok.any():
        i = int(np.flatnonzero(ok)[0])
        return (float(mns[i]), float(cand[i]))
    return None


def scale_pairs(bits: int) -> List[Tuple[float, float, int, str]]:
    """(mn, mx, intended scale pattern, kind) for every reachable pattern."""
    q = (1 << bits) - 1
    exact = {}
    out = []
    for i, v in enumerate(POS16):
        pr = pair_for_range(q * v)
        if pr is not None:
            exact[i + 1] = pr
            out.append((pr[0], pr[1], i + 1, "exact"))
    def inside(mn, mx, p):  # q v_(p-1) < mx - mn <= q v_p, both ends finite fp16
        lo = q * POS16[p - 2] if p >= 2 else 0.0
        return _is_f16(mn) and _is_f16(mx) and lo < mx - mn <= q * POS16[p - 1]

    for p in range(1, len(POS16) + 1):
        # just above v_(p-1): widen the pair of p - 1 by one step of its minimum
        if p >= 2 and (p - 1) in exact:
            mn, mx = exact[p - 1]
            mn2 = _step(mn, up=False)
            if inside(mn2, mx, p):
                out.append((mn2, mx, p, "above"))
        # just below v_p: narrow the pair of p by one step of its minimum
        if p in exact:
            mn, mx = exact[p]
            mn2 = _step(mn, up=True)
            if inside(mn2, mx, p) and mx - mn2 < q * POS16[p - 1]:
                out.append((mn2, mx, p, "below"))
        # midpoint of v_(p-1) and v_p (p = 1: one fp16 step over 2^b - 1)
        D = q * (POS16[p - 2] + POS16[p - 1]) / 2 if p >= 2 else 2.0 ** -24
        pr = pair_for_range(D)
        if pr is not None and inside(pr[0], pr[1], p):
            out.append((pr[0], pr[1], p, "mid"))
    return out


def tie_pairs(bits: int) -> List[Tuple[float, float, int, str]]:
    """Groups with scale s (fp16) and zero z whose inner points sit on k + 1/2."""
    q = (1 << bits) - 1
    out = []
    for s in (0.25, 1.0, 2.0 ** -20, 0.5, 2.0 ** -24, 3.0):
        for z in (-3.0, 0.0, 1.5):
            mn, mx = z, z + q * s
            if _is_f16(mn) and _is_f16(mx):
                p = int(np.flatnonzero(POS16 == s)[0]) + 1
                out.append((mn, mx, p, "tie"))
    return out


def group_values(mn: float, mx: float, p: int, n: int, rng: np.random.Generator) -> np.ndarray:
    """n fp16 values in [mn, mx] holding both ends, the exact ties
    mn + (k + 1/2) v_p that fp16 represents, and random fill."""
    s = POS16[p - 1]
    vals = [mn, mx]
    k = 0
    while len(vals) < n // 2 and mn + (k + 0.5) * s < mx:
        t = mn + (k + 0.5) * s
        if _is_f16(t):
            vals.append(t)
        k += 1 if k < 4 else max(1, k)  # a few low codes, then spread out
    while len(vals) < n:
        vals.append(float(np.clip(np.float16(rng.uniform(mn, mx)), mn, mx)))
    v = np.array(vals[:n], dtype=np.float64)
    rng.shuffle(v)
    out = v.astype(np.float16)
    assert (out.astype(np.float64) == v).all()
    return out


def crafted_kv(bits: int, hkv: int = 8, d: int = 128, group: int = 32, seed: int = 0):
    """K, V fp16 [L][hkv][d] whose key groups (group tokens of one channel) and
    value groups (group channels of one token) are the crafted groups of this
    width, repeated cyclically to fill whole key groups; plus the labels
    (mn, mx, pattern, kind) in instance order."""
    rng = np.random.default_rng([0x51, bits, seed])
    cases = scale_pairs(bits) + tie_pairs(bits)
    groups = [group_values(mn, mx, p, group, rng) for mn, mx, p, _ in cases]
    n = len(groups)
    assert np.gcd(n, 7919) == 1
    ng = d // group
    per_kgroup = hkv * d                 # key instances per `group` tokens
    per_token = hkv * ng                 # value instances per token
    L = group * max(-(-n // per_kgroup), -(-n // (per_token * group)))
    K = np.empty((L, hkv, d), dtype=np.float16)
    V = np.empty((L, hkv, d), dtype=np.float16)
    for i in range((L // group) * per_kgroup):
        g = groups[i % n]
        j, h, c = i // per_kgroup, (i // d) % hkv, i % d
        K[j * group:(j + 1) * group, h, c] = g
    for i in range(L * per_token):
        g = groups[(i * 7919) % n]       # another order than the keys
        t, h, gg = i // per_token, (i // ng) % hkv, i % ng
        V[t, h, gg * group:(gg + 1) * group] = g
    return K, V, cases
