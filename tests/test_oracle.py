"""Pins of the CPU oracle against facts it does not compute itself.

- fp16 decoding and the fp16 ceiling: exhaustive over every fp16 pattern,
  checked against NumPy's binary16 conversion.
- The quantizer: an exact-rational brute force (fractions.Fraction, the fp16
  grid enumerated by NumPy, Python's half-to-even round) on many small groups,
  forced ties and subnormal scales included; plus the error bound
  |x - x^| <= s/2 and the constant-group round trip.
- The byte layout: images written out by hand from the layout's definition.
- Attention: torch's scaled_dot_product_attention in fp64 (a library routine)
  on tiny shapes, and closed forms: a single token returns its value row,
  identical keys return the mean of V with uniform weights, weights sum to 1,
  a constant key shift leaves the output unchanged (softmax shift invariance,
  Motivation, "Decode-Time Analysis of Accuracy Loss"), GQA equals MHA with
  repeated kv heads, token order does not matter.
"""
import bisect
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

# ---------------------------------------------------------------- fp16 basics

ALL_U16 = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
POS_FINITE = np.arange(1, 0x7C00, dtype=np.uint32).astype(np.uint16)
POS_VALUES = POS_FINITE.view(np.float16).astype(np.float64)
POS_FRACS = [Fraction(float(v)) for v in POS_VALUES]  # exact, increasing


def test_half_value_matches_numpy_for_every_pattern():
    ref = ALL_U16.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_value(int(h)) for h in ALL_U16])
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()
    # sign of zero survives
    assert np.signbit(oracle.half_value(0x8000)) and not np.signbit(oracle.half_value(0))


def test_half_ceil_exhaustive():
    # every representable value maps to itself
    for h, v in zip(POS_FINITE, POS_VALUES):
        assert oracle.half_ceil(v) == int(h)
    # midpoints and values just above a representable value go up one step;
    # values just below stay
    for i in range(len(POS_VALUES) - 1):
        lo, hi = POS_VALUES[i], POS_VALUES[i + 1]
        assert oracle.half_ceil((lo + hi) / 2) == int(POS_FINITE[i + 1])
        assert oracle.half_ceil(np.nextafter(lo, np.inf)) == int(POS_FINITE[i + 1])
        assert oracle.half_ceil(np.nextafter(hi, 0.0)) == int(POS_FINITE[i + 1])
    assert oracle.half_ceil(0.0) == 0
    assert oracle.half_ceil(1e-300) == 1  # smallest subnormal
    assert oracle.half_ceil(65504.0) == 0x7BFF
    with pytest.raises(oracle.OracleError):
        oracle.half_ceil(np.nextafter(65504.0, np.inf))
    with pytest.raises(oracle.OracleError):
        oracle.half_ceil(float("inf"))
    with pytest.raises(oracle.OracleError):
        oracle.half_ceil(-1.0)


# -------------------------------------------------- quantizer vs brute force

def bf_ceil16(s: Fraction):
    if s == 0:
        return Fraction(0)
    i = bisect.bisect_left(POS_FRACS, s)
    return POS_FRACS[i] if i < len(POS_FRACS) else None


def bf_quantize(xs: np.ndarray, bits: int):
    vals = [Fraction(float(x)) for x in xs.astype(np.float64)]
    mn, mx = min(vals), max(vals)
    s = bf_ceil16((mx - mn) / (2 ** bits - 1))
    if s is None:
        return None
    codes = [0] * len(vals) if s == 0 else [round((v - mn) / s) for v in vals]
    return s, mn, codes


def _groups(rng: np.random.Generator):
    """Small fp16 groups covering the shapes the quantizer meets."""
    out = []
    for n in (1, 2, 3, 5, 32, 64):
        for kind in ("normal", "outlier", "tiny", "huge", "student", "int"):
            for _ in range(6 if n <= 5 else 3):
                if kind == "normal":
                    x = rng.standard_normal(n)
                elif kind == "outlier":
                    x = rng.standard_normal(n) * np.where(rng.random(n) < 0.2, 10.0, 1.0)
                elif kind == "tiny":          # subnormal fp16 range -> subnormal scales
                    x = rng.standard_normal(n) * 3e-6
                elif kind == "huge":
                    x = rng.uniform(-16000, 16000, n)
                elif kind == "student":
                    x = rng.standard_t(3, n)
                else:
                    x = rng.integers(-8, 9, n).astype(np.float64)
                out.append(x.astype(np.float16))
    return out


def _tie_groups():
    """Groups whose (x - z) / s lands exactly on k + 1/2 for every bit width."""
    out = []
    for bits in (1, 2, 4, 8):
        qmax = 2 ** bits - 1
        for s in (0.25, 1.0, 2.0 ** -20, 0.5):
            z = -3.0 if s >= 0.25 else 0.0
            xs = [z, z + qmax * s] + [z + (k + 0.5) * s for k in range(min(qmax, 6))]
            out.append((bits, np.array(xs, dtype=np.float64).astype(np.float16)))
    return out


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_quantizer_matches_exact_rational_brute_force(bits):
    rng = np.random.default_rng([7, bits])
    groups = _groups(rng) + [x for b, x in _tie_groups() if b == bits]
    for x in groups:
        ref = bf_quantize(x, bits)
        s, z, codes = oracle.quantize_group(x, bits)
        assert ref is not None
        rs, rz, rc = ref
        assert Fraction(oracle.half_value(s)) == rs
        assert Fraction(oracle.half_value(z)) == rz and z != 0x8000
        assert list(codes) == rc, (x, bits)


def test_ties_round_to_even():
    # b = 2, s = 0.25, z = 0: 0.375 / 0.25 = 1.5 -> 2 and 0.125 / 0.25 = 0.5 -> 0
    x = np.array([0.0, 0.75, 0.375, 0.125, 0.625], dtype=np.float16)
    s, z, codes = oracle.quantize_group(x, 2)
    assert oracle.half_value(s) == 0.25 and oracle.half_value(z) == 0.0
    assert list(codes) == [0, 3, 2, 0, 2]


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_error_bound_and_code_range(bits):
    rng = np.random.default_rng([11, bits])
    qmax = 2 ** bits - 1
    for x in _groups(rng):
        s, z, codes = oracle.quantize_group(x, bits)
        sv, zv = Fraction(oracle.half_value(s)), Fraction(oracle.half_value(z))
        vals = [Fraction(float(v)) for v in x.astype(np.float64)]
        assert all(0 <= c <= qmax for c in codes)
        for v, c in zip(vals, codes):
            assert abs(v - (zv + c * sv)) <= sv / 2
        assert codes[int(np.argmin(x))] == 0
        if oracle.half_value(s) >= 2.0 ** -14:  # normal scale: the maximum maps to the top code
            assert codes[int(np.argmax(x))] == qmax


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_constant_group_round_trips_exactly(bits):
    for v in (0.0, -0.0, 1.5, -65504.0, 6e-8, 3.14159):
        x = np.full(32, v, dtype=np.float16)
        s, z, codes = oracle.quantize_group(x, bits)
        assert s == 0 and (codes == 0).all()
        assert oracle.half_value(z) == float(x[0])
        assert z != 0x8000


def test_range_errors():
    with pytest.raises(oracle.OracleError) as e:   # range 131008 > 65504 at one bit
        oracle.quantize_group(np.array([-65504, 65504], dtype=np.float16), 1)
    assert e.value.status == oracle.ERR_RANGE
    s, _, _ = oracle.quantize_group(np.array([-65504, 65504], dtype=np.float16), 2)
    assert oracle.half_value(s) == oracle.half_value(oracle.half_ceil(131008 / 3))
    with pytest.raises(oracle.OracleError):
        oracle.quantize_group(np.array([1.0, np.inf], dtype=np.float16), 4)
    with pytest.raises(oracle.OracleError):
        oracle.quantize_group(np.array([1.0, np.nan], dtype=np.float16), 4)


# ------------------------------------------------------- layout, by hand

def _h(v):
    """fp16 bytes (little-endian) of a value."""
    return list(np.array([v], dtype=np.float16).view(np.uint8))


def test_layout_one_bit_by_hand():
    # d = 8, one key group of 2 tokens, one value group of 8 channels, L = 3,
    # no window -> Lq = 2 and one fp16 tail token.
    K = np.zeros((3, 8), dtype=np.float16)
    K[0] = [1, 0, 1, 1, 0, 0, 0, 0]
    K[1] = [0, 1, 0, 0, 1, 1, 1, 1]
    K[2] = [9, 9, 9, 9, 9, 9, 9, 9]
    V = np.zeros((3, 8), dtype=np.float16)
    V[0] = [2, 2, 2, 2, 2, 2, 2, 4]     # z = 2, s = 2 -> codes 0000 0001
    V[1] = [-1, -1, -1, -1, -1, -1, -1, -1]  # constant -> s = 0, z = -1
    V[2] = [5, 6, 7, 8, 9, 10, 11, 12]
    img = oracle.build_head(K, V, 1, 1, 2, 8, 0)
    expect = []
    expect += [0x0D, 0xF2]                       # key code rows (1 byte each)
    expect += _h(1.0) * 8 + _h(0.0) * 8          # key scales then zeros
    expect += [0x80, 0x00]                       # value code rows
    expect += _h(2.0) + _h(2.0) + _h(0.0) + _h(-1.0)  # (s, z) per token
    expect += sum((_h(9.0) for _ in range(8)), [])     # key tail
    expect += sum((_h(float(v)) for v in V[2]), [])    # value tail
    assert list(img) == expect


def test_layout_two_bit_by_hand():
    # d = 8, key group of 4 tokens: per channel values (code, 0, 3, 1) give
    # z = 0, s = 1, so token 0's codes are its values.
    K = np.zeros((4, 8), dtype=np.float16)
    K[0] = [3, 0, 1, 2, 2, 1, 0, 3]
    K[1] = 0
    K[2] = 3
    K[3] = 1
    V = np.tile(np.array([0, 1, 2, 3, 3, 2, 1, 0], dtype=np.float16), (4, 1))
    img = oracle.build_head(K, V, 2, 2, 4, 4, 0)
    rows = [list(img[i * 2:(i + 1) * 2]) for i in range(4)]
    assert rows[0] == [0x93, 0xC6]   # 3,0,1,2 -> 0b10_01_00_11 ; 2,1,0,3 -> 0b11_00_01_10
    assert rows[1] == [0x00, 0x00]
    assert rows[2] == [0xFF, 0xFF]
    assert rows[3] == [0x55, 0x55]
    meta = img[8:8 + 32]
    assert list(meta[:16]) == _h(1.0) * 8 and list(meta[16:]) == _h(0.0) * 8
    # values: group [0,1,2,3] -> s = 1, z = 0, codes 0..3 ; group [3,2,1,0] -> codes 3..0
    vrows = img[40:48]
    assert list(vrows[:2]) == [0xE4, 0x1B]
    vmeta = img[48:48 + 16]
    assert list(vmeta[:8]) == _h(1.0) + _h(0.0) + _h(1.0) + _h(0.0)


def test_layout_eight_and_four_bit_rows():
    # d = 8, key group of 2 tokens at 8 bits, one value group of 8 channels at 4 bits
    K = np.zeros((2, 8), dtype=np.float16)
    K[1] = [255, 1, 2, 3, 4, 5, 6, 7]
    img = oracle.build_head(K, K, 8, 4, 2, 8, 0)
    # key rows are 8 bytes; channel 0 has values (0, 255) -> s = 1, codes (0, 255)
    assert img[0] == 0 and img[8] == 255
    # value rows start after 16 key-code bytes and 32 key-meta bytes, 4 bytes each;
    # token 0 is a constant group, token 1 packs two 4-bit codes per byte, low nibble first
    s, z, codes = oracle.quantize_group(K[1], 4)
    assert list(img[48:52]) == [0, 0, 0, 0]
    assert list(img[52:56]) == [int(codes[2 * i]) | (int(codes[2 * i + 1]) << 4) for i in range(4)]
    assert list(img[56:60]) == _h(0.0) + _h(0.0)
    assert list(img[60:64]) == [s & 0xFF, s >> 8, z & 0xFF, z >> 8]


def test_dequant_of_a_hand_written_image():
    # d = 8, b = 1, key group 2, value group 4, L = 2 (all quantized)
    img = []
    img += [0b00000101, 0b11111010]                      # key rows
    img += _h(0.5) * 8 + _h(-1.0) * 8                    # key s, z
    img += [0b11110000, 0b00001111]                      # value rows
    img += _h(0.25) + _h(1.0) + _h(3.0) + _h(-2.0)       # token 0 groups
    img += _h(0.0) + _h(7.0) + _h(1.0) + _h(0.0)         # token 1 groups
    Kh, Vh = oracle.dequant_head(np.array(img, dtype=np.uint8), 2, 8, 1, 1, 2, 4, 0)
    assert Kh[0].tolist() == [-0.5, -1, -0.5, -1, -1, -1, -1, -1]
    assert Kh[1].tolist() == [-1, -0.5, -1, -0.5, -0.5, -0.5, -0.5, -0.5]
    assert Vh[0].tolist() == [1, 1, 1, 1, 1, 1, 1, 1]
    assert Vh[1].tolist() == [7, 7, 7, 7, 0, 0, 0, 0]


@pytest.mark.parametrize("bk,bv,gk,gv,R,L", [
    (1, 1, 32, 32, 0, 100), (2, 2, 32, 32, 0, 64), (4, 2, 64, 32, 0, 130),
    (8, 8, 32, 16, 0, 33), (1, 4, 32, 32, 40, 111), (2, 1, 16, 128, 128, 150),
    (1, 1, 32, 32, 0, 0), (1, 1, 32, 32, 0, 31), (4, 4, 32, 32, 200, 150)])
def test_image_round_trip_bound_and_sizes(bk, bv, gk, gv, R, L):
    d = 128
    rng = np.random.default_rng([L, bk, bv, gk])
    K = (rng.standard_normal((L, d)) * np.where(rng.random(d) < 0.05, 10, 1)).astype(np.float16)
    V = rng.standard_normal((L, d)).astype(np.float16)
    img = oracle.build_head(K, V, bk, bv, gk, gv, R)
    Lq = oracle.quantized_len(L, gk, R)
    assert Lq == (max(0, L - R) // gk) * gk
    assert img.size == Lq * d * (bk + bv) // 8 + (Lq // gk) * 4 * d + Lq * (d // gv) * 4 + (L - Lq) * 4 * d
    Kh, Vh = oracle.dequant_head(img, L, d, bk, bv, gk, gv, R)
    # tail is exact
    assert (Kh[Lq:] == K[Lq:].astype(np.float64)).all() and (Vh[Lq:] == V[Lq:].astype(np.float64)).all()
    # quantized part: error within half a scale of its own group
    for j in range(Lq // gk):
        blk = K[j * gk:(j + 1) * gk].astype(np.float64)
        rngk = blk.max(0) - blk.min(0)
        assert (np.abs(Kh[j * gk:(j + 1) * gk] - blk) <= rngk / (2 ** bk - 1) * (1 + 2 ** -10) / 2 + 1e-30).all()
    for t in range(Lq):
        for g in range(d // gv):
            seg = V[t, g * gv:(g + 1) * gv].astype(np.float64)
            bound = (seg.max() - seg.min()) / (2 ** bv - 1) * (1 + 2 ** -10) / 2
            assert (np.abs(Vh[t, g * gv:(g + 1) * gv] - seg) <= bound + 1e-30).all()


def test_appends_commute_with_the_layout():
    # the image depends only on the final token sequence: a prefix's image is
    # a sub-image of the full one (finished groups never change)
    d, gk, gv = 128, 32, 32
    rng = np.random.default_rng(5)
    K = rng.standard_normal((100, d)).astype(np.float16)
    V = rng.standard_normal((100, d)).astype(np.float16)
    full = oracle.build_head(K, V, 2, 2, gk, gv, 0)
    part = oracle.build_head(K[:64], V[:64], 2, 2, gk, gv, 0)
    rowb = d * 2 // 8
    assert (full[:64 * rowb] == part[:64 * rowb]).all()


# ----------------------------------------------------------------- attention

def _sdpa_ref(q16, Kh, Vh):
    """torch scaled_dot_product_attention in fp64 on the CPU, MHA form."""
    Hq, d = q16.shape
    Hkv = Kh.shape[0]
    q = torch.from_numpy(q16.astype(np.float64)).view(1, Hq, 1, d)
    k = torch.from_numpy(Kh).repeat_interleave(Hq // Hkv, dim=0).unsqueeze(0)
    v = torch.from_numpy(Vh).repeat_interleave(Hq // Hkv, dim=0).unsqueeze(0)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v)
    return o.view(Hq, d).numpy()


@pytest.mark.parametrize("L,d,Hq,Hkv", [(1, 8, 1, 1), (2, 8, 4, 1), (3, 128, 4, 4), (31, 128, 8, 2),
                                        (32, 8, 5, 1), (33, 128, 10, 2), (65, 128, 32, 8)])
def test_attention_matches_torch_sdpa(L, d, Hq, Hkv):
    rng = np.random.default_rng([L, d, Hq])
    q = rng.standard_normal((Hq, d)).astype(np.float16)
    Kh = rng.standard_normal((Hkv, L, d)) * 2
    Vh = rng.standard_normal((Hkv, L, d))
    out = oracle.attention(q, Kh, Vh)
    np.testing.assert_allclose(out, _sdpa_ref(q, Kh, Vh), rtol=1e-12, atol=1e-13)


def test_attention_closed_forms():
    rng = np.random.default_rng(3)
    d, L = 128, 50
    q = rng.standard_normal((4, d)).astype(np.float16)
    # one token: output is that token's value row, exactly
    Kh = rng.standard_normal((1, 1, d))
    Vh = rng.standard_normal((1, 1, d))
    assert (oracle.attention(q, Kh, Vh) == np.repeat(Vh[0], 4, 0)).all()
    # identical keys: uniform weights, mean of V
    Kh = np.repeat(rng.standard_normal((1, 1, d)), L, axis=1)
    Vh = rng.standard_normal((1, L, d))
    out, w = oracle.attention(q, Kh, Vh, return_weights=True)
    np.testing.assert_allclose(w, 1.0 / L, rtol=1e-13)
    np.testing.assert_allclose(out, np.repeat(Vh[0].mean(0, keepdims=True), 4, 0), rtol=1e-12, atol=1e-14)
    # weights sum to 1 on random data
    Kh = rng.standard_normal((1, L, d)) * 5
    _, w = oracle.attention(q, Kh, Vh, return_weights=True)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-13)
    # a dominating key: output tends to that value row
    Kh = rng.standard_normal((1, L, d)) * 0.01
    q1 = np.ones((1, d), dtype=np.float16)
    Kh[0, 17] = 100.0
    out = oracle.attention(q1, Kh, Vh)
    np.testing.assert_allclose(out[0], Vh[0, 17], rtol=1e-12, atol=1e-12)
    # no tokens: zeros by convention
    assert (oracle.attention(q, np.zeros((1, 0, d)), np.zeros((1, 0, d))) == 0).all()


def test_attention_shift_gqa_and_permutation_invariance():
    rng = np.random.default_rng(4)
    d, L, Hq, Hkv = 128, 77, 8, 2
    q = rng.standard_normal((Hq, d)).astype(np.float16)
    Kh = rng.standard_normal((Hkv, L, d)) * 3
    Vh = rng.standard_normal((Hkv, L, d))
    base = oracle.attention(q, Kh, Vh)
    # adding the same vector to every key shifts every score of a head by a constant
    u = rng.standard_normal((Hkv, 1, d)) * 4
    np.testing.assert_allclose(oracle.attention(q, Kh + u, Vh), base, rtol=1e-10, atol=1e-12)
    # GQA equals MHA with each kv head repeated for its query heads
    rep = oracle.attention(q, np.repeat(Kh, Hq // Hkv, 0), np.repeat(Vh, Hq // Hkv, 0))
    np.testing.assert_allclose(rep, base, rtol=1e-14, atol=1e-15)
    # the order of the cached tokens does not matter
    perm = rng.permutation(L)
    np.testing.assert_allclose(oracle.attention(q, Kh[:, perm], Vh[:, perm]), base, rtol=1e-12, atol=1e-14)


def test_decode_seq_pipeline_consistent():
    from workloads import Workload, gen_kv, gen_q
    w = Workload("tiny", 1, 8, 2, 128, (150,), (2,), (2,), 32, 32, 20, cfg_id=99)
    K, V = gen_kv(w, 0, 0)
    q = gen_q(w)
    out = oracle.decode_seq(q, K, V, 2, 2, 32, 32, 20)
    Khs, Vhs = [], []
    for h in range(2):
        img = oracle.build_head(K[:, h], V[:, h], 2, 2, 32, 32, 20)
        Kh, Vh = oracle.dequant_head(img, 150, 128, 2, 2, 32, 32, 20)
        Khs.append(Kh)
        Vhs.append(Vh)
    np.testing.assert_allclose(out, _sdpa_ref(q, np.stack(Khs), np.stack(Vhs)), rtol=1e-12, atol=1e-13)


# ------------------------------------------------------- chunk queries (causal)

@pytest.mark.parametrize("L,n_q,d,Hq,Hkv", [(1, 1, 8, 1, 1), (5, 5, 8, 4, 1), (33, 7, 128, 4, 1),
                                            (65, 16, 128, 8, 2), (40, 3, 128, 10, 2)])
def test_chunk_attention_matches_masked_sdpa(L, n_q, d, Hq, Hkv):
    # torch SDPA over all n_q queries at once with an explicit boolean mask
    # (query i sees tokens t <= L - n_q + i): a different formulation
    rng = np.random.default_rng([L, n_q, d, Hq])
    q = rng.standard_normal((n_q, Hq, d)).astype(np.float16)
    Kh = rng.standard_normal((Hkv, L, d)) * 2
    Vh = rng.standard_normal((Hkv, L, d))
    out = oracle.chunk_attention(q, Kh, Vh)
    qt = torch.from_numpy(q.astype(np.float64)).permute(1, 0, 2).unsqueeze(0)     # [1][Hq][n_q][d]
    k = torch.from_numpy(Kh).repeat_interleave(Hq // Hkv, dim=0).unsqueeze(0)     # [1][Hq][L][d]
    v = torch.from_numpy(Vh).repeat_interleave(Hq // Hkv, dim=0).unsqueeze(0)
    mask = torch.arange(L)[None, :] <= (L - n_q + torch.arange(n_q))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, k, v, attn_mask=mask)
    np.testing.assert_allclose(out, ref[0].permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_chunk_attention_causality_and_end_cases():
    rng = np.random.default_rng(12)
    d, L, n_q, Hq, Hkv = 128, 60, 9, 8, 2
    q = rng.standard_normal((n_q, Hq, d)).astype(np.float16)
    Kh = rng.standard_normal((Hkv, L, d)) * 3
    Vh = rng.standard_normal((Hkv, L, d))
    base = oracle.chunk_attention(q, Kh, Vh)
    # the last query sees the whole cache: plain decode attention
    assert (base[-1] == oracle.attention(q[-1], Kh, Vh)).all()
    # a token past a query's position changes nothing for that query, and
    # changes every query that sees it
    t = L - n_q + 4
    K2, V2 = Kh.copy(), Vh.copy()
    K2[:, t] += 5.0
    V2[:, t] -= 7.0
    pert = oracle.chunk_attention(q, K2, V2)
    assert (pert[:4] == base[:4]).all()
    assert all(np.abs(pert[i] - base[i]).max() > 1e-6 for i in range(4, n_q))
    # n_q = L: the first query sees only token 0, its output is that value row
    qa = rng.standard_normal((L, Hq, d)).astype(np.float16)
    full = oracle.chunk_attention(qa, Kh, Vh)
    assert (full[0] == np.repeat(Vh[:, 0], Hq // Hkv, axis=0)).all()
    with pytest.raises(oracle.OracleError):
        oracle.chunk_attention(qa[:1].repeat(L + 1, 0), Kh, Vh)
