"""NumPy front-end of the CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product library.  Argument
marshalling only; every step of the computation is in oracle.c.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, ERR_ARG, ERR_RANGE = 0, 1, 4


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"oracle {what} failed with status {status}")
        self.status = status


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    L_, I_, SZ = ctypes.c_long, ctypes.c_int, ctypes.c_size_t
    lib.orc_half_value.argtypes = [ctypes.c_uint16]
    lib.orc_half_value.restype = ctypes.c_double
    lib.orc_half_ceil.argtypes = [ctypes.c_double, P]
    lib.orc_half_ceil.restype = I_
    lib.orc_quantize_group.argtypes = [P, L_, L_, I_, P, P, P]
    lib.orc_quantize_group.restype = I_
    lib.orc_quantized_len.argtypes = [L_, I_, I_]
    lib.orc_quantized_len.restype = L_
    lib.orc_head_bytes.argtypes = [L_, I_, I_, I_, I_, I_, I_]
    lib.orc_head_bytes.restype = SZ
    lib.orc_build_head.argtypes = [P, P, L_, L_, I_, I_, I_, I_, I_, I_, P]
    lib.orc_build_head.restype = I_
    lib.orc_dequant_head.argtypes = [P, L_, I_, I_, I_, I_, I_, I_, P, P]
    lib.orc_dequant_head.restype = I_
    lib.orc_attention.argtypes = [P, P, P, L_, I_, I_, I_, P, P]
    lib.orc_attention.restype = I_
    lib.orc_num_threads.argtypes = []
    lib.orc_num_threads.restype = I_
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _as_u16(x) -> np.ndarray:
    x = np.ascontiguousarray(x)
    if x.dtype == np.float16:
        return x.view(np.uint16)
    if x.dtype == np.uint16:
        return x
    raise TypeError(f"expected float16 or uint16 array, got {x.dtype}")


def half_value(h: int) -> float:
    return _load().orc_half_value(int(h) & 0xFFFF)


def half_ceil(s: float) -> int:
    out = np.zeros(1, dtype=np.uint16)
    st = _load().orc_half_ceil(float(s), _ptr(out))
    if st != OK:
        raise OracleError(st, "half_ceil")
    return int(out[0])


def quantize_group(x, bits: int) -> Tuple[int, int, np.ndarray]:
    """One group of fp16 values -> (scale bits, zero bits, codes)."""
    xu = _as_u16(x).ravel()
    s = np.zeros(1, dtype=np.uint16)
    z = np.zeros(1, dtype=np.uint16)
    codes = np.zeros(max(1, xu.size), dtype=np.uint8)
    st = _load().orc_quantize_group(_ptr(xu), xu.size, 1, int(bits), _ptr(s), _ptr(z), _ptr(codes))
    if st != OK:
        raise OracleError(st, "quantize_group")
    return int(s[0]), int(z[0]), codes[:xu.size]


def quantized_len(L: int, key_group: int, window: int) -> int:
    return int(_load().orc_quantized_len(int(L), int(key_group), int(window)))


def head_bytes(L: int, d: int, bits_k: int, bits_v: int, key_group: int, value_group: int,
               window: int) -> int:
    return int(_load().orc_head_bytes(L, d, bits_k, bits_v, key_group, value_group, window))


def build_head(K, V, bits_k: int, bits_v: int, key_group: int, value_group: int,
               window: int) -> np.ndarray:
    """Canonical image of one kv head; K, V are fp16 [L][d]."""
    Ku, Vu = _as_u16(K), _as_u16(V)
    L, d = Ku.shape
    n = head_bytes(L, d, bits_k, bits_v, key_group, value_group, window)
    out = np.zeros(max(n, 1), dtype=np.uint8)
    st = _load().orc_build_head(_ptr(Ku), _ptr(Vu), L, d, d, bits_k, bits_v, key_group,
                                value_group, window, _ptr(out))
    if st != OK:
        raise OracleError(st, "build_head")
    return out[:n]


def build_seq(K, V, bits_k: int, bits_v: int, key_group: int, value_group: int,
              window: int, heads: Optional[List[int]] = None) -> List[np.ndarray]:
    """Canonical images of the kv heads of one sequence; K, V are fp16 [L][Hkv][d]."""
    Ku, Vu = _as_u16(K), _as_u16(V)
    L, H, d = Ku.shape
    heads = range(H) if heads is None else heads
    return [build_head(np.ascontiguousarray(Ku[:, h, :]), np.ascontiguousarray(Vu[:, h, :]),
                       bits_k, bits_v, key_group, value_group, window) for h in heads]


def dequant_head(img: np.ndarray, L: int, d: int, bits_k: int, bits_v: int, key_group: int,
                 value_group: int, window: int) -> Tuple[np.ndarray, np.ndarray]:
    """fp64 K^, V^ [L][d] from a canonical image."""
    img = np.ascontiguousarray(img, dtype=np.uint8)
    if img.size != head_bytes(L, d, bits_k, bits_v, key_group, value_group, window):
        raise ValueError("image size does not match the layout")
    Kh = np.zeros((L, d), dtype=np.float64)
    Vh = np.zeros((L, d), dtype=np.float64)
    buf = img if img.size else np.zeros(1, dtype=np.uint8)
    st = _load().orc_dequant_head(_ptr(buf), L, d, bits_k, bits_v, key_group, value_group,
                                  window, _ptr(Kh), _ptr(Vh))
    if st != OK:
        raise OracleError(st, "dequant_head")
    return Kh, Vh


def attention(q, Khat: np.ndarray, Vhat: np.ndarray, return_weights: bool = False):
    """fp64 decode attention. q fp16 [Hq][d]; Khat, Vhat fp64 [Hkv][L][d]."""
    qu = _as_u16(q)
    Hq, d = qu.shape
    Kh = np.ascontiguousarray(Khat, dtype=np.float64)
    Vh = np.ascontiguousarray(Vhat, dtype=np.float64)
    Hkv, L, d2 = Kh.shape
    assert d2 == d and Vh.shape == Kh.shape
    out = np.zeros((Hq, d), dtype=np.float64)
    w = np.zeros((Hq, max(L, 1)), dtype=np.float64) if return_weights else None
    kb = Kh if Kh.size else np.zeros(1)
    vb = Vh if Vh.size else np.zeros(1)
    st = _load().orc_attention(_ptr(qu), _ptr(kb), _ptr(vb), L, Hq, Hkv, d, _ptr(out),
                               _ptr(w) if w is not None else None)
    if st != OK:
        raise OracleError(st, "attention")
    if return_weights:
        return out, w[:, :L]
    return out


def chunk_attention(q, Khat: np.ndarray, Vhat: np.ndarray):
    """fp64 attention of the last n_q positions of a cache, causal among them.

    Chunked prefill and the verification step of speculative decoding
    (Related Work) evaluate several consecutive query positions at once;
    each is the scaled dot-product attention of the decoder (Introduction)
    over the cache up to and including its own position.  q fp16
    [n_q][Hq][d]; Khat, Vhat fp64 [Hkv][L][d] with L >= n_q.  Query i is
    position L - n_q + i and attends to tokens [0, L - n_q + i]: the
    decode attention above on that prefix.
    """
    qu = _as_u16(q)
    n_q = qu.shape[0]
    L = Khat.shape[1]
    if not 1 <= n_q <= L:
        raise OracleError(ERR_ARG, "chunk_attention: need 1 <= n_q <= L")
    out = np.zeros((n_q,) + qu.shape[1:], dtype=np.float64)
    for i in range(n_q):
        visible = L - n_q + 1 + i
        out[i] = attention(qu[i], Khat[:, :visible], Vhat[:, :visible])
    return out


def chunk_seq(q, K, V, bits_k: int, bits_v: int, key_group: int, value_group: int,
              window: int, heads: Optional[List[int]] = None):
    """Quantize one sequence's cache, dequantize it and run chunk_attention.

    q fp16 [n_q][Hq][d]; K, V fp16 [L][Hkv][d].  Rows of kv heads outside
    ``heads`` are left NaN.
    """
    qu = _as_u16(q)
    L, Hkv, d = K.shape
    n_q, Hq = qu.shape[0], qu.shape[1]
    gq = Hq // Hkv
    heads = list(range(Hkv)) if heads is None else list(heads)
    out = np.full((n_q, Hq, d), np.nan)
    for h in heads:
        img = build_head(np.ascontiguousarray(K[:, h, :]), np.ascontiguousarray(V[:, h, :]),
                         bits_k, bits_v, key_group, value_group, window)
        Kh, Vh = dequant_head(img, L, d, bits_k, bits_v, key_group, value_group, window)
        out[:, h * gq:(h + 1) * gq] = chunk_attention(qu[:, h * gq:(h + 1) * gq], Kh[None], Vh[None])
    return out


def decode_seq(q, K, V, bits_k: int, bits_v: int, key_group: int, value_group: int,
               window: int, heads: Optional[List[int]] = None):
    """Quantize one sequence's cache, dequantize it and attend.

    q fp16 [Hq][d]; K, V fp16 [L][Hkv][d].  ``heads`` restricts the work to
    some kv heads: the result then holds only their query heads (rows of the
    other heads are left NaN).
    """
    qu = _as_u16(q)
    L, Hkv, d = K.shape
    Hq = qu.shape[0]
    gq = Hq // Hkv
    heads = list(range(Hkv)) if heads is None else list(heads)
    out = np.full((Hq, d), np.nan)
    for h in heads:
        img = build_head(np.ascontiguousarray(K[:, h, :]), np.ascontiguousarray(V[:, h, :]),
                         bits_k, bits_v, key_group, value_group, window)
        Kh, Vh = dequant_head(img, L, d, bits_k, bits_v, key_group, value_group, window)
        out[h * gq:(h + 1) * gq] = attention(qu[h * gq:(h + 1) * gq], Kh[None], Vh[None])
    return out


def num_threads() -> int:
    return int(_load().orc_num_threads())
