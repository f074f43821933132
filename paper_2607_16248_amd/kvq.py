"""Python binding of libkvq.so (ctypes): same names as the C ABI in include/kvq.h.

Argument marshalling only.  Tensors are passed by their device pointers and
the current HIP stream of torch; every step of the computation runs in the
library's kernels.  There is no fallback: without the built library every
call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvq.so")

OK, ERR_ARG, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_RANGE, ERR_STATE, ERR_HIP = range(7)
STATUS_NAMES = ["KVQ_OK", "KVQ_ERR_ARG", "KVQ_ERR_UNSUPPORTED", "KVQ_ERR_CAPACITY",
                "KVQ_ERR_RANGE", "KVQ_ERR_STATE", "KVQ_ERR_HIP"]

EXPORTED = ["kvq_cache_bytes", "kvq_cache_init", "kvq_cache_destroy", "kvq_cache_reset",
            "kvq_seq_len", "kvq_seq_release", "kvq_free_pages",
            "kvq_append", "kvq_workspace_bytes", "kvq_decode_attention", "kvq_decode_attention_noalloc",
            "kvq_append_decode",
            "kvq_decode_partials", "kvq_decode_merge", "kvq_chunk_workspace_bytes", "kvq_chunk_attention",
            "kvq_dequant", "kvq_export_bytes", "kvq_export", "kvq_check",
            "kvq_set_split_tokens", "kvq_last_error", "kvq_version",
            "kvq_read_probe", "kvq_read_probe_sink_bytes",
            "dgap_workspace_bytes", "dgap_info_floats", "dgap_restore"]


class KvqError(RuntimeError):
    def __init__(self, status: int, message: str):
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{name}: {message}")
        self.status = status


class CacheDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("key_group", ctypes.c_int32),
                ("value_group", ctypes.c_int32), ("fp16_window", ctypes.c_int32),
                ("bits_k", ctypes.POINTER(ctypes.c_uint8)), ("bits_v", ctypes.POINTER(ctypes.c_uint8)),
                ("page_tokens", ctypes.c_int32), ("num_pages", ctypes.c_int32)]


class DgapParams(ctypes.Structure):
    """dgap_params of include/dgap.h (weights are device pointers)."""
    _fields_ = [("vocab", ctypes.c_int32), ("k", ctypes.c_int32), ("hidden_det", ctypes.c_int32),
                ("hidden_corr", ctypes.c_int32), ("tau", ctypes.c_float), ("det_b2", ctypes.c_float),
                ("corr_b2", ctypes.c_float), ("pad", ctypes.c_int32),
                ("det_w1", ctypes.c_void_p), ("det_b1", ctypes.c_void_p), ("det_w2", ctypes.c_void_p),
                ("corr_w1", ctypes.c_void_p), ("corr_b1", ctypes.c_void_p), ("corr_w2", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_16248_amd/build.py "
                          "(the HIP library has no fallback)")
    L = ctypes.CDLL(LIB_PATH)
    P, S, I32, I64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int64
    D = ctypes.POINTER(CacheDesc)
    sig = {
        "kvq_cache_bytes": ([D], S),
        "kvq_cache_init": ([ctypes.POINTER(P), D, P, S], ctypes.c_int),
        "kvq_cache_destroy": ([P], None),
        "kvq_cache_reset": ([P, P], ctypes.c_int),
        "kvq_seq_len": ([P, I32], I64),
        "kvq_seq_release": ([P, I32], ctypes.c_int),
        "kvq_free_pages": ([P], I64),
        "kvq_append": ([P, P, P, I32, ctypes.POINTER(I32), P], ctypes.c_int),
        "kvq_workspace_bytes": ([P], S),
        "kvq_decode_attention": ([P, P, P, P, S, P], ctypes.c_int),
        "kvq_decode_attention_noalloc": ([P, P, P, P], ctypes.c_int),
        "kvq_chunk_workspace_bytes": ([P, ctypes.c_int32], S),
        "kvq_chunk_attention": ([P, P, ctypes.c_int32, P, P, S, P], ctypes.c_int),
        "kvq_append_decode": ([P, P, P, I32, ctypes.POINTER(I32), P, P, P, S, P], ctypes.c_int),
        "kvq_decode_partials": ([P, P, P, S, P], ctypes.c_int),
        "kvq_decode_merge": ([P, P, P, P], ctypes.c_int),
        "kvq_dequant": ([P, I32, I32, I32, P, P, P], ctypes.c_int),
        "kvq_export_bytes": ([P, I32, I32], S),
        "kvq_export": ([P, I32, I32, P, S, P], ctypes.c_int),
        "kvq_check": ([P, P], ctypes.c_int),
        "kvq_set_split_tokens": ([P, I32], ctypes.c_int),
        "kvq_last_error": ([], ctypes.c_char_p),
        "kvq_version": ([], ctypes.c_char_p),
        "kvq_read_probe": ([P, S, P, P], ctypes.c_int),
        "kvq_read_probe_sink_bytes": ([], S),
        "dgap_workspace_bytes": ([I32, I32, I32], S),
        "dgap_info_floats": ([I32], S),
        "dgap_restore": ([ctypes.POINTER(DgapParams), P, I32, P, S, P, P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(status: int):
    if status != OK:
        raise KvqError(status, kvq_last_error())


def _ptr(x) -> Optional[int]:
    """Device address of a tensor, or an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        if not torch.cuda.is_available():
            return None
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_desc(batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int, max_tokens: int,
              key_group: int, value_group: int, fp16_window: int, bits_k: Sequence[int],
              bits_v: Sequence[int], page_tokens: int = 0, num_pages: int = 0):
    """A descriptor plus the host arrays it points to (keep both alive)."""
    bk = (ctypes.c_uint8 * max(1, len(bits_k)))(*bits_k)
    bv = (ctypes.c_uint8 * max(1, len(bits_v)))(*bits_v)
    d = CacheDesc(batch, num_q_heads, num_kv_heads, head_dim, max_tokens, key_group, value_group,
                  fp16_window, ctypes.cast(bk, ctypes.POINTER(ctypes.c_uint8)),
                  ctypes.cast(bv, ctypes.POINTER(ctypes.c_uint8)), page_tokens, num_pages)
    d._keep = (bk, bv)
    return d


def kvq_cache_bytes(desc: CacheDesc) -> int:
    return int(lib().kvq_cache_bytes(ctypes.byref(desc)))


def kvq_cache_init(desc: CacheDesc, arena, arena_bytes: Optional[int] = None) -> int:
    """Handle (an int) over ``arena`` (a device tensor or address)."""
    if arena_bytes is None:
        arena_bytes = arena.numel() * arena.element_size()
    h = ctypes.c_void_p()
    _check(lib().kvq_cache_init(ctypes.byref(h), ctypes.byref(desc), _ptr(arena), int(arena_bytes)))
    return h.value


def kvq_cache_destroy(cache: int) -> None:
    lib().kvq_cache_destroy(cache)


def kvq_cache_reset(cache: int, stream=None) -> None:
    _check(lib().kvq_cache_reset(cache, _stream(stream)))


def kvq_seq_len(cache: int, seq: int) -> int:
    return int(lib().kvq_seq_len(cache, seq))


def kvq_seq_release(cache: int, seq: int) -> None:
    _check(lib().kvq_seq_release(cache, seq))


def kvq_free_pages(cache: int) -> int:
    return int(lib().kvq_free_pages(cache))


def kvq_append(cache: int, K, V, n_new: Sequence[int], n_max: Optional[int] = None, stream=None) -> None:
    """K, V: fp16 [batch][n_max][Hkv][d] on the device; n_new: per-sequence counts."""
    n = (ctypes.c_int32 * max(1, len(n_new)))(*n_new)
    if n_max is None:
        n_max = int(K.shape[1]) if K is not None and not isinstance(K, int) else max(n_new, default=0)
    _check(lib().kvq_append(cache, _ptr(K), _ptr(V), int(n_max), n, _stream(stream)))


def kvq_workspace_bytes(cache: int) -> int:
    return int(lib().kvq_workspace_bytes(cache))


def kvq_decode_attention(cache: int, q, out, ws, ws_bytes: Optional[int] = None, stream=None) -> None:
    """q: fp16 [batch][Hq][d]; out: fp32 [batch][Hq][d]; ws: scratch bytes."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().kvq_decode_attention(cache, _ptr(q), _ptr(out), _ptr(ws), int(ws_bytes), _stream(stream)))


def kvq_decode_attention_noalloc(cache: int, q, out, stream=None) -> None:
    """kvq_decode_attention with the library's own scratch array as workspace."""
    _check(lib().kvq_decode_attention_noalloc(cache, _ptr(q), _ptr(out), _stream(stream)))


def kvq_chunk_workspace_bytes(cache: int, n_q: int) -> int:
    return int(lib().kvq_chunk_workspace_bytes(cache, int(n_q)))


def kvq_chunk_attention(cache: int, q, n_q: int, out, ws, ws_bytes: Optional[int] = None, stream=None) -> None:
    """The last n_q tokens of every sequence attend causally: q fp16 [batch][n_q][Hq][d],
    out fp32 [batch][n_q][Hq][d]."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().kvq_chunk_attention(cache, _ptr(q), int(n_q), _ptr(out), _ptr(ws), int(ws_bytes),
                                     _stream(stream)))


def kvq_append_decode(cache: int, K, V, n_new: Sequence[int], q, out, ws, ws_bytes: Optional[int] = None,
                      n_max: Optional[int] = None, stream=None) -> None:
    """kvq_append then kvq_decode_attention in one call (two launches when no key group fills)."""
    n = (ctypes.c_int32 * max(1, len(n_new)))(*n_new)
    if n_max is None:
        n_max = int(K.shape[1]) if K is not None and not isinstance(K, int) else max(n_new, default=0)
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().kvq_append_decode(cache, _ptr(K), _ptr(V), int(n_max), n, _ptr(q), _ptr(out), _ptr(ws),
                                   int(ws_bytes), _stream(stream)))


def kvq_decode_partials(cache: int, q, ws, ws_bytes: Optional[int] = None, stream=None) -> None:
    """Phase 1 of decode: per-split softmax records into ``ws``."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().kvq_decode_partials(cache, _ptr(q), _ptr(ws), int(ws_bytes), _stream(stream)))


def kvq_read_probe(src, nbytes: int, sink, stream=None) -> None:
    """Diagnostics: read ``nbytes`` of the device buffer ``src`` once (streaming-read rate)."""
    _check(lib().kvq_read_probe(_ptr(src), int(nbytes), _ptr(sink), _stream(stream)))


def kvq_read_probe_sink_bytes() -> int:
    return int(lib().kvq_read_probe_sink_bytes())


def kvq_decode_merge(cache: int, ws, out, stream=None) -> None:
    """Phase 2 of decode: merge the records of ``ws`` into ``out``."""
    _check(lib().kvq_decode_merge(cache, _ptr(ws), _ptr(out), _stream(stream)))


def kvq_dequant(cache: int, seq: int, tok0: int, ntok: int, K_out, V_out, stream=None) -> None:
    _check(lib().kvq_dequant(cache, seq, tok0, ntok, _ptr(K_out), _ptr(V_out), _stream(stream)))


def kvq_export_bytes(cache: int, seq: int, kv_head: int) -> int:
    return int(lib().kvq_export_bytes(cache, seq, kv_head))


def kvq_export(cache: int, seq: int, kv_head: int, dst, nbytes: Optional[int] = None, stream=None) -> None:
    if nbytes is None:
        nbytes = dst.numel() * dst.element_size()
    _check(lib().kvq_export(cache, seq, kv_head, _ptr(dst), int(nbytes), _stream(stream)))


def kvq_check(cache: int, stream=None) -> None:
    _check(lib().kvq_check(cache, _stream(stream)))


def kvq_set_split_tokens(cache: int, tokens: int) -> None:
    _check(lib().kvq_set_split_tokens(cache, int(tokens)))


def kvq_last_error() -> str:
    return lib().kvq_last_error().decode()


def kvq_version() -> str:
    return lib().kvq_version().decode()


class KVCache:
    """A cache over a torch-allocated, zero-filled device arena."""

    def __init__(self, batch, num_q_heads, num_kv_heads, max_tokens, bits_k, bits_v,
                 key_group=32, value_group=32, fp16_window=0, head_dim=128, device="cuda",
                 page_tokens=0, num_pages=0):
        import torch
        bits_k = list(bits_k) if hasattr(bits_k, "__len__") else [bits_k] * batch
        bits_v = list(bits_v) if hasattr(bits_v, "__len__") else [bits_v] * batch
        self.desc = make_desc(batch, num_q_heads, num_kv_heads, head_dim, max_tokens, key_group,
                              value_group, fp16_window, bits_k, bits_v, page_tokens, num_pages)
        self.page_tokens, self.num_pages = page_tokens, num_pages
        self.batch, self.num_q_heads, self.num_kv_heads = batch, num_q_heads, num_kv_heads
        self.head_dim, self.key_group, self.value_group = head_dim, key_group, value_group
        self.fp16_window, self.bits_k, self.bits_v, self.max_tokens = fp16_window, bits_k, bits_v, max_tokens
        nbytes = kvq_cache_bytes(self.desc)
        if nbytes == 0:
            # surface the descriptor error through init
            kvq_cache_init(self.desc, 256, 0)
        self.arena = torch.zeros(nbytes, dtype=torch.uint8, device=device)
        self.handle = kvq_cache_init(self.desc, self.arena)
        self.ws = None

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                kvq_cache_destroy(h)
            except TypeError:  # interpreter shutdown: module globals are already torn down
                pass
            self.handle = None

    def append(self, K, V, n_new=None, stream=None):
        if n_new is None:
            n_new = [int(K.shape[1])] * self.batch
        kvq_append(self.handle, K, V, n_new, stream=stream)

    def workspace(self):
        import torch
        need = kvq_workspace_bytes(self.handle)
        if self.ws is None or self.ws.numel() < need:
            self.ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.arena.device)
        return self.ws

    def decode(self, q, out=None, stream=None):
        import torch
        if out is None:
            out = torch.empty((self.batch, self.num_q_heads, self.head_dim), dtype=torch.float32,
                              device=q.device)
        kvq_decode_attention(self.handle, q, out, self.workspace(), stream=stream)
        return out

    def chunk(self, q, out=None, stream=None):
        """Causal attention of the last q.shape[1] tokens of every sequence."""
        import torch
        n_q = int(q.shape[1])
        if out is None:
            out = torch.empty((self.batch, n_q, self.num_q_heads, self.head_dim), dtype=torch.float32,
                              device=q.device)
        need = kvq_chunk_workspace_bytes(self.handle, n_q)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.arena.device)
        kvq_chunk_attention(self.handle, q, n_q, out, ws, stream=stream)
        return out

    def append_decode(self, K, V, q, n_new=None, out=None, stream=None):
        import torch
        if n_new is None:
            n_new = [int(K.shape[1])] * self.batch
        if out is None:
            out = torch.empty((self.batch, self.num_q_heads, self.head_dim), dtype=torch.float32,
                              device=q.device)
        kvq_append_decode(self.handle, K, V, n_new, q, out, self.workspace(), stream=stream)
        return out

    def seq_len(self, seq):
        return kvq_seq_len(self.handle, seq)

    def release(self, seq):
        kvq_seq_release(self.handle, seq)

    def free_pages(self):
        return kvq_free_pages(self.handle)

    def export(self, seq, kv_head):
        import torch
        n = kvq_export_bytes(self.handle, seq, kv_head)
        dst = torch.zeros(max(n, 1), dtype=torch.uint8, device=self.arena.device)
        kvq_export(self.handle, seq, kv_head, dst, n)
        torch.cuda.synchronize()
        return dst[:n].cpu().numpy()

    def dequant(self, seq, tok0, ntok):
        import torch
        Ko = torch.empty((max(ntok, 1), self.num_kv_heads, self.head_dim), dtype=torch.float32,
                         device=self.arena.device)
        Vo = torch.empty_like(Ko)
        kvq_dequant(self.handle, seq, tok0, ntok, Ko, Vo)
        return Ko[:ntok], Vo[:ntok]

    def check(self):
        kvq_check(self.handle)

    def reset(self):
        kvq_cache_reset(self.handle)


# ------------------------------------------------------------------ DGAP

def dgap_workspace_bytes(batch: int, vocab: int, k: int) -> int:
    return int(lib().dgap_workspace_bytes(batch, vocab, k))


def dgap_info_floats(k: int) -> int:
    return int(lib().dgap_info_floats(k))


def dgap_params(vocab: int, k: int, tau: float, det_w1, det_b1, det_w2, det_b2: float,
                corr_w1, corr_b1, corr_w2, corr_b2: float) -> DgapParams:
    """Params from device fp32 tensors (det_w1 [12][hd], corr_w1 [17][hc], ...)."""
    return DgapParams(int(vocab), int(k), int(det_b1.numel()) if det_b1 is not None else 0,
                      int(corr_b1.numel()) if corr_b1 is not None else 0, float(tau), float(det_b2),
                      float(corr_b2), 0, _ptr(det_w1), _ptr(det_b1), _ptr(det_w2), _ptr(corr_w1),
                      _ptr(corr_b1), _ptr(corr_w2))


def dgap_restore(params: DgapParams, logits, batch: int, ws, ws_bytes: Optional[int] = None, info=None,
                 stream=None) -> None:
    """One DGAP step on ``batch`` rows of device fp32 logits, in place."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().dgap_restore(ctypes.byref(params), _ptr(logits), int(batch), _ptr(ws), int(ws_bytes),
                              _ptr(info), _stream(stream)))
