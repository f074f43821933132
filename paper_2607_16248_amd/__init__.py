"""Packed low-bit KV cache and single-token decode attention for MI355X (gfx950).

The computation lives in the HIP library libkvq.so (C ABI: include/kvq.h and
include/dgap.h, DGAP's logit-side step);
:mod:`paper_2607_16248_amd.kvq` is its thin ctypes binding.
"""
from .kvq import (KVCache, KvqError, kvq_append, kvq_append_decode, kvq_cache_bytes, kvq_cache_destroy,  # noqa: F401
                  kvq_cache_init, kvq_cache_reset, kvq_check, kvq_chunk_attention, kvq_chunk_workspace_bytes,
                  kvq_decode_attention, kvq_decode_attention_noalloc,
                  kvq_decode_merge, kvq_decode_partials, kvq_dequant,
                  kvq_export, kvq_export_bytes, kvq_free_pages, kvq_last_error, kvq_seq_len, kvq_seq_release,
                  kvq_set_split_tokens,
                  kvq_version, kvq_workspace_bytes, make_desc)
from .kvq import dgap_info_floats, dgap_params, dgap_restore, dgap_workspace_bytes  # noqa: F401
