/*
 * kvq — packed low-bit KV cache and attention over it for AMD Instinct
 * MI355X (gfx950): single-token decode, chunk queries (the last n_q tokens,
 * causal) and a paged layout for serving.  Plain C ABI.
 *
 * The computation is attention over a persistent low-bit KV cache.  The
 * paper evaluates KbVb caches, b-bit keys and b-bit values with
 * b in {1, 2, 4, 8} (Motivation, "Accuracy Loss under Aggressive KV
 * Quantization", Methodology paragraph), keeps that cache unchanged for the
 * whole decode (Methodology, "DGAP Overview", online restoration framework)
 * and decodes one token per step through scaled dot-product attention,
 * softmax(q K^T / sqrt(d)) V (Introduction; Experimental Setup, Testbed:
 * batch-1 decoding).  The paper does not define the quantizer; this library
 * implements asymmetric min-max quantization (the asymmetric key/value
 * format the paper builds on, Related Work) with these choices:
 *   - keys: one group per channel over key_group consecutive tokens;
 *     values: one group per token over value_group consecutive channels;
 *   - zero-point z = the group minimum (an fp16 value); scale s = the
 *     smallest fp16 value >= (max - min) / (2^b - 1); code =
 *     round-half-even((x - z) / s); dequantized value z + code * s; a
 *     constant group has s = 0 and codes 0;
 *   - a token is quantized once it and its whole key group lie more than
 *     fp16_window tokens before the end of the sequence: the first
 *     Lq = key_group * floor(max(0, L - fp16_window) / key_group) tokens are
 *     packed, the remaining L - Lq (< fp16_window + key_group) stay fp16.
 *
 * Conventions for every call:
 *   - Device pointers are HIP device pointers owned by the caller; the
 *     library never allocates or frees device memory.  `stream` is a
 *     hipStream_t passed as void*; NULL is the default stream.  Calls that
 *     take a stream are asynchronous and stream-ordered unless stated.
 *   - A non-OK status leaves the cache unchanged and launches nothing,
 *     except KVQ_ERR_HIP, which reports a failed launch or copy.
 *     kvq_last_error() then describes the failure (thread-local string).
 *   - One cache may be used from one stream at a time.  Distinct caches are
 *     independent.
 */
#ifndef KVQ_H
#define KVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KVQ_OK = 0,
  KVQ_ERR_ARG = 1,          /* invalid argument or descriptor */
  KVQ_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. head_dim != 128) */
  KVQ_ERR_CAPACITY = 3,     /* an append would exceed max_tokens; workspace too small */
  KVQ_ERR_RANGE = 4,        /* input outside the quantizer's domain (see kvq_check) */
  KVQ_ERR_STATE = 5,        /* call not valid in the cache's current state */
  KVQ_ERR_HIP = 6           /* a HIP runtime call failed */
} kvq_status;

/* Shape and quantizer settings of a cache.  All sequences share the shape
 * and capacity; bit widths may differ per sequence. */
typedef struct {
  int32_t batch;          /* sequences, >= 1 */
  int32_t num_q_heads;    /* Hq, a multiple of num_kv_heads; Hq / Hkv in {1, 2, 4, 5, 8} */
  int32_t num_kv_heads;   /* Hkv >= 1 */
  int32_t head_dim;       /* d; only 128 is supported */
  int32_t max_tokens;     /* capacity L_max per sequence, >= 1 */
  int32_t key_group;      /* tokens per key group: 32, 64 or 128 */
  int32_t value_group;    /* channels per value group: 8, 16, 32, 64 or 128 */
  int32_t fp16_window;    /* recent tokens kept in fp16, >= 0 */
  const uint8_t* bits_k;  /* host array [batch] of key bits, each 1, 2, 4 or 8 */
  const uint8_t* bits_v;  /* host array [batch] of value bits, each 1, 2, 4 or 8 */
  /* Paged layout (serving): 0 = one contiguous region per sequence.  Else
   * the packed codes and scales of every page_tokens consecutive tokens of
   * a sequence (all kv heads) live in one page of a pool shared by the
   * batch, found through a block table; pages are taken as sequences grow
   * and returned by kvq_seq_release.  A power of two >= key_group; every
   * sequence must then use the same bit widths. */
  int32_t page_tokens;
  /* Pages in the pool (paged layout only); 0 = enough for every sequence
   * at max_tokens.  Fewer pages let the batch share a smaller pool. */
  int32_t num_pages;
} kvq_cache_desc;

/* Opaque host-side handle.  It owns no device memory. */
typedef struct kvq_cache kvq_cache;

/* Device arena size in bytes needed for `desc`; 0 if desc is invalid. */
size_t kvq_cache_bytes(const kvq_cache_desc* desc);

/* Create a handle over a caller-allocated device arena of at least
 * kvq_cache_bytes(desc) bytes, 256-byte aligned.  Host-only: touches no
 * device memory.  The arena's first 256 bytes must be zero (allocate it
 * zero-filled, or call kvq_cache_reset before the first append).  All
 * sequences start empty.  The descriptor is copied. */
kvq_status kvq_cache_init(kvq_cache** out, const kvq_cache_desc* desc, void* arena,
                          size_t arena_bytes);

/* Free the handle (not the arena).  NULL is allowed. */
void kvq_cache_destroy(kvq_cache* cache);

/* Empty every sequence and clear the device error flag (a small fill
 * kernel on `stream`, no memset node). */
kvq_status kvq_cache_reset(kvq_cache* cache, void* stream);

/* Current length L of a sequence (host bookkeeping), or -1 if out of range. */
int64_t kvq_seq_len(const kvq_cache* cache, int32_t seq);

/* Empty one sequence (host bookkeeping only, no launch): its length
 * becomes 0 and, in a paged cache, its pages return to the pool, so the
 * slot can take a new sequence while the others keep decoding. */
kvq_status kvq_seq_release(kvq_cache* cache, int32_t seq);

/* Free pages in the pool of a paged cache; -1 for a contiguous cache or
 * a NULL handle. */
int64_t kvq_free_pages(const kvq_cache* cache);

/* Append tokens and quantize every key group that leaves the fp16 window
 * (the fused quantize-on-append step).  Defines the b-bit key and value
 * storage of a KbVb cache (Motivation, "Accuracy Loss under Aggressive KV
 * Quantization", Methodology paragraph), with the asymmetric min-max rule
 * stated at the top of this header (Related Work, "KV-cache quantization and
 * distribution preservation": asymmetric key/value formats).
 *   K, V : device fp16 [batch][n_max][Hkv][d]; sequence i appends rows
 *          0 .. n_new[i]-1 of its slice.  Read only.
 *   n_new: host int32 [batch], 0 <= n_new[i] <= n_max.
 * KVQ_ERR_CAPACITY if any L + n_new exceeds max_tokens, or if a paged
 * cache's pool has too few free pages for the new packed tokens (nothing
 * appended).
 * Inputs must be finite fp16 whose group range fits the fp16 scale
 * (|x| <= 32752 always does); a violation is reported later by kvq_check.
 * Prefill is an append with n_new = prompt length. */
kvq_status kvq_append(kvq_cache* cache, const void* K, const void* V, int32_t n_max,
                      const int32_t* n_new, void* stream);

/* Bytes of workspace kvq_decode_attention needs for any lengths up to
 * max_tokens under the current split setting. */
size_t kvq_workspace_bytes(const kvq_cache* cache);

/* Single-token decode attention over every cached token of every sequence,
 * the decoder's scaled dot-product attention softmax(Q K^T / sqrt(d_k)) V
 * (Introduction) at one query per sequence per step (Experimental Setup,
 * Testbed: batch-1 decoding):
 *   out[i][h][:] = softmax(q[i][h] . K^[i][kv(h)]^T / sqrt(d)) V^[i][kv(h)]
 * with kv(h) = h / (Hq / Hkv), K^ and V^ the dequantized cache (fp16 tail
 * tokens exact).  q: device fp16 [batch][Hq][d], finite (a NaN or infinity
 * in q gives undefined outputs for its rows).  out: device fp32
 * [batch][Hq][d].  ws: device scratch of ws_bytes >= kvq_workspace_bytes,
 * 16-byte aligned, contents undefined on entry and exit.  A sequence with
 * no tokens yields zeros.  Split-K over tokens (flash-decoding) followed
 * by a merge pass; results do not depend on the stream or on other
 * sequences, and are bitwise reproducible for a fixed split setting. */
kvq_status kvq_decode_attention(const kvq_cache* cache, const void* q, float* out, void* ws,
                                size_t ws_bytes, void* stream);

/* kvq_decode_attention without a caller workspace, for callers that cannot
 * allocate device memory (code under graph capture, serving loops that
 * forbid allocation): the split records live in a scratch array of
 * KVQ_NOALLOC_SCRATCH_BYTES (16 MiB) that the library holds on every GPU it
 * runs on until the process ends.  It allocates nothing and launches the
 * same kernels with the same split plan, so out equals kvq_decode_attention's
 * bit for bit.  Every call on one GPU uses that GPU's one array: calls that
 * overlap on one GPU (different streams, or different threads) race and give
 * undefined outputs; calls ordered on one stream are safe.  The array keeps
 * the last call's records; nothing in it needs to start at zero.
 * Errors: KVQ_ERR_ARG (null pointers), KVQ_ERR_CAPACITY when the call would
 * need more workspace than the array holds (kvq_workspace_bytes at the
 * current lengths; nothing launched), KVQ_ERR_HIP. */
#define KVQ_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
kvq_status kvq_decode_attention_noalloc(const kvq_cache* cache, const void* q, float* out, void* stream);

/* One decode step in one call: the same result, cache state and error
 * behaviour as kvq_append(cache, K, V, n_max, n_new, stream) followed by
 * kvq_decode_attention(cache, q, out, ws, ws_bytes, stream) (the decode is
 * that of the Introduction's attention; the append is the quantize-on-append
 * of kvq_append).  When the new tokens complete no key group (every step
 * but one in key_group for single-token decode), the tokens stay fp16 and
 * the decode launch itself stores them into the fp16 tail before it attends
 * over them: two launches instead of three.  Otherwise it runs the two
 * calls.  K, V: as for kvq_append, 4-byte aligned.  ws_bytes must cover the
 * lengths after the append (kvq_workspace_bytes covers any length).  Every
 * argument, capacity and workspace check happens before anything is
 * launched, and a failed check leaves the cache unchanged. */
kvq_status kvq_append_decode(kvq_cache* cache, const void* K, const void* V, int32_t n_max,
                             const int32_t* n_new, const void* q, float* out, void* ws, size_t ws_bytes,
                             void* stream);

/* The two phases of kvq_decode_attention, for callers that combine partial
 * results themselves (for example across devices) and for timing.
 * kvq_decode_partials writes, for every sequence i, query head h and split
 * k, one record of 132 floats at ws + ((base_i + k) * Hq + h) * 132:
 *   [0] m = max over the split's tokens of the base-2 score
 *       log2(e) * q.k / sqrt(d),  [1] l = sum of 2^(score - m),
 *   [2..3] unused,  [4..131] acc[c] = sum of 2^(score - m) * V^[c],
 * where base_i is the number of splits of sequences 0..i-1.  The split plan
 * depends only on the lengths and the split setting.  kvq_decode_merge
 * reads those records and writes out exactly as kvq_decode_attention does;
 * no append may come between the two calls. */
kvq_status kvq_decode_partials(const kvq_cache* cache, const void* q, void* ws, size_t ws_bytes,
                               void* stream);
kvq_status kvq_decode_merge(const kvq_cache* cache, const void* ws, float* out, void* stream);

/* Most queries per sequence in one kvq_chunk_attention call. */
#define KVQ_MAX_CHUNK 1024

/* Workspace bytes kvq_chunk_attention needs for n_q queries per sequence
 * (n_q times kvq_workspace_bytes); 0 if n_q is outside [1, KVQ_MAX_CHUNK]. */
size_t kvq_chunk_workspace_bytes(const kvq_cache* cache, int32_t n_q);

/* Attention of the last n_q tokens of every sequence over its cache, causal
 * among them: the same scaled dot-product attention as
 * kvq_decode_attention, for the several query positions that chunked
 * prefill and the verification step of speculative decoding evaluate at
 * once (Related Work: paged serving and I/O-aware attention kernels; the
 * quantized caches built for speculative decoding).  Query i of sequence s
 * is the token at position L_s - n_q + i (already appended) and attends to
 * tokens [0, L_s - n_q + i]:
 *   out[s][i][h][:] = softmax over t <= L_s - n_q + i of
 *                     (q[s][i][h] . K^[s][kv(h)][t] / sqrt(d)) V^[s][kv(h)]
 * q: device fp16 [batch][n_q][Hq][d]; out: device fp32 [batch][n_q][Hq][d];
 * ws: device scratch of ws_bytes >= kvq_chunk_workspace_bytes(cache, n_q),
 * 16-byte aligned, contents undefined on entry and exit.  Every sequence
 * must hold at least n_q tokens.  With n_q = 1 the result equals
 * kvq_decode_attention's.  The queries of a kv head are read in groups of
 * up to 8 (query, head) rows, each group one pass over the cache.
 * Errors: KVQ_ERR_ARG (n_q out of range, a sequence shorter than n_q, null
 * pointers, misaligned workspace), KVQ_ERR_CAPACITY (workspace too small),
 * KVQ_ERR_HIP. */
kvq_status kvq_chunk_attention(const kvq_cache* cache, const void* q, int32_t n_q, float* out, void* ws,
                               size_t ws_bytes, void* stream);

/* Dequantize tokens [tok0, tok0 + ntok) of one sequence into device fp32
 * K_out, V_out [ntok][Hkv][d]: fmaf(code, s, z) for packed tokens (the
 * exact z + code*s rounded once to fp32) and the fp16 value for tail
 * tokens.  These are the dequantized keys and values K^, V^ that decode
 * attends over (the KbVb cache of Motivation, "Accuracy Loss under
 * Aggressive KV Quantization", read back through the rule at the top of
 * this header).  For checking; not on the decode path.  Errors:
 * KVQ_ERR_ARG (seq out of range, a token range outside [0, L), null
 * outputs), KVQ_ERR_HIP. */
kvq_status kvq_dequant(const kvq_cache* cache, int32_t seq, int32_t tok0, int32_t ntok,
                       float* K_out, float* V_out, void* stream);

/* Size of the canonical byte image of (seq, kv_head) at its current length:
 *   key codes [Lq][d*bk/8] | key meta [Lq/key_group][2][d] fp16 (scales,
 *   then zeros) | value codes [Lq][d*bv/8] | value meta [Lq][d/value_group]
 *   [2] fp16 (scale, zero) | key tail [L-Lq][d] fp16 | value tail [L-Lq][d]
 * where a code row holds channel c at row bits [c*b, c*b+b), least
 * significant bit first (row bit i = bit i%8 of byte i/8), little-endian
 * fp16.  Returns 0 for an invalid (seq, kv_head). */
size_t kvq_export_bytes(const kvq_cache* cache, int32_t seq, int32_t kv_head);

/* Copy the canonical image of (seq, kv_head) into device memory `dst` of
 * `bytes` >= kvq_export_bytes(...): the persistent low-bit cache the paper
 * keeps unchanged across decode steps (Methodology, "DGAP Overview", online
 * restoration framework), in the byte order above, for checking and for
 * saving a cache.  Device-to-device copies and a reorder kernel on
 * `stream`.  Errors: KVQ_ERR_ARG (seq or kv_head out of range, null dst),
 * KVQ_ERR_CAPACITY (bytes too small), KVQ_ERR_HIP. */
kvq_status kvq_export(const kvq_cache* cache, int32_t seq, int32_t kv_head, void* dst,
                      size_t bytes, void* stream);

/* Synchronize `stream` and read the device error flag: KVQ_ERR_RANGE if an
 * append met a non-finite input or a group range beyond the fp16 scale,
 * else KVQ_OK.  The flag is sticky until kvq_cache_reset. */
kvq_status kvq_check(const kvq_cache* cache, void* stream);

/* Tokens per split of the decode kernel: a positive multiple of key_group
 * giving at most 512 splits per sequence at capacity, or 0 to let the
 * library choose from the current lengths (the default).  Changing it
 * changes kvq_workspace_bytes. */
kvq_status kvq_set_split_tokens(kvq_cache* cache, int32_t tokens);

/* Diagnostics: the device's streaming-read rate, for comparing the decode
 * kernels' algorithmic bytes with a measured ceiling beside the nominal HBM
 * peak.  Reads `bytes` (a multiple of 16) from the device buffer `src`
 * (16-byte aligned) once, with 16-byte loads in a grid-stride loop, and
 * writes one XOR fold per workgroup to `sink` (device, at least
 * kvq_read_probe_sink_bytes() bytes, contents meaningless).  Asynchronous on
 * `stream`; time it with events.  Errors: KVQ_ERR_ARG (null pointer,
 * misaligned or ragged size), KVQ_ERR_HIP. */
kvq_status kvq_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream);
size_t kvq_read_probe_sink_bytes(void);

/* Message for the last non-OK status on this thread ("" if none). */
const char* kvq_last_error(void);

/* Library version string. */
const char* kvq_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KVQ_H */
