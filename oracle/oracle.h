/*
 * CPU oracle for the packed low-bit KV-cache decode path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library may include,
 * link or call this code; only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no source with the HIP
 * implementation.
 *
 * What it computes:
 *  - the quantizer: b-bit asymmetric min-max with an fp16 scale and an fp16
 *    zero-point per group; key groups run along tokens for one channel,
 *    value groups along channels for one token.  The paper names the
 *    precision settings ("KbVb", Motivation, "Accuracy Loss under Aggressive
 *    KV Quantization", Methodology paragraph) and points to asymmetric
 *    key/value formats as the quantizers it builds on (Introduction; Related
 *    Work, "KV-cache quantization and distribution preservation") but never
 *    writes the quantizer down; the exact rule implemented is stated at each
 *    function below.
 *  - the canonical byte image of one (sequence, kv head) of the cache;
 *  - dequantization of that image; and
 *  - decode attention softmax(q K^T / sqrt(d)) V (Introduction, the scaled
 *    dot-product attention formula) in fp64 over the dequantized cache.
 *
 * fp16 values travel as their IEEE binary16 bit patterns (uint16_t).
 */
#ifndef KVQ_ORACLE_H
#define KVQ_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_OK = 0, ORC_ERR_ARG = 1, ORC_ERR_RANGE = 4 };

/* Exact value of an fp16 bit pattern (NaN/inf map to NaN/inf). */
double orc_half_value(uint16_t h);

/* Smallest fp16 value >= s, for finite s >= 0 (subnormals included).
 * Writes its bit pattern to *out; ORC_ERR_RANGE if s > 65504 or not finite. */
int orc_half_ceil(double s, uint16_t* out);

/* Quantize one group of n fp16 values x[0], x[stride], ... to `bits` bits.
 * Writes the scale (*s), zero-point (*z) and n codes.  ORC_ERR_RANGE for a
 * non-finite input or a scale beyond the fp16 range. */
int orc_quantize_group(const uint16_t* x, long n, long stride, int bits,
                       uint16_t* s, uint16_t* z, uint8_t* codes);

/* Number of tokens held quantized: key_group * floor(max(0, L - window) / key_group). */
long orc_quantized_len(long L, int key_group, int window);

/* Size in bytes of the canonical image of one (sequence, kv head). */
size_t orc_head_bytes(long L, int d, int bits_k, int bits_v, int key_group,
                      int value_group, int window);

/* Build the canonical image of one (sequence, kv head) from its L tokens.
 * K, V point at token 0, channel 0 of that head; consecutive tokens are
 * row_stride elements apart.  `out` receives orc_head_bytes(...) bytes. */
int orc_build_head(const uint16_t* K, const uint16_t* V, long L, long row_stride, int d,
                   int bits_k, int bits_v, int key_group, int value_group, int window,
                   uint8_t* out);

/* Dequantize a canonical image back to fp64 K^ and V^, each [L][d]. */
int orc_dequant_head(const uint8_t* img, long L, int d, int bits_k, int bits_v,
                     int key_group, int value_group, int window,
                     double* Khat, double* Vhat);

/* Decode attention for one sequence in fp64.
 * q: fp16 [Hq][d].  Khat, Vhat: fp64 [Hkv][L][d].  out: fp64 [Hq][d].
 * weights: optional fp64 [Hq][L] (the softmax weights), may be NULL.
 * Query head h reads kv head h / (Hq / Hkv).  L == 0 yields out = 0. */
int orc_attention(const uint16_t* q, const double* Khat, const double* Vhat, long L,
                  int Hq, int Hkv, int d, double* out, double* weights);

/* Number of threads the attention loop runs on (OpenMP), 1 without it. */
int orc_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
