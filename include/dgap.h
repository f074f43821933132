/*
 * dgap — the logit-side runtime step of DGAP on AMD Instinct MI355X
 * (gfx950).  Plain C ABI, in the same library as kvq.h.
 *
 * DGAP restores the local top-K candidate distribution of a decoder that
 * keeps a low-bit KV cache (Methodology, "DGAP Overview", online restoration
 * framework).  At each decode step it computes runtime features phi from the
 * quantized logits z^ alone, scores them with a detector,
 * r = sigmoid(f_theta(phi)) ("Distribution-Risk Detector"), and, only when
 * r > tau, predicts updates Delta for the window S = TopK(z^, K_b) with a
 * corrector g_psi from candidate features and phi, merging them back:
 * z~_j = z^_j + Delta_j for j in S, z~_j = z^_j otherwise ("Selective Top-K
 * Distribution Corrector", sparse merge).  The paper uses MLPs for both
 * modules and tau = 0.60 (ablations).  It leaves the features, the MLP
 * shapes and K_b open; this library fixes:
 *   - TopK: the K largest logits, largest first, equal logits by lower
 *     vocabulary index;
 *   - phi (DGAP_FEATURES = 12), with v_1 >= ... >= v_K the window's logits,
 *     p = softmax(z^) over the vocabulary and P_k = p at v_k, natural logs:
 *       0 entropy H = -sum p log p,  1 H / log V,  2 log P_1,
 *       3 sum_k P_k,  4 sum_{k<=8} P_k,  5 sum p^2,  6 v_1 - v_2,
 *       7 v_2 - v_3,  8 (v_1 - v_K) / (K - 1),  9 min_{k<8} (v_k - v_{k+1}),
 *       10 population standard deviation of v_1..v_K,
 *       11 entropy of P_1..P_K renormalized to sum 1 (0 log 0 = 0);
 *   - xi_k (DGAP_CAND_INPUTS = 5) for candidate k = 1..K: v_k - v_1,
 *     v_k - log-sum-exp(z^), (k - 1) / (K - 1), v_{k-1} - v_k (0 for k = 1),
 *     v_k - v_{k+1} (0 for k = K);
 *   - f_theta(phi) = w2 . relu(W1^T phi + b1) + b2 and
 *     g_psi(xi_k, phi) = w2' . relu(W1'^T [xi_k, phi] + b1') + b2', one
 *     hidden layer each, g_psi shared by the K candidates.
 *
 * Conventions: device pointers are caller-owned HIP device buffers; the
 * library allocates nothing; `stream` is a hipStream_t as void*, calls are
 * asynchronous and stream-ordered.  A non-OK status other than KVQ_ERR_HIP
 * launches nothing and leaves every buffer unchanged; kvq_last_error()
 * describes the failure.
 */
#ifndef DGAP_H
#define DGAP_H

#include <stddef.h>
#include <stdint.h>

#include "kvq.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DGAP_FEATURES 12
#define DGAP_CAND_INPUTS 5
#define DGAP_MIN_K 8
#define DGAP_MAX_K 256
#define DGAP_MAX_HIDDEN 64

/* Shapes, threshold and weights (device pointers, fp32, row-major). */
typedef struct {
  int32_t vocab;        /* V, K <= V <= 2^24 */
  int32_t k;            /* K_b, DGAP_MIN_K .. DGAP_MAX_K */
  int32_t hidden_det;   /* detector hidden units, 1 .. DGAP_MAX_HIDDEN */
  int32_t hidden_corr;  /* corrector hidden units, 1 .. DGAP_MAX_HIDDEN */
  float tau;            /* risk threshold: correct when r > tau */
  float det_b2;         /* detector output bias */
  float corr_b2;        /* corrector output bias */
  int32_t pad;
  const float* det_w1;  /* [DGAP_FEATURES][hidden_det] */
  const float* det_b1;  /* [hidden_det] */
  const float* det_w2;  /* [hidden_det] */
  const float* corr_w1; /* [DGAP_CAND_INPUTS + DGAP_FEATURES][hidden_corr]: rows 0..4 take xi, 5..16 phi */
  const float* corr_b1; /* [hidden_corr] */
  const float* corr_w2; /* [hidden_corr] */
} dgap_params;

/* Workspace bytes dgap_restore needs for `batch` rows of `vocab` logits and
 * window k; 0 if the shape is not supported. */
size_t dgap_workspace_bytes(int32_t batch, int32_t vocab, int32_t k);

/* Floats per row of dgap_restore's optional info output:
 *   [0] r, [1] 1 if the row was corrected else 0, [2] log-sum-exp of the
 *   row, [3] 0, [4 .. 4+12) phi, [16 .. 16+k) the window's vocabulary
 *   indices in TopK order (int32 bit patterns), [16+k .. 16+2k) Delta in the
 *   same order (0 when the row was not corrected). */
size_t dgap_info_floats(int32_t k);

/* One DGAP step on `batch` rows of fp32 logits, in place: logits is a
 * device array [batch][vocab], finite values; only the K entries of a
 * corrected row's window change.  ws: device scratch of ws_bytes >=
 * dgap_workspace_bytes, 16-byte aligned, contents undefined on entry and
 * exit.  info: NULL or a device array [batch][dgap_info_floats(k)].
 * Errors: KVQ_ERR_ARG (null params, pointers or weights, shapes out of
 * range, small or misaligned workspace), KVQ_ERR_UNSUPPORTED (vocab above
 * 2^24, or more than 32768 window candidates: ceil(vocab / 2048) * k),
 * KVQ_ERR_HIP (launch failure).  Results are bitwise reproducible. */
kvq_status dgap_restore(const dgap_params* p, float* logits, int32_t batch, void* ws, size_t ws_bytes,
                        float* info, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DGAP_H */
