// Internal definitions shared by the host library and the HIP kernels.
//
// Device arena:
//   [0, 256)            header; word 0 is the sticky error flag
//   per sequence i, per kv head h, one block of head_stride(i) bytes:
//     kc  key codes    [Cq][16*bk]       token rows, canonical bit order
//     km  key meta     [Cq/Gk][2][128]   fp16 scales then zeros per key group
//     vc  value codes  [Cq][16*bv]
//     vm  value meta   [Cq][128/Gv][2]   fp16 (scale, zero) per value group
//     tk  key ring     [W][128]          fp16 tokens not yet packed
//     tv  value ring   [W][128]
//   Cq = Gk * floor(max(0, L_max - R) / Gk) is the most tokens ever packed;
//   W = R + Gk ring slots hold the < R + Gk fp16 tokens, token p in slot p % W.
//   Every region starts on a 256-byte boundary.
//
// The packed regions use the canonical byte order of the export image, so an
// export is a handful of device-to-device copies.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace kvq {

constexpr int kHeadDim = 128;
constexpr int kMaxSeqPerLaunch = 64;   // sequences described in one kernel-argument block
// row_x of the rows of a chunk row group past its whole queries: any value
// at least the largest n_q (KVQ_MAX_CHUNK = 1024) makes such a row spare,
// and kSpareRow * Hq stays far inside 32 bits
constexpr int32_t kSpareRow = 1024;
constexpr int kRecFloats = 132;        // split record: m, l, 2 pad, acc[128]
constexpr uint64_t kAlign = 256;
constexpr uint64_t kHeaderBytes = 256;

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

struct HeadLayout {
  uint64_t kc, km, vc, vm, tk, tv;  // byte offsets inside a (seq, head) block
  uint64_t vb;                      // bound on the value scales packed so far (fp16 bits, in a uint32)
  uint64_t stride;                  // block size
};

inline HeadLayout head_layout(int bk, int bv, int64_t cq, int gk, int gv, int64_t w, bool with_bound = true) {
  HeadLayout L{};
  uint64_t o = 0;
  L.kc = o; o = align_up(o + (uint64_t)cq * 16 * bk, kAlign);
  L.km = o; o = align_up(o + (uint64_t)(cq / gk) * 2 * kHeadDim * 2, kAlign);
  L.vc = o; o = align_up(o + (uint64_t)cq * 16 * bv, kAlign);
  L.vm = o; o = align_up(o + (uint64_t)cq * (kHeadDim / gv) * 4, kAlign);
  L.tk = o; o = align_up(o + (uint64_t)w * kHeadDim * 2, kAlign);
  L.tv = o; o = align_up(o + (uint64_t)w * kHeadDim * 2, kAlign);
  L.vb = o; o = with_bound ? align_up(o + 4, kAlign) : o;
  L.stride = o;
  return L;
}

// ---------------------------------------------------------------- paging
//
// Paged caches keep the packed codes and scales of page_tokens consecutive
// tokens of a sequence (all kv heads) in one page of a shared pool; a block
// table maps (sequence, logical page) to a pool page.  Within a page, head
// h's packed data sit at h * page_head_bytes in the head layout of
// page_tokens tokens.  The fp16 ring of every (sequence, head) stays in a
// contiguous region of its own.  table == nullptr: contiguous caches.
struct PageMap {
  const int32_t* table;      // [batch][max_pages] pool page of each logical page
  uint64_t pool0;            // arena offset of pool page 0
  uint64_t page_bytes;       // Hkv * page_head_bytes
  uint64_t page_head_bytes;
  uint64_t pool_bytes;       // pages * page_bytes
  int32_t page_tokens, max_pages;
  int32_t page_shift, gk_shift;  // log2(page_tokens), log2(key_group)
};

#ifdef __HIPCC__
#define KVQ_PAGE_HD __host__ __device__
#else
#define KVQ_PAGE_HD
#endif
// Arena offset of the packed segment that holds token tok of (sequence seq,
// kv head h), and tok's position in it.  Contiguous caches: the head's
// region (head0 + h * head_stride) and tok itself.
KVQ_PAGE_HD inline uint64_t packed_seg(const PageMap& pm, uint64_t head0, uint64_t head_stride, int seq,
                                               int h, int tok, int& t_in) {
  if (pm.table == nullptr) {
    t_in = tok;
    return head0 + (uint64_t)h * head_stride;
  }
  const int pg = tok >> pm.page_shift;
  t_in = tok & (pm.page_tokens - 1);
  return pm.pool0 + (uint64_t)pm.table[(size_t)seq * pm.max_pages + pg] * pm.page_bytes +
         (uint64_t)h * pm.page_head_bytes;
}

// Block-table entries written by one launch (graph-safe: no memset/copy node).
constexpr int kTableSetMax = 240;
struct TableSet {
  int32_t* table;
  int32_t n, pad;
  int32_t idx[kTableSetMax];
  int32_t val[kTableSetMax];
};

// ---------------------------------------------------------------- append

struct AppendSeq {
  uint64_t head0;     // arena offset of (seq, head 0)
  int32_t seq;        // index into the input batch
  int32_t L_old, Lq_old, Lq_new, L_new;
  int32_t wg_begin;   // first workgroup of this sequence
  int32_t n_quant;    // key groups to pack per head
  int32_t do_copy;    // 1 if this launch writes ring slots
};

struct AppendArgs {
  uint8_t* arena;
  const uint16_t* K;  // fp16 [batch][n_max][Hkv][128]
  const uint16_t* V;
  uint64_t head_stride;
  uint32_t kc, km, vc, vm, tk, tv, vb;
  int32_t n_max, hkv, gk, gv, W, nseq, total_wg;
  int32_t quantize;   // 1: pack groups in this launch
  int32_t matrix;     // 1: matrix layout (kvq_layout.h) for this bit class
  PageMap pm;
  AppendSeq seq[kMaxSeqPerLaunch];
};

// ---------------------------------------------------------------- decode

struct DecodeSeq {
  uint64_t head0;
  int32_t seq;        // batch index (q / out row)
  int32_t L, Lq;
  int32_t nq;         // packed splits per head
  int32_t nsplit;     // nq + (L > Lq)
  int32_t wg_begin;
  int32_t ws_base;    // first split record of this sequence
  int32_t L_old;      // tokens [L_old, L) arrive in this call (fused append), else L_old = L
};

// Query rows.  A launch attends nqry queries per sequence: query j is the
// token at position L - nqry + j and sees tokens [0, L - nqry + 1 + j)
// (nqry = 1: single-token decode over the whole cache).  The rows of one kv
// head h are (query j, head h*gqh + x); a workgroup takes a row group of qpr
// consecutive queries times the gqh heads (GQ = qpr*gqh rows, the kernel's
// template size), row group rg of nrg = ceil(nqry / qpr) (the last one
// may repeat the last query in its spare rows).  q and out are
// [batch][nqry][Hq][128]; a split record row is j*Hq + head.
struct DecodeArgs {
  const uint8_t* arena;
  const uint16_t* q;  // fp16 [batch][nqry][Hq][128]
  float* ws;          // split records [.][nqry * Hq][kRecFloats]
  // fused append: fp16 [batch][n_max][Hkv][128] rows of the tokens [L_old, L),
  // written into the ring by the fp16 tail split of their (sequence, head)
  // before it attends over them; null when the call appends nothing
  const uint16_t* K_new;
  const uint16_t* V_new;
  int32_t n_max, pad;
  uint64_t head_stride;
  uint32_t kc, km, vc, vm, tk, tv, vb;
  int32_t hq, hkv, gk, gv, W, split_tokens, nseq, total_wg;
  float qscale;       // log2(e) / sqrt(d)
  DecodeSeq seq[kMaxSeqPerLaunch];
  // (read by chunk and paged launches only; after the per-sequence entries
  // so that single-token decode reads the same argument lines as before)
  int32_t nqry, qpr, nrg, gqh;
  // row g of a row group is chunk query rg*qpr + row_x[g] and head
  // h*gqh + (row_off[g] - row_x[g]*Hq): row_off[g] = row_x[g]*Hq + g % gqh;
  // rows past the group's qpr*gqh have row_x = kSpareRow (always spare)
  // (host-computed, so the kernels divide nothing)
  int32_t row_off[32], row_x[32];
  PageMap pm;
};

struct MergeSeq {
  int32_t seq, nsplit, ws_base, pad;
};

struct MergeArgs {
  const float* ws;
  float* out;         // fp32 [batch][hq][128]
  int32_t hq, nseq;   // hq: record rows per split (query heads times queries)
  MergeSeq seq[kMaxSeqPerLaunch];
};

// ---------------------------------------------------------------- DGAP

constexpr int kDgapChunk = 2048;            // logits per scan workgroup
constexpr int kDgapMaxK = 256;              // largest window
constexpr int kDgapMaxCandidates = 32768;   // chunks * K per row, held by one workgroup
constexpr int kDgapFeatures = 12;
constexpr int kDgapCandInputs = 5;
constexpr int kDgapInfoHead = 16;           // info floats before the window's indices
constexpr int kDgapMaxHidden = 64;

struct DgapArgs {
  float* logits;       // [batch][vocab], corrected in place
  float* info;         // [batch][kDgapInfoHead + 2k] or null
  float* ws_stats;     // [batch][nchunk][4]: chunk max m, sum e, sum (m - z) e, sum e^2 (e = e^(z - m))
  uint64_t* ws_cand;   // [batch][nchunk][k] candidate keys (0 = empty)
  const float* det_w1;
  const float* det_b1;
  const float* det_w2;
  const float* corr_w1;
  const float* corr_b1;
  const float* corr_w2;
  int32_t vocab, k, nchunk, hidden_det, hidden_corr;
  float tau, det_b2, corr_b2;
};

// ---------------------------------------------------------------- dequant

struct DequantArgs {
  const uint8_t* arena;
  uint64_t head0;       // (seq, head 0) block (paged: the sequence's ring region)
  float* K_out;
  float* V_out;
  uint64_t head_stride;
  uint32_t kc, km, vc, vm, tk, tv;
  int32_t hkv, gk, gv, W, bk, bv, Lq, tok0, ntok;
  int32_t matrix, seq;
  PageMap pm;
};

// ---------------------------------------------------------------- export

// Matrix-layout codes and value meta of one (seq, head) rewritten in the
// canonical order: 32-token blocks [0, Lq / 32).
struct ExportArgs {
  const uint8_t* blk;   // (seq, head) block
  uint8_t* kc_out;      // canonical key codes [Lq][16*bk]
  uint8_t* vc_out;      // canonical value codes [Lq][16*bv]
  uint8_t* vm_out;      // canonical value meta [Lq][128/gv][2] fp16
  uint32_t kc, vc, vm;
  int32_t bk, bv, gv, nblocks;
};

// Launchers (defined next to their kernels).  Return a hipError_t as int.
int launch_append(const AppendArgs& a, int bk, int bv, void* stream);
int launch_table_set(const TableSet& t, void* stream);
// Zero the given 32-bit words of the arena (byte offsets), up to kTableSetMax per launch.
struct WordReset {
  uint8_t* arena;
  int32_t n, pad;
  uint64_t off[kTableSetMax];
};
int launch_word_reset(const WordReset& r, void* stream);
int launch_decode(const DecodeArgs& a, int bk, int bv, int gq, void* stream);
int launch_decode_matrix(const DecodeArgs& a, int bk, int bv, int gq, void* stream);
// Matrix-core decode (and the matrix layout) for this bit class: 4, 5 or 8
// query heads per kv head, 1- or 2-bit codes, value groups >= 32 channels,
// and a (sequence, head) block that one buffer resource covers.
bool matrix_decode_supported(int bk, int bv, int gq, int gk, int gv, uint64_t head_bytes);
// Waves per SIMD of the matrix-core kernel for this bit class (2, 3 or 4);
// the vector kernel runs two.
int matrix_decode_occupancy(int bk, int bv, int gk, int gq);
// Chunk queries over row groups of 16 or 32 rows (chunk_mfma.hip).
int launch_chunk_matrix(const DecodeArgs& a, int bk, int bv, int rows, void* stream);
// The matrix-core decode kernels of one bit class (decode_mfma.hip, one
// object per class); launch_decode_matrix (matrix_dispatch.cpp) picks one.
template <int BK, int BV>
int launch_matrix_class(const DecodeArgs& a, int gq, void* stream);
int launch_export(const ExportArgs& a, void* stream);
int launch_merge(const MergeArgs& a, void* stream);
int launch_dgap(const struct DgapArgs& a, int batch, void* stream);
int launch_dequant(const DequantArgs& a, void* stream);
int launch_fill_zero(void* dst, size_t words, void* stream);
// Streaming-read probe: kvq_read_probe's kernel and its grid size.
int launch_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream);
int read_probe_blocks();

// Bytes of the per-device scratch array behind kvq_decode_attention_noalloc.
constexpr size_t kScratchBytes = (size_t)16 << 20;
// Device address of the current device's scratch array (looked up once per
// device); returns a hipError_t as int.
int scratch_workspace(void** ptr);

}  // namespace kvq
