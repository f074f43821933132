// Matrix-core decode attention for caches with 1- or 2-bit keys and values,
// or 4- or 8-bit keys and values, and 1, 2, 4, 5 or 8 query heads per kv head
// (gfx950, v_mfma_f32_16x16x32_f16).
//
// Same result as the vector kernel: softmax(q K^T / sqrt(d)) V over the
// dequantized cache (Introduction: scaled dot-product attention), split-K
// over tokens with an online softmax in base 2.  At one or two bits a token
// of one kv head carries 64-96 bytes but 2 * 4 * 128 multiply-adds, more than
// the vector ALUs can retire at HBM speed, so both contractions go to the
// matrix cores with fp32 accumulation:
//
//   scores:  S[row][t] = sum_c Q'[row][c] * code[t][c] + sum_c q~[row][c] * z[c]
//     A = Q' = q~ (.) s split into fp16 hi + lo parts (two product terms,
//         each exact: q~ and s are fp16, their product fits two halves),
//         row = 4*head + x for 4 heads (x = 0, 2 carry hi, x = 1, 3 lo) or
//         2*head + x for up to 8 heads (x = 0 hi, 1 lo),
//     B = key codes as exact fp16.
//     A lane of the result holds one token of one or two heads (elements
//     x), so every lane takes its own exponentials and a 16-lane row reduces
//     the block maximum of its heads.  The zero-point term uses A = q~ and B = z
//     broadcast over tokens.  q~ = q * 2^-e with |q~| < 1 keeps every fp16
//     operand finite; the scale 2^e * log2(e) / sqrt(d) is applied to the
//     fp32 result.
//   values:  O^T[c][col] = sum_t code[t][c] * P'[t][col] (+ z term on VALU)
//     A = value codes (exact fp16), B = P' = p * s_v rounded once to fp16
//     (relative error <= 2^-11 per weight, the rounding of the P operand in
//     any fp16 attention kernel), column col = 4*head + value group (one
//     MFMA per 4 heads and 16 channels); the weights p reach the B layout
//     through LDS.  A tile of 16 channels keeps only the columns of its
//     value group (the rest of its B operand is zero), so tiles of
//     different groups share one accumulator: two accumulators hold the
//     128 channels of 4 heads.  Eight heads take two such head quads; five
//     heads take columns (head, group) = (col % 5, col / 5) for groups 0-2
//     and a second operand for group 3 (at 8 bits: a second quad with head
//     4 alone).  With two operands per block the registers hold one
//     accumulator per tile instead of sharing them.
//
// Packed key codes become operands with a shift or two and one AND per
// element pair: a set bit at mantissa position w of a half is the exact fp16
// subnormal 2^(w - 24), and the shifts put every code among the top mantissa
// positions, where the matrix cores keep the products of such subnormals to
// near fp32 precision (see unpack_bits).  An element pair's weight (2^i at
// one bit, 1 or 4 at two bits) depends only on the channel and is folded
// into q~ once per decode; the common code unit goes into the fp32 scale.
// A 1-bit value operand (8 tokens of one channel) is unpacked like a key
// operand (one shift, four ANDs); its element-pair weight 2^i is folded into
// the softmax weights of those tokens through the exponent offset of their
// lanes, so it costs no instruction in the loop.  A 2-bit value operand comes
// from a 256-entry LDS table indexed by bytes of packed codes (4 halves
// 0..3 per byte, exact normal numbers), one LDS read per byte instead of
// several vector instructions.
// At 4 and 8 bits a dword holds whole codes, and one instruction per
// element pair turns them into subnormal halves (see whole8); a token then
// carries 160-288 bytes for the same arithmetic, and the matrix cores keep
// the vector ALUs free for the conversions.
// The layouts that place the bits are in kvq_layout.h.
#include <hip/hip_runtime.h>

#include "decode_common.h"
#include "kvq_internal.h"
#include "kvq_layout.h"
#include "mfma_common.h"

namespace kvq {
namespace {

using namespace dec;

using namespace mfma_ops;

// Headroom of the softmax reference above the largest score seen (log2
// units): weights of later tokens within it need no rescale.
constexpr float kLazyMargin = 3.f;
// dwords per Q' row in LDS: 64 + 4 of padding, so that the eight rows one
// 8-lane group of a 16-byte read touches start in different bank quads
constexpr int kQRow = 68;
// floats per head row of the weights handed from the score to the value
// layout: 32 + 16 of padding (rows 2r and 2r+1 fall in different bank halves)
constexpr int kPRow = 48;
// Blocks per zero-point table (a multiple of the main loop's unroll of 3):
// the table holds the zero-point terms of the kChunk / BPG key groups a wave
// processes next.
constexpr int kChunk = 48;

// Maximum over the four lane rows (lanes l, l^16, l^32, l^48) with the
// gfx950 row-swap permutes.
__device__ __forceinline__ float max_across_rows(float v) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  v = fmaxf(__builtin_bit_cast(float, (uint32_t)s32[0]), __builtin_bit_cast(float, (uint32_t)s32[1]));
  const uint32_t w = __builtin_bit_cast(uint32_t, v);
  const auto s16 = __builtin_amdgcn_permlane16_swap(w, w, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)s16[0]), __builtin_bit_cast(float, (uint32_t)s16[1]));
}

// v[i] as a chain of selects (keeps v in registers; an indexed read would
// move the array to scratch memory).
template <int K, int N>
__device__ __forceinline__ float pick_from(const float (&v)[N], int i) {
  if constexpr (K == N - 1)
    return v[K];
  else
    return i == K ? v[K] : pick_from<K + 1, N>(v, i);
}
template <int N>
__device__ __forceinline__ float pickn(const float (&v)[N], int i) {
  return pick_from<0, N>(v, i);
}

// Everything one 32-token block reads from memory.
template <int BK, int BV>
struct BlockData {
  uint32_t s;          // key scales of channels 2*lane, 2*lane+1 (this block's key group)
  uint32_t kx[2][BK];  // key codes of tokens 16*mb + (lane & 15)
  uint32_t vx[2 * BV]; // value codes of this lane
  u4_t sv, zv;         // value scales / zeros of this lane's 8 tokens and group, element order
  u4_t sv3, zv3;       // five heads: the same for value group 3 (loaded only there)
};

// Per-lane byte offsets of one block's loads (the per-block parts are scalar).
struct LaneOffsets {
  uint32_t km, kc, vc, vs, vz, vs3, vz3;
};

template <int BK, int BV, bool G3>
__device__ __forceinline__ void load_block(__amdgpu_buffer_rsrc_t r, const LaneOffsets& lo, uint32_t km,
                                           uint32_t kc, uint32_t vc, uint32_t vm, BlockData<BK, BV>& o) {
  o.s = ld32(r, lo.km, km);
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    if constexpr (BK == 1) {
      o.kx[mb][0] = ld32(r, lo.kc + mb * 16 * 16 * BK, kc);
    } else if constexpr (BK == 2) {
      const uint2 v = ld64(r, lo.kc + mb * 16 * 16 * BK, kc);
      o.kx[mb][0] = v.x;
      o.kx[mb][1] = v.y;
    } else {
#pragma unroll
      for (int w = 0; w < BK / 4; ++w) {
        const u4_t v = ld128(r, lo.kc + mb * 16 * 16 * BK + 16 * w, kc);
        o.kx[mb][4 * w] = v[0]; o.kx[mb][4 * w + 1] = v[1]; o.kx[mb][4 * w + 2] = v[2]; o.kx[mb][4 * w + 3] = v[3];
      }
    }
  }
  if constexpr (BV == 1) {
    const uint2 v = ld64(r, lo.vc, vc);
    o.vx[0] = v.x;
    o.vx[1] = v.y;
  } else {
#pragma unroll
    for (int w = 0; w < BV / 2; ++w) {
      const u4_t v = ld128(r, lo.vc + 16 * w, vc);
      o.vx[4 * w] = v[0]; o.vx[4 * w + 1] = v[1]; o.vx[4 * w + 2] = v[2]; o.vx[4 * w + 3] = v[3];
    }
  }
  o.sv = ld128(r, lo.vs, vm);
  o.zv = ld128(r, lo.vz, vm);
  if constexpr (G3) {
    o.sv3 = ld128(r, lo.vs3, vm);
    o.zv3 = ld128(r, lo.vz3, vm);
  }
}

// The value of quad member K, broadcast to the whole quad (quad_perm
// [K,K,K,K]; every lane has a source, so no fill value is needed).
template <int K>
__device__ __forceinline__ float quad_bcast(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), K * 0x55, 0xF, 0xF, false));
}

// Query heads per kv head the score rows carry: 4 (rows 4h + x, x = hi, lo,
// hi, lo) or 8 (rows 2h + x, x = hi, lo); 5 heads use the 8-head layout with
// three empty heads.
template <int GQ>
struct MatrixHeads {
  static constexpr int value = GQ <= 4 ? 4 : 8;
};
// Waves per SIMD the instantiation is compiled for (matrix_waves, shared
// with the host's split plan).
template <int BK, int BV, int BPG, int GQ>
struct MatrixOcc {
  static constexpr int value = matrix_waves(BK, BV, BPG, GQ);
};
// Blocks in flight per wave: at four waves per SIMD, with the eight-head
// accumulators and with 8-bit blocks (41 registers each), the registers hold
// two block buffers (loads one block ahead), otherwise three.
template <int BK, int BV, int BPG, int GQ>
struct MatrixStages {
  static constexpr int value = (MatrixOcc<BK, BV, BPG, GQ>::value >= 4 || GQ > 4 || BK + BV >= 16) ? 2 : 3;
};


// CAUSAL: chunk queries (rows see tokens below their own limit); the
// single-token decode instantiations carry no masking code.  PAGED: the
// packed data live in the pages of a block table (PageMap).
template <int BK, int BV, int BPG, int GQ, bool CAUSAL, bool PAGED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MatrixOcc<BK, BV, BPG, GQ>::value))) void
decode_mfma_kernel(DecodeArgs a) {
  constexpr int NH = MatrixHeads<GQ>::value;  // heads in the score rows
  constexpr int HPL = NH / 4;                 // heads per lane in the score layout
  constexpr int NQ = NH / 4;                  // head quads in the value columns
  constexpr int RS = 16 / NH;                 // score rows per head
  constexpr int kDzRows = (kChunk * NH + kQRow - 1) / kQRow;
  // per wave: Q' hi rows, lo rows, then the zero-point terms of up to
  // kChunk key groups (16-byte aligned: rows are read with 16-byte loads)
  __shared__ __attribute__((aligned(16))) uint32_t q_lds[kWaves][(2 * NH + kDzRows) * kQRow];
  // the prepared query, shared by the waves: q~ of head g in row g (the B
  // operand of the zero-point terms), the lane words of q~ with the key
  // pair weights, and the fp32 score scale of each head
  __shared__ __attribute__((aligned(16))) uint32_t qq_s[NH * kQRow];
  __shared__ uint32_t qt_s[NH][64];
  __shared__ float cs_s[NH];
  __shared__ __attribute__((aligned(16))) float p_lds[kWaves][kPRow * NH];  // weights to the value layout; fp16 tail split
  __shared__ Reduce<GQ> red;
  // value operand halves of each byte of packed 2-bit codes (its 2-bit fields)
  constexpr int kTabWords = BV == 2 ? ValueTable2::kWords : 4;
  __shared__ __attribute__((aligned(16))) uint32_t vtab[kTabWords];

  const Work wk = find_work<CAUSAL>(a);
  const DecodeSeq& S = a.seq[wk.si];
  const uint8_t* blk = a.arena + S.head0 + (uint64_t)wk.h * a.head_stride;
  // wave index as a scalar so that per-wave loop bounds stay in SGPRs
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // The bound on this head's value scales (it sets the weight shift below).
  // Issued first as a vector load, held there by the compiler barrier, and
  // consumed after the query is prepared, so its latency hides behind the
  // first blocks' loads (a scalar load would be waited for with the loads of
  // the arguments, before those go out).
  uint32_t vbound = __builtin_amdgcn_raw_buffer_load_b32(head_rsrc(blk + a.vb, 4), 0, 0, 0);
  asm volatile("" ::: "memory");

  if (wk.sp >= S.nq) {  // fp16 tail tokens: vector path
    float qs0[GQ], qs1[GQ];
    load_q_scaled<GQ, CAUSAL>(a, S, wk.h, wk.rg, lane, qs0, qs1);
    State<GQ> st;
    init_state<GQ>(st);
    static_assert(kHeadDim * QStride<GQ>::value <= (2 * NH + kDzRows) * kQRow, "tail query fits the Q' area");
    static_assert(32 * GQ <= kPRow * NH, "tail weights fit the weight area");
    tail_split<GQ, CAUSAL>(a, S, wk.h, wk.rg, blk, qs0, qs1, reinterpret_cast<float*>(q_lds[wv]), p_lds[wv], st,
                           lane, wv);
    stage_state<GQ>(st, red, lane, wv);
    __syncthreads();
    write_record<GQ, CAUSAL>(a, S, wk.h, wk.rg, wk.sp, red);
    return;
  }

  // Value layout: lane (col, row) = column (head 4q + hc, value group xc),
  // tokens of K-group row.  Score A rows: row col = head hs, half part.
  const int col = lane & 15, row = lane >> 4;     // MFMA column, lane row
  const int hc = col >> 2, xc = col & 3, part = col & 1, hs = col / RS;
  const int ng = kHeadDim / a.gv;
  // Five heads (with one accumulator per tile): the value columns of one B
  // operand are (head h1, group g1) = (col % 5, col / 5) for the groups 0 ..
  // G1 - 1, G1 = min(ng, 3) (15 columns at most; the rest repeat a column),
  // and with four groups a second operand holds (col, group 3) for col < 5.
  // 8 value MFMAs per block instead of two head quads' 16.
  constexpr bool kFive = GQ == 5 && NH / 4 == 2 && BK + BV <= 8;
  const int g1 = min(col / 5, min(ng, 3) - 1), h1 = col % 5;
  const int gsel = kFive ? g1 : xc & (ng - 1);
  // row g of the row group reads q row qbase + row_q_offset(g) (0 for row 0)
  const uint16_t* qbase = CAUSAL ? a.q + q_index<GQ, CAUSAL>(a, S, wk.h, wk.rg, 0) * kHeadDim
                                 : a.q + ((size_t)S.seq * a.hq + (size_t)wk.h * GQ) * kHeadDim;
  // Packed data: the (sequence, head) region, or in a paged cache this kv
  // head's region of the page that holds the block (a buffer resource per
  // block, so that offsets stay inside one page whatever the pool size).
  // The split's first 64 pages are looked up once, one per lane; a block
  // reads its page index from that lane (pages further on, in splits of more
  // than 64 pages, come from the table directly).
  constexpr bool paged = PAGED;
  const __amdgpu_buffer_rsrc_t rs = head_rsrc(blk, paged ? 0 : a.head_stride);
  const int32_t* ptab = paged ? a.pm.table + (size_t)S.seq * a.pm.max_pages : nullptr;
  const uint8_t* pool_h = paged ? a.arena + a.pm.pool0 + (uint64_t)wk.h * a.pm.page_head_bytes : nullptr;
  const int pg0 = paged ? (wk.sp * a.split_tokens) >> a.pm.page_shift : 0;
  int lane_pg = 0;
  if constexpr (PAGED) {
    if (pg0 + lane < a.pm.max_pages) lane_pg = ptab[pg0 + lane];
  }
  // the resource of the region holding token tok, and tok's position in it;
  // seg_of takes a wave-uniform token
  auto seg_of = [&](int tok, int& tin) -> __amdgpu_buffer_rsrc_t {
    if (!paged) {
      tin = tok;
      return rs;
    }
    const int pg = tok >> a.pm.page_shift;
    tin = tok & (a.pm.page_tokens - 1);
    const int k = pg - pg0;
    const int pool_pg = k < 64 ? __builtin_amdgcn_readlane(lane_pg, k) : ptab[pg];
    return head_rsrc(pool_h + (uint64_t)pool_pg * a.pm.page_bytes, a.pm.page_head_bytes);
  };
  LaneOffsets lo;
  lo.km = 4 * lane;
  lo.kc = col * 16 * BK + row * 4 * BK;
  lo.vc = lane * 8 * BV;
  lo.vs = (gsel * 32 + 8 * row) * 2;
  lo.vz = lo.vs + ng * 64;
  lo.vs3 = (3 * 32 + 8 * row) * 2;
  lo.vz3 = lo.vs3 + ng * 64;

  // This wave's 32-token blocks: key groups j0 + ws + kWaves*n, each of
  // BPG blocks; block i is key group j0 + kWaves*(i / BPG), part i % BPG.
  // The wave slot ws rotates by two with the workgroup's dispatch round
  // (ids 256 apart share a compute unit, one wave of each on every SIMD):
  // when a split's key groups do not divide by kWaves, the extra groups of
  // the two workgroups of a compute unit go to different SIMDs instead of
  // piling onto the first.
  const int t0 = wk.sp * a.split_tokens;
  const int t1 = min(S.Lq, t0 + a.split_tokens);
  const int wslot = (wv + 2 * ((int)blockIdx.x >> 8)) & (kWaves - 1);
  const int j0 = t0 / a.gk + wslot, jend = t1 / a.gk;
  const int ngroups = j0 < jend ? (jend - j0 + kWaves - 1) / kWaves : 0;
  const int nblocks = ngroups * BPG;
  const int last = nblocks - 1;
  const int vstride = 128 * ng;
  auto load = [&](int i, BlockData<BK, BV>& o) {
    const int j = j0 + kWaves * (i / BPG);
    int tok;
    const __amdgpu_buffer_rsrc_t r = seg_of(j * a.gk + (i % BPG) * 32, tok);
    const int jg = paged ? tok >> a.pm.gk_shift : j;  // key group within the segment
    load_block<BK, BV, kFive>(r, lo, a.km + (uint32_t)jg * (2 * kHeadDim * 2), a.kc + (uint32_t)tok * 16 * BK,
                       a.vc + (uint32_t)(tok / 32) * 512 * BV, a.vm + (uint32_t)(tok / 32) * vstride, o);
  };
  // Key zero-points of the wave's key groups k0 .. k0 + 15 as the A operand
  // of their zero-point terms (row = group; past the last group: the last).
  // A paged cache reads them with 64-bit addresses (one page per lane).
  auto load_z = [&](int k0, h8_t (&zq)[4]) {
    const int j = j0 + kWaves * min(k0 + col, ngroups - 1);
    if constexpr (PAGED) {
      const int tok = j * a.gk;
      const uint8_t* zrow = pool_h + (uint64_t)ptab[tok >> a.pm.page_shift] * a.pm.page_bytes + a.km +
                            (uint64_t)((tok & (a.pm.page_tokens - 1)) >> a.pm.gk_shift) * (2 * kHeadDim * 2) +
                            kHeadDim * 2;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        zq[kb] = __builtin_bit_cast(h8_t, *reinterpret_cast<const u4_t*>(zrow + (32 * kb + 8 * row) * 2));
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        zq[kb] = __builtin_bit_cast(
            h8_t, ld128(rs, (uint32_t)j * (2 * kHeadDim * 2) + kHeadDim * 2 + (32 * kb + 8 * row) * 2, a.km));
    }
  };
  // The query heads this wave prepares for the workgroup (heads wv,
  // wv + kWaves, ...), and the value table words this thread copies: both
  // loads go out before the first blocks', so that the barrier below does
  // not wait behind the bulk of the data.
  constexpr int kOwn = (NH + kWaves - 1) / kWaves;
  uint32_t qw[kOwn];
#pragma unroll
  for (int i = 0; i < kOwn; ++i) {
    const int g = wv + kWaves * i;
    qw[i] = g < GQ ? reinterpret_cast<const uint32_t*>(qbase + (size_t)(CAUSAL ? row_q_offset(a, wk.rg, g) : g) * kHeadDim)[lane]
                   : 0u;
  }
  constexpr int kTabLoads = BV == 2 ? ValueTable2::kWords / 4 : 0;
  u4_t tabw = {0u, 0u, 0u, 0u};
  if constexpr (kTabLoads > 0) {
    if ((int)threadIdx.x < kTabLoads) tabw = reinterpret_cast<const u4_t*>(kValueTable2.w)[threadIdx.x];
  }
  asm volatile("" ::: "memory");

  // the first two blocks and the first zero-points load while the query is prepared
  constexpr int kStages = MatrixStages<BK, BV, BPG, GQ>::value;
  BlockData<BK, BV> b0, b1, b2;
  h8_t zq[4];
  if (nblocks > 0) {
    load(0, b0);
    if constexpr (kStages == 3) load(min(1, last), b1);
    load_z(0, zq);
  }

  // q~ = q * 2^-e per head with max |q~| < 1.  For the code MFMA each lane's
  // channel pair (2*lane, 2*lane+1) also carries 2^-w, w = the bit weight of
  // those channels in the unpacked key operand.  Each wave prepares its own
  // heads into LDS; empty heads get zero rows (scores 0).
  const float wq = BK == 1 ? ldexpf(1.f, -(lane & 3)) : BK == 2 ? ((lane & 1) ? 0.25f : 1.f) : 1.f;
#pragma unroll
  for (int i = 0; i < kOwn; ++i) {
    const int g = wv + kWaves * i;
    if (g >= NH) break;
    if (g < GQ) {
      const float q0 = h2f(qw[i] & 0xFFFF), q1 = h2f(qw[i] >> 16);
      const float mx = wave_max(fmaxf(fabsf(q0), fabsf(q1)));
      int e = 0;
      frexpf(mx, &e);
      const float inv = ldexpf(1.f, -e);
      qt_s[g][lane] = h2u((h2_t){(_Float16)(q0 * inv * wq), (_Float16)(q1 * inv * wq)});
      qq_s[g * kQRow + lane] = h2u((h2_t){(_Float16)(q0 * inv), (_Float16)(q1 * inv)});
      if (lane == 0) cs_s[g] = ldexpf(a.qscale, e - CodeUnit<BK>::value);  // undoes 2^-e and the code unit
    } else {
      qt_s[g][lane] = 0u;
      qq_s[g * kQRow + lane] = 0u;
      if (lane == 0) cs_s[g] = 1.f;
    }
  }
  if constexpr (kTabLoads > 0) {
    if ((int)threadIdx.x < kTabLoads) reinterpret_cast<u4_t*>(vtab)[threadIdx.x] = tabw;
  }
  uint32_t* ql = q_lds[wv];
  float* dzt = reinterpret_cast<float*>(ql + 2 * NH * kQRow);  // [group k mod (kChunk / BPG)][head]
#pragma unroll
  for (int g = GQ; g < NH; ++g) {  // empty heads: zero Q' rows
    ql[g * kQRow + lane] = 0u;
    ql[(NH + g) * kQRow + lane] = 0u;
  }
  __syncthreads();
  uint32_t qt[NH];
#pragma unroll
  for (int g = 0; g < NH; ++g) qt[g] = g < GQ ? qt_s[g][lane] : 0u;
  const uint32_t* qq = qq_s;
  // score layout: token col of the 16-token tile, heads HPL*row + hh
  float cs[HPL];
#pragma unroll
  for (int hh = 0; hh < HPL; ++hh) cs[hh] = cs_s[HPL * row + hh];
  // Chunk queries: row g sees tokens below lim[g]; blocks that reach glim
  // (the row group's smallest limit) mask their later tokens per row.
  // Single-token decode: glim = L, past every packed block.
  const int glim = group_limit(a, S, wk.rg);
  int lim[HPL];
#pragma unroll
  for (int hh = 0; hh < HPL; ++hh) {
    const int g = HPL * row + hh;
    lim[hh] = g < GQ ? row_limit(a, S, wk.rg, g) : S.L;
  }

  // Zero-point terms sum_c z[c] q~[c] of 16 key groups and the NH heads, in
  // one MFMA chain (A = z of group col, B = q~ of head col / RS), scaled like
  // the code products, into table rows s .. s + 15; lanes of column RS*head
  // hold groups 4*row .. 4*row + 3.
  auto dz_rows = [&](int s, const h8_t (&zq)[4]) {
    f4_t t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      t = mfma(zq[kb], *reinterpret_cast<const h8_t*>(&qq[hs * kQRow + 16 * kb + 4 * row]), t);
    if (col % RS == 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) dzt[(s + 4 * row + e) * NH + hs] = t[e] * ldexpf(1.f, CodeUnit<BK>::value);
    }
  };
  // The table for the wave's groups k0 .. k0 + kChunk / BPG - 1; zq holds
  // the zero-points of the first 16 (the rest load here: only long splits
  // have them).
  constexpr int kChunkGroups = kChunk / BPG;
  auto fill_table = [&](int k0, const h8_t (&zq)[4]) {
    wave_lds_sync();  // the q~ rows are written, earlier reads of the table are done
    dz_rows(0, zq);
    for (int s = 16; s < kChunkGroups && k0 + s < ngroups; s += 16) {
      h8_t zn[4];
      load_z(k0 + s, zn);
      dz_rows(s, zn);
    }
  };
  if (nblocks > 0) fill_table(0, zq);

  // the weight shift of this (sequence, kv head): the largest S <= 30 with
  // 2^S * bound < 2^15 (bound = the largest value scale packed so far)
  float pshift = (float)kMaxPShift;
  {
    asm volatile("" : "+v"(vbound));
    const uint32_t vbits = vbound & 0xFFFFu;
    if (vbits >= 0x7C00u) {
      pshift = 0.f;
    } else if (vbits != 0u) {
      int ex = 0;
      frexpf(h2f(vbits), &ex);  // bound < 2^ex
      pshift = (float)min(kMaxPShift, max(0, 15 - ex));
    }
  }

  // Score layout: m[hh] = the softmax reference of head HPL*row + hh
  // (uniform over the row), l[hh] = the sum of the lane's own weights.
  // Value layout: zacc[q][t] = the zero-point term of head 4q + hc, group xc
  // over the lane's tokens (element pair t of the 1-bit value operand: the
  // weights of pair t carry 2^-t there); acc[q] the code term.
  //
  // 1-bit values: the unpacked operand of element pair i is code * 2^(i - 18),
  // so the weights of its tokens are taken as 2^-i * p.  Score lane col holds
  // block token 16*mb + col, which is element 4*mb + (col & 3) of the value
  // operand, pair i = 2*mb + pw with pw = (col & 3) >> 1: the exponent offset
  // nm[hh][mb] = -(m + i) gives the weighted p at no extra cost, and l adds
  // 4x the second tile's weight and is rescaled by 2^pw after the loop.
  constexpr bool kPairW = BV == 1;
  constexpr int NZ = kPairW ? 4 : 1;
  const float pw = kPairW ? (float)((col & 3) >> 1) : 0.f;
  float m[HPL], l[HPL], nm[HPL][2], zacc[NQ][NZ];
  // Packed value accumulators: the column group xc of a tile's MFMA keeps
  // only the columns of its value group, so the four tiles 2j + e (j =
  // 0..3) with distinct column groups share accumulator e (the other
  // columns of their B operand are zero).  Tile pair (2j, 2j + 1) takes
  // column group tile_col(j); lane column xc owns that pair iff they match.
  // With two head quads (five or eight heads, two waves per SIMD) the
  // registers hold one accumulator per tile instead: every column of a
  // tile's product is kept, the columns of other value groups are dropped
  // after the loop, and the B operand needs no per-tile zeroing (32 fewer
  // selects per block).  Not with 8-bit codes, whose blocks leave too few
  // registers (250-256 with eight accumulators, and slower).
  constexpr bool kWide = NQ == 2 && BK + BV <= 8;
  constexpr int NA = kWide ? 8 : 2;
  f4_t acc[NQ][NA];
#pragma unroll
  for (int hh = 0; hh < HPL; ++hh) {
    m[hh] = -__builtin_inff();
    l[hh] = 0.f;
    nm[hh][0] = nm[hh][1] = __builtin_inff();
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
#pragma unroll
    for (int t = 0; t < NZ; ++t) zacc[q][t] = 0.f;
#pragma unroll
    for (int e = 0; e < NA; ++e) acc[q][e] = (f4_t){0.f, 0.f, 0.f, 0.f};
  }
  // Column group of tile pair j: value group g = j * ng / 4 of channels
  // 32j .. 32j + 31 sits in column groups x with x % ng = g; the pairs
  // sharing an accumulator take distinct ones.
  auto tile_col = [&](int j) { return ng == 2 ? (j >> 1) + 2 * (j & 1) : j; };
  bool own[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) own[j] = xc == tile_col(j);

  float* pl = p_lds[wv];

  f4_t dz = {0.f, 0.f, 0.f, 0.f};
  h8_t bp[4];
  auto process = [&](const BlockData<BK, BV>& cur, int i) {
    if (BPG == 1 || i % BPG == 0) {
      const int k = i / BPG;  // the wave's key group
      // Q' = q~ (.) s of the block's key group, hi and lo halves, re-laid
      // out through LDS
      wave_lds_sync();
#pragma unroll
      for (int g = 0; g < GQ; ++g) {  // (the rows of empty heads stay zero)
        const h2_t q2 = u2h(qt[g]), s2 = u2h(cur.s);
        const h2_t hi = q2 * s2;
        const h2_t lo = __builtin_elementwise_fma(q2, s2, -hi);
        ql[g * kQRow + lane] = h2u(hi);
        ql[(NH + g) * kQRow + lane] = h2u(lo);
      }
      wave_lds_sync();
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        bp[kb] = *reinterpret_cast<const h8_t*>(&ql[(part * NH + hs) * kQRow + 16 * kb + 4 * row]);
      // the group's zero-point terms enter the hi rows of the scores
      const float* dzr = dzt + (k % kChunkGroups) * NH + HPL * row;
      if constexpr (HPL == 1)
        dz = (f4_t){dzr[0], 0.f, 0.f, 0.f};
      else
        dz = (f4_t){dzr[0], 0.f, dzr[1], 0.f};
    }

    // unscaled scores of token 16*mb + col for heads HPL*row + hh
    f4_t d[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      d[mb] = dz;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if constexpr (BK == 1) {
          d[mb] = mfma(bp[kb], unpack_bits(cur.kx[mb][0], kb), d[mb]);
        } else if constexpr (BK == 2) {
          d[mb] = mfma(bp[kb], unpack_pairs2(cur.kx[mb][kb >> 1], kb & 1), d[mb]);
        } else {
          d[mb] = mfma(bp[kb], whole8<BK>(&cur.kx[mb][(BK / 4) * kb]), d[mb]);
        }
      }
    }
    float raw[HPL][2];
#pragma unroll
    for (int hh = 0; hh < HPL; ++hh)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) raw[hh][mb] = d[mb][2 * hh] + d[mb][2 * hh + 1];  // hi + lo rows
    const int tok = (j0 + kWaves * (i / BPG)) * a.gk + (i % BPG) * 32;
    const bool masked = CAUSAL && tok + 32 > glim;
    if (masked) {
#pragma unroll
      for (int hh = 0; hh < HPL; ++hh)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
          if (tok + 16 * mb + col >= lim[hh]) raw[hh][mb] = -__builtin_inff();
    }

    // online softmax (base 2) per head over these 32 tokens; cs > 0, so the
    // maximum is taken before scaling.  The reference m moves only when a
    // score exceeds it, and then to kLazyMargin above the block maximum of
    // the head: every weight stays <= 1, and the rescale of the accumulators
    // (and its exponential) is skipped while later scores stay under the
    // reference.  Each lane compares its own two scores; only a block with a
    // score above its reference reduces the maxima across the row's lanes.
    // With the weight shift m and every score are kept pshift lower, so the
    // weights reach 2^pshift; m is the reference of the record.
    const float ninf = -__builtin_inff();
    float bm[HPL];
    bool up = false;
#pragma unroll
    for (int hh = 0; hh < HPL; ++hh) {
      const float b = fmaxf(raw[hh][0], raw[hh][1]);
      bm[hh] = fmaf(b, cs[hh], -pshift);
      up |= bm[hh] > m[hh];
    }
    if (__builtin_amdgcn_ballot_w64(up)) {
      float alpha[HPL];
#pragma unroll
      for (int hh = 0; hh < HPL; ++hh) {
        float b = bm[hh];  // scaling by cs > 0 (and the shift) keeps the order
        b = fmaxf(b, dpp_mov<kQuadXor1>(ninf, b));
        b = fmaxf(b, dpp_mov<kQuadXor2>(ninf, b));
        b = fmaxf(b, dpp_mov<kHalfMirror>(ninf, b));
        b = fmaxf(b, dpp_mov<kMirror>(ninf, b));
        const float mnew = b > m[hh] ? b + kLazyMargin : m[hh];
        // 1 where the reference stays; a chunk row with no visible token yet
        // keeps m = -inf (single-token rows all move at the first block)
        alpha[hh] = CAUSAL && mnew == m[hh] ? 1.f : __builtin_amdgcn_exp2f(m[hh] - mnew);
        l[hh] *= alpha[hh];
        m[hh] = mnew;
        nm[hh][0] = -(mnew + pw);
        nm[hh][1] = kPairW ? nm[hh][0] - 2.f : nm[hh][0];
      }
      // the same factors in the value layout: head H = 4q + hc sits in the
      // score lanes of row H / HPL, as their element H % HPL
#pragma unroll
      for (int q = 0; q < (kFive ? 1 : NQ); ++q) {
        // five heads: both value operands of a lane hold its column's head
        // h1 (see kFive), one accumulator per tile; else quad 1 is head 4
        // alone
        const int H = kFive ? h1 : (GQ == 5 && q == 1) ? 4 : 4 * q + hc;
        float av;
        if constexpr (HPL == 1) {
          av = __shfl(alpha[0], 16 * H);
        } else {
          const float a0 = __shfl(alpha[0], 16 * (H >> 1)), a1 = __shfl(alpha[1], 16 * (H >> 1));
          av = (H & 1) ? a1 : a0;
        }
#pragma unroll
        for (int e = 0; e < NA; ++e) acc[q][e] *= av;
#pragma unroll
        for (int t = 0; t < NZ; ++t) {
          zacc[q][t] *= av;
          if constexpr (kFive) zacc[1][t] *= av;
        }
      }
    }
    // to the value layout: lane (col, row) needs tokens 4*row + 0..3 and
    // 16 + 4*row + 0..3 of heads 4q + hc
    float e[HPL][2];
#pragma unroll
    for (int hh = 0; hh < HPL; ++hh) {
      e[hh][0] = __builtin_amdgcn_exp2f(fmaf(raw[hh][0], cs[hh], nm[hh][0]));
      e[hh][1] = __builtin_amdgcn_exp2f(fmaf(raw[hh][1], cs[hh], nm[hh][1]));
      if (masked) {  // masked tokens weigh 0, also while m is still -inf
        e[hh][0] = raw[hh][0] == -__builtin_inff() ? 0.f : e[hh][0];
        e[hh][1] = raw[hh][1] == -__builtin_inff() ? 0.f : e[hh][1];
      }
      l[hh] += kPairW ? fmaf(e[hh][1], 4.f, e[hh][0]) : e[hh][0] + e[hh][1];
    }
    wave_lds_sync();
#pragma unroll
    for (int hh = 0; hh < HPL; ++hh) {
      pl[(HPL * row + hh) * kPRow + col] = e[hh][0];
      pl[(HPL * row + hh) * kPRow + 16 + col] = e[hh][1];
    }
    wave_lds_sync();
    if constexpr (kFive) {
      // Five heads: lane column col carries head h1 = col % 5 in both value
      // operands, group g1 in the first and group 3 in the second (four
      // groups); tiles of group 3 take the second, all others the first.
      const f4_t pa = *reinterpret_cast<const f4_t*>(&pl[h1 * kPRow + 4 * row]);
      const f4_t pb = *reinterpret_cast<const f4_t*>(&pl[h1 * kPRow + 16 + 4 * row]);
      const float p[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};
      u4_t b1, b3;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const h2_t s2 = u2h(cur.sv[t]);
        float f0 = fmaf(p[2 * t], (float)s2.x, 0.f), f1 = fmaf(p[2 * t + 1], (float)s2.y, 0.f);
        keep_f32(f0, f1);
        b1[t] = h2u((h2_t){(_Float16)f0, (_Float16)f1});
        const h2_t z2 = u2h(cur.zv[t]);
        float& za = zacc[0][kPairW ? t : 0];
        za = fmaf(p[2 * t], (float)z2.x, fmaf(p[2 * t + 1], (float)z2.y, za));
      }
      b3 = b1;
      if (ng == 4) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const h2_t s2 = u2h(cur.sv3[t]);
          float f0 = fmaf(p[2 * t], (float)s2.x, 0.f), f1 = fmaf(p[2 * t + 1], (float)s2.y, 0.f);
          keep_f32(f0, f1);
          b3[t] = h2u((h2_t){(_Float16)f0, (_Float16)f1});
          const h2_t z2 = u2h(cur.zv3[t]);
          float& za = zacc[1][kPairW ? t : 0];
          za = fmaf(p[2 * t], (float)z2.x, fmaf(p[2 * t + 1], (float)z2.y, za));
        }
      }
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        h8_t av;
        if constexpr (BV == 1) {
          av = unpack_bits(cur.vx[mb >> 2], mb & 3);
        } else if constexpr (BV == 2) {
          const uint32_t x = cur.vx[mb >> 1] >> (16 * (mb & 1));
          const uint2 t0 = *reinterpret_cast<const uint2*>(&vtab[(x & 0xFFu) * 2]);
          const uint2 t1 = *reinterpret_cast<const uint2*>(&vtab[((x >> 8) & 0xFFu) * 2]);
          av = __builtin_bit_cast(h8_t, (u4_t){t0.x, t0.y, t1.x, t1.y});
        } else {
          av = whole8<BV>(&cur.vx[(BV / 4) * mb]);
        }
        acc[0][mb] = mfma(av, __builtin_bit_cast(h8_t, mb >= 6 ? b3 : b1), acc[0][mb]);
      }
    }
#pragma unroll
    for (int q = 0; q < (kFive ? 0 : NQ); ++q) {
      // Five heads: the second quad carries head 4 alone (columns 0-3, the
      // rest zero).
      const bool solo = GQ == 5 && q == 1;
      const int Hp = solo ? 4 : 4 * q + hc;
      const f4_t pa = *reinterpret_cast<const f4_t*>(&pl[Hp * kPRow + 4 * row]);
      const f4_t pb = *reinterpret_cast<const f4_t*>(&pl[Hp * kPRow + 16 + 4 * row]);
      const float p[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};

      // P' = p * s_v rounded once to fp16 (the product is one mixed-precision
      // fma from the fp32 p and the fp16 scale, then a round to nearest)
      u4_t bhi;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const h2_t s2 = u2h(cur.sv[t]);
        float f0 = fmaf(p[2 * t], (float)s2.x, 0.f), f1 = fmaf(p[2 * t + 1], (float)s2.y, 0.f);
        keep_f32(f0, f1);
        const uint32_t hw = h2u((h2_t){(_Float16)f0, (_Float16)f1});
        bhi[t] = !kWide && solo && hc != 0 ? 0u : hw;
        const h2_t z2 = u2h(cur.zv[t]);
        float& za = zacc[q][kPairW ? t : 0];
        za = fmaf(p[2 * t], (float)z2.x, fmaf(p[2 * t + 1], (float)z2.y, za));
      }
      u4_t bm[4];
      if constexpr (!kWide) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int t = 0; t < 4; ++t) bm[j][t] = own[j] ? bhi[t] : 0u;
      }
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        h8_t av;
        if constexpr (BV == 1) {
          av = unpack_bits(cur.vx[mb >> 2], mb & 3);
        } else if constexpr (BV == 2) {
          const uint32_t x = cur.vx[mb >> 1] >> (16 * (mb & 1));
          const uint2 t0 = *reinterpret_cast<const uint2*>(&vtab[(x & 0xFFu) * 2]);
          const uint2 t1 = *reinterpret_cast<const uint2*>(&vtab[((x >> 8) & 0xFFu) * 2]);
          av = __builtin_bit_cast(h8_t, (u4_t){t0.x, t0.y, t1.x, t1.y});
        } else {
          av = whole8<BV>(&cur.vx[(BV / 4) * mb]);
        }
        if constexpr (kWide)
          acc[q][mb] = mfma(av, __builtin_bit_cast(h8_t, bhi), acc[q][mb]);
        else
          acc[q][mb & 1] = mfma(av, __builtin_bit_cast(h8_t, bm[mb >> 1]), acc[q][mb & 1]);
      }
    }
  };

  // Three buffers, loads two blocks ahead of the arithmetic (two buffers,
  // one block ahead, at four waves per SIMD).  The loads are
  // unconditional (past the end they re-read the last block) so every path
  // through the loop has the same loads in flight and the memory waits stay
  // exact; the main loop has no early exit, the last one or two blocks run
  // after it.
  // The zero-point table covers kChunk blocks; long splits refill it
  // between chunks.
  if (nblocks > 0) {
    int i = 0;
    for (int c0 = 0; c0 < nblocks; c0 += kChunk) {
      if (c0 > 0) {
        h8_t zn[4];
        load_z(c0 / BPG, zn);
        fill_table(c0 / BPG, zn);
      }
      const int cend = min(nblocks, c0 + kChunk);
      if constexpr (kStages == 3) {
        for (; i + 3 <= cend; i += 3) {
          load(min(i + 2, last), b2);
          process(b0, i);
          load(min(i + 3, last), b0);
          process(b1, i + 1);
          load(min(i + 4, last), b1);
          process(b2, i + 2);
        }
      } else {
        for (; i + 2 <= cend; i += 2) {
          load(min(i + 1, last), b1);
          process(b0, i);
          load(min(i + 2, last), b0);
          process(b1, i + 1);
        }
      }
    }
    if (i < nblocks) process(b0, i);
    if (kStages == 3 && i + 1 < nblocks) process(b1, i + 1);
  }

  // Lane coordinates again, from the lane id: recomputing them here keeps
  // the loop's register budget free of epilogue-only values.
  const int ln = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int ecol = ln & 15, erow = ln >> 4, ehc = ecol >> 2, exc = ecol & 3;
  // l: sum the 16 lanes of the head's row (1-bit values: the lane's weights
  // carry 2^-pw); zacc: sum over the lane rows (the tokens of a group column)
#pragma unroll
  for (int hh = 0; hh < HPL; ++hh) {
    if constexpr (kPairW) l[hh] *= (ecol & 2) ? 2.f : 1.f;
    l[hh] += dpp_mov<kQuadXor1>(0.f, l[hh]);
    l[hh] += dpp_mov<kQuadXor2>(0.f, l[hh]);
    l[hh] += dpp_mov<kHalfMirror>(0.f, l[hh]);
    l[hh] += dpp_mov<kMirror>(0.f, l[hh]);
  }
  // 1-bit, 4- and 8-bit value codes enter the products as code * 2^CodeUnit
  // (2-bit table halves are the codes themselves)
  const float kAccScale = BV == 2 ? 1.f : ldexpf(1.f, -CodeUnit<BV>::value);
  if constexpr (kFive) {
    // tile mb (value group g = (mb / 2) * ng / 4): the first operand's lanes
    // with column 5g .. 5g + 4 (g < min(ng, 3)), or the second's with column
    // 0 .. 4 (g = 3); head = column % 5
    float zs[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      zs[q] = zacc[q][0];
#pragma unroll
      for (int t = 1; t < NZ; ++t) zs[q] = fmaf(zacc[q][t], (float)(1 << t), zs[q]);
      zs[q] += __shfl_xor(zs[q], 16);
      zs[q] += __shfl_xor(zs[q], 32);
    }
    const int H = ecol % 5;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int g = (mb >> 1) * ng / 4;
      const bool second = ng == 4 && g == 3;
      const bool mine = second ? ecol < 5 : (ecol < 5 * min(ng, 3) && ecol / 5 == g);
      if (mine) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          red.acc[wv][H * kHeadDim + 16 * mb + 4 * erow + i] = acc[0][mb][i] * kAccScale + zs[second ? 1 : 0];
      }
    }
  }
#pragma unroll
  for (int q = 0; q < (kFive ? 0 : NQ); ++q) {
    float zs = zacc[q][0];
#pragma unroll
    for (int t = 1; t < NZ; ++t) zs = fmaf(zacc[q][t], (float)(1 << t), zs);
    zs += __shfl_xor(zs, 16);
    zs += __shfl_xor(zs, 32);
    const bool solo = GQ == 5 && q == 1;  // head 4 in columns 0-3
    const int H = solo ? 4 : 4 * q + ehc;
    // accumulator e of column group exc holds tile 2j + e, tile_col(j) = exc
    const int ej = ng == 2 ? 2 * (exc & 1) + (exc >> 1) : exc;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      f4_t v = acc[q][e];
      if constexpr (kWide) {  // the tile 2*ej + e (a select chain keeps acc in registers)
#pragma unroll
        for (int j = 1; j < 4; ++j) v = ej == j ? acc[q][2 * j + e] : v;
      }
      if (solo ? ehc == 0 : H < GQ) {
        const int mb = 2 * ej + e;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          red.acc[wv][H * kHeadDim + 16 * mb + 4 * erow + i] = v[i] * kAccScale + zs;
      }
    }
  }
  if (ecol == 0) {
#pragma unroll
    for (int hh = 0; hh < HPL; ++hh) {
      const int H = HPL * erow + hh;
      if (H < GQ) {
        red.m[wv][H] = m[hh];
        red.l[wv][H] = l[hh];
      }
    }
  }
  __syncthreads();
  write_record<GQ, CAUSAL>(a, S, wk.h, wk.rg, wk.sp, red);
}

template <int BK, int BV, int BPG, int GQ, bool CAUSAL, bool PAGED>
void launch_k(const DecodeArgs& a, void* stream) {
  hipLaunchKernelGGL((decode_mfma_kernel<BK, BV, BPG, GQ, CAUSAL, PAGED>), dim3(a.total_wg), dim3(64 * kWaves), 0,
                     (hipStream_t)stream, a);
}

template <int BK, int BV, int BPG, int GQ>
int launch_t(const DecodeArgs& a, void* stream) {
  const bool causal = a.nqry > 1, paged = a.pm.table != nullptr;
  if (causal && paged) launch_k<BK, BV, BPG, GQ, true, true>(a, stream);
  else if (causal) launch_k<BK, BV, BPG, GQ, true, false>(a, stream);
  else if (paged) launch_k<BK, BV, BPG, GQ, false, true>(a, stream);
  else launch_k<BK, BV, BPG, GQ, false, false>(a, stream);
  return (int)hipGetLastError();
}

template <int BK, int BV, int BPG>
int launch_gq(const DecodeArgs& a, int gq, void* stream) {
  switch (gq) {
    case 1:  // one or two query heads per kv head: the four-head layout with empty heads
      return launch_t<BK, BV, BPG, 1>(a, stream);
    case 2:
      return launch_t<BK, BV, BPG, 2>(a, stream);
    case 4: return launch_t<BK, BV, BPG, 4>(a, stream);
    case 5: return launch_t<BK, BV, BPG, 5>(a, stream);
    case 8: return launch_t<BK, BV, BPG, 8>(a, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

template <int BK, int BV>
int launch_bpg(const DecodeArgs& a, int gq, void* stream) {
  switch (a.gk / 32) {
    case 1: return launch_gq<BK, BV, 1>(a, gq, stream);
    case 2: return launch_gq<BK, BV, 2>(a, gq, stream);
    case 4: return launch_gq<BK, BV, 4>(a, gq, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

}  // namespace

// This source is compiled once per bit class (KVQ_BK key bits, KVQ_BV value
// bits, set by the build), so that the classes' kernels build in parallel;
// each object holds one class's launcher (launch_decode_matrix dispatches).
template <>
int launch_matrix_class<KVQ_BK, KVQ_BV>(const DecodeArgs& a, int gq, void* stream) {
  return launch_bpg<KVQ_BK, KVQ_BV>(a, gq, stream);
}

}  // namespace kvq
