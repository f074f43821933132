// Matrix-core chunk attention over 16 or 32 (query, head) rows of one kv head.
//
// Chunk queries (the last n_q cached tokens attend causally over the cache:
// the decoder's own attention, softmax(q K^T / sqrt(d)) V, applied to several
// positions at once; Introduction: scaled dot-product attention) give a kv
// head 4*n_q or 8*n_q query rows.  The decode kernel lays its 4-8 heads out
// as columns (head, value group), so a 16-column value product keeps a
// quarter of its output; here the rows are the M dimension of both products
// and no output is discarded:
//
//   scores:  S[row][t] = sum_c Q'[row][c] * code[t][c] + sum_c q~[row][c] * z[c]
//     A = Q' = q~ (.) s of 16 rows as two operands, the fp16 hi and lo parts
//         (each product exact), chained into one accumulator,
//     B = key codes as exact fp16 (the decode kernel's B operand),
//     D: lane (token n, row block rb) holds rows 4*rb .. 4*rb + 3.
//   values:  O[row][c] = sum_t P'_g[row][t] * code[t][c] + Z[row][g]
//     A = P'_g = p * s_v (value group g of the tile's channels), one fp16
//         rounding (fp16 fma of the hi part onto the product of the lo part),
//     B = value codes (the register layout the decode kernel's value operand
//         already has: 8 tokens of one channel per lane),
//     D: lane (channel n, row block rb) holds rows 4*rb .. 4*rb + 3 (the
//         same rows as the score lane: the rescale needs no shuffle).
//   zero points:  Z[row][g] = sum_t p[row][t] * z_v[t][g], two MFMAs (A = the
//     hi and lo parts of p, B = the staged value zeros, columns = groups).
//
// The value meta of a block (scales and zeros of every group) is staged in
// LDS, since each lane's rows need the scales of all groups.  Per 32-token
// block and wave: 16 score MFMAs, 2 zero-point MFMAs, 8 value MFMAs for 16
// rows, against 24 for 8 rows (with half of their value columns unused) in
// the decode kernel's eight-head layout.  A workgroup of 32 rows runs two
// row halves of 16 over the same blocks: every unpacked key and value
// operand then feeds both halves' MFMAs, so the unpacking (one vector
// instruction per operand dword) is paid once per 32 rows.
#include <hip/hip_runtime.h>

#include "decode_common.h"
#include "kvq_internal.h"
#include "kvq_layout.h"
#include "mfma_common.h"

namespace kvq {
namespace {

using namespace dec;
using namespace mfma_ops;

constexpr int kRows = 16;           // rows of one row half (the M dimension of an MFMA)
constexpr float kMargin = 6.f;      // lazy softmax reference headroom (log2 units)
constexpr int kQR = 68;             // dwords per Q' row (64 + 4: rows start in distinct bank quads)
constexpr int kPR = 36;             // floats per weight row (32 + 4)
constexpr int kZG = 16;             // key groups per zero-point table

// LDS areas (bytes) of a workgroup of NU row halves (16 * NU rows).  The
// first holds the cross-wave reduction after the loop, or the staged query
// rows of the fp16-tail splits (per wave).
constexpr int kTailQ = kHeadDim * 8;  // floats of one wave's staged query rows (8 rows)
template <int NU>
struct ChunkSmem {
  static constexpr int R = kRows * NU;
  static constexpr int kOffQA = 0;
  static constexpr int kBytesQA = (int)sizeof(Reduce<8>);  // the reduction takes 8 rows at a time
  static constexpr int kOffPL = (kOffQA + kBytesQA + 15) / 16 * 16;
  static constexpr int kOffVM = kOffPL + kWaves * R * kPR * 4;
  static constexpr int kOffKS = kOffVM + kWaves * 128 * 4;
  static constexpr int kOffDZ = kOffKS + kWaves * 64 * 4;
  static constexpr int kOffQQ = kOffDZ + kWaves * kZG * R * 4;
  static constexpr int kOffCS = kOffQQ + R * kQR * 4;
  static constexpr int kOffLM = kOffCS + R * 4;
  static constexpr int kOffVT = kOffLM + R * 4;
  static constexpr int kBytes = kOffVT + ValueTable2::kWords * 4;
  static_assert(kWaves * kTailQ * 4 <= kBytesQA, "the tail splits' query rows fit the first area");
  static_assert(32 * 8 <= R * kPR, "a tail half's weights fit its wave's weight area");
};

// Everything one 32-token block reads from memory.
template <int BK, int BV>
struct ChunkBlock {
  uint32_t s;          // key scales of channels 2*lane, 2*lane+1
  uint32_t kx[2][BK];  // key codes of tokens 16*mb + (lane & 15)
  uint32_t vx[2 * BV]; // value codes of this lane (channel lane & 15, tokens of K-group lane >> 4)
  uint2 vm;            // bytes 8*lane .. 8*lane + 7 of the block's value meta (staged in LDS)
};

template <int BK, int BV, int NU>
struct ChunkOcc {  // waves per SIMD (registers), shared with the host's split plan
  static constexpr int value = chunk_waves(BK, BV, kRows * NU);
};

// NU row halves of 16 rows share every unpacked code operand: each key and
// value operand feeds NU products (two row halves halve the unpacking per
// row), the Q' and weight work stays per row.
template <int BK, int BV, int BPG, bool PAGED, int NU>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(ChunkOcc<BK, BV, NU>::value))) void
chunk_mfma_kernel(DecodeArgs a) {
  using SM = ChunkSmem<NU>;
  constexpr int R = SM::R;
  constexpr bool kPairW = BV == 1;  // 1-bit value operands carry pair weights 2^t
  __shared__ __attribute__((aligned(16))) uint8_t smem[SM::kBytes];
  uint32_t* const qa_all = reinterpret_cast<uint32_t*>(smem + SM::kOffQA);
  float* const pl_all = reinterpret_cast<float*>(smem + SM::kOffPL);
  uint32_t* const vm_all = reinterpret_cast<uint32_t*>(smem + SM::kOffVM);
  float* const dz_all = reinterpret_cast<float*>(smem + SM::kOffDZ);
  uint32_t* const qq_s = reinterpret_cast<uint32_t*>(smem + SM::kOffQQ);
  float* const cs_s = reinterpret_cast<float*>(smem + SM::kOffCS);
  uint32_t* const vtab = reinterpret_cast<uint32_t*>(smem + SM::kOffVT);
  uint32_t* const ks_all = reinterpret_cast<uint32_t*>(smem + SM::kOffKS);
  int* const lim_s = reinterpret_cast<int*>(smem + SM::kOffLM);
  Reduce<8>& red = *reinterpret_cast<Reduce<8>*>(smem + SM::kOffQA);

  const Work wk = find_work<true>(a);
  const DecodeSeq& S = a.seq[wk.si];
  const uint8_t* blk = a.arena + S.head0 + (uint64_t)wk.h * a.head_stride;
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint32_t vbound = __builtin_amdgcn_raw_buffer_load_b32(head_rsrc(blk + a.vb, 4), 0, 0, 0);
  asm volatile("" ::: "memory");

  if (wk.sp >= S.nq) {  // fp16 tail tokens: the vector path, in parts of 8 rows
    uint32_t* qa = qa_all + wv * kTailQ;
    for (int half = 0; half < 2 * NU; ++half) {
      float qs0[8], qs1[8];
      load_q_scaled<8, true>(a, S, wk.h, wk.rg, lane, qs0, qs1, 8 * half);
      State<8> st;
      init_state<8>(st);
      tail_split<8, true>(a, S, wk.h, wk.rg, blk, qs0, qs1, reinterpret_cast<float*>(qa), pl_all + wv * R * kPR, st,
                          lane, wv, 8 * half);
      __syncthreads();  // every wave is done with its area before the reduction overlays it
      stage_state<8>(st, red, lane, wv);
      __syncthreads();
      write_record<8, true>(a, S, wk.h, wk.rg, wk.sp, red, 8 * half);
      __syncthreads();  // the reduction is read before the next part's query overlays it
    }
    return;
  }

  const int col = lane & 15, row = lane >> 4;
  constexpr int ng = kHeadDim / 32;  // value groups of 32 channels (the host sends no other size here)
  const uint16_t* qbase = a.q + q_index<R, true>(a, S, wk.h, wk.rg, 0) * kHeadDim;
  // packed data: the (sequence, head) region, or the kv head's region of the
  // page that holds a block (as in the decode kernel)
  const __amdgpu_buffer_rsrc_t rs = head_rsrc(blk, PAGED ? 0 : a.head_stride);
  const int32_t* ptab = PAGED ? a.pm.table + (size_t)S.seq * a.pm.max_pages : nullptr;
  const uint8_t* pool_h = PAGED ? a.arena + a.pm.pool0 + (uint64_t)wk.h * a.pm.page_head_bytes : nullptr;
  const int pg0 = PAGED ? (wk.sp * a.split_tokens) >> a.pm.page_shift : 0;
  int lane_pg = 0;
  if constexpr (PAGED) {
    if (pg0 + lane < a.pm.max_pages) lane_pg = ptab[pg0 + lane];
  }
  auto seg_of = [&](int tok, int& tin) -> __amdgpu_buffer_rsrc_t {
    if constexpr (!PAGED) {
      tin = tok;
      return rs;
    } else {
      const int pg = tok >> a.pm.page_shift;
      tin = tok & (a.pm.page_tokens - 1);
      const int k = pg - pg0;
      const int pool_pg = k < 64 ? __builtin_amdgcn_readlane(lane_pg, k) : ptab[pg];
      return head_rsrc(pool_h + (uint64_t)pool_pg * a.pm.page_bytes, a.pm.page_head_bytes);
    }
  };
  const uint32_t lo_kc = col * 16 * BK + row * 4 * BK, lo_vc = lane * 8 * BV, lo_km = 4 * lane, lo_vm = 8 * lane;
  const int vstride = 128 * ng;  // value meta bytes per 32-token block (8 per lane)

  // This wave's 32-token blocks (as in the decode kernel): key groups
  // j0 + ws + kWaves*n of the split, BPG blocks each.
  const int t0 = wk.sp * a.split_tokens;
  const int t1 = min(S.Lq, t0 + a.split_tokens);
  const int wslot = (wv + 2 * ((int)blockIdx.x >> 8)) & (kWaves - 1);
  const int j0 = t0 / a.gk + wslot, jend = t1 / a.gk;
  const int ngroups = j0 < jend ? (jend - j0 + kWaves - 1) / kWaves : 0;
  const int nblocks = ngroups * BPG;
  const int last = nblocks - 1;
  auto load = [&](int i, ChunkBlock<BK, BV>& o) {
    const int j = j0 + kWaves * (i / BPG);
    int tok;
    const __amdgpu_buffer_rsrc_t r = seg_of(j * a.gk + (i % BPG) * 32, tok);
    const int jg = PAGED ? tok >> a.pm.gk_shift : j;
    const uint32_t km = a.km + (uint32_t)jg * (2 * kHeadDim * 2), kc = a.kc + (uint32_t)tok * 16 * BK;
    const uint32_t vc = a.vc + (uint32_t)(tok / 32) * 512 * BV, vm = a.vm + (uint32_t)(tok / 32) * vstride;
    o.s = ld32(r, lo_km, km);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      if constexpr (BK == 1) {
        o.kx[mb][0] = ld32(r, lo_kc + mb * 16 * 16 * BK, kc);
      } else if constexpr (BK == 2) {
        const uint2 v = ld64(r, lo_kc + mb * 16 * 16 * BK, kc);
        o.kx[mb][0] = v.x;
        o.kx[mb][1] = v.y;
      } else {
#pragma unroll
        for (int w = 0; w < BK / 4; ++w) {
          const u4_t v = ld128(r, lo_kc + mb * 16 * 16 * BK + 16 * w, kc);
          o.kx[mb][4 * w] = v[0]; o.kx[mb][4 * w + 1] = v[1]; o.kx[mb][4 * w + 2] = v[2]; o.kx[mb][4 * w + 3] = v[3];
        }
      }
    }
    if constexpr (BV == 1) {
      const uint2 v = ld64(r, lo_vc, vc);
      o.vx[0] = v.x;
      o.vx[1] = v.y;
    } else {
#pragma unroll
      for (int w = 0; w < BV / 2; ++w) {
        const u4_t v = ld128(r, lo_vc + 16 * w, vc);
        o.vx[4 * w] = v[0]; o.vx[4 * w + 1] = v[1]; o.vx[4 * w + 2] = v[2]; o.vx[4 * w + 3] = v[3];
      }
    }
    o.vm = ld64(r, lo_vm, vm);
  };
  // key zero-points of the wave's key groups k0 .. k0 + 15 (A operand of the
  // zero-point terms, row = group; past the last group: the last)
  auto load_z = [&](int k0, h8_t (&zq)[4]) {
    const int j = j0 + kWaves * min(k0 + col, max(ngroups - 1, 0));
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

  // query words of the rows this wave prepares (rows wv, wv + 4, ...) and the
  // 2-bit value table: loaded before the first blocks
  uint32_t qw[R / kWaves];
#pragma unroll
  for (int i = 0; i < R / kWaves; ++i)
    qw[i] = reinterpret_cast<const uint32_t*>(qbase + (size_t)row_q_offset(a, wk.rg, wv + kWaves * i) * kHeadDim)[lane];
  constexpr int kTabLoads = BV == 2 ? ValueTable2::kWords / 4 : 0;
  u4_t tabw = {0u, 0u, 0u, 0u};
  if constexpr (kTabLoads > 0) {
    if ((int)threadIdx.x < kTabLoads) tabw = reinterpret_cast<const u4_t*>(kValueTable2.w)[threadIdx.x];
  }
  asm volatile("" ::: "memory");

  ChunkBlock<BK, BV> b0, b1;
  h8_t zq[4];
  if (nblocks > 0) {
    load(0, b0);
    load_z(0, zq);
  }

  // q~ = q * 2^-e per row with max |q~| < 1
#pragma unroll
  for (int i = 0; i < R / kWaves; ++i) {
    const int g = wv + kWaves * i;
    const float q0 = h2f(qw[i] & 0xFFFF), q1 = h2f(qw[i] >> 16);
    const float mx = wave_max(fmaxf(fabsf(q0), fabsf(q1)));
    int e = 0;
    frexpf(mx, &e);
    const float inv = ldexpf(1.f, -e);
    qq_s[g * kQR + lane] = h2u((h2_t){(_Float16)(q0 * inv), (_Float16)(q1 * inv)});
    if (lane == 0) {
      cs_s[g] = ldexpf(a.qscale, e - CodeUnit<BK>::value);
      lim_s[g] = row_limit(a, S, wk.rg, g);
    }
  }
  if constexpr (kTabLoads > 0) {
    if ((int)threadIdx.x < kTabLoads) reinterpret_cast<u4_t*>(vtab)[threadIdx.x] = tabw;
  }
  __syncthreads();
  // q~ of row 16u + col in the A layout of the score product (channels 32*kb
  // + 8*row + e), with the key operand's pair weights: element pair t of a
  // 1-bit operand carries 2^t, odd pairs of a 2-bit operand 4
  h8_t qa[NU][4];
#pragma unroll
  for (int u = 0; u < NU; ++u)
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const u4_t v = *reinterpret_cast<const u4_t*>(&qq_s[(kRows * u + col) * kQR + 16 * kb + 4 * row]);
      u4_t w;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const _Float16 f = (_Float16)(BK == 1 ? ldexpf(1.f, -t) : (BK == 2 && (t & 1)) ? 0.25f : 1.f);
        w[t] = h2u(u2h(v[t]) * (h2_t){f, f});
      }
      qa[u][kb] = __builtin_bit_cast(h8_t, w);
    }
  // the score scale and the token limit of rows 16u + 4*row + r stay in LDS
  // (cs_s, lim_s) and are read per block: registers are scarce at 32 rows
  const int glim = group_limit(a, S, wk.rg);

  uint32_t* const ks = ks_all + wv * 64;
  float* const pl = pl_all + wv * R * kPR;
  uint32_t* const vml = vm_all + wv * 128;
  float* const dzt = dz_all + wv * kZG * R;

  // zero-point terms sum_c z[c] q~[row][c] of 16 key groups: D[group][row]
  // (A = z of group col, B = q~ of row 16u + col), scaled like the code
  // products
  auto fill_dz = [&](const h8_t (&z)[4]) {
    f4_t t[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      t[u] = (f4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        t[u] = mfma(z[kb], *reinterpret_cast<const h8_t*>(&qq_s[(kRows * u + col) * kQR + 16 * kb + 4 * row]), t[u]);
    }
    wave_lds_sync();  // earlier reads of the table are done
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) dzt[(4 * row + r) * R + kRows * u + col] = t[u][r] * ldexpf(1.f, CodeUnit<BK>::value);
  };
  if (nblocks > 0) {
    fill_dz(zq);
    if (ngroups > kZG) load_z(kZG, zq);  // the next table's zero-points
  }

  // The weight shift S of this (sequence, kv head), as in the decode kernel
  // (2^S * bound < 2^15).  Here p itself becomes an fp16 operand, so it is
  // shifted by Sp = min(S, 14) (15 at S = 30) only, and the rest,
  // X = S - Sp <= 15, goes onto the staged value scales: s_v * 2^X < 2, so
  // P' = p * s_v * 2^X is the decode kernel's P' again.  The value
  // accumulators carry 2^X, undone after the loop.
  int shift = kMaxPShift;
  {
    asm volatile("" : "+v"(vbound));
    const uint32_t vbits = vbound & 0xFFFFu;
    if (vbits >= 0x7C00u) {
      shift = 0;
    } else if (vbits != 0u) {
      int ex = 0;
      frexpf(h2f(vbits), &ex);
      shift = min(kMaxPShift, max(0, 15 - ex));
    }
  }
  const int pshift_p = max(min(shift, 14), shift - 15), xshift = shift - pshift_p;
  const float pshift = (float)pshift_p;
  // Factors of the two meta dwords a lane stages: the scales (lanes < 32)
  // carry 2^X, and at one bit also 2^-t for element pair t of the value
  // operand, whose unpacked codes carry 2^t (lane k holds the scales of
  // positions 4k .. 4k + 3 of its group row: pairs 2(k & 1), 2(k & 1) + 1).
  // The zeros (lanes >= 32) stay as they are.  A scale far below the head's
  // bound may turn subnormal here; its products are below 2^-25 absolute.
  h2_t vmf[2];
  {
    const int t0 = kPairW ? 2 * (lane & 1) : 0, t1 = kPairW ? t0 + 1 : 0;
    const _Float16 f0 = (_Float16)ldexpf(1.f, xshift - t0), f1 = (_Float16)ldexpf(1.f, xshift - t1);
    vmf[0] = lane < 32 ? (h2_t){f0, f0} : (h2_t){(_Float16)1.f, (_Float16)1.f};
    vmf[1] = lane < 32 ? (h2_t){f1, f1} : (h2_t){(_Float16)1.f, (_Float16)1.f};
  }

  // Lane state, rows 16u + 4*row + r: the reference m (uniform over the 16
  // lanes of the row block) and the lane's share of l.
  float m[NU][4], l[NU][4];
  f4_t acc[NU][8], zac[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      m[u][r] = -__builtin_inff();
      l[u][r] = 0.f;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[u][t] = (f4_t){0.f, 0.f, 0.f, 0.f};
    zac[u] = (f4_t){0.f, 0.f, 0.f, 0.f};
  }

  f4_t dz[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) dz[u] = (f4_t){0.f, 0.f, 0.f, 0.f};
  auto process = [&](const ChunkBlock<BK, BV>& cur, int i) {
    if (BPG == 1 || i % BPG == 0) {
      const int k = i / BPG;
      if (k > 0 && k % kZG == 0) {  // the next zero-point table
        fill_dz(zq);
        if (k + kZG < ngroups) load_z(k + kZG, zq);
      }
      // the key scales of the block's key group go through LDS (lane L
      // holds channels 2L, 2L+1)
      wave_lds_sync();
      ks[lane] = cur.s;
      wave_lds_sync();
#pragma unroll
      for (int u = 0; u < NU; ++u) dz[u] = *reinterpret_cast<const f4_t*>(&dzt[(k % kZG) * R + kRows * u + 4 * row]);
    }

    // scores of token 16*mb + col, rows 16u + 4*row + r; Q' = q~ (.) s of
    // each 32-channel block kb in the A layout, hi and lo parts; each
    // unpacked key operand serves every row half
    f4_t d[NU][2];
#pragma unroll
    for (int u = 0; u < NU; ++u) d[u][0] = d[u][1] = dz[u];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const u4_t sv = *reinterpret_cast<const u4_t*>(&ks[16 * kb + 4 * row]);
      h8_t ahi[NU], alo[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const u4_t qv = __builtin_bit_cast(u4_t, qa[u][kb]);
        u4_t h, o;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const h2_t hi = u2h(qv[t]) * u2h(sv[t]);
          h[t] = h2u(hi);
          o[t] = h2u(__builtin_elementwise_fma(u2h(qv[t]), u2h(sv[t]), -hi));
        }
        ahi[u] = __builtin_bit_cast(h8_t, h);
        alo[u] = __builtin_bit_cast(h8_t, o);
      }
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        h8_t b;
        if constexpr (BK == 1) b = unpack_bits(cur.kx[mb][0], kb);
        else if constexpr (BK == 2) b = unpack_pairs2(cur.kx[mb][kb >> 1], kb & 1);
        else b = whole8<BK>(&cur.kx[mb][(BK / 4) * kb]);
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          d[u][mb] = mfma(ahi[u], b, d[u][mb]);
          d[u][mb] = mfma(alo[u], b, d[u][mb]);
        }
      }
    }
    const int tok = (j0 + kWaves * (i / BPG)) * a.gk + (i % BPG) * 32;
    const bool masked = tok + 32 > glim;
    float raw[NU][4][2];
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) raw[u][r][mb] = d[u][mb][r];
    if (masked) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const int4 lim = *reinterpret_cast<const int4*>(&lim_s[kRows * u + 4 * row]);
        const int lr[4] = {lim.x, lim.y, lim.z, lim.w};
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
            if (tok + 16 * mb + col >= lr[r]) raw[u][r][mb] = -__builtin_inff();
      }
    }
    float cs[NU][4];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const f4_t c4 = *reinterpret_cast<const f4_t*>(&cs_s[kRows * u + 4 * row]);
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[u][r] = c4[r];
    }

    // online softmax (base 2) per row, lazy reference as in the decode
    // kernel; lane row r of the 4 row blocks rescales only when one of
    // those rows moves its reference
    const float ninf = -__builtin_inff();
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float bmr = fmaf(fmaxf(raw[u][r][0], raw[u][r][1]), cs[u][r], -pshift);
        if (__builtin_amdgcn_ballot_w64(bmr > m[u][r])) {
          float b = bmr;
          b = fmaxf(b, dpp_mov<kQuadXor1>(ninf, b));
          b = fmaxf(b, dpp_mov<kQuadXor2>(ninf, b));
          b = fmaxf(b, dpp_mov<kHalfMirror>(ninf, b));
          b = fmaxf(b, dpp_mov<kMirror>(ninf, b));
          const float mnew = b > m[u][r] ? b + kMargin : m[u][r];
          // a row with no visible token yet keeps m = -inf and factor 1
          const float alpha = mnew == m[u][r] ? 1.f : __builtin_amdgcn_exp2f(m[u][r] - mnew);
          l[u][r] *= alpha;
          m[u][r] = mnew;
#pragma unroll
          for (int t = 0; t < 8; ++t) acc[u][t][r] *= alpha;
          zac[u][r] *= alpha;
        }
      }
    float e[NU][4][2];
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
          e[u][r][mb] = __builtin_amdgcn_exp2f(fmaf(raw[u][r][mb], cs[u][r], -m[u][r]));
    if (masked) {  // masked tokens weigh 0, also while m is still -inf
#pragma unroll
      for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) e[u][r][mb] = raw[u][r][mb] == -__builtin_inff() ? 0.f : e[u][r][mb];
    }
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) l[u][r] += e[u][r][0] + e[u][r][1];

    // weights to the A layout (lane: row 16u + col, tokens of K-group row),
    // and the block's value meta to LDS
    wave_lds_sync();
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pl[(kRows * u + 4 * row + r) * kPR + col] = e[u][r][0];
        pl[(kRows * u + 4 * row + r) * kPR + 16 + col] = e[u][r][1];
      }
    *reinterpret_cast<uint2*>(&vml[2 * lane]) = make_uint2(h2u(u2h(cur.vm.x) * vmf[0]), h2u(u2h(cur.vm.y) * vmf[1]));
    wave_lds_sync();
    // p in fp16 hi + lo parts
    u4_t phi[NU], plo[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const f4_t pa = *reinterpret_cast<const f4_t*>(&pl[(kRows * u + col) * kPR + 4 * row]);
      const f4_t pb = *reinterpret_cast<const f4_t*>(&pl[(kRows * u + col) * kPR + 16 + 4 * row]);
      const float p[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float f0 = p[2 * t], f1 = p[2 * t + 1];
        keep_f32(f0, f1);
        uint32_t hw = h2u((h2_t){(_Float16)f0, (_Float16)f1});
        asm("" : "+v"(hw));
        const h2_t hi = u2h(hw);
        float g0 = fmaf(p[2 * t], 1.f, -(float)hi.x), g1 = fmaf(p[2 * t + 1], 1.f, -(float)hi.y);
        keep_f32(g0, g1);
        phi[u][t] = hw;
        plo[u][t] = h2u((h2_t){(_Float16)g0, (_Float16)g1});
      }
    }
    // zero-point terms: B = the staged zeros of group col (columns past the
    // groups: zero)
    {
      u4_t zb = {0u, 0u, 0u, 0u};
      if (col < ng) zb = *reinterpret_cast<const u4_t*>(&vml[16 * ng + 16 * col + 4 * row]);
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        zac[u] = mfma(__builtin_bit_cast(h8_t, phi[u]), __builtin_bit_cast(h8_t, zb), zac[u]);
        zac[u] = mfma(__builtin_bit_cast(h8_t, plo[u]), __builtin_bit_cast(h8_t, zb), zac[u]);
      }
    }
    // P'_g = p * s_v of each value group (32 channels: tiles 2g, 2g + 1), and
    // the products of its tiles; each unpacked value operand serves every
    // row half
    h8_t pg[NU];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      if (mb % 2 == 0) {
        const u4_t sg = *reinterpret_cast<const u4_t*>(&vml[16 * (mb / 2) + 4 * row]);
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          u4_t w;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const h2_t s2 = u2h(sg[t]);
            w[t] = h2u(__builtin_elementwise_fma(u2h(phi[u][t]), s2, u2h(plo[u][t]) * s2));
          }
          pg[u] = __builtin_bit_cast(h8_t, w);
        }
      }
      h8_t bv;
      if constexpr (BV == 1) {
        bv = unpack_bits(cur.vx[mb >> 2], mb & 3);
      } else if constexpr (BV == 2) {
        const uint32_t x = cur.vx[mb >> 1] >> (16 * (mb & 1));
        const uint2 t0 = *reinterpret_cast<const uint2*>(&vtab[(x & 0xFFu) * 2]);
        const uint2 t1 = *reinterpret_cast<const uint2*>(&vtab[((x >> 8) & 0xFFu) * 2]);
        bv = __builtin_bit_cast(h8_t, (u4_t){t0.x, t0.y, t1.x, t1.y});
      } else {
        bv = whole8<BV>(&cur.vx[(BV / 4) * mb]);
      }
#pragma unroll
      for (int u = 0; u < NU; ++u) acc[u][mb] = mfma(pg[u], bv, acc[u][mb]);
    }
  };

  if (nblocks > 0) {
    int i = 0;
    for (; i + 2 <= nblocks; i += 2) {
      load(min(i + 1, last), b1);
      process(b0, i);
      load(min(i + 2, last), b0);
      process(b1, i + 1);
    }
    if (i < nblocks) process(b0, i);
  }

  // l over the 16 lanes of the row block; the zero-point term of (row,
  // group g) sits in lane (g, row block)
  const int ln = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int ecol = ln & 15, erow = ln >> 4;
#pragma unroll
  for (int u = 0; u < NU; ++u)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      l[u][r] += dpp_mov<kQuadXor1>(0.f, l[u][r]);
      l[u][r] += dpp_mov<kQuadXor2>(0.f, l[u][r]);
      l[u][r] += dpp_mov<kHalfMirror>(0.f, l[u][r]);
      l[u][r] += dpp_mov<kMirror>(0.f, l[u][r]);
    }
  const float kAccScale = ldexpf(1.f, (BV == 2 ? 0 : -CodeUnit<BV>::value) - xshift);
  // rows 8*part .. 8*part + 7 (row half part / 2, lane row blocks 2*(part %
  // 2), 2*(part % 2) + 1) pass through the reduction area one part after
  // the other
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    float zg[4][4];  // zero-point terms of rows 16u + 4*erow + r, group g, in this lane
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int r = 0; r < 4; ++r) zg[g][r] = __shfl(zac[u][r], 16 * erow + g);
    for (int half = 0; half < 2; ++half) {
      __syncthreads();  // the area is free
      if ((erow >> 1) == half) {
        const int rb = erow & 1;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            red.acc[wv][(4 * rb + r) * kHeadDim + 16 * mb + ecol] = acc[u][mb][r] * kAccScale + zg[mb / 2][r];
        if (ecol == 0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            red.m[wv][4 * rb + r] = m[u][r];
            red.l[wv][4 * rb + r] = l[u][r];
          }
        }
      }
      __syncthreads();
      write_record<8, true>(a, S, wk.h, wk.rg, wk.sp, red, kRows * u + 8 * half);
    }
  }
}

template <int BK, int BV, int BPG, int NU>
int launch_p(const DecodeArgs& a, void* stream) {
  if (a.pm.table != nullptr)
    hipLaunchKernelGGL((chunk_mfma_kernel<BK, BV, BPG, true, NU>), dim3(a.total_wg), dim3(64 * kWaves), 0,
                       (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL((chunk_mfma_kernel<BK, BV, BPG, false, NU>), dim3(a.total_wg), dim3(64 * kWaves), 0,
                       (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

template <int BK, int BV, int NU>
int launch_g(const DecodeArgs& a, void* stream) {
  switch (a.gk / 32) {
    case 1: return launch_p<BK, BV, 1, NU>(a, stream);
    case 2: return launch_p<BK, BV, 2, NU>(a, stream);
    case 4: return launch_p<BK, BV, 4, NU>(a, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

// 32 rows for 1- and 2-bit classes (the 4-bit blocks leave too few
// registers for two row halves), 16 rows for all.
template <int BK, int BV>
int launch_r(const DecodeArgs& a, int rows, void* stream) {
  if constexpr (chunk_rows32(BK, BV)) {
    if (rows == 32) return launch_g<BK, BV, 2>(a, stream);
  }
  if (rows == 16) return launch_g<BK, BV, 1>(a, stream);
  return (int)hipErrorInvalidValue;
}

}  // namespace

int launch_chunk_matrix(const DecodeArgs& a, int bk, int bv, int rows, void* stream) {
  if (a.total_wg <= 0) return 0;
  if (bk == 1 && bv == 1) return launch_r<1, 1>(a, rows, stream);
  if (bk == 1 && bv == 2) return launch_r<1, 2>(a, rows, stream);
  if (bk == 2 && bv == 1) return launch_r<2, 1>(a, rows, stream);
  if (bk == 2 && bv == 2) return launch_r<2, 2>(a, rows, stream);
  if (bk == 4 && bv == 4) return launch_r<4, 4>(a, rows, stream);
  return (int)hipErrorInvalidValue;  // 8-bit classes take the decode kernel's row groups
}

}  // namespace kvq
