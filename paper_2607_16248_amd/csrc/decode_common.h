// Pieces shared by the decode kernels: wave reductions over DPP, the
// online-softmax state of the vector path, the fp16-tail pass, and the
// combination of per-wave partial results into one split record.
#pragma once

#include <hip/hip_runtime.h>

#include "kvq_internal.h"

namespace kvq {
namespace dec {

constexpr int kWaves = 4;

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_mov(float old, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                               __builtin_bit_cast(int, v), CTRL,
                                                               ROW_MASK, 0xF, false));
}

// DPP controls: quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror,
// row_mirror, row_bcast:15, row_bcast:31.
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140,
              kBcast15 = 0x142, kBcast31 = 0x143;

__device__ __forceinline__ float readlane63(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<kQuadXor1>(0.f, v);
  v += dpp_mov<kQuadXor2>(0.f, v);
  v += dpp_mov<kHalfMirror>(0.f, v);
  v += dpp_mov<kMirror>(0.f, v);
  v += dpp_mov<kBcast15, 0xA>(0.f, v);
  v += dpp_mov<kBcast31, 0xC>(0.f, v);
  return readlane63(v);
}

__device__ __forceinline__ float wave_max(float v) {
  const float ninf = -__builtin_inff();
  v = fmaxf(v, dpp_mov<kQuadXor1>(ninf, v));
  v = fmaxf(v, dpp_mov<kQuadXor2>(ninf, v));
  v = fmaxf(v, dpp_mov<kHalfMirror>(ninf, v));
  v = fmaxf(v, dpp_mov<kMirror>(ninf, v));
  v = fmaxf(v, dpp_mov<kBcast15, 0xA>(ninf, v));
  v = fmaxf(v, dpp_mov<kBcast31, 0xC>(ninf, v));
  return readlane63(v);
}

// LDS written and read back by the same wave: order the accesses.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// floats per channel of the query rows staged for the vector passes
template <int GQ>
struct QStride {
  static constexpr int value = GQ <= 4 ? GQ : GQ <= 8 ? 8 : 16;
};

template <int GQ>
struct State {
  float m[GQ];
  float l[GQ];
  float acc[GQ][8];
};

// Online-softmax update for one pass of 32 tokens held as sig (QK layout:
// lanes 2t, 2t+1 hold token t).  Writes p to LDS, rescales the state.
template <int GQ, bool CHUNK>
__device__ __forceinline__ void softmax_pass(State<GQ>& st, float (&sig)[GQ], int half, int tl,
                                             float* p_lds) {
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    const float mx = wave_max(sig[g]);
    const float mnew = fmaxf(st.m[g], mx);
    // a chunk row with no visible token yet keeps m = -inf: factor 1,
    // weights 0 (single-token decode sees a token in every pass)
    const bool none = CHUNK && mnew == -__builtin_inff();
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(st.m[g] - mnew);
    const float p = none ? 0.f : __builtin_amdgcn_exp2f(sig[g] - mnew);
    st.l[g] = st.l[g] * alpha + (half ? 0.f : p);
#pragma unroll
    for (int k = 0; k < 8; ++k) st.acc[g][k] *= alpha;
    st.m[g] = mnew;
    if (!half) p_lds[tl * GQ + g] = p;
  }
}

// fp16 tail tokens [Lq, L), read from the ring; pass `pass` covers 32 tokens.
template <int GQ, bool CHUNK>
__device__ __forceinline__ void tail_pass(const DecodeArgs& a, const DecodeSeq& S, const uint8_t* blk,
                                          int pass, const float* qp, float* p_lds, State<GQ>& st,
                                          const int (&lim)[GQ], int lane) {
  constexpr int QS = QStride<GQ>::value;
  const int ntail = S.L - S.Lq;
  const int tl = lane >> 1, half = lane & 1;
  const int idx = pass * 32 + tl;
  float sig[GQ];
#pragma unroll
  for (int g = 0; g < GQ; ++g) sig[g] = 0.f;
  if (idx < ntail) {
    const int slot = (S.Lq + idx) % a.W;
    const uint4* kr = reinterpret_cast<const uint4*>(blk + a.tk + ((size_t)slot * kHeadDim + half * 64) * 2);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint4 v = kr[i];
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = h2f((w4[e >> 1] >> ((e & 1) * 16)) & 0xFFFF);
        const float* qv = qp + (half * 64 + i * 8 + e) * QS;
#pragma unroll
        for (int g = 0; g < GQ; ++g) sig[g] = fmaf(qv[g], x, sig[g]);
      }
    }
  }
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    sig[g] += dpp_mov<kQuadXor1>(0.f, sig[g]);
    if (idx >= ntail || (CHUNK && S.Lq + idx >= lim[g])) sig[g] = -__builtin_inff();
  }
  softmax_pass<GQ, CHUNK>(st, sig, half, tl, p_lds);
  wave_lds_sync();
  const int tq = lane >> 4, cc = lane & 15;
  for (int tt = tq; tt < 32; tt += 4) {
    const int i2 = pass * 32 + tt;
    if (i2 >= ntail) break;
    const int slot = (S.Lq + i2) % a.W;
    const uint4 v = *reinterpret_cast<const uint4*>(blk + a.tv + ((size_t)slot * kHeadDim + cc * 8) * 2);
    const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
    const float* pp = p_lds + tt * GQ;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float x = h2f((w4[k >> 1] >> ((k & 1) * 16)) & 0xFFFF);
#pragma unroll
      for (int g = 0; g < GQ; ++g) st.acc[g][k] = fmaf(pp[g], x, st.acc[g][k]);
    }
  }
  wave_lds_sync();
}

// Locate this workgroup's (sequence, kv head, row group, split).
struct Work {
  int si, h, rg, sp;
};

// CHUNK = false: single-token decode (one query, one row group of the kv
// head's GQ query heads), where the row arithmetic reduces to h * GQ + g.
template <bool CHUNK>
__device__ __forceinline__ Work find_work(const DecodeArgs& a) {
  const int wg = blockIdx.x;
  int si = 0;
  for (int i = 1; i < a.nseq; ++i) si = (a.seq[i].wg_begin <= wg) ? i : si;
  const int local = wg - a.seq[si].wg_begin;
  const int ns = a.seq[si].nsplit;
  const int hv = local / ns;
  Work w{si, hv, 0, local % ns};
  if (a.nqry == 1) {
    // single-token decode: the packed splits of every kv head first, the
    // fp16-tail workgroups (split nq, a few tokens each) after them
    const int nq = a.seq[si].nq, packed = a.hkv * nq;
    if (local < packed) {
      w.h = local / nq;
      w.sp = local - w.h * nq;
    } else {
      w.h = local - packed;
      w.sp = nq;
    }
  }
  if (CHUNK && a.nrg > 1) {  // chunk queries: kv head and row group
    const int units = a.hkv * ns;  // (kv head, split) pairs
    if (units % 8 == 0) {
      // Row groups of one (kv head, split) unit read the same tokens: give
      // them workgroup ids 8 apart, so that they land on one XCD (ids go
      // round-robin over the 8) and their re-reads hit its L2.
      const int q = local >> 3, u = ((q / a.nrg) << 3) + (local & 7);
      w.rg = q % a.nrg;
      w.h = u / ns;
      w.sp = u % ns;
    } else {
      w.h = hv / a.nrg;
      w.rg = hv - w.h * a.nrg;
    }
  }
  return w;
}

// Chunk queries: when qpr does not divide nqry, the last row group holds
// fewer queries; its rows past the last query repeat the last query (they
// read its q row and see its tokens, so every access stays in bounds) and
// write no record.
__device__ __forceinline__ bool row_padded(const DecodeArgs& a, int rg, int g) {
  return rg * a.qpr + a.row_x[g] >= a.nqry;
}
// the query row g computes: rg * qpr + row_x[g], or the last query
__device__ __forceinline__ int row_query(const DecodeArgs& a, int rg, int g) {
  return min(rg * a.qpr + a.row_x[g], a.nqry - 1);
}
// offset of row g's q row from that of the row group's row 0 (a valid query)
__device__ __forceinline__ int row_q_offset(const DecodeArgs& a, int rg, int g) {
  return a.row_off[g] - (rg * a.qpr + a.row_x[g] - row_query(a, rg, g)) * a.hq;
}

// Row g of the workgroup's row group: its index in q / out
// ([batch][nqry][Hq]), its record row within a split (query * Hq + head),
// and the end of the tokens it sees.
template <int GQ, bool CHUNK>
__device__ __forceinline__ size_t q_index(const DecodeArgs& a, const DecodeSeq& S, int h, int rg, int g) {
  if constexpr (!CHUNK) return (size_t)S.seq * a.hq + (size_t)h * GQ + g;
  return ((size_t)S.seq * a.nqry + rg * a.qpr) * a.hq + h * a.gqh + row_q_offset(a, rg, g);
}

template <int GQ, bool CHUNK>
__device__ __forceinline__ int rec_row(const DecodeArgs& a, int h, int rg, int g) {
  if constexpr (!CHUNK) return h * GQ + g;
  return rg * a.qpr * a.hq + h * a.gqh + a.row_off[g];
}

__device__ __forceinline__ int row_limit(const DecodeArgs& a, const DecodeSeq& S, int rg, int g) {
  return S.L - a.nqry + 1 + row_query(a, rg, g);
}

// The smallest limit of the row group: every token below it is visible to
// every row.
__device__ __forceinline__ int group_limit(const DecodeArgs& a, const DecodeSeq& S, int rg) {
  return S.L - a.nqry + 1 + rg * a.qpr;
}

// (g0: the first row of the group the GQ rows start at; the chunk kernel
// takes its fp16 tail in parts of 8 rows)
template <int GQ>
__device__ __forceinline__ void row_limits(const DecodeArgs& a, const DecodeSeq& S, int h, int rg, int (&lim)[GQ],
                                           int g0 = 0) {
#pragma unroll
  for (int g = 0; g < GQ; ++g) lim[g] = row_limit(a, S, rg, g0 + g);
}

// Per-wave partial results of GQ query heads, staged for the combine.
template <int GQ>
struct Reduce {
  float m[kWaves][GQ], l[kWaves][GQ];
  float acc[kWaves][GQ * kHeadDim];
};

// Vector-path state (lanes (tq, cc) hold 8 channels for a quarter of the
// tokens; l is spread over lanes) into the staging area of wave wv.
template <int GQ>
__device__ __forceinline__ void stage_state(State<GQ>& st, Reduce<GQ>& r, int lane, int wv) {
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    st.l[g] = wave_sum(st.l[g]);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      st.acc[g][k] += __shfl_xor(st.acc[g][k], 16);
      st.acc[g][k] += __shfl_xor(st.acc[g][k], 32);
    }
  }
  if (lane < 16) {
#pragma unroll
    for (int g = 0; g < GQ; ++g)
#pragma unroll
      for (int k = 0; k < 8; ++k) r.acc[wv][g * kHeadDim + lane * 8 + k] = st.acc[g][k];
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < GQ; ++g) { r.m[wv][g] = st.m[g]; r.l[wv][g] = st.l[g]; }
  }
}

// After a barrier: merge the waves' partial results and write the record of
// split sp for the GQ query heads of kv head h.
template <int GQ, bool CHUNK>
__device__ __forceinline__ void write_record(const DecodeArgs& a, const DecodeSeq& S, int h, int rg, int sp,
                                             const Reduce<GQ>& r, int g0 = 0) {
  for (int idx = threadIdx.x; idx < GQ * kHeadDim; idx += blockDim.x) {
    const int g = idx / kHeadDim, c = idx % kHeadDim;
    if (CHUNK && row_padded(a, rg, g0 + g)) continue;  // a repeat of the last query
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, r.m[w][g]);
    float val = 0.f, lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      // a wave that saw no visible token of a chunk row has m = -inf, l = 0
      // (in single-token decode some wave of every split has a block, so M
      // is finite and exp2(-inf - M) = 0 already)
      const float f = CHUNK && r.m[w][g] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(r.m[w][g] - M);
      val = fmaf(f, r.acc[w][idx], val);
      lsum = fmaf(f, r.l[w][g], lsum);
    }
    const size_t rows = CHUNK ? (size_t)a.hq * a.nqry : (size_t)a.hq;
    float* rec = a.ws + ((size_t)(S.ws_base + sp) * rows + rec_row<GQ, CHUNK>(a, h, rg, g0 + g)) * kRecFloats;
    rec[4 + c] = val;
    if (c == 0) { rec[0] = M; rec[1] = lsum; }
  }
}

// The fp16 tail split: every wave takes passes of 32 tokens.
template <int GQ, bool CHUNK>
__device__ __forceinline__ void tail_split(const DecodeArgs& a, const DecodeSeq& S, int h, int rg,
                                           const uint8_t* blk, const float (&qs0)[GQ], const float (&qs1)[GQ],
                                           float* qp, float* pl, State<GQ>& st, int lane, int wv, int g0 = 0) {
  constexpr int QS = QStride<GQ>::value;
  // Fused append: this workgroup alone reads the ring of (sequence, head h)
  // in this launch; it first stores the tokens appended by the call, which
  // all stay fp16 (the host takes this path only when no key group fills).
  if (a.K_new != nullptr && S.L_old < S.L) {
    uint32_t* rk = reinterpret_cast<uint32_t*>(const_cast<uint8_t*>(blk) + a.tk);
    uint32_t* rv = reinterpret_cast<uint32_t*>(const_cast<uint8_t*>(blk) + a.tv);
    const uint32_t* ik = reinterpret_cast<const uint32_t*>(a.K_new);
    const uint32_t* iv = reinterpret_cast<const uint32_t*>(a.V_new);
    constexpr int kRow = kHeadDim / 2;  // dwords per token row
    for (int idx = threadIdx.x; idx < (S.L - S.L_old) * kRow; idx += blockDim.x) {
      const int t = idx / kRow, c = idx % kRow;
      const size_t src = (((size_t)S.seq * a.n_max + t) * a.hkv + h) * kRow + c;
      const size_t dst = (size_t)((S.L_old + t) % a.W) * kRow + c;
      rk[dst] = ik[src];
      rv[dst] = iv[src];
    }
    __syncthreads();  // the stores are visible to the whole workgroup
  }
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    qp[(2 * lane) * QS + g] = qs0[g];
    qp[(2 * lane + 1) * QS + g] = qs1[g];
  }
  wave_lds_sync();
  int lim[GQ];
  row_limits<GQ>(a, S, h, rg, lim, g0);
  for (int pass = wv; pass * 32 < S.L - S.Lq; pass += kWaves)
    tail_pass<GQ, CHUNK>(a, S, blk, pass, qp, pl, st, lim, lane);
}

template <int GQ>
__device__ __forceinline__ void init_state(State<GQ>& st) {
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    st.m[g] = -__builtin_inff();
    st.l[g] = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) st.acc[g][k] = 0.f;
  }
}

// This lane's two channels (2*lane, 2*lane+1) of the GQ query heads,
// pre-scaled to base 2.
template <int GQ, bool CHUNK>
__device__ __forceinline__ void load_q_scaled(const DecodeArgs& a, const DecodeSeq& S, int h, int rg, int lane,
                                              float (&qs0)[GQ], float (&qs1)[GQ], int g0 = 0) {
#pragma unroll
  for (int g = 0; g < GQ; ++g) {
    const uint32_t w = reinterpret_cast<const uint32_t*>(a.q + q_index<GQ, CHUNK>(a, S, h, rg, g0 + g) * kHeadDim)[lane];
    qs0[g] = h2f(w & 0xFFFF) * a.qscale;
    qs1[g] = h2f(w >> 16) * a.qscale;
  }
}

}  // namespace dec
}  // namespace kvq
