// C ABI of the packed low-bit KV-cache library: argument checks, host-side
// length bookkeeping, the split plan of the decode kernel, and launches.
//
// Everything before a launch is plain host code that touches no device and
// calls no HIP function, so argument and capacity errors are detected (and
// testable) without a GPU and leave the cache unchanged.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <utility>
#include <vector>

#include "dgap.h"
#include "kvq.h"
#include "kvq_internal.h"
#include "kvq_layout.h"

using kvq::HeadLayout;

static_assert(kvq::kScratchBytes == KVQ_NOALLOC_SCRATCH_BYTES, "scratch array size as the header states");
static_assert(kvq::kSpareRow >= KVQ_MAX_CHUNK, "a spare row lies past every chunk query");

struct kvq_cache {
  kvq_cache_desc d{};
  std::vector<uint8_t> bk, bv;
  uint8_t* arena = nullptr;
  size_t arena_bytes = 0;
  int64_t cq = 0;   // most tokens ever packed per sequence
  int32_t W = 0;    // ring slots per head
  std::vector<uint64_t> head0;
  std::vector<HeadLayout> lay;
  std::vector<int32_t> L, Lq;
  std::vector<uint8_t> matrix;  // 1: matrix layout and the matrix-core decode kernel
  std::vector<int> occupancy;    // resident decode workgroups per compute unit, per sequence's kernel
  int32_t split_tokens = 0;
  // paged layout: block table on the device (pm.table), page lists and the
  // free pool on the host
  bool paged = false;
  kvq::PageMap pm{};
  std::vector<std::vector<int32_t>> pages;  // per sequence: pool page of each logical page
  std::vector<int32_t> free_pages;           // taken from the back
};

namespace {

thread_local std::string g_err;

constexpr int kMaxSplits = 512;          // packed splits per sequence and kv head
constexpr int kMinGroupsPerSplit = 4;    // one key group per wave at least
// Decode workgroups that fit the current device at once (one round of the
// grid): compute units times the resident workgroups per unit (one 4-wave
// workgroup per wave slot of a SIMD).
int64_t target_workgroups(int per_cu) {
  static thread_local int cached_dev = -1;
  static thread_local int64_t cus = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256 * per_cu;
  if (dev != cached_dev) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached_dev = dev;
    cus = n;
  }
  return cus * per_cu;
}

kvq_status fail(kvq_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

kvq_status ok() {
  g_err.clear();
  return KVQ_OK;
}

bool valid_bits(int b) { return b == 1 || b == 2 || b == 4 || b == 8; }

kvq_status check_desc(const kvq_cache_desc* d) {
  if (!d) return fail(KVQ_ERR_ARG, "descriptor is NULL");
  if (d->batch < 1) return fail(KVQ_ERR_ARG, "batch must be >= 1 (got %d)", d->batch);
  if (d->num_kv_heads < 1) return fail(KVQ_ERR_ARG, "num_kv_heads must be >= 1");
  if (d->num_q_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(KVQ_ERR_ARG, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)",
                d->num_q_heads, d->num_kv_heads);
  const int gq = d->num_q_heads / d->num_kv_heads;
  if (!(gq == 1 || gq == 2 || gq == 4 || gq == 5 || gq == 8))
    return fail(KVQ_ERR_UNSUPPORTED, "num_q_heads / num_kv_heads = %d; supported: 1, 2, 4, 5, 8", gq);
  if (d->head_dim < 1) return fail(KVQ_ERR_ARG, "head_dim must be positive");
  if (d->head_dim != kvq::kHeadDim) return fail(KVQ_ERR_UNSUPPORTED, "head_dim %d; only 128 is supported", d->head_dim);
  if (d->max_tokens < 1) return fail(KVQ_ERR_ARG, "max_tokens must be >= 1");
  if (!(d->key_group == 32 || d->key_group == 64 || d->key_group == 128))
    return fail(KVQ_ERR_ARG, "key_group %d; must be 32, 64 or 128", d->key_group);
  const int gv = d->value_group;
  if (!(gv == 8 || gv == 16 || gv == 32 || gv == 64 || gv == 128))
    return fail(KVQ_ERR_ARG, "value_group %d; must be 8, 16, 32, 64 or 128", gv);
  if (d->fp16_window < 0) return fail(KVQ_ERR_ARG, "fp16_window must be >= 0");
  if ((int64_t)d->fp16_window + d->key_group > (int64_t)1 << 30) return fail(KVQ_ERR_ARG, "fp16_window too large");
  if (!d->bits_k || !d->bits_v) return fail(KVQ_ERR_ARG, "bits_k and bits_v must be host arrays of length batch");
  for (int i = 0; i < d->batch; ++i) {
    if (!valid_bits(d->bits_k[i]) || !valid_bits(d->bits_v[i]))
      return fail(KVQ_ERR_ARG, "sequence %d: bits (%d, %d) must each be 1, 2, 4 or 8", i, d->bits_k[i], d->bits_v[i]);
  }
  const int P = d->page_tokens;
  if (P < 0 || (P > 0 && (P < d->key_group || P > (1 << 20) || (P & (P - 1)) != 0)))
    return fail(KVQ_ERR_ARG, "page_tokens %d: must be 0 or a power of two in [key_group = %d, 2^20]", P, d->key_group);
  if (d->num_pages < 0 || (d->num_pages > 0 && P == 0))
    return fail(KVQ_ERR_ARG, "num_pages %d: must be >= 0, and 0 unless page_tokens > 0", d->num_pages);
  if (P > 0) {
    for (int i = 1; i < d->batch; ++i)
      if (d->bits_k[i] != d->bits_k[0] || d->bits_v[i] != d->bits_v[0])
        return fail(KVQ_ERR_UNSUPPORTED, "a paged cache needs one bit width pair for every sequence");
  }
  return KVQ_OK;
}

int64_t packed_capacity(const kvq_cache_desc* d) {
  const int64_t past = (int64_t)d->max_tokens - d->fp16_window;
  return past <= 0 ? 0 : past / d->key_group * d->key_group;
}

int32_t quantized_len(int64_t L, const kvq_cache_desc& d) {
  const int64_t past = L - d.fp16_window;
  return past <= 0 ? 0 : (int32_t)(past / d.key_group * d.key_group);
}

HeadLayout layout_of(const kvq_cache_desc* d, int bk, int bv) {
  return kvq::head_layout(bk, bv, packed_capacity(d), d->key_group, d->value_group,
                          (int64_t)d->fp16_window + d->key_group);
}

// Arena of a paged cache: header | fp16 rings [batch][Hkv] | block table
// [batch][max_pages] int32 | pool [num_pages][Hkv][page head layout].
struct PagedArena {
  HeadLayout page, ring, seq_lay;  // seq_lay: packed offsets of the page, ring offsets and stride
  uint64_t table_off = 0, pool0 = 0, page_bytes = 0, total = 0;
  int32_t max_pages = 0, num_pages = 0;
};

PagedArena paged_arena(const kvq_cache_desc* d) {
  PagedArena A;
  const int bk = d->bits_k[0], bv = d->bits_v[0], P = d->page_tokens;
  const int64_t W = (int64_t)d->fp16_window + d->key_group;
  A.page = kvq::head_layout(bk, bv, P, d->key_group, d->value_group, 0, false);
  A.ring = kvq::head_layout(bk, bv, 0, d->key_group, d->value_group, W);
  A.seq_lay = A.page;
  A.seq_lay.tk = A.ring.tk;
  A.seq_lay.tv = A.ring.tv;
  A.seq_lay.vb = A.ring.vb;
  A.seq_lay.stride = A.ring.stride;
  A.max_pages = (int32_t)((packed_capacity(d) + P - 1) / P);
  A.num_pages = d->num_pages > 0 ? d->num_pages : d->batch * A.max_pages;
  const uint64_t rings = (uint64_t)d->batch * d->num_kv_heads * A.ring.stride;
  A.table_off = kvq::align_up(kvq::kHeaderBytes + rings, kvq::kAlign);
  A.pool0 = kvq::align_up(A.table_off + (uint64_t)d->batch * A.max_pages * 4, kvq::kAlign);
  A.page_bytes = (uint64_t)d->num_kv_heads * A.page.stride;
  A.total = A.pool0 + (uint64_t)A.num_pages * A.page_bytes;
  return A;
}

int log2_exact(int v) {
  int s = 0;
  while ((1 << s) < v) ++s;
  return s;
}

// Split length of one launch's sequences (one bit class): the launch fills
// two workgroups per compute unit (two waves per SIMD), a full round of
// the kernels that fit two and part of one for those that fit three or
// four.  Longer splits with fewer waves measured as fast or faster there:
// every wave pays a prologue (query, zero-point table, first loads) and an
// epilogue, all waves' first loads queue behind each other, and the merge
// reads fewer records.  Fewer than two per unit (one wave per SIMD on some
// units) measured 15-36% slower.  Classes launch one after another, so each
// gets the whole device.
int32_t split_tokens_for(const kvq_cache* c, const std::vector<int>& seqs, int nqry, int nrg, int occ_rows) {
  const int gk = c->d.key_group;
  if (c->split_tokens > 0) return c->split_tokens;
  int64_t total = 0, lq_max = 0, tails = 0;
  int occ = 4;
  for (int i : seqs) {
    total += (int64_t)c->Lq[i] * c->d.num_kv_heads * nrg;
    lq_max = std::max<int64_t>(lq_max, c->Lq[i]);
    if (c->L[i] > c->Lq[i]) tails += (int64_t)c->d.num_kv_heads * nrg;
    occ = std::min(occ, occ_rows > 0 && c->matrix[i] ? occ_rows : c->occupancy[i]);
  }
  // The fp16-tail workgroups (one per sequence and kv head with tail tokens)
  // must not wait for a free slot (that would add a whole split's time to
  // the launch).  Single-token decode of one sequence with kernels that fit
  // more than two workgroups per compute unit takes a full round of packed
  // splits (whole blocks per wave) and its tail workgroups, a few tokens
  // each and last in id order, in spare slots; otherwise the round leaves
  // them room (with several sequences each one's tail workgroups follow its
  // own packed splits, so the ids past the round would be packed splits;
  // chunk queries' tail workgroups hold the queries' own tokens: started
  // last, they would end last).
  const int64_t round = target_workgroups(std::min(occ, 2));
  const bool tails_spare = nqry == 1 && occ > 2 && seqs.size() == 1;
  const int64_t target = tails_spare ? round : std::max<int64_t>(round - tails, round / 2);
  int64_t st = (total + target - 1) / target;
  if (nrg > 1 && !seqs.empty()) {
    // chunk queries: every row group of a (kv head, split) unit reads the
    // unit's tokens; units of at most ~1 MiB let the row groups that share
    // an XCD find them in its L2 (more workgroup rounds instead)
    const int i0 = seqs[0];
    const int64_t tok_bytes = 16 * (c->bk[i0] + c->bv[i0]) + 512 / gk + 4 * (kvq::kHeadDim / c->d.value_group);
    st = std::min<int64_t>(st, ((int64_t)1 << 20) / tok_bytes);
  }
  st = std::max<int64_t>(st, (lq_max + kMaxSplits - 1) / kMaxSplits);
  st = (st + gk - 1) / gk * gk;
  st = std::max<int64_t>(st, (int64_t)gk * kMinGroupsPerSplit);
  if (nrg == 1) {
    // Short sequences: two 32-token blocks per wave at least, while the
    // launch still gives every compute unit a workgroup (a wave's first
    // loads and its epilogue cost about as much as a block)
    const int64_t two = ((int64_t)2 * 32 * kMinGroupsPerSplit + gk - 1) / gk * gk;
    if (two > st && (total + two - 1) / two >= round / 2) st = two;
  }
  return (int32_t)std::min<int64_t>(st, (int64_t)1 << 30);
}

int64_t splits_bound(const kvq_cache* c) {
  const int64_t cq = c->cq;
  int64_t nq;
  if (c->split_tokens > 0)
    nq = (cq + c->split_tokens - 1) / c->split_tokens;
  else
    nq = std::min<int64_t>(kMaxSplits, (cq + (int64_t)c->d.key_group * kMinGroupsPerSplit - 1) /
                                           ((int64_t)c->d.key_group * kMinGroupsPerSplit));
  return nq + 1;
}

kvq_status hip_fail(int e, const char* what) {
  return fail(KVQ_ERR_HIP, "%s: %s", what, hipGetErrorString((hipError_t)e));
}

// Sequences grouped by (key bits, value bits), each class in chunks that fit
// one kernel-argument block.
std::vector<std::pair<std::pair<int, int>, std::vector<int>>> bit_classes(const kvq_cache* c,
                                                                          const std::vector<int>& seqs) {
  std::map<std::pair<int, int>, std::vector<int>> m;
  for (int i : seqs) m[{c->bk[i], c->bv[i]}].push_back(i);
  std::vector<std::pair<std::pair<int, int>, std::vector<int>>> out;
  for (auto& kv : m) {
    for (size_t b = 0; b < kv.second.size(); b += kvq::kMaxSeqPerLaunch) {
      const size_t e = std::min(kv.second.size(), b + kvq::kMaxSeqPerLaunch);
      out.push_back({kv.first, std::vector<int>(kv.second.begin() + b, kv.second.begin() + e)});
    }
  }
  return out;
}

}  // namespace

namespace kvq {
int matrix_decode_occupancy(int bk, int bv, int gk, int gq) { return matrix_waves(bk, bv, gk / 32, gq); }

bool matrix_decode_supported(int bk, int bv, int gq, int gk, int gv, uint64_t head_bytes) {
  return matrix_heads(gq, gk) && matrix_bits(bk, bv) && gv >= 32 && head_bytes <= 0xFFFFFFFFull;
}
}  // namespace kvq

extern "C" {

size_t kvq_cache_bytes(const kvq_cache_desc* d) {
  if (check_desc(d) != KVQ_OK) return 0;
  if (d->page_tokens > 0) return (size_t)paged_arena(d).total;
  uint64_t total = kvq::kHeaderBytes;
  for (int i = 0; i < d->batch; ++i) total += (uint64_t)d->num_kv_heads * layout_of(d, d->bits_k[i], d->bits_v[i]).stride;
  return (size_t)total;
}

kvq_status kvq_cache_init(kvq_cache** out, const kvq_cache_desc* d, void* arena, size_t arena_bytes) {
  if (!out) return fail(KVQ_ERR_ARG, "out is NULL");
  *out = nullptr;
  const kvq_status st = check_desc(d);
  if (st != KVQ_OK) return st;
  if (!arena) return fail(KVQ_ERR_ARG, "arena is NULL");
  if (reinterpret_cast<uintptr_t>(arena) % kvq::kAlign != 0) return fail(KVQ_ERR_ARG, "arena must be 256-byte aligned");
  const size_t need = kvq_cache_bytes(d);
  if (arena_bytes < need)
    return fail(KVQ_ERR_CAPACITY, "arena holds %zu bytes, the cache needs %zu", arena_bytes, need);
  kvq_cache* c = new kvq_cache();
  c->d = *d;
  c->bk.assign(d->bits_k, d->bits_k + d->batch);
  c->bv.assign(d->bits_v, d->bits_v + d->batch);
  c->d.bits_k = c->bk.data();
  c->d.bits_v = c->bv.data();
  c->arena = static_cast<uint8_t*>(arena);
  c->arena_bytes = arena_bytes;
  c->cq = packed_capacity(d);
  c->W = d->fp16_window + d->key_group;
  uint64_t off = kvq::kHeaderBytes;
  uint64_t packed_bytes = 0;  // what the matrix kernel's 32-bit offsets must reach (one buffer resource)
  if (d->page_tokens > 0) {
    const PagedArena A = paged_arena(d);
    c->paged = true;
    c->pm.table = reinterpret_cast<const int32_t*>(c->arena + A.table_off);
    c->pm.pool0 = A.pool0;
    c->pm.page_bytes = A.page_bytes;
    c->pm.page_head_bytes = A.page.stride;
    c->pm.pool_bytes = (uint64_t)A.num_pages * A.page_bytes;
    c->pm.page_tokens = d->page_tokens;
    c->pm.max_pages = A.max_pages;
    c->pm.page_shift = log2_exact(d->page_tokens);
    c->pm.gk_shift = log2_exact(d->key_group);
    for (int i = 0; i < d->batch; ++i) {
      c->lay.push_back(A.seq_lay);
      c->head0.push_back(off);
      off += (uint64_t)d->num_kv_heads * A.ring.stride;
    }
    c->pages.assign(d->batch, {});
    for (int pg = A.num_pages - 1; pg >= 0; --pg) c->free_pages.push_back(pg);
    packed_bytes = A.page.stride;  // one page's region of one kv head, whatever the pool size
  } else {
    for (int i = 0; i < d->batch; ++i) {
      c->lay.push_back(layout_of(d, c->bk[i], c->bv[i]));
      c->head0.push_back(off);
      off += (uint64_t)d->num_kv_heads * c->lay.back().stride;
    }
  }
  c->L.assign(d->batch, 0);
  c->Lq.assign(d->batch, 0);
  for (int i = 0; i < d->batch; ++i)
    c->matrix.push_back(kvq::matrix_decode_supported(c->bk[i], c->bv[i], d->num_q_heads / d->num_kv_heads,
                                                     d->key_group,
                                                     d->value_group, c->paged ? packed_bytes : c->lay[i].stride)
                            ? 1
                            : 0);
  // the split plan of a launch fills one round of its kernel's workgroups
  for (int i = 0; i < d->batch; ++i)
    c->occupancy.push_back(c->matrix[i] ? kvq::matrix_decode_occupancy(c->bk[i], c->bv[i], d->key_group,
                                                                       d->num_q_heads / d->num_kv_heads)
                                        : 2);
  *out = c;
  return ok();
}

void kvq_cache_destroy(kvq_cache* c) { delete c; }

kvq_status kvq_cache_reset(kvq_cache* c, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  const int e = kvq::launch_fill_zero(c->arena, kvq::kHeaderBytes / 4, stream);
  if (e) return hip_fail(e, "reset");
  std::fill(c->L.begin(), c->L.end(), 0);
  std::fill(c->Lq.begin(), c->Lq.end(), 0);
  if (c->paged) {
    for (auto& pl : c->pages) {
      for (int32_t pg : pl) c->free_pages.push_back(pg);
      pl.clear();
    }
  }
  return ok();
}

int64_t kvq_seq_len(const kvq_cache* c, int32_t seq) {
  if (!c || seq < 0 || seq >= c->d.batch) return -1;
  return c->L[seq];
}

kvq_status kvq_seq_release(kvq_cache* c, int32_t seq) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (seq < 0 || seq >= c->d.batch) return fail(KVQ_ERR_ARG, "seq %d out of range", seq);
  c->L[seq] = 0;
  c->Lq[seq] = 0;
  if (c->paged) {
    for (int32_t pg : c->pages[seq]) c->free_pages.push_back(pg);
    c->pages[seq].clear();
  }
  return ok();
}

int64_t kvq_free_pages(const kvq_cache* c) {
  if (!c || !c->paged) return -1;
  return (int64_t)c->free_pages.size();
}

kvq_status kvq_append(kvq_cache* c, const void* K, const void* V, int32_t n_max, const int32_t* n_new,
                      void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (!n_new) return fail(KVQ_ERR_ARG, "n_new is NULL");
  if (n_max < 0) return fail(KVQ_ERR_ARG, "n_max must be >= 0");
  const kvq_cache_desc& d = c->d;
  bool any = false;
  for (int i = 0; i < d.batch; ++i) {
    if (n_new[i] < 0 || n_new[i] > n_max)
      return fail(KVQ_ERR_ARG, "sequence %d: n_new = %d outside [0, n_max = %d]", i, n_new[i], n_max);
    if ((int64_t)c->L[i] + n_new[i] > d.max_tokens)
      return fail(KVQ_ERR_CAPACITY, "sequence %d: %d + %d tokens exceed max_tokens = %d", i, c->L[i], n_new[i],
                  d.max_tokens);
    any |= n_new[i] > 0;
  }
  if (!any) return ok();
  if (!K || !V) return fail(KVQ_ERR_ARG, "K and V must be device pointers");

  std::vector<int> seqs;
  std::vector<int32_t> L_new(d.batch), Lq_new(d.batch);
  bool fused = true;
  int64_t pages_needed = 0;
  for (int i = 0; i < d.batch; ++i) {
    L_new[i] = c->L[i] + n_new[i];
    Lq_new[i] = quantized_len(L_new[i], d);
    if (n_new[i] > 0) seqs.push_back(i);
    if ((int64_t)L_new[i] - c->Lq[i] > c->W) fused = false;
    if (c->paged)
      pages_needed += (Lq_new[i] + d.page_tokens - 1) / d.page_tokens - (int64_t)c->pages[i].size();
  }
  if (c->paged && pages_needed > (int64_t)c->free_pages.size())
    return fail(KVQ_ERR_CAPACITY, "the append needs %lld more pages, the pool has %zu free", (long long)pages_needed,
                c->free_pages.size());
  {
    // a sequence's first packed group starts a fresh bound on its value
    // scales (after kvq_seq_release or kvq_cache_reset the old one is stale)
    kvq::WordReset r{};
    r.arena = c->arena;
    for (int i = 0; i < d.batch; ++i) {
      if (c->Lq[i] != 0 || Lq_new[i] == 0) continue;
      for (int h = 0; h < d.num_kv_heads; ++h) {
        r.off[r.n++] = c->head0[i] + (uint64_t)h * c->lay[i].stride + c->lay[i].vb;
        if (r.n == kvq::kTableSetMax) {
          const int e = kvq::launch_word_reset(r, stream);
          if (e) return hip_fail(e, "bound reset launch");
          r.n = 0;
        }
      }
    }
    const int e = kvq::launch_word_reset(r, stream);
    if (e) return hip_fail(e, "bound reset launch");
  }
  if (c->paged && pages_needed > 0) {
    // take the pages and write their block-table entries (ordered before the append launch)
    kvq::TableSet t{};
    t.table = const_cast<int32_t*>(c->pm.table);
    for (int i = 0; i < d.batch; ++i) {
      const int32_t want = (Lq_new[i] + d.page_tokens - 1) / d.page_tokens;
      while ((int32_t)c->pages[i].size() < want) {
        const int32_t pg = c->free_pages.back();
        c->free_pages.pop_back();
        t.idx[t.n] = i * c->pm.max_pages + (int32_t)c->pages[i].size();
        t.val[t.n] = pg;
        ++t.n;
        c->pages[i].push_back(pg);
        if (t.n == kvq::kTableSetMax) {
          const int e = kvq::launch_table_set(t, stream);
          if (e) return hip_fail(e, "block table launch");
          t.n = 0;
        }
      }
    }
    const int e = kvq::launch_table_set(t, stream);
    if (e) return hip_fail(e, "block table launch");
  }

  // fused: one launch packs groups and fills ring slots (no slot is both
  // read and written); otherwise pack first, then fill the ring.
  const int phases = fused ? 1 : 2;
  for (int ph = 0; ph < phases; ++ph) {
    const bool quant = fused || ph == 0, copy = fused || ph == 1;
    for (auto& cls : bit_classes(c, seqs)) {
      kvq::AppendArgs a{};
      const HeadLayout& lay = c->lay[cls.second[0]];
      a.arena = c->arena;
      a.K = static_cast<const uint16_t*>(K);
      a.V = static_cast<const uint16_t*>(V);
      a.head_stride = lay.stride;
      a.kc = (uint32_t)lay.kc; a.km = (uint32_t)lay.km; a.vc = (uint32_t)lay.vc;
      a.vm = (uint32_t)lay.vm; a.tk = (uint32_t)lay.tk; a.tv = (uint32_t)lay.tv; a.vb = (uint32_t)lay.vb;
      a.n_max = n_max; a.hkv = d.num_kv_heads; a.gk = d.key_group; a.gv = d.value_group; a.W = c->W;
      a.quantize = quant ? 1 : 0;
      a.matrix = c->matrix[cls.second[0]];
      a.pm = c->pm;
      int wg = 0, n = 0;
      for (int i : cls.second) {
        kvq::AppendSeq& s = a.seq[n++];
        s.head0 = c->head0[i];
        s.seq = i;
        s.L_old = c->L[i]; s.Lq_old = c->Lq[i]; s.L_new = L_new[i]; s.Lq_new = Lq_new[i];
        s.n_quant = (Lq_new[i] - c->Lq[i]) / d.key_group;
        s.do_copy = (copy && L_new[i] > std::max(Lq_new[i], c->L[i])) ? 1 : 0;
        s.wg_begin = wg;
        wg += (quant ? s.n_quant * d.num_kv_heads : 0) + (s.do_copy ? d.num_kv_heads : 0);
      }
      a.nseq = n;
      a.total_wg = wg;
      const int e = kvq::launch_append(a, cls.first.first, cls.first.second, stream);
      if (e) return hip_fail(e, "append launch");
    }
  }
  for (int i = 0; i < d.batch; ++i) {
    c->L[i] = L_new[i];
    c->Lq[i] = Lq_new[i];
  }
  return ok();
}

size_t kvq_workspace_bytes(const kvq_cache* c) {
  if (!c) return 0;
  return (size_t)c->d.batch * c->d.num_q_heads * (size_t)splits_bound(c) * kvq::kRecFloats * sizeof(float);
}

}  // extern "C"

// The split plan and the launches of decode, shared by the entry points below.
namespace {

// Query rows of a launch (see DecodeArgs): nqry queries per sequence in row
// groups of qpr queries, rows = qpr * (Hq / Hkv) rows per workgroup.
struct Rows {
  int nqry = 1, qpr = 1, nrg = 1, rows = 1;
};

// Single-token decode: one row group of the kv head's query heads.  Chunk
// queries on the vector kernel: the largest of its row groups (8, 5, 4, 2,
// 1 rows) made of whole queries, with a whole number of groups.  On the
// matrix cores (32 rows in the chunk kernel for 1- and 2-bit classes, 16 for
// those and 4-bit classes, with value groups of 32 channels; 8, 5 or 4 in
// the decode kernel), the row group of whole queries with the smallest
// estimated time: ceil(nqry / qpr) passes over the kv head's cache at a
// per-pass cost that grows with the rows; the last group may repeat the last
// query in its spare rows, and a chunk kernel group of five heads leaves the
// rows past its 3 or 6 queries spare.
// Relative cost of one pass per row count: µs per row group of 131072-token
// K1V1 Llama-3.1-8B layers when a chunk launch takes several (4-row 18,
// 8-row 21, 16-row 30, 32-row 38; a launch's first pass costs 10-20 µs
// more).
int pass_cost(int rows) { return rows >= 32 ? 38 : rows >= 16 ? 30 : rows >= 8 ? 21 : rows >= 5 ? 19 : 18; }

Rows rows_for(const kvq_cache* c, bool matrix, int nqry, int bk, int bv) {
  const int gqh = c->d.num_q_heads / c->d.num_kv_heads;
  Rows r;
  r.rows = gqh;
  if (nqry <= 1) return r;
  r.nqry = nqry;
  if (!matrix) {
    for (int rg : {8, 5, 4, 2, 1}) {
      if (rg % gqh == 0 && nqry % (rg / gqh) == 0) {
        r.qpr = rg / gqh;
        r.nrg = nqry / r.qpr;
        r.rows = rg;
        return r;
      }
    }
    r.qpr = 1;  // not reached: rg = gqh always qualifies
    r.nrg = nqry;
    return r;
  }
  const bool rows16 = c->d.value_group == 32 && bk + bv <= 8;
  r.qpr = 1;  // one query per group (rows = gqh) unless a candidate is cheaper
  r.nrg = nqry;
  int best = -1;
  for (int rg : {32, 16, 8, 5, 4}) {
    if (rg >= 16 && !rows16) continue;
    if (rg == 32 && !kvq::chunk_rows32(bk, bv)) continue;
    // the decode kernel's row layouts hold whole sets of heads; the chunk
    // kernel's 16 or 32 rows take floor(rows / gqh) queries (five heads: 3
    // or 6) and leave the remaining rows spare
    if (rg < 16 && rg % gqh != 0) continue;
    const int qpr = rg / gqh, nrg = (nqry + qpr - 1) / qpr;
    const int cost = nrg * pass_cost(rg);
    if (best < 0 || cost < best) {
      best = cost;
      r.qpr = qpr;
      r.nrg = nrg;
      r.rows = rg;
    }
  }
  return r;  // 4 rows (1, 2 or 4 heads), 5 or 8 always qualify
}

struct SplitPlan {
  std::vector<int32_t> st, nq, ns, base;  // per sequence: split length, packed splits, all splits, first record
  int64_t records = 0;
  int nqry = 1;
};

SplitPlan plan_splits(const kvq_cache* c, int nqry = 1) {
  SplitPlan p;
  p.nqry = nqry;
  const int B = c->d.batch;
  p.st.assign(B, 0);
  std::map<std::pair<int, int>, std::vector<int>> classes;
  for (int i = 0; i < B; ++i) classes[{c->bk[i], c->bv[i]}].push_back(i);
  for (auto& cl : classes) {
    const bool matrix = c->matrix[cl.second[0]] != 0;
    const Rows r = rows_for(c, matrix, nqry, cl.first.first, cl.first.second);
    const int occ = nqry > 1 && matrix
                        ? kvq::matrix_decode_occupancy(cl.first.first, cl.first.second, c->d.key_group, r.rows)
                        : 0;
    const int32_t st = split_tokens_for(c, cl.second, nqry, r.nrg, occ);
    for (int i : cl.second) p.st[i] = st;
  }
  p.nq.resize(B);
  p.ns.resize(B);
  p.base.resize(B);
  for (int i = 0; i < B; ++i) {
    p.nq[i] = (c->Lq[i] + p.st[i] - 1) / p.st[i];
    p.ns[i] = p.nq[i] + (c->L[i] > c->Lq[i] ? 1 : 0);
    p.base[i] = (int32_t)p.records;
    p.records += p.ns[i];
  }
  return p;
}

// Append inputs of a fused append + decode: the tokens [L_old[i], L[i]) of
// each sequence come from K/V rows and are written into the ring by the
// decode launch itself.
struct FusedAppend {
  const void* K;
  const void* V;
  int32_t n_max;
  const std::vector<int32_t>* L_old;
};

kvq_status run_partials(const kvq_cache* c, const SplitPlan& p, const void* q, void* ws, size_t ws_bytes,
                        void* stream, const FusedAppend* app = nullptr) {
  const kvq_cache_desc& d = c->d;
  const size_t need = (size_t)p.records * d.num_q_heads * p.nqry * kvq::kRecFloats * sizeof(float);
  if (!q) return fail(KVQ_ERR_ARG, "q must be a device pointer");
  if (need > 0 && !ws) return fail(KVQ_ERR_ARG, "workspace is NULL");
  if (ws_bytes < need) return fail(KVQ_ERR_CAPACITY, "workspace holds %zu bytes, this call needs %zu", ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 16 != 0) return fail(KVQ_ERR_ARG, "workspace must be 16-byte aligned");
  std::vector<int> seqs;
  for (int i = 0; i < d.batch; ++i)
    if (c->L[i] > 0) seqs.push_back(i);
  const float qscale = (float)(1.4426950408889634 / std::sqrt((double)d.head_dim));
  for (auto& cls : bit_classes(c, seqs)) {
    kvq::DecodeArgs a{};
    const HeadLayout& lay = c->lay[cls.second[0]];
    a.arena = c->arena;
    a.q = static_cast<const uint16_t*>(q);
    a.ws = static_cast<float*>(ws);
    a.head_stride = lay.stride;
    a.kc = (uint32_t)lay.kc; a.km = (uint32_t)lay.km; a.vc = (uint32_t)lay.vc;
    a.vm = (uint32_t)lay.vm; a.tk = (uint32_t)lay.tk; a.tv = (uint32_t)lay.tv; a.vb = (uint32_t)lay.vb;
    a.hq = d.num_q_heads; a.hkv = d.num_kv_heads; a.gk = d.key_group; a.gv = d.value_group; a.W = c->W;
    a.split_tokens = p.st[cls.second[0]];
    a.qscale = qscale;
    const Rows r = rows_for(c, c->matrix[cls.second[0]] != 0, p.nqry, cls.first.first, cls.first.second);
    a.nqry = r.nqry; a.qpr = r.qpr; a.nrg = r.nrg; a.gqh = d.num_q_heads / d.num_kv_heads;
    // rows past qpr whole queries (a chunk kernel group of five heads) are
    // spare: row_x = kvq::kSpareRow marks them (a repeat of the last query)
    for (int g = 0; g < 32; ++g) {
      a.row_x[g] = g < r.qpr * a.gqh ? g / a.gqh : kvq::kSpareRow;
      a.row_off[g] = a.row_x[g] * d.num_q_heads + g % a.gqh;
    }
    a.pm = c->pm;
    if (app) {
      a.K_new = static_cast<const uint16_t*>(app->K);
      a.V_new = static_cast<const uint16_t*>(app->V);
      a.n_max = app->n_max;
    }
    int wg = 0, n = 0;
    for (int i : cls.second) {
      kvq::DecodeSeq& s = a.seq[n++];
      s.head0 = c->head0[i];
      s.seq = i; s.L = c->L[i]; s.Lq = c->Lq[i];
      s.L_old = app ? (*app->L_old)[i] : c->L[i];
      s.nq = p.nq[i]; s.nsplit = p.ns[i]; s.ws_base = p.base[i];
      s.wg_begin = wg;
      wg += p.ns[i] * d.num_kv_heads * r.nrg;
    }
    a.nseq = n;
    a.total_wg = wg;
    const int e = !c->matrix[cls.second[0]] ? kvq::launch_decode(a, cls.first.first, cls.first.second, r.rows, stream)
                  : r.rows >= 16 ? kvq::launch_chunk_matrix(a, cls.first.first, cls.first.second, r.rows, stream)
                                       : kvq::launch_decode_matrix(a, cls.first.first, cls.first.second, r.rows, stream);
    if (e) return hip_fail(e, "decode launch");
  }
  return KVQ_OK;
}

kvq_status run_merge(const kvq_cache* c, const SplitPlan& p, const void* ws, float* out, void* stream) {
  const kvq_cache_desc& d = c->d;
  if (!out) return fail(KVQ_ERR_ARG, "out must be a device pointer");
  if (p.records > 0 && !ws) return fail(KVQ_ERR_ARG, "workspace is NULL");
  for (int b = 0; b < d.batch; b += kvq::kMaxSeqPerLaunch) {
    kvq::MergeArgs m{};
    m.ws = static_cast<const float*>(ws);
    m.out = out;
    m.hq = d.num_q_heads * p.nqry;  // out [batch][nqry][Hq] = [batch][nqry * Hq]
    int n = 0;
    for (int i = b; i < std::min(d.batch, b + kvq::kMaxSeqPerLaunch); ++i) {
      m.seq[n].seq = i; m.seq[n].nsplit = p.ns[i]; m.seq[n].ws_base = p.base[i];
      ++n;
    }
    m.nseq = n;
    const int e = kvq::launch_merge(m, stream);
    if (e) return hip_fail(e, "merge launch");
  }
  return KVQ_OK;
}

}  // namespace

extern "C" {

kvq_status kvq_decode_attention(const kvq_cache* c, const void* q, float* out, void* ws, size_t ws_bytes,
                                void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (!q || !out) return fail(KVQ_ERR_ARG, "q and out must be device pointers");
  const SplitPlan p = plan_splits(c);
  kvq_status st = run_partials(c, p, q, ws, ws_bytes, stream);
  if (st != KVQ_OK) return st;
  st = run_merge(c, p, ws, out, stream);
  if (st != KVQ_OK) return st;
  return ok();
}

kvq_status kvq_decode_attention_noalloc(const kvq_cache* c, const void* q, float* out, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (!q || !out) return fail(KVQ_ERR_ARG, "q and out must be device pointers");
  const SplitPlan p = plan_splits(c);
  const size_t need = (size_t)p.records * c->d.num_q_heads * kvq::kRecFloats * sizeof(float);
  if (need > kvq::kScratchBytes)
    return fail(KVQ_ERR_CAPACITY, "this decode needs %zu bytes of workspace, more than the %zu bytes of the "
                "library's scratch array; use kvq_decode_attention with a caller workspace", need, kvq::kScratchBytes);
  void* ws = nullptr;
  const int e = kvq::scratch_workspace(&ws);
  if (e) return hip_fail(e, "scratch array address");
  kvq_status st = run_partials(c, p, q, ws, kvq::kScratchBytes, stream);
  if (st != KVQ_OK) return st;
  st = run_merge(c, p, ws, out, stream);
  if (st != KVQ_OK) return st;
  return ok();
}

kvq_status kvq_append_decode(kvq_cache* c, const void* K, const void* V, int32_t n_max, const int32_t* n_new,
                             const void* q, float* out, void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (!n_new) return fail(KVQ_ERR_ARG, "n_new is NULL");
  if (n_max < 0) return fail(KVQ_ERR_ARG, "n_max must be >= 0");
  if (!q || !out) return fail(KVQ_ERR_ARG, "q and out must be device pointers");
  const kvq_cache_desc& d = c->d;
  bool any = false, flush = false;
  for (int i = 0; i < d.batch; ++i) {
    if (n_new[i] < 0 || n_new[i] > n_max)
      return fail(KVQ_ERR_ARG, "sequence %d: n_new = %d outside [0, n_max = %d]", i, n_new[i], n_max);
    if ((int64_t)c->L[i] + n_new[i] > d.max_tokens)
      return fail(KVQ_ERR_CAPACITY, "sequence %d: %d + %d tokens exceed max_tokens = %d", i, c->L[i], n_new[i],
                  d.max_tokens);
    any |= n_new[i] > 0;
    flush |= quantized_len(c->L[i] + n_new[i], d) != c->Lq[i];
  }
  if (any && (!K || !V)) return fail(KVQ_ERR_ARG, "K and V must be device pointers");
  if (any && (reinterpret_cast<uintptr_t>(K) % 4 != 0 || reinterpret_cast<uintptr_t>(V) % 4 != 0))
    return fail(KVQ_ERR_ARG, "K and V must be 4-byte aligned");

  // plan with the lengths after the append; nothing is launched or changed
  // unless the workspace fits
  const std::vector<int32_t> L_old = c->L, Lq_old = c->Lq;
  for (int i = 0; i < d.batch; ++i) {
    c->L[i] = L_old[i] + n_new[i];
    c->Lq[i] = quantized_len(c->L[i], d);
  }
  const SplitPlan p = plan_splits(c);
  const size_t need = (size_t)p.records * d.num_q_heads * kvq::kRecFloats * sizeof(float);
  const char* bad = nullptr;
  kvq_status bad_st = KVQ_ERR_ARG;
  if (need > 0 && !ws) bad = "workspace is NULL";
  else if (ws_bytes < need) bad = "workspace too small for the lengths after the append", bad_st = KVQ_ERR_CAPACITY;
  else if (reinterpret_cast<uintptr_t>(ws) % 16 != 0) bad = "workspace must be 16-byte aligned";
  if (bad || flush) {
    c->L = L_old;
    c->Lq = Lq_old;
  }
  if (bad) return fail(bad_st, "%s (needs %zu bytes, has %zu)", bad, need, ws_bytes);
  if (flush) {  // a key group fills: the append kernel packs it, then a plain decode
    kvq_status st = kvq_append(c, K, V, n_max, n_new, stream);
    if (st != KVQ_OK) return st;
    return kvq_decode_attention(c, q, out, ws, ws_bytes, stream);
  }
  const FusedAppend app{K, V, n_max, &L_old};
  kvq_status st = run_partials(c, p, q, ws, ws_bytes, stream, any ? &app : nullptr);
  if (st != KVQ_OK) return st;
  st = run_merge(c, p, ws, out, stream);
  if (st != KVQ_OK) return st;
  return ok();
}

kvq_status kvq_decode_partials(const kvq_cache* c, const void* q, void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  const kvq_status st = run_partials(c, plan_splits(c), q, ws, ws_bytes, stream);
  return st == KVQ_OK ? ok() : st;
}

kvq_status kvq_decode_merge(const kvq_cache* c, const void* ws, float* out, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  const kvq_status st = run_merge(c, plan_splits(c), ws, out, stream);
  return st == KVQ_OK ? ok() : st;
}

size_t kvq_chunk_workspace_bytes(const kvq_cache* c, int32_t n_q) {
  if (!c || n_q < 1 || n_q > KVQ_MAX_CHUNK) return 0;
  return kvq_workspace_bytes(c) * (size_t)n_q;
}

kvq_status kvq_chunk_attention(const kvq_cache* c, const void* q, int32_t n_q, float* out, void* ws,
                               size_t ws_bytes, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (n_q < 1 || n_q > KVQ_MAX_CHUNK) return fail(KVQ_ERR_ARG, "n_q = %d outside [1, %d]", n_q, KVQ_MAX_CHUNK);
  if (!q || !out) return fail(KVQ_ERR_ARG, "q and out must be device pointers");
  for (int i = 0; i < c->d.batch; ++i)
    if (c->L[i] < n_q)
      return fail(KVQ_ERR_ARG, "sequence %d holds %d tokens, fewer than the %d chunk queries", i, c->L[i], n_q);
  const SplitPlan p = plan_splits(c, n_q);
  kvq_status st = run_partials(c, p, q, ws, ws_bytes, stream);
  if (st != KVQ_OK) return st;
  st = run_merge(c, p, ws, out, stream);
  if (st != KVQ_OK) return st;
  return ok();
}

kvq_status kvq_dequant(const kvq_cache* c, int32_t seq, int32_t tok0, int32_t ntok, float* K_out, float* V_out,
                       void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (seq < 0 || seq >= c->d.batch) return fail(KVQ_ERR_ARG, "seq %d out of range", seq);
  if (tok0 < 0 || ntok < 0 || (int64_t)tok0 + ntok > c->L[seq])
    return fail(KVQ_ERR_ARG, "token range [%d, %lld) outside [0, %d)", tok0, (long long)tok0 + ntok, c->L[seq]);
  if (ntok == 0) return ok();
  if (!K_out || !V_out) return fail(KVQ_ERR_ARG, "outputs must be device pointers");
  const HeadLayout& lay = c->lay[seq];
  kvq::DequantArgs a{};
  a.arena = c->arena;
  a.head0 = c->head0[seq];
  a.seq = seq;
  a.pm = c->pm;
  a.K_out = K_out; a.V_out = V_out;
  a.head_stride = lay.stride;
  a.kc = (uint32_t)lay.kc; a.km = (uint32_t)lay.km; a.vc = (uint32_t)lay.vc;
  a.vm = (uint32_t)lay.vm; a.tk = (uint32_t)lay.tk; a.tv = (uint32_t)lay.tv;
  a.hkv = c->d.num_kv_heads; a.gk = c->d.key_group; a.gv = c->d.value_group; a.W = c->W;
  a.bk = c->bk[seq]; a.bv = c->bv[seq]; a.Lq = c->Lq[seq]; a.tok0 = tok0; a.ntok = ntok;
  a.matrix = c->matrix[seq];
  const int e = kvq::launch_dequant(a, stream);
  if (e) return hip_fail(e, "dequant launch");
  return ok();
}

size_t kvq_export_bytes(const kvq_cache* c, int32_t seq, int32_t h) {
  if (!c || seq < 0 || seq >= c->d.batch || h < 0 || h >= c->d.num_kv_heads) return 0;
  const size_t Lq = c->Lq[seq], tail = c->L[seq] - c->Lq[seq], D = kvq::kHeadDim;
  return Lq * 16 * c->bk[seq] + Lq / c->d.key_group * 2 * D * 2 + Lq * 16 * c->bv[seq] +
         Lq * (D / c->d.value_group) * 4 + tail * D * 2 * 2;
}

kvq_status kvq_export(const kvq_cache* c, int32_t seq, int32_t h, void* dst, size_t bytes, void* stream) {
  const size_t need = kvq_export_bytes(c, seq, h);
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (seq < 0 || seq >= c->d.batch || h < 0 || h >= c->d.num_kv_heads)
    return fail(KVQ_ERR_ARG, "(seq %d, kv head %d) out of range", seq, h);
  if (bytes < need) return fail(KVQ_ERR_CAPACITY, "destination holds %zu bytes, the image has %zu", bytes, need);
  if (need == 0) return ok();
  if (!dst) return fail(KVQ_ERR_ARG, "destination is NULL");
  const HeadLayout& lay = c->lay[seq];
  const uint8_t* blk = c->arena + c->head0[seq] + (uint64_t)h * lay.stride;
  uint8_t* o = static_cast<uint8_t*>(dst);
  const size_t Lq = c->Lq[seq], L = c->L[seq], D = kvq::kHeadDim;
  const size_t part[4][2] = {{lay.kc, Lq * 16 * c->bk[seq]},
                             {lay.km, Lq / c->d.key_group * 2 * D * 2},
                             {lay.vc, Lq * 16 * c->bv[seq]},
                             {lay.vm, Lq * (D / c->d.value_group) * 4}};
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (c->paged) {
    // page by page into the same canonical image: the page's tokens
    // [t0, t0 + n) of every part, codes and value meta re-ordered by the
    // export kernel in the matrix layout
    uint8_t* okc = o;
    uint8_t* okm = okc + part[0][1];
    uint8_t* ovc = okm + part[1][1];
    uint8_t* ovm = ovc + part[2][1];
    const size_t P = c->d.page_tokens, gk = c->d.key_group, ng = D / c->d.value_group;
    const int bk = c->bk[seq], bv = c->bv[seq];
    for (size_t lp = 0; lp * P < Lq; ++lp) {
      const size_t t0 = lp * P, n = std::min(Lq - t0, P);
      const uint8_t* seg =
          c->arena + c->pm.pool0 + (uint64_t)c->pages[seq][lp] * c->pm.page_bytes + (uint64_t)h * c->pm.page_head_bytes;
      const hipError_t e = hipMemcpyAsync(okm + t0 / gk * 2 * D * 2, seg + lay.km, n / gk * 2 * D * 2,
                                          hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "export copy");
      if (c->matrix[seq]) {
        kvq::ExportArgs x{};
        x.blk = seg;
        x.kc_out = okc + t0 * 16 * bk;
        x.vc_out = ovc + t0 * 16 * bv;
        x.vm_out = ovm + t0 * ng * 4;
        x.kc = (uint32_t)lay.kc; x.vc = (uint32_t)lay.vc; x.vm = (uint32_t)lay.vm;
        x.bk = bk; x.bv = bv; x.gv = c->d.value_group; x.nblocks = (int32_t)(n / 32);
        const int ek = kvq::launch_export(x, stream);
        if (ek) return hip_fail(ek, "export launch");
      } else {
        const size_t src[3][3] = {{lay.kc, t0 * 16 * bk, n * 16 * bk},
                                  {lay.vc, t0 * 16 * bv, n * 16 * bv},
                                  {lay.vm, t0 * ng * 4, n * ng * 4}};
        uint8_t* dst[3] = {okc, ovc, ovm};
        for (int k = 0; k < 3; ++k) {
          const hipError_t e2 = hipMemcpyAsync(dst[k] + src[k][1], seg + src[k][0], src[k][2],
                                               hipMemcpyDeviceToDevice, s);
          if (e2 != hipSuccess) return hip_fail(e2, "export copy");
        }
      }
    }
    o = ovm + part[3][1];
  } else if (c->matrix[seq]) {
    // key meta is stored canonically; codes and value meta are re-ordered by a kernel
    if (part[1][1]) {
      const hipError_t e = hipMemcpyAsync(o + part[0][1], blk + part[1][0], part[1][1], hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "export copy");
    }
    kvq::ExportArgs x{};
    x.blk = blk;
    x.kc_out = o;
    x.vc_out = o + part[0][1] + part[1][1];
    x.vm_out = x.vc_out + part[2][1];
    x.kc = (uint32_t)lay.kc; x.vc = (uint32_t)lay.vc; x.vm = (uint32_t)lay.vm;
    x.bk = c->bk[seq]; x.bv = c->bv[seq]; x.gv = c->d.value_group; x.nblocks = (int32_t)(Lq / 32);
    const int e = kvq::launch_export(x, stream);
    if (e) return hip_fail(e, "export launch");
    o += part[0][1] + part[1][1] + part[2][1] + part[3][1];
  } else {
    for (auto& p : part) {
      if (p[1] == 0) continue;
      const hipError_t e = hipMemcpyAsync(o, blk + p[0], p[1], hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "export copy");
      o += p[1];
    }
  }
  const size_t W = c->W, n = L - Lq, first = Lq % W;
  for (uint64_t ring : {lay.tk, lay.tv}) {
    const size_t a1 = std::min(n, W - first), a2 = n - a1;
    if (a1) {
      const hipError_t e = hipMemcpyAsync(o, blk + ring + first * D * 2, a1 * D * 2, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "export copy");
      o += a1 * D * 2;
    }
    if (a2) {
      const hipError_t e = hipMemcpyAsync(o, blk + ring, a2 * D * 2, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "export copy");
      o += a2 * D * 2;
    }
  }
  return ok();
}

kvq_status kvq_check(const kvq_cache* c, void* stream) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  uint32_t flag = 0;
  e = hipMemcpy(&flag, c->arena, sizeof flag, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "read error flag");
  if (flag == (uint32_t)KVQ_ERR_RANGE)
    return fail(KVQ_ERR_RANGE, "an append met a non-finite input or a group range beyond the fp16 scale");
  return ok();
}

kvq_status kvq_set_split_tokens(kvq_cache* c, int32_t tokens) {
  if (!c) return fail(KVQ_ERR_ARG, "cache is NULL");
  if (tokens < 0 || (tokens > 0 && tokens % c->d.key_group != 0))
    return fail(KVQ_ERR_ARG, "split tokens %d must be 0 or a positive multiple of key_group %d", tokens,
                c->d.key_group);
  if (tokens > 0 && (c->cq + tokens - 1) / tokens > kMaxSplits)
    return fail(KVQ_ERR_ARG, "split tokens %d would give more than %d splits at capacity", tokens, kMaxSplits);
  c->split_tokens = tokens;
  return ok();
}

// ------------------------------------------------------------------ DGAP

size_t dgap_workspace_bytes(int32_t batch, int32_t vocab, int32_t k) {
  if (batch < 1 || k < DGAP_MIN_K || k > DGAP_MAX_K || vocab < k || vocab > (1 << 24)) return 0;
  const int64_t nchunk = (vocab + kvq::kDgapChunk - 1) / kvq::kDgapChunk;
  if (nchunk * k > kvq::kDgapMaxCandidates) return 0;
  const uint64_t stats = ((uint64_t)batch * nchunk * 4 * sizeof(float) + kvq::kAlign - 1) / kvq::kAlign * kvq::kAlign;
  return (size_t)(stats + (uint64_t)batch * nchunk * k * sizeof(uint64_t));
}

size_t dgap_info_floats(int32_t k) { return (size_t)kvq::kDgapInfoHead + 2 * (size_t)(k > 0 ? k : 0); }

kvq_status dgap_restore(const dgap_params* p, float* logits, int32_t batch, void* ws, size_t ws_bytes, float* info,
                        void* stream) {
  if (!p) return fail(KVQ_ERR_ARG, "params is NULL");
  if (batch < 1) return fail(KVQ_ERR_ARG, "batch must be >= 1 (got %d)", batch);
  if (p->k < DGAP_MIN_K || p->k > DGAP_MAX_K)
    return fail(KVQ_ERR_ARG, "k = %d outside [%d, %d]", p->k, DGAP_MIN_K, DGAP_MAX_K);
  if (p->vocab < p->k) return fail(KVQ_ERR_ARG, "vocab %d smaller than k %d", p->vocab, p->k);
  if (p->hidden_det < 1 || p->hidden_det > DGAP_MAX_HIDDEN || p->hidden_corr < 1 || p->hidden_corr > DGAP_MAX_HIDDEN)
    return fail(KVQ_ERR_ARG, "hidden sizes (%d, %d) outside [1, %d]", p->hidden_det, p->hidden_corr, DGAP_MAX_HIDDEN);
  if (!(p->tau == p->tau)) return fail(KVQ_ERR_ARG, "tau is NaN");
  if (!p->det_w1 || !p->det_b1 || !p->det_w2 || !p->corr_w1 || !p->corr_b1 || !p->corr_w2)
    return fail(KVQ_ERR_ARG, "a weight pointer is NULL");
  if (!logits) return fail(KVQ_ERR_ARG, "logits is NULL");
  const size_t need = dgap_workspace_bytes(batch, p->vocab, p->k);
  if (need == 0)
    return fail(KVQ_ERR_UNSUPPORTED, "vocab %d with k %d: at most 2^24 logits and %d window candidates per row",
                p->vocab, p->k, kvq::kDgapMaxCandidates);
  if (!ws) return fail(KVQ_ERR_ARG, "workspace is NULL");
  if (ws_bytes < need) return fail(KVQ_ERR_CAPACITY, "workspace holds %zu bytes, this call needs %zu", ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 16 != 0) return fail(KVQ_ERR_ARG, "workspace must be 16-byte aligned");
  kvq::DgapArgs a{};
  a.logits = logits;
  a.info = info;
  a.vocab = p->vocab;
  a.k = p->k;
  a.nchunk = (p->vocab + kvq::kDgapChunk - 1) / kvq::kDgapChunk;
  a.hidden_det = p->hidden_det;
  a.hidden_corr = p->hidden_corr;
  a.tau = p->tau;
  a.det_b2 = p->det_b2;
  a.corr_b2 = p->corr_b2;
  a.det_w1 = p->det_w1; a.det_b1 = p->det_b1; a.det_w2 = p->det_w2;
  a.corr_w1 = p->corr_w1; a.corr_b1 = p->corr_b1; a.corr_w2 = p->corr_w2;
  const uint64_t stats = ((uint64_t)batch * a.nchunk * 4 * sizeof(float) + kvq::kAlign - 1) / kvq::kAlign * kvq::kAlign;
  a.ws_stats = static_cast<float*>(ws);
  a.ws_cand = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + stats);
  const int e = kvq::launch_dgap(a, batch, stream);
  if (e) return hip_fail(e, "dgap launch");
  return ok();
}

const char* kvq_last_error(void) { return g_err.c_str(); }

kvq_status kvq_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (!src || !sink) return fail(KVQ_ERR_ARG, "src and sink must be device pointers");
  if (bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16 != 0)
    return fail(KVQ_ERR_ARG, "src must be 16-byte aligned and bytes a multiple of 16");
  const int e = kvq::launch_read_probe(src, bytes, sink, stream);
  if (e) return hip_fail(e, "read probe launch");
  return ok();
}

size_t kvq_read_probe_sink_bytes(void) { return (size_t)kvq::read_probe_blocks() * sizeof(uint32_t); }

const char* kvq_version(void) { return "kvq 0.1.0 gfx950"; }

}  // extern "C"
