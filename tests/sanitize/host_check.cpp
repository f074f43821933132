// Drives the library's host code (argument checks, length bookkeeping, page
// lists, split plans, export offsets) through the C ABI with host buffers
// standing in for device memory, under AddressSanitizer and UBSan.  Every
// status is checked; "host checks ok" on success.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "dgap.h"
#include "kvq.h"

extern int g_launches;
extern int g_row_plans;

static int g_fail = 0;
#define EXPECT(cond)                                                    \
  do {                                                                  \
    if (!(cond)) {                                                      \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, kvq_last_error()); \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

struct Buf {  // 256-byte aligned host buffer
  void* p = nullptr;
  size_t n = 0;
  explicit Buf(size_t bytes) : n(bytes) {
    p = std::aligned_alloc(256, (bytes + 255) / 256 * 256 + 256);
    std::memset(p, 0, (bytes + 255) / 256 * 256 + 256);
  }
  ~Buf() { std::free(p); }
  template <class T> T* as() { return static_cast<T*>(p); }
};

static kvq_cache_desc desc(int batch, int hq, int hkv, int maxt, int gk, int gv, int R, const uint8_t* bk,
                           const uint8_t* bv, int P = 0, int pages = 0) {
  kvq_cache_desc d{};
  d.batch = batch; d.num_q_heads = hq; d.num_kv_heads = hkv; d.head_dim = 128; d.max_tokens = maxt;
  d.key_group = gk; d.value_group = gv; d.fp16_window = R; d.bits_k = bk; d.bits_v = bv;
  d.page_tokens = P; d.num_pages = pages;
  return d;
}

// One cache through every call: appends in ragged pieces, decodes, chunk
// queries, exports of every (sequence, head), dequantization, release, reset.
static void exercise(const kvq_cache_desc& d) {
  const size_t bytes = kvq_cache_bytes(&d);
  EXPECT(bytes > 0);
  Buf arena(bytes);
  kvq_cache* c = nullptr;
  EXPECT(kvq_cache_init(&c, &d, arena.p, bytes) == KVQ_OK);
  if (!c) return;
  kvq_cache* small = nullptr;
  EXPECT(kvq_cache_init(&small, &d, arena.p, bytes - 1) != KVQ_OK && small == nullptr);
  const int B = d.batch, H = d.num_kv_heads, Hq = d.num_q_heads, T = d.max_tokens;
  const int n_max = 97;
  Buf K((size_t)B * n_max * H * 128 * 2), V((size_t)B * n_max * H * 128 * 2);
  Buf q((size_t)B * 64 * Hq * 128 * 2), out((size_t)B * 64 * Hq * 128 * 4);
  std::vector<int32_t> n(B);
  int step = 0;
  for (; step < 1000; ) {
    bool any = false;
    for (int s = 0; s < B; ++s) {
      const int64_t L = kvq_seq_len(c, s);
      const int want = (step * 37 + s * 11) % n_max + 1;
      n[s] = (int)std::min<int64_t>(want, T - L - (s == 0 ? 3 : 0));
      if (n[s] < 0) n[s] = 0;
      any |= n[s] > 0;
    }
    if (!any || g_fail > 20) break;
    std::vector<int64_t> before(B);
    for (int s = 0; s < B; ++s) before[s] = kvq_seq_len(c, s);
    if (d.num_pages > 0) {
      const kvq_status st = kvq_append(c, K.p, V.p, n_max, n.data(), nullptr);
      if (st == KVQ_ERR_CAPACITY) {
        // a shared pool ran out: nothing changed; release the longest sequence
        int longest = 0;
        for (int s = 0; s < B; ++s) {
          EXPECT(kvq_seq_len(c, s) == before[s]);
          if (before[s] > before[longest]) longest = s;
        }
        const int64_t free0 = kvq_free_pages(c);
        EXPECT(kvq_seq_release(c, longest) == KVQ_OK);
        EXPECT(kvq_free_pages(c) > free0);
        ++step;
        continue;
      }
      EXPECT(st == KVQ_OK);
    } else {
      const kvq_status st = (step % 3 == 2)
                                ? kvq_append_decode(c, K.p, V.p, n_max, n.data(), q.p, out.as<float>(), nullptr, 0, nullptr)
                                : kvq_append(c, K.p, V.p, n_max, n.data(), nullptr);
      if (step % 3 == 2) {
        EXPECT(st != KVQ_OK);  // no workspace given: nothing changes
        for (int s = 0; s < B; ++s) EXPECT(kvq_seq_len(c, s) == before[s]);
        EXPECT(kvq_append(c, K.p, V.p, n_max, n.data(), nullptr) == KVQ_OK);
      } else {
        EXPECT(st == KVQ_OK);
      }
    }
    const size_t wsb = kvq_workspace_bytes(c);
    Buf ws(wsb + 16);
    EXPECT(kvq_decode_attention(c, q.p, out.as<float>(), ws.p, wsb, nullptr) == KVQ_OK);
    EXPECT(kvq_decode_attention(c, q.p, out.as<float>(), ws.p, 16, nullptr) == KVQ_ERR_CAPACITY);  // < one record
    EXPECT(kvq_decode_partials(c, q.p, ws.p, wsb, nullptr) == KVQ_OK);
    EXPECT(kvq_decode_merge(c, ws.p, out.as<float>(), nullptr) == KVQ_OK);
    EXPECT(kvq_decode_attention_noalloc(c, q.p, out.as<float>(), nullptr) == KVQ_OK);
    int64_t Lmin = T;
    for (int s = 0; s < B; ++s) Lmin = std::min<int64_t>(Lmin, kvq_seq_len(c, s));
    for (int nq : {1, 2, 3, 5, 7, 13, 33, 64}) {
      if (nq > Lmin) continue;
      const size_t cw = kvq_chunk_workspace_bytes(c, nq);
      Buf cws(cw + 16);
      EXPECT(kvq_chunk_attention(c, q.p, nq, out.as<float>(), cws.p, cw, nullptr) == KVQ_OK);
    }
    ++step;
  }
  for (int s = 0; s < B; ++s)
    for (int h = 0; h < H; ++h) {
      const size_t eb = kvq_export_bytes(c, s, h);
      Buf img(eb + 1);
      EXPECT(kvq_export(c, s, h, img.p, eb, nullptr) == KVQ_OK);
      if (eb > 0) EXPECT(kvq_export(c, s, h, img.p, eb - 1, nullptr) == KVQ_ERR_CAPACITY);
    }
  const int64_t L0 = kvq_seq_len(c, 0);
  Buf Ko((size_t)(L0 + 1) * H * 128 * 4), Vo((size_t)(L0 + 1) * H * 128 * 4);
  EXPECT(kvq_dequant(c, 0, 0, (int32_t)L0, Ko.as<float>(), Vo.as<float>(), nullptr) == KVQ_OK);
  EXPECT(kvq_dequant(c, 0, 1, (int32_t)L0, Ko.as<float>(), Vo.as<float>(), nullptr) != KVQ_OK);
  EXPECT(kvq_check(c, nullptr) == KVQ_OK);
  EXPECT(kvq_set_split_tokens(c, d.key_group * 4) == KVQ_OK);
  {
    const size_t wsb = kvq_workspace_bytes(c);
    Buf ws(wsb + 16);
    EXPECT(kvq_decode_attention(c, q.p, out.as<float>(), ws.p, wsb, nullptr) == KVQ_OK);
  }
  EXPECT(kvq_set_split_tokens(c, d.key_group + 1) == KVQ_ERR_ARG);
  if (B > 1) {
    EXPECT(kvq_seq_release(c, 1) == KVQ_OK);
    EXPECT(kvq_seq_len(c, 1) == 0);
  }
  EXPECT(kvq_seq_release(c, B) == KVQ_ERR_ARG);
  EXPECT(kvq_cache_reset(c, nullptr) == KVQ_OK);
  for (int s = 0; s < B; ++s) EXPECT(kvq_seq_len(c, s) == 0);
  kvq_cache_destroy(c);
}

int main() {
  const uint8_t b1[4] = {1, 1, 1, 1}, b2[4] = {2, 2, 2, 2}, mixk[4] = {1, 2, 4, 8}, mixv[4] = {2, 1, 8, 4},
                b4[4] = {4, 4, 4, 4}, b8[4] = {8, 8, 8, 8};
  // invalid descriptors: zero size, no launch
  {
    kvq_cache_desc d = desc(2, 32, 8, 100, 32, 32, 0, b1, b1);
    d.head_dim = 64;
    EXPECT(kvq_cache_bytes(&d) == 0);
    d = desc(2, 30, 8, 100, 32, 32, 0, b1, b1);
    EXPECT(kvq_cache_bytes(&d) == 0);
    d = desc(2, 32, 8, 100, 48, 32, 0, b1, b1);
    EXPECT(kvq_cache_bytes(&d) == 0);
    d = desc(2, 32, 8, 100, 32, 24, 0, b1, b1);
    EXPECT(kvq_cache_bytes(&d) == 0);
    const uint8_t bad[2] = {3, 1};
    d = desc(2, 32, 8, 100, 32, 32, 0, bad, b1);
    EXPECT(kvq_cache_bytes(&d) == 0);
    d = desc(2, 32, 8, 100, 32, 32, 0, b1, b1, 48);
    EXPECT(kvq_cache_bytes(&d) == 0);
    d = desc(2, 32, 8, 100, 32, 32, 0, mixk, mixv, 64);  // paged caches need one width pair
    EXPECT(kvq_cache_bytes(&d) == 0);
    EXPECT(kvq_cache_bytes(nullptr) == 0);
    kvq_cache* c = nullptr;
    EXPECT(kvq_cache_init(&c, nullptr, nullptr, 0) == KVQ_ERR_ARG);
  }
  exercise(desc(3, 32, 8, 700, 32, 32, 0, b1, b1));            // matrix layout, four heads
  exercise(desc(2, 40, 8, 500, 32, 32, 128, b2, b2));          // five heads, fp16 window
  exercise(desc(4, 32, 8, 400, 64, 32, 40, mixk, mixv));       // mixed widths, canonical layouts
  exercise(desc(2, 16, 8, 300, 32, 16, 0, b2, b1));            // two heads per kv head, small value groups
  exercise(desc(2, 64, 8, 600, 128, 64, 7, b4, b4));           // eight heads, key groups of 128
  exercise(desc(3, 32, 8, 900, 32, 32, 0, b8, b8, 64));        // paged
  exercise(desc(2, 32, 8, 800, 32, 32, 50, b1, b1, 128, 9));   // paged, shared pool smaller than capacity
  exercise(desc(1, 8, 8, 200, 32, 128, 0, b1, b1));            // one head per kv head
  // DGAP argument checks
  {
    EXPECT(dgap_workspace_bytes(1, 32768, 64) > 0);
    EXPECT(dgap_workspace_bytes(1, 32768, 4) == 0);
    dgap_params p{};
    p.vocab = 1000; p.k = 16; p.hidden_det = 8; p.hidden_corr = 8; p.tau = 0.6f;
    std::vector<float> w(4096, 0.f);
    p.det_w1 = p.det_b1 = p.det_w2 = p.corr_w1 = p.corr_b1 = p.corr_w2 = w.data();
    std::vector<float> logits(2 * 1000, 0.f);
    const size_t wsb = dgap_workspace_bytes(2, 1000, 16);
    Buf ws(wsb + 16);
    EXPECT(dgap_restore(&p, logits.data(), 2, ws.p, wsb, nullptr, nullptr) == KVQ_OK);
    EXPECT(dgap_restore(&p, logits.data(), 2, ws.p, wsb - 1, nullptr, nullptr) != KVQ_OK);
    EXPECT(dgap_restore(nullptr, logits.data(), 2, ws.p, wsb, nullptr, nullptr) == KVQ_ERR_ARG);
  }
  if (g_fail) {
    std::fprintf(stderr, "%d host checks failed\n", g_fail);
    return 1;
  }
  std::printf("host checks ok (%d launches, %d chunk row plans checked)\n", g_launches, g_row_plans);
  return 0;
}
