// Host-side exercise of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer: the pool allocator, argument validation, work
// lists, table checks and trace layouts, with randomised inputs.  No kernel
// runs: the launchers are stubs.  Exits non-zero on the first failed check;
// the sanitizers abort on the first memory or undefined-behaviour error.
#include "paged_attn.h"

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

static int g_fail = 0;
#define CHECK(cond)                                                                        \
  do {                                                                                     \
    if (!(cond)) {                                                                         \
      std::fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__, #cond,         \
                   pa_last_error());                                                       \
      ++g_fail;                                                                            \
    }                                                                                      \
  } while (0)

static void* const kK = reinterpret_cast<void*>(0x10000);
static void* const kV = reinterpret_cast<void*>(0x20000);

static void allocator(std::mt19937& rng) {
  pa_kv_pool* p = nullptr;
  CHECK(kv_pool_create(0, 16, 8, 128, kK, kV, &p) == PA_EINVAL && !p);
  CHECK(kv_pool_create(64, 16, 8, 96, kK, kV, &p) == PA_EUNSUPPORTED);
  CHECK(kv_pool_create(64, 16, 8, 128, kK, kV, &p) == PA_OK && p);
  std::vector<int32_t> held;
  std::vector<int32_t> count(64, 0);
  for (int it = 0; it < 4000; ++it) {
    const int op = rng() % 4;
    int32_t nfree = 0;
    CHECK(kv_pool_num_free(p, &nfree) == PA_OK);
    if (op == 0) {
      const int32_t n = rng() % 9;
      std::vector<int32_t> ids(n + 1, -1);
      const int rc = kv_pool_alloc(p, n, ids.data());
      if (n > nfree) {
        CHECK(rc == PA_ENOMEM);
      } else {
        CHECK(rc == PA_OK);
        for (int i = 0; i < n; ++i) {
          CHECK(ids[i] >= 0 && ids[i] < 64 && count[ids[i]] == 0);
          if (ids[i] >= 0 && ids[i] < 64) count[ids[i]] = 1;
          held.push_back(ids[i]);
        }
      }
    } else if (op == 1 && !held.empty()) {
      const int32_t id = held[rng() % held.size()];
      CHECK(kv_pool_retain(p, 1, &id) == PA_OK);
      ++count[id];
      held.push_back(id);
    } else if (op == 2 && !held.empty()) {
      const size_t at = rng() % held.size();
      const int32_t id = held[at];
      CHECK(kv_pool_release(p, 1, &id) == PA_OK);
      --count[id];
      held.erase(held.begin() + at);
    } else {
      // state violations change nothing
      int32_t free_id = -1;
      for (int32_t i = 0; i < 64; ++i)
        if (count[i] == 0) { free_id = i; break; }
      if (free_id >= 0) {
        CHECK(kv_pool_release(p, 1, &free_id) == PA_ESTATE);
        CHECK(kv_pool_retain(p, 1, &free_id) == PA_ESTATE);
      }
      const int32_t bad[2] = {64, -1};
      CHECK(kv_pool_claim(p, 1, &bad[0]) == PA_EINVAL);
      CHECK(kv_pool_release(p, 1, &bad[1]) == PA_EINVAL);
    }
    for (int32_t i = 0; i < 64; i += 13) {
      int32_t c = -1;
      CHECK(kv_pool_refcount(p, i, &c) == PA_OK && c == count[i]);
    }
    int64_t shared = -1, expect = 0;
    for (int32_t i = 0; i < 64; ++i) expect += count[i] >= 2;
    CHECK(kv_pool_num_shared(p, &shared) == PA_OK && shared == expect);
  }
  int64_t strides[4], bytes = 0;
  CHECK(kv_pool_layout(p, strides, &bytes) == PA_OK && bytes == 64LL * 8 * 16 * 128 * 2);
  CHECK(kv_pool_destroy(p) == PA_OK);
  CHECK(kv_pool_destroy(nullptr) == PA_OK);
}

static void schedules(std::mt19937& rng) {
  for (int it = 0; it < 300; ++it) {
    const int32_t batch = rng() % 40;
    const int32_t S = 16 * (1 + rng() % 64);
    const int32_t max_ctx = 1 + rng() % 5000;
    const int32_t prefix = (rng() % 3 == 0) ? 16 * (rng() % (max_ctx / 16 + 1)) : 0;
    std::vector<int32_t> ctx(batch + 1);
    for (auto& c : ctx) c = (int32_t)(rng() % (max_ctx + 40)) - 20;   // some out of range
    const int64_t parts = prefix ? (max_ctx - prefix + S - 1) / S : (max_ctx + S - 1) / S;
    std::vector<int32_t> items((size_t)std::max<int64_t>(1, parts * batch) + 1, -1);
    int32_t n = -1;
    const int rc = paged_attn_schedule(ctx.data(), batch, max_ctx, S, prefix, items.data(),
                                       (int32_t)items.size() - 1, &n);
    CHECK(rc == PA_OK);
    if (rc != PA_OK) continue;
    CHECK(n >= 0 && n <= (int32_t)items.size() - 1 && items[items.size() - 1] == -1);
    std::vector<char> seen((size_t)std::max<int64_t>(1, parts * batch + 1), 0);
    for (int i = 0; i < n; ++i) {
      CHECK(items[i] >= 0 && items[i] < std::max<int64_t>(1, parts * batch));
      if (items[i] >= 0 && items[i] < (int64_t)seen.size()) {
        CHECK(!seen[items[i]]);
        seen[items[i]] = 1;
      }
    }
    // too small a list is an error that still reports the size
    if (n > 0) {
      int32_t m = -1;
      CHECK(paged_attn_schedule(ctx.data(), batch, max_ctx, S, prefix, items.data(), n - 1, &m) ==
                PA_EINVAL && m == n);
    }
  }
}

static void tables(std::mt19937& rng) {
  pa_kv_pool* p = nullptr;
  CHECK(kv_pool_create(200, 16, 8, 128, kK, kV, &p) == PA_OK);
  for (int it = 0; it < 300; ++it) {
    const int32_t batch = 1 + rng() % 12, stride = 1 + rng() % 20;
    const int32_t prefix = 16 * (rng() % (stride + 1));
    std::vector<int32_t> bt((size_t)batch * stride), ctx(batch);
    for (int32_t j = 0; j < stride; ++j) bt[j] = rng() % 200;
    for (int32_t b = 0; b < batch; ++b) {
      ctx[b] = rng() % (16 * stride + 1);
      for (int32_t j = 0; j < stride; ++j)
        bt[(size_t)b * stride + j] = (16 * j < prefix) ? bt[j] : (int32_t)(rng() % 200);
    }
    int32_t bad = 0;
    CHECK(paged_attn_check_tables(p, bt.data(), stride, ctx.data(), batch, prefix, nullptr, 0, 0,
                                  &bad) == PA_OK && bad == -1);
    if (batch > 1 && prefix > 0) {
      const int32_t b = 1 + rng() % (batch - 1);
      const int32_t j = rng() % (prefix / 16);
      bt[(size_t)b * stride + j] = (bt[j] + 1) % 200;
      const bool reads = 16 * j < std::min(ctx[b], prefix);
      const int rc = paged_attn_check_tables(p, bt.data(), stride, ctx.data(), batch, prefix,
                                             nullptr, 0, 0, &bad);
      CHECK(reads ? (rc == PA_EINVAL && bad == b) : rc == PA_OK);
    }
  }
  CHECK(kv_pool_destroy(p) == PA_OK);
}

static void validation() {
  pa_kv_pool* p = nullptr;
  CHECK(kv_pool_create(10, 16, 8, 128, kK, kV, &p) == PA_OK);
  void* q = reinterpret_cast<void*>(0x30000);
  const int32_t* bt = reinterpret_cast<const int32_t*>(0x40000);
  const int32_t* ctx = reinterpret_cast<const int32_t*>(0x50000);
  void* out = reinterpret_cast<void*>(0x60000);
  float* po = reinterpret_cast<float*>(0x70000);
  float* pl = reinterpret_cast<float*>(0x80000);
  CHECK(paged_attn_decode(p, q, bt, 8, ctx, 2, 24, 0.1f, 128, 0, out, nullptr, nullptr, nullptr) ==
        PA_EUNSUPPORTED);                                        // 3 query heads per KV head
  CHECK(paged_attn_decode(p, q, bt, 7, ctx, 2, 32, 0.1f, 128, 0, out, nullptr, nullptr, nullptr) ==
        PA_EINVAL);                                              // table too narrow
  CHECK(paged_attn_decode(p, q, bt, 8, ctx, 2, 32, 0.1f, 128, 64, out, nullptr, nullptr, nullptr) ==
        PA_EINVAL);                                              // split without partials
  CHECK(paged_attn_decode(p, q, bt, 8, ctx, 2, 32, 0.1f, 128, 64, out, po, pl, nullptr) == PA_EHIP);
  CHECK(paged_attn_decode(p, q, bt, 8, ctx, 0, 32, 0.1f, 128, 64, out, po, pl, nullptr) == PA_OK);
  int64_t lay[7];
  CHECK(paged_attn_cascade_trace_layout(p, 10, 32, 2300, 512, 2048, 512, 0, 0, lay) == PA_OK);
  CHECK(lay[6] == lay[4] + 3LL * 10 * 8 * 32);
  std::vector<int32_t> trace((size_t)lay[6]);
  CHECK(paged_attn_decode_cascade_trace(p, q, bt, 160, ctx, 10, 32, 0.1f, 2300, 512, 2048, 512,
                                        nullptr, 0, 0, 0, nullptr, 0, po, pl, trace.data(),
                                        lay[6] - 1, nullptr) == PA_EINVAL);
  CHECK(paged_attn_decode_cascade_trace(p, q, bt, 160, ctx, 10, 32, 0.1f, 2300, 512, 2048, 512,
                                        nullptr, 0, 0, 0, nullptr, 0, po, pl, trace.data(), lay[6],
                                        nullptr) == PA_EHIP);
  void* kn = reinterpret_cast<void*>(0x90000);
  void* vn = reinterpret_cast<void*>(0xa0000);
  CHECK(paged_attn_decode_append(p, q, nullptr, vn, bt, 8, ctx, 2, 32, 0.1f, 128, 64, nullptr, 0,
                                 out, po, pl, nullptr) == PA_EINVAL);   // k_new missing
  CHECK(paged_attn_decode_append(p, q, reinterpret_cast<char*>(kn) + 8, vn, bt, 8, ctx, 2, 32, 0.1f,
                                 128, 64, nullptr, 0, out, po, pl, nullptr) == PA_EINVAL);  // misaligned
  CHECK(paged_attn_decode_append(p, q, kn, vn, bt, 8, ctx, 2, 32, 0.1f, 128, 64, nullptr, 0, out, po,
                                 pl, nullptr) == PA_EHIP);
  CHECK(paged_attn_decode_cascade_append(p, q, kn, vn, bt, 160, ctx, 10, 32, 0.1f, 2300, 512, 2048,
                                         512, nullptr, 0, 0, -1, nullptr, 0, po, pl, nullptr) ==
        PA_EINVAL);                                                   // negative group_len
  CHECK(paged_attn_decode_cascade_append(p, q, kn, vn, bt, 160, ctx, 10, 32, 0.1f, 2300, 512, 2048,
                                         512, nullptr, 0, 0, 0, nullptr, 0, po, pl, nullptr) ==
        PA_EHIP);
  CHECK(paged_attn_reduce(po, pl, ctx, 2, 32, 128, 0, 4, out, nullptr) == PA_EINVAL);
  CHECK(paged_attn_extend(p, q, ctx, 10, bt, 600, ctx, 2, 32, 0.1f, 9000, 10, out, nullptr) ==
        PA_EUNSUPPORTED);
  CHECK(kv_pool_destroy(p) == PA_OK);
}

int main() {
  std::mt19937 rng(2510);
  allocator(rng);
  schedules(rng);
  tables(rng);
  validation();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host ABI checks passed\n");
  return 0;
}
