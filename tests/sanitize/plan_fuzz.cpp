// Host sanitizer driver: the planner's host mirror and the C-ABI argument
// checks over random shapes, every output buffer allocated at exactly the
// size the header states, so that AddressSanitizer sees any overrun and
// UndefinedBehaviorSanitizer any overflow or bad shift.  Each plan is also
// checked for coverage: every tile's pages are covered once, in order, by
// its units, and partial slots are distinct.  Prints "ok <plans>" on success.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <memory>
#include <random>
#include <vector>

#include "splash_attn.h"

namespace {

int fails = 0;
#define EXPECT(c)                                                        \
  do {                                                                   \
    if (!(c)) {                                                          \
      std::fprintf(stderr, "FAILED %s at line %d\n", #c, __LINE__);      \
      ++fails;                                                           \
    }                                                                    \
  } while (0)

splash_mla_desc desc_for(int B, int H, int max_pages, int num_pages) {
  splash_mla_desc d = {};
  d.batch = B;
  d.num_heads = H;
  d.dim_qk = 576;
  d.dim_v = 512;
  d.page_size = 64;
  d.max_pages_per_seq = max_pages;
  d.num_pages = num_pages;
  d.kv_dtype = SPLASH_KV_BF16;
  d.softmax_scale = 0.0721687823f;
  return d;
}

}  // namespace

int main(int argc, char** argv) {
  const int plans = argc > 1 ? std::atoi(argv[1]) : 400;
  std::mt19937 rng(12345);
  auto uni = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int done = 0;
  for (int it = 0; it < plans; ++it) {
    const int B = uni(0, 1 << uni(0, 11));      // up to 2048 requests
    const int q = uni(1, 8);
    const int H = 16 * uni(1, 8);
    const int kind = uni(0, 2);
    std::vector<int32_t> lens(std::max(B, 1));
    int mx = q;
    for (int b = 0; b < B; ++b) {
      int s;
      if (kind == 0) s = uni(q, 4096);
      else if (kind == 1) s = uni(q, 1 << uni(7, 18));  // up to 262,144 keys
      else s = uni(0, 9) == 0 ? uni(65536, 200000) : uni(q, 300);
      lens[b] = s;
      mx = std::max(mx, s);
    }
    const int max_pages = (mx + 63) / 64;
    const splash_mla_desc d = desc_for(B, H, max_pages, 1 << 20);
    const int T = B * q;
    const int max_partials = uni(0, 3) == 0 ? 0 : uni(1, 4096);
    const int G = uni(1, 1024);
    const int max_units = splash_mla_max_units(B, q, max_partials);
    std::unique_ptr<int32_t[]> units(new int32_t[(size_t)std::max(max_units, 1) * 4]);
    std::unique_ptr<int32_t[]> indptr(new int32_t[T + 1]);
    std::unique_ptr<int32_t[]> worker(new int32_t[G + 1]);
    int32_t stats[7];
    const int st = splash_mla_plan_host(lens.data(), q, &d, G, max_partials, units.get(), max_units, indptr.get(),
                                        stats, worker.get());
    if (st == SPLASH_ERR_WORKSPACE_TOO_SMALL) continue;  // a history beyond what the partials can hold
    EXPECT(st == SPLASH_OK);
    if (st != SPLASH_OK) {
      std::fprintf(stderr, "  B=%d q=%d H=%d G=%d max_partials=%d: %s\n", B, q, H, G, max_partials,
                   splash_last_error());
      continue;
    }
    ++done;
    // coverage: each tile's units tile [0, pages) in order; slots distinct
    std::vector<int> next(T, 0), seen_slot((size_t)stats[1] + 1, 0);
    for (int u = 0; u < stats[0]; ++u) {
      const int32_t* r = units.get() + 4 * u;
      EXPECT(r[0] >= 0 && r[0] < T);
      if (r[0] < 0 || r[0] >= T) continue;
      EXPECT(r[1] < r[2]);
      if (r[3] >= 0) {
        EXPECT(r[3] < stats[1]);
        if (r[3] >= 0 && r[3] < stats[1]) seen_slot[r[3]]++;
      }
    }
    for (int s = 0; s < stats[1]; ++s) EXPECT(seen_slot[s] == 1);
    std::vector<std::vector<std::pair<int, int>>> per(T);
    for (int u = 0; u < stats[0]; ++u) {
      const int32_t* r = units.get() + 4 * u;
      if (r[0] >= 0 && r[0] < T) per[r[0]].push_back({r[1], r[2]});
    }
    for (int t = 0; t < T; ++t) {
      const int b = t / q, i = t - b * q;
      const int L = lens[b] - q + i + 1;
      const int pages = L > 0 ? (L + 63) / 64 : 0;
      std::sort(per[t].begin(), per[t].end());
      int at = 0;
      for (auto& pr : per[t]) {
        EXPECT(pr.first == at);
        at = pr.second;
      }
      EXPECT(at == pages);
      EXPECT(indptr[t] <= indptr[t + 1]);
    }
    (void)next;
  }
  // C-ABI argument checks: all return before any HIP call
  splash_mla_desc bad = desc_for(4, 16, 8, 24);
  bad.dim_qk = 512;
  EXPECT(splash_mla_attend((void*)16, (void*)16, (int32_t*)16, (int32_t*)16, 1, (void*)16, (float*)16, &bad,
                           (void*)16, 1 << 20, nullptr) == SPLASH_ERR_INVALID_ARGUMENT);
  splash_mla_desc good = desc_for(4, 16, 8, 24);
  EXPECT(splash_mla_attend((void*)17, (void*)16, (int32_t*)16, (int32_t*)16, 1, (void*)16, (float*)16, &good,
                           (void*)16, 1 << 20, nullptr) == SPLASH_ERR_MISALIGNED);
  EXPECT(splash_mla_attend((void*)16, (void*)16, (int32_t*)16, (int32_t*)16, 0, (void*)16, (float*)16, &good,
                           (void*)16, 1 << 20, nullptr) == SPLASH_ERR_INVALID_ARGUMENT);
  EXPECT(splash_mla_workspace_size(1 << 20, 8, 128, 0) > 0);
  // a batch whose forced partials exceed the no-allocation scratch is
  // refused before the scratch is looked up
  const splash_mla_desc huge = desc_for(600, 128, 2000, 1 << 20);
  EXPECT(splash_mla_attend_noalloc((void*)16, (void*)16, (int32_t*)16, (int32_t*)16, 1, (void*)16, (float*)16,
                                   &huge, nullptr) == SPLASH_ERR_WORKSPACE_TOO_SMALL);
  if (fails) return 1;
  std::printf("ok %d\n", done);
  return 0;
}
