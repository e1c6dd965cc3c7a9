// Host-only checks of the C ABI: planning of every entry point over random
// shapes (ragged plans and their tables, pyramid schedules, workspace sizes)
// and the early argument errors.  No GPU work: built with AddressSanitizer on
// the host code by tests/test_host_asan.py.
#include <cstdio>
#include <cstdint>
#include <vector>
#include <random>
#include "grkv.h"
int main() {
  std::mt19937 rng(1);
  int bad = 0;
  for (int trial = 0; trial < 2000; ++trial) {
    const int U = 1 + rng() % 300, G = 1 + rng() % 4, w = 1 + rng() % 40;
    const int64_t n = w + 1 + rng() % 40000;
    grkv_problem pr{U, G, (rng() % 2) ? 128 : 64, (rng() % 4) ? GRKV_BF16 : GRKV_F32};
    std::vector<int32_t> b(U);
    for (auto& x : b) x = w + (int32_t)(rng() % (n - w + 1));
    if (rng() % 3 == 0) for (auto& x : b) x = b[0];
    const size_t ws = grkv_workspace_bytes_ragged(&pr, n, w, b.data());
    if ((int64_t)G * w <= 256 && ws == 0) ++bad;
    std::vector<int32_t> pb(U);
    const int layers = 1 + rng() % 40;
    std::vector<int32_t> pyr((size_t)layers * 8);
    const int mean = w + (int)(rng() % (n - w + 1));
    if (grkv_pyramid_budgets(layers, 8, mean, w, n, (rng() % 100) / 100.f, pyr.data()) != GRKV_OK) ++bad;
    for (int32_t x : pyr) if (x < w || x > n) ++bad;
  }
  for (int trial = 0; trial < 3000; ++trial) {
    const int U = 1 + rng() % 300, G = 1 + rng() % 9, w = 1 + rng() % 70;
    const int64_t n = w + (rng() % 50000);
    grkv_problem pr{U, G, (rng() % 3) ? 128 : ((rng() % 2) ? 64 : 96), (rng() % 4) ? GRKV_BF16 : GRKV_F32};
    const int c = w + (int)(rng() % (n - w + 2));   // sometimes above n
    const size_t a = grkv_workspace_bytes(&pr, n, w, c);
    grkv_layout lay;
    const int st = grkv_workspace_layout(&pr, n, w, c, &lay);
    if ((st == GRKV_OK) != (a != 0)) ++bad;
    if (st == GRKV_OK && lay.total != a) ++bad;
    const size_t k1 = grkv_workspace_bytes_kv(&pr, n, w, c, 1 + rng() % 4);
    if (k1 != 0 && k1 < a) ++bad;
    // pointer and argument errors return before any HIP call
    grkv_outputs o{};
    if (grkv_compress(nullptr, nullptr, nullptr, n, w, c, 7, 0.01f, nullptr, &pr, nullptr, &o) != GRKV_ERR_INVALID) ++bad;
  }
  // sum past 2^31 - 1
  grkv_problem pr{3, 4, 128, GRKV_BF16};
  int32_t big[3] = {1 << 30, 1 << 30, 1 << 30};
  if (grkv_workspace_bytes_ragged(&pr, (int64_t)1 << 30, 32, big) != 0) ++bad;
  std::printf("host checks done, bad = %d\n", bad);
  return bad != 0;
}
