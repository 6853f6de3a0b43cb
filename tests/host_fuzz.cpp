// Host-only fuzz of bridger_forest_create_ex and the query entry points: random valid forests
// (perfect and ragged shapes, vector leaves, infinite thresholds) and corrupted ones (children
// out of range, cycles, features out of range, NaN thresholds, bad tree offsets and classes),
// each created on a host-only handle and, when accepted, queried and destroyed.  Built with
// AddressSanitizer and UndefinedBehaviorSanitizer on the host code by tests/test_host_fuzz.py;
// no device is touched.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>
#include "bridger.h"

int main(int argc, char **argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  std::mt19937_64 rng(12345);
  auto U = [&](int lo, int hi) { return (int)(lo + rng() % (uint64_t)(hi - lo + 1)); };
  int ok = 0, bad = 0;
  for (int it = 0; it < iters; ++it) {
    const int T = U(1, 6), F = U(1, 40), K = U(1, 5);
    std::vector<int64_t> offs(T + 1, 0);
    std::vector<int32_t> feat, left, right, tc;
    std::vector<float> thr, val;
    const bool vec = U(0, 3) == 0;
    for (int t = 0; t < T; ++t) {
      // a random valid tree (BFS ids), then maybe corrupt it
      const int n_int = U(0, 20);
      const int n = 2 * n_int + 1;
      std::vector<int> l(n, -1), r(n, -1);
      int next = 1;
      std::vector<int> q{0};
      for (size_t qi = 0; qi < q.size() && next + 1 < n + 1 && next < n; ++qi) {
        if (next + 1 >= n + 1) break;
        l[q[qi]] = next; r[q[qi]] = next + 1;
        q.push_back(next); q.push_back(next + 1);
        next += 2;
      }
      const int nn = next;
      offs[t + 1] = offs[t] + nn;
      for (int i = 0; i < nn; ++i) {
        feat.push_back(U(0, F - 1));
        float th = (float)(rng() % 1000) / 100.0f - 5.0f;
        if (U(0, 50) == 0) th = INFINITY;
        thr.push_back(th);
        left.push_back(l[i]); right.push_back(r[i]);
        for (int k = 0; k < (vec ? K : 1); ++k) val.push_back((float)(rng() % 100) / 10.0f);
      }
      tc.push_back(U(0, K - 1));
    }
    const int64_t N = offs[T];
    // corruptions
    const int c = U(0, 12);
    if (c == 1 && N > 0) left[U(0, (int)N - 1)] = U(-3, 60);
    if (c == 2 && N > 0) right[U(0, (int)N - 1)] = U(-3, 60);
    if (c == 3 && N > 0) feat[U(0, (int)N - 1)] = U(-5, F + 5);
    if (c == 4 && N > 0) thr[U(0, (int)N - 1)] = NAN;
    if (c == 5) offs[U(1, T)] -= U(0, 3);
    if (c == 6 && T > 0) tc[U(0, T - 1)] = U(-2, K + 2);
    const int agg = U(0, 2) == 0 ? 1 : 0;
    const int xf = U(0, 3) == 0 ? (K == 1 ? 1 : 2) : 0;
    std::vector<float> base(K);
    for (auto &b : base) b = (float)(rng() % 10);
    bridger_forest_t h = nullptr;
    uint32_t flags = BRIDGER_CREATE_HOST_ONLY | (vec ? BRIDGER_CREATE_VECTOR_LEAVES : 0u);
    // a corrupted offsets array can make N inconsistent with the arrays: only pass it when the
    // offsets stay within the arrays (the ABI cannot check array lengths)
    bool offs_ok = offs[0] == 0;
    for (int t = 0; t < T; ++t) offs_ok = offs_ok && offs[t + 1] >= offs[t] && offs[t + 1] <= N;
    if (!offs_ok) continue;
    bridger_status s = bridger_forest_create_ex(T, offs.data(), feat.data(), thr.data(), left.data(),
                                                right.data(), val.data(), F, K,
                                                (vec || U(0, 1)) ? nullptr : tc.data(), agg, xf,
                                                U(0, 1) ? base.data() : nullptr, flags, &h);
    if (s == BRIDGER_OK) {
      ++ok;
      int32_t a, b2, c2, d, e;
      bridger_forest_info(h, &a, &b2, &c2, &d, &e);
      int32_t rpw, cb, tpc, nc, lds;
      double hb, sb, lb;
      bridger_forest_plan(h, U(0, 100000), &rpw, &cb, &tpc, &nc, &lds, &hb, &sb, &lb);
      int32_t bb; int64_t nt;
      bridger_forest_bin_info(h, &bb, &nt);
      for (int which = 0; which < 8; ++which) {
        const void *p = nullptr; int64_t bytes = 0;
        bridger_forest_packed(h, which, &p, &bytes);
        volatile uint8_t sink = 0;
        for (int64_t i = 0; i < bytes; i += 97) sink ^= ((const uint8_t *)p)[i];
      }
      for (int k = 0; k < 6; ++k) bridger_forest_set_kernel(h, k);
      double pa[64], pb[64];
      for (int i = 0; i < 64; ++i) { pa[i] = 1.0; pb[i] = 2.0; }
      if (F <= 64) bridger_forest_set_preprocess(h, U(0, 5), pa, pb);
      bridger_forest_destroy(h);
    } else {
      ++bad;
      if (h) { printf("handle set on failure\n"); return 1; }
    }
  }
  printf("ok %d rejected %d\n", ok, bad);
  return 0;
}
