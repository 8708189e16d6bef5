// Runs every oracle entry point on small seeded inputs (ragged blocks, GQA,
// causal and not, listed-row and compact layouts, clamping, empty lists), for
// a build with AddressSanitizer and UndefinedBehaviorSanitizer: any invalid
// access or undefined operation aborts the process.  Prints "ok" at the end.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

extern "C" {
int ora_bf16_round(const double*, int64_t, uint16_t*);
int ora_pool(const uint16_t*, int64_t, int64_t, int64_t, int64_t, int32_t, uint16_t*, int32_t);
int ora_pooled_scores(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t, int64_t, int64_t,
                      int32_t, int32_t, int64_t, int64_t, int64_t, double*, int64_t*);
int ora_pooled_scores_rows(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t, int64_t,
                           int64_t, int32_t, int32_t, const int64_t*, int64_t, double*, int32_t);
int64_t ora_topk_count(double, int64_t);
int ora_select(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t, int64_t, int64_t, int32_t,
               int32_t, int32_t, double, int64_t, int32_t*, int32_t*, int64_t*, const int64_t*,
               int64_t, int32_t, int32_t);
int ora_select_mins_tiled(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t, int64_t,
                          int64_t, int32_t, int32_t, double, int64_t, int64_t, int64_t, int32_t*,
                          int32_t*, int64_t*, const int64_t*, int64_t, int32_t, int32_t);
int ora_mins_progressive_row(const double*, int64_t, double, int64_t, int64_t, int32_t*, int64_t*);
int ora_sparse_attn(const uint16_t*, const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t,
                    int64_t, int64_t, int32_t, int32_t, double, const int32_t*, int64_t,
                    const int32_t*, double*, double*, const int64_t*, int64_t, int32_t, int32_t);
int ora_dense_attn(const uint16_t*, const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t,
                   int64_t, int64_t, int32_t, double, double*, double*, int32_t);
int ora_kept_mass(const uint16_t*, const uint16_t*, int64_t, int64_t, int64_t, int64_t, int64_t,
                  int32_t, int32_t, double, const int32_t*, int64_t, const int32_t*, double*,
                  const int64_t*, int64_t, int32_t);
int ora_sparse_attn_online(const uint16_t*, const uint16_t*, const uint16_t*, int64_t, int64_t,
                           int64_t, int64_t, int64_t, int32_t, int32_t, double, const int32_t*,
                           int64_t, const int32_t*, int32_t, double*, double*, int32_t);
}

static int failures = 0;
static void expect(bool ok, const char* what) {
  if (!ok) {
    std::printf("FAILED: %s\n", what);
    ++failures;
  }
}

int main() {
  std::mt19937_64 rng(7);
  std::normal_distribution<double> nd(0.0, 1.0);
  const int64_t B = 1, Hq = 4, Hkv = 2, N = 150, D = 16;
  auto bits = [&](int64_t n) {
    std::vector<double> x(n);
    for (auto& v : x) v = nd(rng);
    std::vector<uint16_t> b(n);
    expect(ora_bf16_round(x.data(), n, b.data()) == 0, "bf16_round");
    return b;
  };
  std::vector<uint16_t> q = bits(B * Hq * N * D), k = bits(B * Hkv * N * D), v = bits(B * Hkv * N * D);
  for (int32_t P : {1, 16, 64, 200}) {
    const int64_t Np = (N + P - 1) / P;
    std::vector<uint16_t> qp(B * Hq * Np * D);
    expect(ora_pool(q.data(), B, Hq, N, D, P, qp.data(), 2) == 0, "pool");
    for (int32_t causal : {0, 1}) {
      std::vector<double> sc(N);
      int64_t L = 0;
      expect(ora_pooled_scores(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, 0, 3, Np - 1,
                               sc.data(), &L) == 0, "pooled_scores");
      std::vector<int64_t> rows = {0, Np - 1, B * Hq * Np - 1};
      std::vector<double> scr(rows.size() * N);
      expect(ora_pooled_scores_rows(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, rows.data(),
                                    rows.size(), scr.data(), 2) == 0, "pooled_scores_rows");
      const int64_t cap = N;
      std::vector<int32_t> idx(B * Hq * Np * cap), cnt(B * Hq * Np);
      for (int32_t mode : {0, 1, 2}) {
        for (double prm : {0.05, 0.5, 1.0}) {
          int64_t ncl = 0;
          const double pm = mode == 2 ? prm * 2.0 : prm;
          expect(ora_select(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, mode, pm, cap, idx.data(),
                            cnt.data(), &ncl, nullptr, 0, 0, 2) == 0, "select");
          std::vector<int32_t> ci(rows.size() * 7), cc(rows.size());
          const int rc = ora_select(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, mode, pm, 7,
                                    ci.data(), cc.data(), &ncl, rows.data(), rows.size(), 1, 2);
          expect(rc == 0 || (mode == 0 && rc == 3), "select compact, small cap");
        }
      }
      int64_t ncl = 0;
      expect(ora_select_mins_tiled(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, 0.3, 16, 4, 9,
                                   idx.data(), cnt.data(), &ncl, nullptr, 0, 0, 2) == 0, "mins_tiled");
      // attention on the last topK lists, with an empty list in block 0
      expect(ora_select(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, 0, 0.3, cap, idx.data(),
                        cnt.data(), &ncl, nullptr, 0, 0, 2) == 0, "select for attention");
      cnt[0] = 0;
      std::vector<double> o(B * Hq * N * D), lse(B * Hq * N), kept(B * Hq * N);
      expect(ora_sparse_attn(q.data(), k.data(), v.data(), B, Hq, Hkv, N, D, P, causal, 0.0, idx.data(),
                             cap, cnt.data(), o.data(), lse.data(), nullptr, 0, 0, 2) == 0, "sparse_attn");
      std::vector<double> oc(rows.size() * P * D), lc(rows.size() * P);
      std::vector<int32_t> ri(rows.size() * cap), rcn(rows.size());
      for (size_t t = 0; t < rows.size(); ++t) {
        rcn[t] = cnt[rows[t]];
        for (int64_t c = 0; c < cap; ++c) ri[t * cap + c] = idx[rows[t] * cap + c];
      }
      expect(ora_sparse_attn(q.data(), k.data(), v.data(), B, Hq, Hkv, N, D, P, causal, 0.0, ri.data(),
                             cap, rcn.data(), oc.data(), lc.data(), rows.data(), rows.size(), 1, 2) == 0,
             "sparse_attn compact");
      expect(ora_sparse_attn_online(q.data(), k.data(), v.data(), B, Hq, Hkv, N, D, P, causal, 0.0,
                                    idx.data(), cap, cnt.data(), 5, o.data(), lse.data(), 2) == 0,
             "sparse_attn_online");
      expect(ora_kept_mass(q.data(), k.data(), B, Hq, Hkv, N, D, P, causal, 0.0, idx.data(), cap,
                           cnt.data(), kept.data(), nullptr, 0, 2) == 0, "kept_mass");
      expect(ora_dense_attn(q.data(), k.data(), v.data(), B, Hq, Hkv, N, D, causal, 0.0, o.data(),
                            lse.data(), 2) == 0, "dense_attn");
    }
  }
  std::vector<double> s(300);
  for (auto& x : s) x = nd(rng);
  std::vector<int32_t> out(300);
  int64_t n = 0;
  expect(ora_mins_progressive_row(s.data(), 300, 0.5, 16, 4, out.data(), &n) == 0, "mins_progressive");
  expect(ora_topk_count(0.15, 75600) == 11340, "topk_count");
  // rejected arguments return an error without touching the buffers
  expect(ora_select(q.data(), k.data(), B, Hq, 3, N, D, 16, 0, 0, 0.5, 10, nullptr, nullptr, nullptr,
                    nullptr, 0, 0, 1) != 0, "select rejects");
  expect(ora_sparse_attn(q.data(), k.data(), v.data(), B, Hq, Hkv, N, D, 0, 0, 0.0, nullptr, 1, nullptr,
                         nullptr, nullptr, nullptr, 0, 0, 1) != 0, "sparse_attn rejects");
  std::printf(failures ? "failures: %d\n" : "ok\n", failures);
  return failures ? 1 : 0;
}
