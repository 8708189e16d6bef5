// Calls the C ABI's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer, without a GPU: every argument check of every
// entry point (with addresses that are never dereferenced), the host-side
// queries (max_count, workspace sizes over a range of shapes), and the
// per-head filter-ratio programme on random tables.  Calls with valid
// arguments reach the launch code and must fail with VECATTN_ERR_DEVICE (no
// device here).  Prints "ok" at the end.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "vecattn.h"

static int failures = 0;
static void expect(bool ok, const char* what) {
  if (!ok) {
    std::printf("FAILED: %s\n", what);
    ++failures;
  }
}

static vecattn_tdesc desc(int64_t B, int64_t H, int64_t N, int64_t D) {
  return vecattn_tdesc{B, H, N, D, H * N * D, N * D, D};
}

int main() {
  void* const fake = reinterpret_cast<void*>(uintptr_t(0x100000));
  int32_t* const ifake = static_cast<int32_t*>(fake);
  expect(vecattn_version() >= 100, "version");
  for (int s = 0; s < 6; ++s) expect(vecattn_status_string(static_cast<vecattn_status>(s)) != nullptr, "status");

  for (int64_t N : {int64_t(1), int64_t(63), int64_t(64), int64_t(1000), int64_t(75600), int64_t(1) << 30})
    for (int32_t P : {1, 64, 128, 1000})
      for (int32_t flags : {0, 1, 2, 3, 4, 7})
        for (int32_t mode : {0, 1, 2, 3}) {
          int64_t out = 0;
          const double prm = mode < 2 ? 0.3 : 1.5;
          expect(vecattn_select_max_count(N, P, flags, mode, prm, &out) == VECATTN_OK, "max_count");
          expect(out >= 1 && out <= N, "max_count range");
        }
  for (int64_t N : {int64_t(1), int64_t(100), int64_t(75600), int64_t(131072)}) {
    for (int64_t Hkv : {int64_t(1), int64_t(4), int64_t(40)}) {
      vecattn_tdesc q = desc(1, 40, N, 128), k = desc(1, Hkv, N, 128);
      size_t bytes = 0;
      const vecattn_status st = vecattn_select_workspace_size(&q, &k, 64, 0, 1, N, &bytes);
      expect(st == (40 % Hkv == 0 ? VECATTN_OK : VECATTN_ERR_INVALID_ARG), "workspace_size");
      expect(vecattn_select_workspace_bytes(&q, &k, 64, 1, N) == (st == VECATTN_OK ? bytes : 0),
             "workspace_bytes");
    }
  }

  // Argument errors: nothing is touched or launched.
  vecattn_tdesc q = desc(1, 4, 256, 128), k = desc(1, 2, 256, 128), bad = desc(1, 3, 256, 128);
  vecattn_tdesc d96 = desc(1, 4, 256, 96);
  expect(vecattn_select(nullptr, &q, fake, &k, 64, 0, 0, 0.25, ifake, 64, ifake, nullptr, fake,
                        1 << 30, nullptr) == VECATTN_ERR_INVALID_ARG, "select null");
  expect(vecattn_select(fake, &q, fake, &bad, 64, 0, 0, 0.25, ifake, 64, ifake, nullptr, fake,
                        1 << 30, nullptr) == VECATTN_ERR_INVALID_ARG, "select heads");
  expect(vecattn_select(fake, &d96, fake, &d96, 64, 0, 0, 0.25, ifake, 64, ifake, nullptr, fake,
                        1 << 30, nullptr) == VECATTN_ERR_UNSUPPORTED, "select D");
  expect(vecattn_select(fake, &q, fake, &k, 64, 0, 0, 0.25, ifake, 63, ifake, nullptr, fake,
                        1 << 30, nullptr) == VECATTN_ERR_CAPACITY, "select cap");
  expect(vecattn_select_noalloc(fake, &q, fake, &k, 64, 8, 0, 0.25, ifake, 64, ifake, nullptr,
                                nullptr) == VECATTN_ERR_INVALID_ARG, "noalloc bits");
  double params[4] = {0.1, 0.2, 0.3, 1.5};
  expect(vecattn_select_per_head(fake, &q, fake, &k, 64, 0, 0, params, 16, 16, ifake, 256, ifake,
                                 nullptr, fake, 1 << 30, nullptr) == VECATTN_ERR_INVALID_ARG,
         "per_head");
  expect(vecattn_select_mins_tiled(fake, &q, fake, &k, 64, 0, 0.5, 24, 16, ifake, 256, ifake,
                                   nullptr, fake, 1 << 30, nullptr) == VECATTN_ERR_INVALID_ARG,
         "mins_tiled tile");
  int64_t cu[3] = {0, 100, 200};
  expect(vecattn_select_varlen(fake, &q, fake, &k, cu, 2, 64, 0, 0, 0.25, ifake, 64, ifake, nullptr,
                               fake, 1 << 30, nullptr) == VECATTN_ERR_INVALID_ARG, "varlen end");
  vecattn_tdesc big = vecattn_tdesc{1, 40, (int64_t(1) << 24), 128, int64_t(40) << 31, int64_t(1) << 31,
                                    128};
  expect(vecattn_sparse_attn(fake, &big, fake, &big, fake, &big, ifake, 16, ifake, 64, 0, 0.0f, fake,
                             &big, nullptr, nullptr) == VECATTN_ERR_UNSUPPORTED, "attn offsets");
  expect(vecattn_sparse_attn(fake, &q, fake, &k, fake, &bad, ifake, 16, ifake, 64, 0, 0.0f, fake, &q,
                             nullptr, nullptr) == VECATTN_ERR_INVALID_ARG, "attn v");
  expect(vecattn_sparse_attn_varlen(fake, &q, fake, &k, fake, &k, cu, 2, ifake, 16, ifake, 64, 0, 0.0f,
                                    fake, &q, nullptr, nullptr) == VECATTN_ERR_INVALID_ARG,
         "attn varlen");
  expect(vecattn_check_lists(ifake, -1, 16, ifake, 256, ifake, nullptr) == VECATTN_ERR_INVALID_ARG,
         "check_lists");
  expect(vecattn_head_sparsity(nullptr, 1, 4, 256, 64, 0, static_cast<double*>(fake), nullptr) ==
             VECATTN_ERR_INVALID_ARG, "head_sparsity");
  expect(vecattn_recall(fake, &q, fake, &k, ifake, 0, ifake, 64, 0, 0.0f, static_cast<float*>(fake),
                        nullptr) == VECATTN_ERR_INVALID_ARG, "recall cap");
  vecattn_tdesc qp = desc(1, 4, 4, 128);
  expect(vecattn_pool(fake, &q, 0, fake, &qp, nullptr) == VECATTN_ERR_INVALID_ARG, "pool block");
  expect(vecattn_attn_order(ifake, 16, ifake, 1, 4, 256, 0, ifake, nullptr) ==
             VECATTN_ERR_INVALID_ARG, "order block");
  expect(vecattn_attn_order(ifake, 16, ifake, int64_t(1) << 20, 1 << 12, 256, 64, ifake, nullptr) ==
             VECATTN_ERR_INVALID_ARG, "order rows");
  expect(vecattn_sparse_attn_ordered(fake, &q, fake, &k, fake, &bad, ifake, 16, ifake, ifake, 64, 0,
                                     0.0f, fake, &q, nullptr, nullptr) == VECATTN_ERR_INVALID_ARG,
         "ordered attn v");

  // Valid arguments reach the launch code: without a device it reports DEVICE.
  std::vector<uint8_t> dummy(64);
  expect(vecattn_pool(fake, &q, 64, fake, &qp, nullptr) == VECATTN_ERR_DEVICE, "pool launch");
  expect(vecattn_sparse_attn(fake, &q, fake, &k, fake, &k, ifake, 16, ifake, 64, 1, 0.0f, fake, &q,
                             nullptr, nullptr) == VECATTN_ERR_DEVICE, "attn launch");
  expect(vecattn_select_noalloc(fake, &q, fake, &k, 64, 0, 0, 0.25, ifake, 64, ifake, nullptr,
                                nullptr) == VECATTN_ERR_DEVICE, "noalloc launch");
  expect(vecattn_attn_order(ifake, 16, ifake, 1, 4, 256, 64, ifake, nullptr) == VECATTN_ERR_DEVICE,
         "order launch");

  // Eq. 5's programme on random tables.
  std::mt19937_64 rng(11);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  for (int t = 0; t < 50; ++t) {
    const int H = 1 + static_cast<int>(rng() % 40), C = 1 + static_cast<int>(rng() % 16);
    std::vector<double> sp(H * C), pf(H * C);
    for (int j = 0; j < H * C; ++j) {
      sp[j] = u(rng);
      pf[j] = u(rng) - 0.5;
    }
    std::vector<int32_t> choice(H);
    double best = 0.0;
    const vecattn_status st =
        vecattn_plan_filter_ratios(H, C, sp.data(), pf.data(), u(rng), 1 + static_cast<int>(rng() % 2000),
                                   choice.data(), &best);
    expect(st == VECATTN_OK || st == VECATTN_ERR_CAPACITY, "plan");
  }
  std::printf(failures ? "failures: %d\n" : "ok\n", failures);
  return failures ? 1 : 0;
}
