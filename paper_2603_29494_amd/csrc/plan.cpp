// Per-head filter ratios (paper Sec. 3.1.2, Eq. 5): choose one candidate filter
// ratio per head so that the heads' mean sparsity reaches a target and the
// summed per-head performance is largest.  Host code; the tables sp_h and
// Perf_h come from offline sampling.
//
// Eq. 5 indexes the table by the mean sparsity of the first h heads; this
// keeps the equivalent sum instead, quantised to 1/grid per head, with
// "at least" semantics (the base row DP[0][.] = 0 then means: no sparsity
// still required costs nothing):
//   best_h(S) = max_c best_{h-1}(max(0, S - q_{h,c})) + Perf_h(c),
//   best_0(0) = 0, best_0(S > 0) = -inf,  q_{h,c} = round(sp_h(c) * grid),
// and the answer is best_H(ceil(target * H * grid)).  Ties go to the lower
// candidate index.
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "launch.h"

namespace vecattn {

int plan_filter_ratios(int32_t H, int32_t C, const double* sp, const double* perf, double target,
                       int32_t grid, int32_t* choice, double* best) {
  const int64_t T = static_cast<int64_t>(std::ceil(target * static_cast<double>(H) * grid - 1e-9));
  const int64_t Tn = T > 0 ? T : 0;
  const double ninf = -std::numeric_limits<double>::infinity();
  std::vector<int64_t> q(static_cast<size_t>(H) * C);
  for (int64_t t = 0; t < static_cast<int64_t>(H) * C; ++t)
    q[t] = static_cast<int64_t>(std::llround(sp[t] * grid));
  // f[h][S] for S in [0, Tn]; arg[h][S] = the candidate chosen for head h.
  std::vector<double> prev(Tn + 1, ninf), cur(Tn + 1);
  std::vector<int32_t> arg(static_cast<size_t>(H) * (Tn + 1), -1);
  prev[0] = 0.0;
  for (int32_t h = 0; h < H; ++h) {
    for (int64_t S = 0; S <= Tn; ++S) {
      double v = ninf;
      int32_t a = -1;
      for (int32_t c = 0; c < C; ++c) {
        const int64_t rest = S - q[static_cast<size_t>(h) * C + c];
        const double b = prev[rest > 0 ? rest : 0];
        if (b == ninf) continue;
        const double x = b + perf[static_cast<size_t>(h) * C + c];
        if (x > v) {
          v = x;
          a = c;
        }
      }
      cur[S] = v;
      arg[static_cast<size_t>(h) * (Tn + 1) + S] = a;
    }
    prev.swap(cur);
  }
  if (prev[Tn] == ninf) return 1;  // the target is out of reach
  *best = prev[Tn];
  int64_t S = Tn;
  for (int32_t h = H - 1; h >= 0; --h) {
    const int32_t c = arg[static_cast<size_t>(h) * (Tn + 1) + S];
    choice[h] = c;
    const int64_t rest = S - q[static_cast<size_t>(h) * C + c];
    S = rest > 0 ? rest : 0;
  }
  return 0;
}

}  // namespace vecattn
