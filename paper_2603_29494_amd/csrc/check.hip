// Index-list checker: counts the rows whose (I, C) pair breaks the input
// contract of the sparse attention (Eq. 4 gathers the listed keys; the kernel
// relies on every listed key being in range and on each list ascending).
#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

__global__ __launch_bounds__(64) void k_zero_one(int32_t* __restrict__ x) {
  if (threadIdx.x == 0) x[0] = 0;
}

// One wave per row.  A row is bad when its count is outside [0, cap], or one of
// its first `count` entries is outside [0, n_keys) or not above the entry
// before it.  Entries past the count are not read.
__global__ __launch_bounds__(256) void k_check_lists(const int32_t* __restrict__ idx,
                                                     const int32_t* __restrict__ counts,
                                                     int64_t rows, int64_t cap, int64_t n_keys,
                                                     int32_t* __restrict__ n_bad) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t c = counts[row];
  bool bad = c < 0 || c > cap;
  if (!bad) {
    const int32_t* list = idx + row * cap;
    for (int64_t j = lane; j < c; j += 64) {
      const int64_t v = list[j];
      const int64_t prev = j > 0 ? static_cast<int64_t>(list[j - 1]) : int64_t(-1);
      bad = bad || v < 0 || v >= n_keys || v <= prev;
    }
  }
  if (__ballot(bad) != 0ull && lane == 0) atomicAdd(n_bad, 1);
}

}  // namespace

hipError_t launch_check_lists(const int32_t* idx, const int32_t* counts, int64_t rows, int64_t cap,
                              int64_t n_keys, int32_t* n_bad, hipStream_t stream) {
  hipLaunchKernelGGL(k_zero_one, dim3(1), dim3(64), 0, stream, n_bad);
  if (rows > 0)
    hipLaunchKernelGGL(k_check_lists, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0,
                       stream, idx, counts, rows, cap, n_keys, n_bad);
  return hipGetLastError();
}

}  // namespace vecattn
