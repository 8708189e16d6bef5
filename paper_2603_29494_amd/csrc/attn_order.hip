// Block schedule for the sparse attention (Eq. 4 / Algorithm 2 take the query
// blocks in any order; this one only decides which order runs fastest).
//
// For each (b, h) the N_p blocks are sorted by a 64-bit key, ascending:
//   bits 63..33  2^30 - count      (longest list first)
//   bits 32..24  signature         (mean key position of the list, in 512ths
//                                   of N, from 8 sampled entries)
//   bits 23..0   block index       (keys are distinct: the order is unique)
// A head of more than kOrderMaxBlocks blocks is sorted in consecutive
// segments of that many blocks (each segment in place, the key holding the
// index within the segment).
// Longest-first is the classic longest-processing-time rule, so the
// workgroups of a head finish together; it also puts lists of like length
// side by side, and lists of like length walk the keys at a like pace, which
// keeps the gathers of the workgroups running together on an XCD within what
// its L2 holds.  Among lists of one length (all of them, for topK) the
// signature puts lists over like key ranges side by side.
#include <algorithm>

#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

constexpr int kOrderThreads = 1024;

__global__ __launch_bounds__(kOrderThreads) void k_attn_order(
    const int32_t* __restrict__ idx, int64_t cap, const int32_t* __restrict__ counts, int32_t Np,
    int64_t N, int32_t* __restrict__ order) {
  const int64_t bh = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ uint64_t key[kOrderMaxBlocks];
  for (int64_t seg = 0; seg < Np; seg += kOrderMaxBlocks) {
    const int ns = static_cast<int>(std::min<int64_t>(Np - seg, kOrderMaxBlocks));
    const int32_t* cnt = counts + bh * Np + seg;
    int32_t* out = order + bh * Np + seg;
    int n2 = 2;
    while (n2 < ns) n2 <<= 1;
    __syncthreads();  // the previous segment's keys have been written out
    for (int i = tid; i < n2; i += kOrderThreads) {
      uint64_t kk = ~uint64_t(0);  // padding sorts last
      if (i < ns) {
        const int64_t c = std::min<int64_t>(std::max<int64_t>(cnt[i], 0), cap);
        const int32_t* list = idx + (bh * Np + seg + i) * cap;
        int64_t sum = 0;  // of 8 entries in [0, N), N <= 2^30
        if (c > 0) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int64_t e = list[((2 * j + 1) * c) / 16];
            sum += std::min<int64_t>(std::max<int64_t>(e, 0), N - 1);
          }
        }
        // mean * 512 / N = sum * 64 / N, below 512
        const uint64_t sig = static_cast<uint64_t>(std::min<int64_t>((sum * 64) / N, 511));
        kk = (static_cast<uint64_t>((int64_t(1) << 30) - c) << 33) | (sig << 24) |
             static_cast<uint64_t>(i);
      }
      key[i] = kk;
    }
    __syncthreads();
    // Bitonic sort of n2 keys, ascending.
    for (int k = 2; k <= n2; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int t = tid; t < n2 / 2; t += kOrderThreads) {
          const int a = (t / j) * 2 * j + (t % j);
          const int b = a + j;
          const uint64_t x = key[a], y = key[b];
          if ((x > y) == ((a & k) == 0)) {
            key[a] = y;
            key[b] = x;
          }
        }
        __syncthreads();
      }
    }
    for (int i = tid; i < ns; i += kOrderThreads)
      out[i] = static_cast<int32_t>(seg + static_cast<int64_t>(key[i] & 0xFFFFFF));
  }
}

}  // namespace

hipError_t launch_attn_order(const int32_t* idx, int64_t cap, const int32_t* counts, int64_t rows,
                             int32_t Np, int64_t N, int32_t* order, hipStream_t stream) {
  if (rows == 0 || Np == 0) return hipSuccess;
  hipLaunchKernelGGL(k_attn_order, dim3(static_cast<unsigned>(rows)), dim3(kOrderThreads), 0,
                     stream, idx, cap, counts, Np, N, order);
  return hipGetLastError();
}

}  // namespace vecattn
