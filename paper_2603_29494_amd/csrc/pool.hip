// Query pooling, paper Eq. 2 (Sec. 3.1.1): the pooled query of a block is the
// mean of the block's query rows.  One thread owns 8 consecutive head-dim
// values of one block, sums the block's rows in fp64 in row order (bf16 values
// have 8 significant bits, so these sums are exact unless the values span more
// than ~2^38 in magnitude) and rounds the mean to bf16 once.
#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

__global__ __launch_bounds__(256) void k_pool(const uint16_t* __restrict__ q, int64_t q_sB,
                                              int64_t q_sH, int64_t q_sN, int32_t H, int32_t N,
                                              int32_t D, int32_t P, int32_t Np,
                                              uint16_t* __restrict__ qp, int64_t p_sB,
                                              int64_t p_sH, int64_t p_sN, int64_t total) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const int chunks = D / 8;
  const int c = static_cast<int>(t % chunks);
  int64_t rest = t / chunks;
  const int i = static_cast<int>(rest % Np);
  rest /= Np;
  const int h = static_cast<int>(rest % H);
  const int b = static_cast<int>(rest / H);
  const int r0 = i * P;
  const int r1 = min(N, r0 + P);
  const uint16_t* base = q + b * q_sB + h * q_sH + 8 * c;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  auto add_row = [&](const u32x4 w) __attribute__((always_inline)) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += static_cast<double>(bf16_bits_to_f32(w[e] & 0xFFFFu));
      acc[2 * e + 1] += static_cast<double>(bf16_bits_to_f32(w[e] >> 16));
    }
  };
  // Eight rows are loaded before any is summed, so that a thread keeps eight
  // loads in flight; the sums still run in row order.
  int r = r0;
  for (; r + 8 <= r1; r += 8) {
    u32x4 w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      w[j] = *reinterpret_cast<const u32x4*>(base + static_cast<int64_t>(r + j) * q_sN);
#pragma unroll
    for (int j = 0; j < 8; ++j) add_row(w[j]);
  }
  for (; r < r1; ++r) add_row(*reinterpret_cast<const u32x4*>(base + static_cast<int64_t>(r) * q_sN));
  const double n = static_cast<double>(r1 - r0);
  u32x4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t lo = f64_to_bf16_rne(acc[2 * e] / n);
    const uint32_t hi = f64_to_bf16_rne(acc[2 * e + 1] / n);
    out[e] = lo | (hi << 16);
  }
  *reinterpret_cast<u32x4*>(qp + b * p_sB + h * p_sH + static_cast<int64_t>(i) * p_sN + 8 * c) = out;
}

}  // namespace

hipError_t launch_pool(const Tensor4& q, int32_t block, void* qp, int64_t qp_sB, int64_t qp_sH,
                       int64_t qp_sN, hipStream_t stream) {
  const int32_t Np = static_cast<int32_t>((q.N + block - 1) / block);
  const int64_t total = q.B * q.H * static_cast<int64_t>(Np) * (q.D / 8);
  if (total == 0) return hipSuccess;
  const int threads = 256;
  const dim3 grid(static_cast<unsigned>((total + threads - 1) / threads));
  hipLaunchKernelGGL(k_pool, grid, dim3(threads), 0, stream, static_cast<const uint16_t*>(q.ptr),
                     q.sB, q.sH, q.sN, static_cast<int32_t>(q.H), static_cast<int32_t>(q.N),
                     static_cast<int32_t>(q.D), block, Np, static_cast<uint16_t*>(qp), qp_sB,
                     qp_sH, qp_sN, total);
  return hipGetLastError();
}

}  // namespace vecattn
