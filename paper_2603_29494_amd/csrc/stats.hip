// Statistics of a selection, for the offline studies of the paper:
//   - the sparsity of each head (Eq. 5's sp_h, Sec. 3.1.2), from the counts;
//   - the recall of the selected pattern (Sec. 2.2): the share of the exact
//     attention map's mass that each query row's block list keeps.
#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

// One workgroup per query head: sparsity[h] = 1 - (selected keys of the
// head's blocks over the batch) / (B * sum_i L_i), L_i the eligible keys of
// block i (N, or min(N, (i + 1) P) when causal).  Integer sums, one division.
__global__ __launch_bounds__(256) void k_head_sparsity(const int32_t* __restrict__ counts,
                                                       int64_t B, int64_t Hq, int64_t Np, int64_t N,
                                                       int32_t P, int32_t causal,
                                                       double* __restrict__ out) {
  __shared__ int64_t s_c[256], s_l[256];
  const int64_t h = blockIdx.x;
  int64_t c = 0, l = 0;
  for (int64_t t = threadIdx.x; t < B * Np; t += 256) {
    const int64_t b = t / Np, i = t % Np;
    c += counts[(b * Hq + h) * Np + i];
    if (b == 0) l += causal ? min(N, (i + 1) * static_cast<int64_t>(P)) : N;
  }
  s_c[threadIdx.x] = c;
  s_l[threadIdx.x] = l;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (static_cast<int>(threadIdx.x) < o) {
      s_c[threadIdx.x] += s_c[threadIdx.x + o];
      s_l[threadIdx.x] += s_l[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0)
    out[h] = 1.0 - static_cast<double>(s_c[0]) / (static_cast<double>(B) * static_cast<double>(s_l[0]));
}

// Recall of the selected pattern.  One workgroup (4 waves) per 64 query rows
// of a block, as in the sparse attention: the block's list becomes a bitmask
// of the keys in LDS, then every visible key is scored in tiles of 64 keys
// (S^T = K_tile Q^T on v_mfma_f32_32x32x16_bf16; wave (rw, kw) owns 32 rows x
// 32 keys of a tile) and two online softmax sums share one running maximum:
// over all visible keys, and over the listed ones.  The two key halves merge
// at the end; kept = listed sum / total sum.
template <int D>
__global__ __launch_bounds__(256) void k_recall(
    const uint16_t* __restrict__ q, int64_t q_sB, int64_t q_sH, int64_t q_sN,
    const uint16_t* __restrict__ k, int64_t k_sB, int64_t k_sH, int64_t k_sN,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ counts, int64_t cap, int32_t Hq,
    int32_t group, int32_t N, int32_t P, int32_t Np, int32_t chunks, int32_t causal,
    float scale_log2, int64_t total, float* __restrict__ kept) {
  constexpr int DS = D / 16;
  extern __shared__ uint32_t s_bits[];  // ceil(N / 32) words: bit j = key j is listed
  __shared__ float s_merge[3][64];
  const int64_t w = blockIdx.x;
  if (w >= total) return;
  const int chunk = static_cast<int>(w % chunks);
  const int64_t rest = w / chunks;
  const int i = static_cast<int>(rest % Np);
  const int64_t bh = rest / Np;
  const int b = static_cast<int>(bh / Hq), h = static_cast<int>(bh % Hq), hk = h / group;
  const int row0 = i * P + chunk * 64;
  const int row_end = min(N, min(i * P + P, row0 + 64));
  const int count = static_cast<int>(min<int64_t>(max(counts[bh * Np + i], 0), cap));
  const int32_t* list = idx + (bh * Np + i) * cap;
  const int tid = threadIdx.x;
  const int nw = (N + 31) / 32;
  for (int t = tid; t < nw; t += 256) s_bits[t] = 0u;
  __syncthreads();
  for (int t = tid; t < count; t += 256) {
    const int j = list[t];
    if (j >= 0 && j < N) atomicOr(&s_bits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();

  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 5, ln = lane & 31;
  const int rw = wave & 1, kw = wave >> 1;
  const int my_row = row0 + 32 * rw + ln;
  bf16x8 qf[DS];
  {
    const bool have = my_row < row_end;
    const u32x4* qr = reinterpret_cast<const u32x4*>(
        q + b * q_sB + h * q_sH + static_cast<int64_t>(have ? my_row : row0) * q_sN);
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const u32x4 t = have ? qr[2 * s + g] : u32x4{0, 0, 0, 0};
      qf[s] = __builtin_bit_cast(bf16x8, t);
    }
  }
  const uint16_t* kh = k + b * k_sB + hk * k_sH;
  // Keys past the chunk's last row are never visible under causal masking.
  const int nkeys = causal ? row_end : N;
  const int ntiles = (nkeys + 63) / 64;
  float m = kNegInf, la = 0.0f, ls = 0.0f;
  for (int t = 0; t < ntiles; ++t) {
    const int kb = t * 64 + 32 * kw;  // this wave's 32 keys (a multiple of 32)
    const u32x4* kr = reinterpret_cast<const u32x4*>(kh + static_cast<int64_t>(min(kb + ln, N - 1)) * k_sN);
    f32x16 sacc = f32x16{};
#pragma unroll
    for (int s = 0; s < DS; ++s)
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kr[2 * s + g]),
                                                     qf[s], sacc, 0, 0, 0);
    const uint32_t word = kb < N ? s_bits[kb >> 5] : 0u;
    float x[16];
    float tmax = kNegInf;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int kl = 8 * (e >> 2) + 4 * g + (e & 3);
      const int j = kb + kl;
      const bool vis = j < N && (!causal || j <= my_row);
      x[e] = vis ? sacc[e] * scale_log2 : kNegInf;
      tmax = fmaxf(tmax, x[e]);
    }
    tmax = wave_max_xor32(tmax);
    const float mn = fmaxf(m, tmax);
    if (mn != kNegInf) {
      const float alpha = m == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m - mn);
      la *= alpha;
      ls *= alpha;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kl = 8 * (e >> 2) + 4 * g + (e & 3);
        const float p = __builtin_amdgcn_exp2f(x[e] - mn);
        la += p;
        ls += ((word >> kl) & 1u) ? p : 0.0f;
      }
      m = mn;
    }
  }
  // The lane pair (g = 0, 1) holds one row with one running maximum.
  la += __shfl_xor(la, 32);
  ls += __shfl_xor(ls, 32);
  if (kw == 1 && g == 0) {
    s_merge[0][32 * rw + ln] = m;
    s_merge[1][32 * rw + ln] = la;
    s_merge[2][32 * rw + ln] = ls;
  }
  __syncthreads();
  if (kw == 1 || g == 1 || my_row >= row_end) return;
  const float m1 = s_merge[0][32 * rw + ln];
  const float M = fmaxf(m, m1);
  const float a0 = m == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m - M);
  const float a1 = m1 == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m1 - M);
  const float tot = a0 * la + a1 * s_merge[1][32 * rw + ln];
  const float sel = a0 * ls + a1 * s_merge[2][32 * rw + ln];
  kept[bh * N + my_row] = tot > 0.0f ? sel / tot : 0.0f;
}

}  // namespace

hipError_t launch_head_sparsity(const int32_t* counts, int64_t B, int64_t Hq, int64_t N,
                                int32_t block, int32_t causal, double* sparsity,
                                hipStream_t stream) {
  const int64_t Np = (N + block - 1) / block;
  hipLaunchKernelGGL(k_head_sparsity, dim3(static_cast<unsigned>(Hq)), dim3(256), 0, stream,
                     counts, B, Hq, Np, N, block, causal, sparsity);
  return hipGetLastError();
}

hipError_t launch_recall(const RecallArgs& a, hipStream_t stream) {
  const int64_t B = a.q.B, Hq = a.q.H, N = a.q.N, D = a.q.D;
  const int32_t P = a.block;
  const int32_t Np = static_cast<int32_t>((N + P - 1) / P);
  const int32_t chunks = (P + 63) / 64;
  const int64_t total = B * Hq * static_cast<int64_t>(Np) * chunks;
  if (total == 0) return hipSuccess;
  const float scale = a.scale != 0.0f ? a.scale : 1.0f / sqrtf(static_cast<float>(D));
  const size_t lds = static_cast<size_t>((N + 31) / 32) * 4;
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* k = static_cast<const uint16_t*>(a.k.ptr);
  auto launch = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(total)), dim3(256), lds, stream, q,
                       a.q.sB, a.q.sH, a.q.sN, k, a.k.sB, a.k.sH, a.k.sN, a.idx, a.counts, a.cap,
                       static_cast<int32_t>(Hq), static_cast<int32_t>(Hq / a.k.H),
                       static_cast<int32_t>(N), P, Np, chunks, a.causal,
                       scale * 1.4426950408889634f, total, a.kept);
    return hipGetLastError();
  };
  return D == 128 ? launch(k_recall<128>) : launch(k_recall<64>);
}

}  // namespace vecattn
