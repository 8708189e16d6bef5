// Important-vector selection (paper Sec. 3.1; the outputs I and C of
// Algorithm 1) for gfx950: row-wise topK (a budget), topP (a cumulative
// softmax-mass threshold) and minS (Eq. 3: within alpha of the row maximum)
// over the estimated map Q_p K^T / sqrt(D), without ever writing that map to
// memory (the TilingSelect principle, Sec. 3.1.3).
//
// Exact selection needs the score of the k-th key (topK) or of the key where
// the mass reaches p (topP).  Every row therefore narrows a score interval
// that must contain its cut, one pass over the keys at a time:
//   HIST     score tiles stay on chip; each key of the row is classified
//            against the interval (above / inside / below); keys inside land
//            in a 128-bin LDS histogram, keys above are counted (and their
//            softmax mass summed for topP).  A resolve kernel picks the bin
//            range that must hold the cut, which becomes the next interval.
//   COLLECT  once the interval holds at most kCand keys: a bit per key at or
//            above the interval, and the (score, index) pairs of the keys
//            inside it; a resolve kernel ranks those candidates, fixes the cut
//            score t* and how many keys tied at t* are kept (lowest indices),
//            and clears the bits of the rejected ones.
//   EMIT     only for rows whose interval still held more than kCand keys:
//            one more pass sets a bit per kept key (score > t*), and one per
//            key tied at the cut when only some ties are kept.
//   COMPACT  bitmasks -> ascending index lists and counts.
// minS rows start from a MAX pass (the row maximum fixes the threshold); with
// a cap no block can exceed they are emitted directly, otherwise the level-0
// pass counts them and the rows over cap continue as topK(cap).
// All passes compute every score with the same MFMA sequence, so a key's
// score is bit-identical in every pass.
//
// Work decomposition of a pass: a workgroup owns 64 pooled rows (query
// blocks) of one head and one split of up to `split` keys; its 4 waves take
// the split's 32-key blocks in turn.  S^T = K_blk Q_p^T uses
// v_mfma_f32_32x32x16_bf16 with the pooled queries held in registers and K
// read from a copy in MFMA operand order that each call writes once.
#include <float.h>

#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

constexpr int kRowsWG = 64;     // pooled rows per workgroup
constexpr int kThreads = 256;
constexpr int kBins = 128;     // bins per histogram level: 64 rows x 129 bins of 32 bits fit the LDS
                               // of three workgroups per CU (topK, minS), of 64 bits (topP: each
                               // bin also sums its mass) that of two
constexpr int kSampleBins = 256;  // bins of the sampled-score histogram that places level 0 (topK)
// topP bin entries: count << 48 | mass in units of 2^-31 (terms exp(tau s -
// ref) <= 1 rounded to that grid); a workgroup adds at most 4096 terms to a
// bin, so neither field can carry into the other.
constexpr int kMassShift = 48;
constexpr double kMassUnit = 0x1p-31;
constexpr float kTopPRange = 40.0f;  // nats below the row maximum the level-0 topP bins span
// topP cut bins are resolved to this share of the row's total mass: the GPU's
// fp32 scores and exp2 already differ from exact masses by ~1e-7 relative.
constexpr double kTopPMassSlack = 0x1p-20;
constexpr int kLevels = 6;      // histogram refinements per round (idle ones cost ~6 us)
constexpr int kCand = 1024;     // candidate capacity per row
constexpr int kRounds = 2;      // a topP row whose count exceeds cap reruns as topK(cap)
constexpr int kMaxHeadParams = 128;  // query heads a per-head parameter list may cover
// Rows entering each later pass are counted (nact[level] for histogram level
// >= 1, nact[kEmitSlot] for the emit pass); a pass that no row needs returns
// at once, without reading row state.
constexpr int kEmitSlot = kLevels + 1;
constexpr int kActiveSlots = 16;

enum Phase : int { PH_IDLE = 0, PH_HIST = 1, PH_COLLECT = 2, PH_DONE = 3, PH_EMIT = 4 };
// MODE_HIST0: first histogram level (the interval is everything).
// MODE_MAX: the largest score of each minS row.
enum Mode : int {
  MODE_HIST = 0, MODE_COLLECT = 1, MODE_EMIT = 2, MODE_HIST0 = 3, MODE_MAX = 5
};
constexpr int kSampleStride = 16;  // 32-key blocks between sampled blocks

struct RowState {
  int phase;
  int level;        // histogram level the next HIST pass runs
  int topp;         // 1: cut by mass, 0: cut by rank
  int k_target;     // topK: number of keys to keep
  int L;            // eligible keys
  int tie_partial;  // 1: only the first k_eq keys tied at t* are kept
  int k_eq;         // keys tied at t* that are kept
  int count;        // final count
  int clamped;      // 1 if the threshold selection was clamped to cap
  int tie_interval; // 1: the keys tied at the cut are all those in [s_lo, s_hi]
  int mins;         // 1: minS row before its count is known (level 0)
  int pad0;
  // Scores below are raw fp32 dot products <q_p, k_j> (the softmax scale tau
  // > 0 preserves their order; it enters only the topP masses).
  float s_lo, s_hi; // current interval: keys with s_lo <= s <= s_hi (exact float bounds)
  float blo, binv;  // bin range of the current level: lo and bins per unit
  float badd;       // bin of s: floor(fma(s, binv, badd)), badd = -blo * binv
  float smax;       // topP: the row's largest score (ref = tau * smax)
  float tstar;      // cut score
  double ref;       // softmax reference (an upper bound of the row's scores)
  double Z;         // total mass (topP)
  double pZ;        // p * Z
  // topP: bounds of the mass of the keys above the current interval, from the
  // per-bin sums of level 0 and the edge bounds of later levels (exact only in
  // the collect pass, which sums it again).
  double mab_lo, mab_hi;
};

struct SelParams {
  const uint16_t* qp;     // pooled queries, [rows][D] contiguous, rows = bh * Np + i
  const uint16_t* k;
  const u32x4* kop;       // K in MFMA operand order: [B * Hkv][nkb][D / 16][64 lanes] x 16 B
  int nkb;                // 32-key blocks per key/value head
  RowState* st;
  uint32_t* hist;         // [rows][kBins]
  uint64_t* hmass;        // [rows][kBins] topP launches: per-bin mass sum in units of kMassUnit
  uint32_t* n_above;      // [rows][nsplit]
  double* m_above;        // [rows][nsplit]
  double* zpart;          // [rows][nsplit]
  uint32_t* cand_n;       // [rows]
  uint32_t* cand_lohi;    // [rows][2] ordered-score min / max of collected candidates
  uint64_t* cand;         // [rows][kCand]
  uint32_t* bsel;         // [rows][W]
  uint32_t* btie;         // [rows][W]
  float* qnorm;           // [rows]
  float* kmax;            // [B * Hkv]
  int32_t* idx;
  int32_t* counts;
  int32_t* n_clamped;
  int64_t cap;
  int64_t rows;
  int B, Hq, Hkv, group, N, P, Np, D, causal, split, nsplit, W, nrb;  // nrb: row blocks per head
  int mode_topp;
  int mode_mins;
  int mins_direct;  // minS with cap >= every block's eligible keys: no count needed
  int mode_tiled;   // cross-tile minS (Algorithm 1)
  int keep_diag;    // every block also keeps the keys of its own rows
  int unpadded;     // entries past a row's count are left unwritten (no -1 padding)
  int quad_rows;    // idx rows start on 16 bytes and no row can exceed cap
  uint32_t* nact;   // [kActiveSlots] rows waiting for each later pass
  int gate;         // slot of nact this launch needs non-zero, or -1
  int tiled_tile;   // keys per tile: 16 or 32
  int tiled_gs;     // keys per group of tiles (a power of two)
  int tiled_sb;     // 32-key blocks per segment a wave walks in order
  int tiled_carry;  // groups span several splits: waves start from a carried maximum
  double sqrt_d;    // 1 / tau: alpha / tau is alpha in raw-score units
  float* qmax;      // [rows][nsplit * 4]: per quarter split, its maximum, then the carried one
  double param;
  int per_head;     // 1: head_param[h] replaces param for query head h
  double head_param[kMaxHeadParams];
  float tau;
  int64_t items;    // score-pass work items
  int64_t per_xcd;  // work items per XCD
};

__device__ __forceinline__ uint32_t ord_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ord_val(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// The selection parameter of a row (rows are ordered (b, h, i)).
__device__ __forceinline__ double row_param(const SelParams& p, int64_t row) {
  return p.per_head ? p.head_param[(row / p.Np) % p.Hq] : p.param;
}

__device__ __forceinline__ int eligible(int i, int P, int N, int causal) {
  return causal ? min(N, (i + 1) * P) : N;
}

__device__ __forceinline__ int topk_count(double r, int L) {
  int k = static_cast<int>(ceil(r * static_cast<double>(L) - 1e-9));
  return min(max(k, 1), L);
}

// exp(tau * s - ref) for topP masses (s a raw score): exp2 in fp32 while the
// exponent is in range (relative error ~1e-7), with an exact power-of-two
// rescale below it.
__device__ __forceinline__ double mass_term(float s, float tau, double ref) {
  const double y = (static_cast<double>(s) * static_cast<double>(tau) - ref) * 1.4426950408889634;
  if (y > -120.0) return static_cast<double>(__builtin_amdgcn_exp2f(static_cast<float>(y)));
  const double n = floor(y);
  return ldexp(static_cast<double>(__builtin_amdgcn_exp2f(static_cast<float>(y - n))), static_cast<int>(n));
}

// Key of a 32-key block that the operand-order copy of K places in A-operand
// row r: rows 8 a + 4 g + b hold keys 16 g + 4 a + b.  The product's
// accumulator entry e of lane group g (row 8 (e / 4) + 4 g + e % 4) is then
// key 16 g + e: a lane's 16 scores are 16 consecutive keys.
__host__ __device__ constexpr int block_key_of_row(int r) {
  return 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3);
}

// Comparisons as lane masks (bit l: lane l; one compare into a scalar register
// pair), for shift_in.
__device__ __forceinline__ uint64_t lanes_ge(float a, float b) { return __ballot(a >= b); }
__device__ __forceinline__ uint64_t lanes_gt(float a, float b) { return __ballot(a > b); }
__device__ __forceinline__ uint64_t lanes_lt(int a, int b) { return __ballot(a < b); }

// 2 w + (this lane's bit of m): one add with the lane mask as carry-in, so a
// lane's word of flags is built with one instruction per key and no per-lane
// bit constants.
__device__ __forceinline__ uint32_t shift_in(uint32_t w, uint64_t m) {
  uint32_t r;
  uint64_t carry;
  asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry) : "v"(w), "s"(m));
  return r;
}

// Bin of s at one level (must be evaluated identically everywhere: the
// scoring passes and the interval search below use this one function).
// One fma, clamped to [0, nb - 1] in float before the conversion
// (out-of-range conversions are undefined); truncation equals floor on the
// clamped, non-negative value.
__device__ __forceinline__ int bin_of(float s, float mul, float add, int nb) {
  const float x = __builtin_amdgcn_fmed3f(__builtin_fmaf(s, mul, add), 0.0f,
                                          static_cast<float>(nb - 1));
  return static_cast<int>(x);
}

// Bins of the next level: bins of width 1 / binv from lo.
__device__ __forceinline__ void set_bins(RowState& s, float lo, float binv) {
  s.blo = lo;
  s.binv = binv;
  s.badd = -lo * binv;
}

// The interval after choosing bins [ba, bb] of the level with bin function
// (mul, add) inside [s_lo, s_hi]: the bin function is monotone in s, so the
// chosen set is again a float interval; its exact ends are found by binary
// search over ordered float keys with the same bin function the passes use.
__device__ __forceinline__ void narrow(float& s_lo, float& s_hi, float mul, float add, int ba, int bb,
                                       int nb) {
  // smallest s with bin >= ba
  uint32_t a = ord_key(-FLT_MAX), z = ord_key(FLT_MAX);
  if (bin_of(ord_val(a), mul, add, nb) < ba) {
    while (z - a > 1) {
      const uint32_t m = a + (z - a) / 2;
      if (bin_of(ord_val(m), mul, add, nb) >= ba) z = m; else a = m;
    }
    s_lo = fmaxf(s_lo, ord_val(z));
  }
  // largest s with bin <= bb
  a = ord_key(-FLT_MAX);
  z = ord_key(FLT_MAX);
  if (bin_of(ord_val(z), mul, add, nb) > bb) {
    while (z - a > 1) {
      const uint32_t m = a + (z - a) / 2;
      if (bin_of(ord_val(m), mul, add, nb) <= bb) a = m; else z = m;
    }
    s_hi = fminf(s_hi, ord_val(a));
  }
}

// ---------------------------------------------------------------------------
// Per-row setup: eligible keys, targets, first interval [-c, c] with
// c >= |q_p| * max |k| (Cauchy-Schwarz, padded for fp32 rounding).
// ---------------------------------------------------------------------------
// K of every key/value head in MFMA operand order, once per call: for each
// 32-key block and head-dim step s2, the 64 lanes' A-operand pieces (lane l:
// key block_key_of_row(l % 32) of the block, head-dim values 16 s2 + 8 (l / 32) .. +7) lie
// contiguously, so a score pass fetches each step with one fully coalesced
// 1 KB load instead of 32 rows x 32 bytes.  Keys past N repeat key N - 1
// (they are never eligible).  One wave per 32-key block.  The same read of K
// gives the largest key norm per key/value head (kmax, zeroed beforehand):
// one atomic per workgroup and head.
template <int D>
__global__ __launch_bounds__(256) void k_k_operand_order(const uint16_t* __restrict__ k, int64_t sB,
                                                         int64_t sH, int64_t sN, int Hkv, int N,
                                                         int nkb, int64_t nblk_total,
                                                         u32x4* __restrict__ kop,
                                                         float* __restrict__ kmax) {
  constexpr int DS = D / 16;
  __shared__ float s_n2[4];
  __shared__ int64_t s_bh[4];
  const int wave = threadIdx.x >> 6;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + wave;
  const int lane = threadIdx.x & 63, g = lane >> 5, ln = lane & 31;
  float n2 = 0.0f;
  int64_t bh = -1;
  if (t < nblk_total) {
    const int blk = static_cast<int>(t % nkb);
    bh = t / nkb;
    const int64_t b = bh / Hkv, hk = bh % Hkv;
    const int key = min(blk * 32 + block_key_of_row(ln), N - 1);
    const u32x4* src = reinterpret_cast<const u32x4*>(k + b * sB + hk * sH + key * sN);
    u32x4* dst = kop + t * (DS * 64) + lane;
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) {
      const u32x4 w = src[2 * s2 + g];
      dst[s2 * 64] = w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x0 = bf16_bits_to_f32(w[e] & 0xFFFFu), x1 = bf16_bits_to_f32(w[e] >> 16);
        n2 = __builtin_fmaf(x0, x0, n2);
        n2 = __builtin_fmaf(x1, x1, n2);
      }
    }
    n2 += __shfl_xor(n2, 32);  // the key's two halves
    for (int o = 16; o > 0; o >>= 1) n2 = fmaxf(n2, __shfl_xor(n2, o));
  }
  if (lane == 0) {
    s_n2[wave] = n2;
    s_bh[wave] = bh;
  }
  __syncthreads();
  if (threadIdx.x == 0) {  // the 4 blocks belong to at most two heads (nkb >= 1: in order)
    for (int w0 = 0; w0 < 4;) {
      if (s_bh[w0] < 0) break;
      float m = s_n2[w0];
      int w1 = w0 + 1;
      while (w1 < 4 && s_bh[w1] == s_bh[w0]) m = fmaxf(m, s_n2[w1++]);
      atomicMax(reinterpret_cast<unsigned int*>(kmax + s_bh[w0]), __float_as_uint(sqrtf(m)));
      w0 = w1;
    }
  }
}

__global__ __launch_bounds__(256) void k_sel_init(SelParams p, int round) {
  // Counters start at zero once per call (rows sent to the emit pass in the
  // first round still count in the second).
  if (round == 0 && blockIdx.x == 0 && threadIdx.x < kActiveSlots) p.nact[threadIdx.x] = 0u;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= p.rows) return;
  RowState& s = p.st[r];
  const int i = static_cast<int>(r % p.Np);
  const int64_t bh = r / p.Np;
  const int b = static_cast<int>(bh / p.Hq), h = static_cast<int>(bh % p.Hq);
  if (round > 0) {
    if (s.phase != PH_IDLE) return;   // only rows sent back for a second round
  } else {
    s.L = eligible(i, p.P, p.N, p.causal);
    s.clamped = 0;
    s.topp = p.mode_topp;
    if (!p.mode_topp && !p.mode_mins) s.k_target = topk_count(row_param(p, r), s.L);
    if (p.mode_topp && row_param(p, r) >= 1.0) {  // p = 1 keeps every eligible key
      s.topp = 0;
      s.k_target = s.L;
    }
  }
  const float c = p.qnorm[r] * p.kmax[b * p.Hkv + h / p.group];
  const float cc = c * 1.0009765625f + 1e-30f;
  s.level = 0;
  s.phase = PH_HIST;
  s.s_lo = -FLT_MAX;
  s.s_hi = FLT_MAX;
  set_bins(s, -cc, static_cast<float>(kBins) / (2.0f * cc));
  s.ref = static_cast<double>(p.tau) * static_cast<double>(cc);  // >= every tau * score
  s.smax = cc;
  s.tie_partial = 0;
  s.k_eq = 0;
  s.tie_interval = 0;
  s.mins = p.mode_mins && round == 0;
  s.mab_lo = 0.0;
  s.mab_hi = 0.0;
  p.cand_n[r] = 0;
  p.cand_lohi[2 * r] = 0xFFFFFFFFu;
  p.cand_lohi[2 * r + 1] = 0u;
}

// ---------------------------------------------------------------------------
// Norms for the bound: |q_p| per pooled row (from its bf16 values); the
// largest |k_j| per key/value head comes from k_k_operand_order, after
// k_kmax_init has zeroed it.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_qnorm(const uint16_t* __restrict__ qp, int64_t rows, int D,
                                               float* __restrict__ out) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * (blockDim.x / 64) + threadIdx.x / 64;
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  float acc = 0.0f;
  for (int d = lane; d < D; d += 64) {
    const float x = bf16_bits_to_f32(qp[r * D + d]);
    acc = __builtin_fmaf(x, x, acc);
  }
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) out[r] = sqrtf(acc);
}

__global__ __launch_bounds__(256) void k_kmax_init(float* kmax, int n) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) kmax[t] = 0.0f;
}

// ---------------------------------------------------------------------------
// The scoring pass.  Work items are ordered (head, split, row tile) with the
// row tile fastest and handed out XCD by XCD, so the row tiles of one head
// that read the same key split run together on one XCD and share its L2.
// ---------------------------------------------------------------------------
// TOPP: the launch selects by mass (rows restarted as topK(cap) may be mixed
// in); otherwise no mass is computed.
// Histogram passes without per-bin masses (every level of topK / minS rows,
// levels >= 1 of topP rows) are held to 168 VGPRs so that three waves share
// each SIMD (their 33 KB of LDS allows it): the latency of the K loads and of the
// MFMA chains is then hidden better (~5% of the selection at the 75k DiT layer).
template <int D, int MODE, bool TOPP>
__global__ __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu((MODE == MODE_HIST || (MODE == MODE_HIST0 && !TOPP)) ? 3 : 1)))
void k_score_pass(SelParams p) {
  constexpr int DS = D / 16;
  constexpr bool HIST = MODE == MODE_HIST || MODE == MODE_HIST0;
  // Bin-major layout, entry (bin, row) at bin * kRowsWG + row: the 32 rows of
  // a wave's update sit in 32 distinct banks whatever their bins (the two
  // lanes of one row share a bank: at most 2-way conflicts; a row-major
  // layout gave ~4-way ones from bins colliding across rows).  Bin NB of a
  // row takes the increments of keys outside the
  // interval, so that every key can be counted without a branch.
  constexpr int NB = kBins;
  constexpr int HS = NB + 1;  // bins per row including the spare one
  // The level-0 topP pass also sums each bin's softmax mass (terms exp2((s -
  // row max) tau log2 e) <= 1 in fixed point), which pins the cut to one or
  // two bins: one 64-bit integer atomic per key carries both the count and the
  // mass (LDS float atomics are far slower).  Later levels split one such bin
  // into bins so narrow that the mass bounds from their score edges suffice;
  // they count keys only, and the mass above their interval is carried from
  // the levels before (bounds in the row state), so no key's mass is computed
  // there.
  constexpr bool MH = MODE == MODE_HIST0 && TOPP;
  constexpr bool MASS = MODE != MODE_HIST && TOPP;  // this pass computes key masses
  __shared__ uint32_t s_hist[HIST && !MH ? kRowsWG * HS : 1];
  __shared__ uint64_t s_hist64[MH ? kRowsWG * HS : 1];
  __shared__ double s_zred[4][kRowsWG];
  __shared__ double s_mred[4][kRowsWG];
  __shared__ uint32_t s_nred[4][kRowsWG];
  __shared__ int s_part[kRowsWG];
  __shared__ int s_any;
  // COLLECT: candidates are staged per row in LDS (rank from an LDS counter)
  // and written out with one global atomic per row at the end; a row that
  // overflows its LDS slots appends the rest directly.
  constexpr bool COL = MODE == MODE_COLLECT;
  constexpr int kStage = 96;  // LDS candidate slots per row
  constexpr int kStageStride = kStage + 1;  // odd in 8-byte units: rows start in different banks
  __shared__ uint64_t s_cand[COL ? kRowsWG * kStageStride : 1];
  __shared__ uint32_t s_ccnt[COL ? kRowsWG : 1];
  __shared__ uint32_t s_clo[COL ? kRowsWG : 1];
  __shared__ uint32_t s_chi[COL ? kRowsWG : 1];
  __shared__ uint32_t s_cbase[COL ? kRowsWG : 1];
  // per lane: its 16 scores, the 16-byte chunk q stored at q ^ ((lane / 4) % 4) so
  // that the 16 lanes of a 16-byte store or load phase use distinct banks
  __shared__ __align__(16) float s_acc[COL ? 4 * 64 * 16 : 1];
  __shared__ uint32_t s_max[MODE == MODE_MAX ? kRowsWG : 1];  // ordered keys of row maxima

  if (p.gate >= 0 && p.nact[p.gate] == 0u) return;  // no row needs this pass
  const int64_t item = xcd_work_item(p.per_xcd);
  if (item >= p.items) return;
  const int rb = static_cast<int>(item % p.nrb);
  const int64_t rest = item / p.nrb;
  const int sp = static_cast<int>(rest % p.nsplit);
  const int64_t bh = rest / p.nsplit;
  const int b = static_cast<int>(bh / p.Hq), h = static_cast<int>(bh % p.Hq);
  const int hk = h / p.group;
  const int i0 = rb * kRowsWG;
  const int nrows = min(kRowsWG, p.Np - i0);
  const int Ltile = eligible(i0 + nrows - 1, p.P, p.N, p.causal);
  const int key0 = sp * p.split;
  if (key0 >= Ltile) return;
  const int key1 = min(key0 + p.split, Ltile);
  const int64_t row0 = bh * p.Np + i0;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, g = lane >> 5, ln = lane & 31;
  if (tid == 0) s_any = 0;
  __syncthreads();
  if (tid < kRowsWG) {
    int part = 0;
    if (tid < nrows) {
      const int ph = p.st[row0 + tid].phase;
      part = (HIST || MODE == MODE_MAX) ? ph == PH_HIST
             : (MODE == MODE_COLLECT)        ? ph == PH_COLLECT
                                             : ph == PH_EMIT;
      if (MODE == MODE_MAX) part = part && (p.st[row0 + tid].mins || p.st[row0 + tid].topp);
    }
    s_part[tid] = part;
    if (part) atomicOr(&s_any, 1);
  }
  if (COL && tid < kRowsWG) {
    s_ccnt[tid] = 0u;
    s_clo[tid] = 0xFFFFFFFFu;
    s_chi[tid] = 0u;
  }
  if (MODE == MODE_MAX && tid < kRowsWG) s_max[tid] = 0u;  // below every ordered key
  __syncthreads();
  if (!s_any) return;  // passes late in the refinement find most workgroups idle
  if (HIST) {
    for (int t = tid; t < kRowsWG * HS; t += kThreads) {
      if (MH) s_hist64[t] = 0ull;
      else s_hist[t] = 0u;
    }
    __syncthreads();
  }

  // This lane's two rows (rl = 32 * rb2 + ln): pooled query as the B operand
  // (head-dim slots 16s + 8g .. +7) and the row's interval in registers.
  bf16x8 qf[2][DS];
  bool part[2];
  int Lr[2];
  float slo[2], shi[2], bmul[2], badd[2], ts[2], smax[2];
  bool tiep[2], tiei[2];
  double ref[2];  // < 0: no masses needed
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const int rl = rb2 * 32 + ln;
    part[rb2] = rl < nrows && s_part[rl];
    const int64_t row = row0 + (rl < nrows ? rl : 0);
    const RowState& s = p.st[row];
    Lr[rb2] = s.L;
    slo[rb2] = s.s_lo;
    shi[rb2] = s.s_hi;
    bmul[rb2] = s.binv;
    badd[rb2] = s.badd;
    smax[rb2] = s.smax;
    ts[rb2] = s.tstar;
    tiep[rb2] = s.tie_partial;
    tiei[rb2] = s.tie_interval;
    ref[rb2] = (TOPP && s.topp) ? s.ref : -1.0;
    const u32x4* src = reinterpret_cast<const u32x4*>(p.qp + row * D);
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) {
      const u32x4 t = rl < nrows ? src[2 * s2 + g] : u32x4{0, 0, 0, 0};
      qf[rb2][s2] = __builtin_bit_cast(bf16x8, t);
    }
  }

  double zacc[2] = {0.0, 0.0}, macc[2] = {0.0, 0.0};
  const float tl2 = p.tau * 1.4426950408889634f;  // raw score -> log2 units
  uint32_t nacc[2] = {0u, 0u};

  const int nblk = (key1 - key0 + 31) / 32;
  // K of a 32-key block as the A operand (lane -> key ln, head-dim slots
  // 16s + 8g .. +7), from the operand-order copy: one coalesced 1 KB load per
  // head-dim step.  The next block of this wave is loaded while the current
  // one is processed (block indices are clamped, so loads past the end are safe).
  auto kload = [&](u32x4 (&dst)[DS], int blk) __attribute__((always_inline)) {
    const int kbi = min(key0 / 32 + blk, p.nkb - 1);
    const u32x4* ksrc =
        p.kop + ((static_cast<int64_t>(b) * p.Hkv + hk) * p.nkb + kbi) * (DS * 64) + lane;
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) dst[s2] = ksrc[s2 * 64];
  };
  auto kproc = [&](const u32x4 (&ka)[DS], int blk) __attribute__((always_inline)) {
    const int kb = key0 + blk * 32;
#pragma unroll
    for (int rb2 = 0; rb2 < 2; ++rb2) {
      // Raw scores s = <q_p, k> of keys kl = 16 g + e of the block.
      f32x16 acc = f32x16{};
#pragma unroll
      for (int s2 = 0; s2 < DS; ++s2)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka[s2]),
                                                      qf[rb2][s2], acc, 0, 0, 0);
      if (!part[rb2]) continue;
      const int lim = Lr[rb2] - kb;  // keys kl < lim are eligible
      // Whole block eligible for every row of the wave (all blocks but the
      // last, unless causal): the per-key test folds away.
      const bool full = !__any(lim < 32);
      auto rowproc = [&](const bool all_elig) __attribute__((always_inline)) {
        auto elig = [&](int kl) __attribute__((always_inline)) { return all_elig || kl < lim; };
        if (MODE == MODE_MAX) {
          float m = kNegInf;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int kl = 16 * g + e;
            if (elig(kl)) m = fmaxf(m, acc[e]);
          }
          m = fmaxf(m, __shfl_xor(m, 32));
          if (g == 0) atomicMax(&s_max[rb2 * 32 + ln], ord_key(m));
          return;
        }
        if (MODE == MODE_COLLECT) {
          // Two words of this lane's 16 keys (bit e: key 16 g + e): at or above
          // the interval (the kept set; the resolve step clears the candidates
          // it rejects) and above it.  Their difference is the lane's candidates.
          uint32_t wge = 0u, wgt = 0u;
#pragma unroll
          for (int e = 15; e >= 0; --e) {
            uint64_t ge = lanes_ge(acc[e], slo[rb2]), gt = lanes_gt(acc[e], shi[rb2]);
            if (!all_elig) {
              const uint64_t ok = lanes_lt(16 * g + e, lim);
              ge &= ok;
              gt &= ok;
            }
            wge = shift_in(wge, ge);
            wgt = shift_in(wgt, gt);
            if (TOPP && ref[rb2] >= 0.0 && elig(16 * g + e) && acc[e] > shi[rb2])
              macc[rb2] += static_cast<double>(__builtin_amdgcn_exp2f((acc[e] - smax[rb2]) * tl2));
          }
          nacc[rb2] += static_cast<uint32_t>(__builtin_popcount(wgt));
          const uint32_t ins = wge & ~wgt;
          const uint32_t wl = wge << (16 * g);
          const uint32_t w = wl | __shfl_xor(wl, 32);
          if (g == 0) p.bsel[(row0 + rb2 * 32 + ln) * p.W + kb / 32] = w;
          if (__any(ins != 0u)) {
            // The lane's scores go through LDS so that a candidate's score can
            // be read by its (per-lane) position.
            float* sc = s_acc + (wave * 64 + lane) * 16;
            const int csw = (lane >> 2) & 3;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
              *reinterpret_cast<f32x4*>(sc + 4 * (q4 ^ csw)) =
                  f32x4{acc[4 * q4], acc[4 * q4 + 1], acc[4 * q4 + 2], acc[4 * q4 + 3]};
            if (ins) {
              const int rl = rb2 * 32 + ln;
              uint32_t rank = atomicAdd(&s_ccnt[rl], static_cast<uint32_t>(__builtin_popcount(ins)));
              uint32_t lo_k = 0xFFFFFFFFu, hi_k = 0u;
              for (uint32_t m = ins; m; m &= m - 1u) {
                const int e = __builtin_ctz(m);
                const uint32_t okey = ord_key(sc[4 * ((e >> 2) ^ csw) + (e & 3)]);
                const uint64_t entry =
                    (static_cast<uint64_t>(okey) << 32) | (~static_cast<uint32_t>(kb + 16 * g + e));
                lo_k = min(lo_k, okey);
                hi_k = max(hi_k, okey);
                if (rank++ < kStage) {
                  s_cand[rl * kStageStride + rank - 1] = entry;
                } else {  // LDS slots of this row full: append directly
                  const int64_t row = row0 + rl;
                  const uint32_t pos = atomicAdd(&p.cand_n[row], 1u);
                  if (pos < kCand) p.cand[row * kCand + pos] = entry;
                }
              }
              atomicMin(&s_clo[rl], lo_k);
              atomicMax(&s_chi[rl], hi_k);
            }
          }
          return;
        }
        if (MODE == MODE_EMIT) {
          uint32_t wsel = 0u, wtie = 0u;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int kl = 16 * g + e;
            const bool ok = elig(kl);
            wsel |= (ok && acc[e] > ts[rb2]) ? 1u << kl : 0u;
            const bool tie = tiei[rb2] ? (acc[e] >= slo[rb2] && acc[e] <= shi[rb2])
                                       : acc[e] == ts[rb2];
            wtie |= (ok && tie) ? 1u << kl : 0u;
          }
          wsel |= __shfl_xor(wsel, 32);
          wtie |= __shfl_xor(wtie, 32);
          if (!tiep[rb2]) wsel |= wtie;
          if (g == 0) {
            const int64_t row = row0 + rb2 * 32 + ln;
            p.bsel[row * p.W + kb / 32] = wsel;
            if (tiep[rb2]) p.btie[row * p.W + kb / 32] = wtie;
          }
          return;
        }
        const int rl = rb2 * 32 + ln;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 16 * g + e;
          const float sc = acc[e];
          const bool ok = elig(kl);
          bool above = false, inside = ok;
          if (MODE != MODE_HIST0) {  // level 0: the interval is everything
            above = ok && sc > shi[rb2];
            inside = ok && !above && sc >= slo[rb2];
            nacc[rb2] += above ? 1u : 0u;
          }
          // topP: the key's softmax term relative to the row maximum, exp(tau
          // s - ref) with ref = tau * max (terms below 2^-126, a share of the
          // mass far below any tolerance, may flush to 0)
          const float mt = MASS ? __builtin_amdgcn_exp2f((sc - smax[rb2]) * tl2) : 0.0f;
          if (MASS && ref[rb2] >= 0.0 && ok) {
            if (MODE == MODE_HIST0) zacc[rb2] += static_cast<double>(mt);
            if (above) macc[rb2] += static_cast<double>(mt);
          }
          if (HIST) {
            const int bn = inside ? bin_of(sc, bmul[rb2], badd[rb2], NB) : NB;
            if (MH) {
              const uint32_t mq = ref[rb2] >= 0.0
                                      ? static_cast<uint32_t>(__builtin_fmaf(mt, 0x1p31f, 0.5f))
                                      : 0u;
              atomicAdd(reinterpret_cast<unsigned long long*>(&s_hist64[bn * kRowsWG + rl]),
                        (1ull << kMassShift) | mq);
            } else {
              atomicAdd(&s_hist[bn * kRowsWG + rl], 1u);
            }
          }
        }
      };
      if (full) rowproc(true);
      else rowproc(false);
    }
  };
  u32x4 k0[DS], k1[DS];
  kload(k0, wave);
  for (int blk = wave; blk < nblk; blk += 8) {
    kload(k1, blk + 4);
    kproc(k0, blk);
    if (blk + 4 >= nblk) break;
    kload(k0, blk + 8);
    kproc(k1, blk + 4);
  }
  if (MODE == MODE_EMIT) return;
  if (MODE == MODE_MAX) {
    __syncthreads();
    if (tid < nrows && s_part[tid]) atomicMax(&p.cand_lohi[2 * (row0 + tid) + 1], s_max[tid]);
    return;
  }

  // Reduce per-row partials: lanes (ln, g = 0 / 1) of each wave, then the 4
  // waves in a fixed order (deterministic sums).
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const double z = zacc[rb2] + __shfl_xor(zacc[rb2], 32);
    const double m = macc[rb2] + __shfl_xor(macc[rb2], 32);
    const uint32_t n = nacc[rb2] + __shfl_xor(nacc[rb2], 32);
    if (g == 0) {
      s_zred[wave][rb2 * 32 + ln] = z;
      s_mred[wave][rb2 * 32 + ln] = m;
      s_nred[wave][rb2 * 32 + ln] = n;
    }
  }
  __syncthreads();
  if (COL) {  // staged candidates: one atomic per row, then the copy
    if (tid < nrows && s_part[tid]) {
      const int64_t row = row0 + tid;
      const uint32_t c = min(s_ccnt[tid], static_cast<uint32_t>(kStage));
      s_cbase[tid] = c ? atomicAdd(&p.cand_n[row], c) : 0u;
      if (s_ccnt[tid]) {
        atomicMin(&p.cand_lohi[2 * row], s_clo[tid]);
        atomicMax(&p.cand_lohi[2 * row + 1], s_chi[tid]);
      }
    }
    __syncthreads();
    for (int t = tid; t < nrows * kStage; t += kThreads) {
      const int rl = t / kStage, j = t % kStage;
      if (!s_part[rl] || j >= static_cast<int>(min(s_ccnt[rl], static_cast<uint32_t>(kStage)))) continue;
      const uint32_t pos = s_cbase[rl] + j;
      if (pos < kCand) p.cand[(row0 + rl) * kCand + pos] = s_cand[rl * kStageStride + j];
    }
  }
  if (tid < nrows && s_part[tid]) {
    const int64_t row = row0 + tid;
    const double z = ((s_zred[0][tid] + s_zred[1][tid]) + s_zred[2][tid]) + s_zred[3][tid];
    const double m = ((s_mred[0][tid] + s_mred[1][tid]) + s_mred[2][tid]) + s_mred[3][tid];
    const uint32_t n = s_nred[0][tid] + s_nred[1][tid] + s_nred[2][tid] + s_nred[3][tid];
    p.n_above[row * p.nsplit + sp] = n;
    p.m_above[row * p.nsplit + sp] = m;
    if (MODE == MODE_HIST0) p.zpart[row * p.nsplit + sp] = z;
  }
  if (HIST) {
    for (int t = tid; t < nrows * NB; t += kThreads) {
      const int rl = t / NB, bn = t % NB;
      const uint64_t v = MH ? s_hist64[bn * kRowsWG + rl] : 0ull;
      const uint32_t c = MH ? static_cast<uint32_t>(v >> kMassShift) : s_hist[bn * kRowsWG + rl];
      if (c && s_part[rl]) {
        atomicAdd(&p.hist[(row0 + rl) * kBins + bn], c);
        const uint64_t m = v & ((1ull << kMassShift) - 1ull);
        if (MH && m)
          atomicAdd(reinterpret_cast<unsigned long long*>(&p.hmass[(row0 + rl) * kBins + bn]),
                    static_cast<unsigned long long>(m));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Level-0 bins of topK rows from a sample of their scores: every
// kSampleStride-th 32-key block of the row's eligible keys.  One workgroup per
// 64 pooled rows walks all of their sampled blocks twice (the second walk hits
// L2), with the score pass's MFMA sequence:
//   1. Moments: for any set of values with mean mu and deviation sigma, at
//      most a fraction 1 / (1 + a^2) lies at or above mu + a sigma, and as much
//      at or below mu - a sigma (Cantelli's inequality); with a = sqrt((L - k)
//      / k) above and sqrt((k - 1) / (L - k + 1)) below, the k-th largest of L
//      scores lies between (widened for sampling).
//   2. A histogram of the sampled scores over that bracket: the k-th largest
//      key's rank among the n sampled ones is about k n / L, with deviation
//      sqrt(n p (1 - p)) for independent samples (p = k / L).  The level-0
//      bins span the sampled values between the ranks k n / L -/+ (12 sd + 4):
//      6 deviations at twice the independent spread, since sampled blocks of
//      32 consecutive keys are correlated.
// Both only place the bins: keys outside fall into the end bins, and a cut
// that lands there costs a level (the next spans that bin's actual extent),
// never a wrong set.  Rows with fewer than 64 (moments) or 256 (histogram)
// sampled keys keep the wider bins.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void k_sample_bracket(SelParams p) {
  constexpr int DS = D / 16;
  __shared__ uint32_t s_hist[(kSampleBins + 1) * kRowsWG];  // bin-major, as in the score pass
  __shared__ float s_m1[4][kRowsWG], s_m2[4][kRowsWG];
  __shared__ uint32_t s_n[4][kRowsWG];
  __shared__ float s_mul[kRowsWG], s_add[kRowsWG];
  __shared__ int s_part[kRowsWG];
  const int64_t item = xcd_work_item(p.per_xcd);
  if (item >= p.items) return;
  const int rb = static_cast<int>(item % p.nrb);
  const int64_t bh = item / p.nrb;
  const int b = static_cast<int>(bh / p.Hq), h = static_cast<int>(bh % p.Hq);
  const int hk = h / p.group;
  const int i0 = rb * kRowsWG;
  const int nrows = min(kRowsWG, p.Np - i0);
  const int Ltile = eligible(i0 + nrows - 1, p.P, p.N, p.causal);
  const int64_t row0 = bh * p.Np + i0;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, g = lane >> 5, ln = lane & 31;
  if (tid < kRowsWG) {
    int part = 0;
    if (tid < nrows) {
      const RowState& st = p.st[row0 + tid];
      part = st.phase == PH_HIST && st.level == 0 && !st.topp;
    }
    s_part[tid] = part;
  }
  for (int t = tid; t < (kSampleBins + 1) * kRowsWG; t += kThreads) s_hist[t] = 0u;
  __syncthreads();

  bf16x8 qf[2][DS];
  bool part[2];
  int Lr[2];
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const int rl = rb2 * 32 + ln;
    part[rb2] = rl < nrows && s_part[rl];
    Lr[rb2] = rl < nrows ? p.st[row0 + rl].L : 0;
    const u32x4* src = reinterpret_cast<const u32x4*>(p.qp + (row0 + (rl < nrows ? rl : 0)) * D);
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) {
      const u32x4 t = rl < nrows ? src[2 * s2 + g] : u32x4{0, 0, 0, 0};
      qf[rb2][s2] = __builtin_bit_cast(bf16x8, t);
    }
  }
  // Sampled block j is key block kSampleStride * j: keys [32 kSampleStride j, +32).
  const int nsb = (Ltile + 32 * kSampleStride - 1) / (32 * kSampleStride);
  auto scores = [&](int j, int rb2, const u32x4 (&ka)[DS]) __attribute__((always_inline)) {
    f32x16 acc = f32x16{};
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka[s2]),
                                                    qf[rb2][s2], acc, 0, 0, 0);
    return acc;
  };
  auto kload = [&](u32x4 (&dst)[DS], int j) __attribute__((always_inline)) {
    const int kbi = min(kSampleStride * j, p.nkb - 1);
    const u32x4* ksrc =
        p.kop + ((static_cast<int64_t>(b) * p.Hkv + hk) * p.nkb + kbi) * (DS * 64) + lane;
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) dst[s2] = ksrc[s2 * 64];
  };
  // This wave's sampled blocks j = wave, wave + 4, ..., each block's K loaded
  // one block ahead (kload clamps the index, so loads past the end are safe).
  auto walk = [&](auto&& body) __attribute__((always_inline)) {
    u32x4 k0[DS], k1[DS];
    kload(k0, wave);
    for (int j = wave; j < nsb; j += 8) {
      kload(k1, j + 4);
      body(j, k0);
      if (j + 4 >= nsb) break;
      kload(k0, j + 8);
      body(j + 4, k1);
    }
  };

  // 1. Moments of the sampled scores.
  float m1[2] = {0.0f, 0.0f}, m2[2] = {0.0f, 0.0f};
  uint32_t cnt[2] = {0u, 0u};
  walk([&](int j, const u32x4 (&ka)[DS]) __attribute__((always_inline)) {
    const int kb = 32 * kSampleStride * j;
#pragma unroll
    for (int rb2 = 0; rb2 < 2; ++rb2) {
      const f32x16 acc = scores(j, rb2, ka);
      const int lim = Lr[rb2] - kb;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kl = 16 * g + e;
        const float sc = kl < lim ? acc[e] : 0.0f;
        m1[rb2] += sc;
        m2[rb2] = __builtin_fmaf(sc, sc, m2[rb2]);
        cnt[rb2] += kl < lim ? 1u : 0u;
      }
    }
  });
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const float a = m1[rb2] + __shfl_xor(m1[rb2], 32);
    const float c = m2[rb2] + __shfl_xor(m2[rb2], 32);
    const uint32_t n = cnt[rb2] + __shfl_xor(cnt[rb2], 32);
    if (g == 0) {
      s_m1[wave][rb2 * 32 + ln] = a;
      s_m2[wave][rb2 * 32 + ln] = c;
      s_n[wave][rb2 * 32 + ln] = n;
    }
  }
  __syncthreads();
  if (tid < kRowsWG) {  // the Cantelli bracket of row tid
    float mul = 0.0f, add = 0.0f;
    if (s_part[tid]) {
      RowState& st = p.st[row0 + tid];
      const double n = static_cast<double>(s_n[0][tid] + s_n[1][tid] + s_n[2][tid] + s_n[3][tid]);
      const double a1 = ((static_cast<double>(s_m1[0][tid]) + s_m1[1][tid]) + s_m1[2][tid]) + s_m1[3][tid];
      const double a2 = ((static_cast<double>(s_m2[0][tid]) + s_m2[1][tid]) + s_m2[2][tid]) + s_m2[3][tid];
      const int L = st.L, k = st.k_target;
      if (n >= 64.0 && k < L) {
        const double mu = a1 / n;
        const double sd = sqrt(fmax(a2 / n - mu * mu, 0.0));
        if (sd > 0.0) {
          const double a_hi = sqrt(static_cast<double>(L - k) / k);
          const double a_lo = sqrt(static_cast<double>(k - 1) / (L - k + 1));
          const double widen = 1.2 + 4.0 / sqrt(n);
          const float lo = fmaxf(static_cast<float>(mu - (widen * a_lo + 0.25) * sd), st.blo);
          const float hi = fminf(static_cast<float>(mu + (widen * a_hi + 0.25) * sd), -st.blo);
          if (hi > lo) set_bins(st, lo, static_cast<float>(kBins) / (hi - lo));
        }
      }
      // sampled scores go into bins of half the level-0 width over the same range
      // (both factors exact powers of two)
      static_assert(kSampleBins == 2 * kBins, "sample bins halve the level-0 bins");
      mul = 2.0f * st.binv;
      add = 2.0f * st.badd;
      if (!(n >= 256.0 && k < L)) s_part[tid] = 0;  // too few samples for the quantile step
    }
    s_mul[tid] = mul;
    s_add[tid] = add;
  }
  __syncthreads();

  // 2. Histogram of the sampled scores over those bins.
  float bmul[2], badd[2];
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const int rl = rb2 * 32 + ln;
    part[rb2] = rl < nrows && s_part[rl];
    bmul[rb2] = s_mul[rl];
    badd[rb2] = s_add[rl];
  }
  walk([&](int j, const u32x4 (&ka)[DS]) __attribute__((always_inline)) {
    const int kb = 32 * kSampleStride * j;
#pragma unroll
    for (int rb2 = 0; rb2 < 2; ++rb2) {
      const f32x16 acc = scores(j, rb2, ka);
      if (!part[rb2]) continue;
      const int lim = Lr[rb2] - kb;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kl = 16 * g + e;
        const int bn = kl < lim ? bin_of(acc[e], bmul[rb2], badd[rb2], kSampleBins) : kSampleBins;
        atomicAdd(&s_hist[bn * kRowsWG + rb2 * 32 + ln], 1u);
      }
    }
  });
  __syncthreads();
  if (tid < kRowsWG && s_part[tid]) {  // the quantile band of row tid
    RowState& st = p.st[row0 + tid];
    uint32_t n = 0;
    for (int bn = 0; bn < kSampleBins; ++bn) n += s_hist[bn * kRowsWG + tid];
    const double pk = static_cast<double>(st.k_target) / st.L;
    const double mid = pk * n;
    const double margin = 12.0 * sqrt(n * pk * (1.0 - pk)) + 4.0;
    const double r_top = mid - margin, r_bot = mid + margin;  // ranks from the top
    int bt = kSampleBins - 1, bb = 0;
    bool have_top = r_top < 1.0;
    double c = 0.0;
    for (int bn = kSampleBins - 1; bn >= 0; --bn) {
      c += s_hist[bn * kRowsWG + tid];
      if (!have_top && c >= r_top) { bt = bn; have_top = true; }
      if (c >= r_bot) { bb = bn; break; }
    }
    const float w = 0.5f / st.binv;  // width of a sample bin
    const float lo = bb == 0 ? st.blo : st.blo + static_cast<float>(bb) * w;
    const float hi = st.blo + static_cast<float>(bt + 1) * w;
    if (hi > lo) set_bins(st, lo, static_cast<float>(kBins) / (hi - lo));
  }
}

// ---------------------------------------------------------------------------
// topP rows: the row maximum from the MAX pass becomes the softmax reference
// (ref = tau * max, so every mass term exp(tau s - ref) is at most 1 and the
// row's terms fit fp32 down to a mass far below any tolerance), and the
// level-0 bins span the kTopPRange nats below the maximum (narrow bins where
// the mass is, so that each bin's mass sum is tight); keys further down hold
// a share of the mass below e^-40 each and fall into bin 0, which a later
// level spans to its actual extent if the cut should lie there.  One thread
// per row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_topp_ref(SelParams p) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= p.rows) return;
  RowState& s = p.st[r];
  if (s.phase != PH_HIST || !s.topp) return;
  const float mx = ord_val(p.cand_lohi[2 * r + 1]);
  p.cand_lohi[2 * r + 1] = 0u;  // ready for the collect pass
  s.smax = mx;
  s.ref = static_cast<double>(mx) * static_cast<double>(p.tau);  // exact product
  const float lo = fmaxf(mx - kTopPRange / p.tau, s.blo);
  set_bins(s, lo, static_cast<float>(kBins) / fmaxf(mx - lo, FLT_MIN));
}

// ---------------------------------------------------------------------------
// minS (Eq. 3): a key is kept when tau * s >= tau * max - alpha, i.e. when its
// raw score s >= max - alpha / tau.  The first interval is [threshold, max]:
// the level-0 pass counts the keys in it; the resolve step either emits them
// all (at most cap) or keeps the cap best (topK(cap), counted as clamped).
// One thread per row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_mins(SelParams p) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= p.rows) return;
  RowState& s = p.st[r];
  if (s.phase != PH_HIST || !s.mins) return;
  const float mx = ord_val(p.cand_lohi[2 * r + 1]);
  p.cand_lohi[2 * r + 1] = 0u;  // ready for the collect pass
  const float top = static_cast<float>(s.ref / static_cast<double>(p.tau));  // >= every |s|
  const double t = static_cast<double>(mx) - row_param(p, r) / static_cast<double>(p.tau);
  float tf = static_cast<float>(t);
  if (static_cast<double>(tf) > t) tf = ord_val(ord_key(tf) - 1u);  // round down: keep ties
  tf = fmaxf(tf, -top);
  const float hi = fmaxf(mx, tf);
  s.s_lo = tf;
  s.s_hi = FLT_MAX;
  if (p.mins_direct) {  // no block can exceed cap: emit s >= threshold at once
    s.mins = 0;
    s.tstar = tf;
    s.tie_partial = 0;
    s.tie_interval = 0;
    s.k_eq = 0;
    s.phase = PH_EMIT;
    atomicAdd(&p.nact[kEmitSlot], 1u);
    return;
  }
  set_bins(s, tf, static_cast<float>(kBins) / fmaxf(hi - tf, FLT_MIN));
}

// ---------------------------------------------------------------------------
// Cross-tile minS (Algorithm 1; Sec. 3.1.3).  Keys fall into groups of gs =
// tile * group_tiles consecutive keys (groups start at key 0); inside a group
// the tiles of `tile` keys are taken in key order and a key of tile t is kept
// when its score is >= (largest score of the group's tiles 0..t) - alpha.
// A workgroup owns 64 pooled rows and one split of keys; each wave walks whole
// segments of the split in key order and keeps the running maximum of each of
// its rows in a register.  A segment is one group (a 32-key block when groups
// are smaller); when groups span more than a split (tiled_carry), each wave
// takes one quarter of the split and starts from the maximum of the group's
// earlier quarters, which the MAXQ pass (EMIT = false) and k_tiled_carry
// provide.  The pass sets one bit per kept key; k_compact lists them.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float tiled_threshold(float m, double a) {
  // Largest float <= m - a (exact, so a key at the threshold is kept).
  const double t = static_cast<double>(m) - a;
  float tf = static_cast<float>(t);
  if (static_cast<double>(tf) > t) tf = ord_val(ord_key(tf) - 1u);
  return tf;
}

template <int D, bool EMIT>
__global__ __launch_bounds__(kThreads) void k_mins_tiled(SelParams p) {
  constexpr int DS = D / 16;
  const int64_t item = xcd_work_item(p.per_xcd);
  if (item >= p.items) return;
  const int rb = static_cast<int>(item % p.nrb);
  const int64_t rest = item / p.nrb;
  const int sp = static_cast<int>(rest % p.nsplit);
  const int64_t bh = rest / p.nsplit;
  const int b = static_cast<int>(bh / p.Hq), h = static_cast<int>(bh % p.Hq);
  const int hk = h / p.group;
  const int i0 = rb * kRowsWG;
  const int nrows = min(kRowsWG, p.Np - i0);
  const int Ltile = eligible(i0 + nrows - 1, p.P, p.N, p.causal);
  const int key0 = sp * p.split;
  if (key0 >= Ltile) return;
  const int key1 = min(key0 + p.split, Ltile);
  const int64_t row0 = bh * p.Np + i0;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 5, ln = lane & 31;
  const int SB = p.tiled_sb;
  const int nblk = (key1 - key0 + 31) / 32;
  if (wave * SB >= nblk) return;  // no segment left for this wave (no barriers below)
  const int nq = 4 * p.nsplit;    // quarters per row in qmax

  // This lane's two rows (rl = 32 * rb2 + ln): pooled query (B operand), the
  // row's eligible keys, running maximum and current threshold.
  bf16x8 qf[2][DS];
  int Lr[2];
  bool have[2];
  float m[2], thr[2];
  const double a_raw = row_param(p, row0) * p.sqrt_d;  // alpha of this head in raw-score units
#pragma unroll
  for (int rb2 = 0; rb2 < 2; ++rb2) {
    const int rl = rb2 * 32 + ln;
    have[rb2] = rl < nrows;
    const int64_t row = row0 + (have[rb2] ? rl : 0);
    Lr[rb2] = have[rb2] ? eligible(i0 + rl, p.P, p.N, p.causal) : 0;
    const u32x4* src = reinterpret_cast<const u32x4*>(p.qp + row * D);
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) {
      const u32x4 t = have[rb2] ? src[2 * s2 + g] : u32x4{0, 0, 0, 0};
      qf[rb2][s2] = __builtin_bit_cast(bf16x8, t);
    }
    m[rb2] = (EMIT && p.tiled_carry && have[rb2]) ? p.qmax[row * nq + sp * 4 + wave] : kNegInf;
    thr[rb2] = tiled_threshold(m[rb2], a_raw);
  }

  auto kload = [&](u32x4 (&dst)[DS], int blk) __attribute__((always_inline)) {
    const int kbi = min(key0 / 32 + blk, p.nkb - 1);  // clamped: loads past the end are safe
    const u32x4* ksrc =
        p.kop + ((static_cast<int64_t>(b) * p.Hkv + hk) * p.nkb + kbi) * (DS * 64) + lane;
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) dst[s2] = ksrc[s2 * 64];
  };
  // The j-th block this wave visits: segments wave, wave + 4, ... of SB blocks.
  auto blk_of = [&](int j) __attribute__((always_inline)) {
    return ((j / SB) * 4 + wave) * SB + j % SB;
  };
  const uint32_t gmask = static_cast<uint32_t>(p.tiled_gs) - 1u;
  const bool two_tiles = p.tiled_tile == 16;

  auto proc = [&](const u32x4 (&ka)[DS], int blk) __attribute__((always_inline)) {
    const int kb = key0 + blk * 32;
#pragma unroll
    for (int rb2 = 0; rb2 < 2; ++rb2) {
      // Raw scores of keys kl = 16 g + e of the block (with 16-key tiles,
      // lane group g holds tile g).
      f32x16 acc = f32x16{};
#pragma unroll
      for (int s2 = 0; s2 < DS; ++s2)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ka[s2]),
                                                      qf[rb2][s2], acc, 0, 0, 0);
      if (!have[rb2]) continue;
      const int lim = Lr[rb2] - kb;  // keys kl < lim are eligible
      if (!EMIT) {
        float tm = kNegInf;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 16 * g + e;
          if (kl < lim) tm = fmaxf(tm, acc[e]);
        }
        m[rb2] = fmaxf(m[rb2], tm);
        continue;
      }
      float tm = kNegInf;  // this lane's 16 keys
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kl = 16 * g + e;
        if (kl < lim) tm = fmaxf(tm, acc[e]);
      }
      const float tm_x = __shfl_xor(tm, 32);  // the other lane group's
      // The running maximum through the tile starting at key toff of the block
      // (both lanes of a row compute the same values).
      auto advance = [&](const float tmax, const int toff) __attribute__((always_inline)) {
        const bool fresh = (static_cast<uint32_t>(kb + toff) & gmask) == 0u;  // a group starts
        const float mn = fmaxf(fresh ? kNegInf : m[rb2], tmax);
        if (__any(mn != m[rb2])) thr[rb2] = tiled_threshold(mn, a_raw);
        m[rb2] = mn;
      };
      float my_thr;
      if (two_tiles) {
        advance(g ? tm_x : tm, 0);  // tile 0: keys 0-15, lane group 0
        const float thr0 = thr[rb2];
        advance(g ? tm : tm_x, 16);  // tile 1: keys 16-31, lane group 1
        my_thr = g ? thr[rb2] : thr0;
      } else {
        advance(fmaxf(tm, tm_x), 0);
        my_thr = thr[rb2];
      }
      uint32_t w = 0u;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kl = 16 * g + e;
        w |= (kl < lim && acc[e] >= my_thr) ? 1u << kl : 0u;
      }
      w |= __shfl_xor(w, 32);
      if (g == 0) p.bsel[(row0 + rb2 * 32 + ln) * p.W + kb / 32] = w;
    }
  };

  u32x4 k0[DS], k1[DS];
  int j = 0;
  kload(k0, blk_of(0));
  for (; blk_of(j + 1) < nblk; j += 2) {
    kload(k1, blk_of(j + 1));
    proc(k0, blk_of(j));
    kload(k0, blk_of(j + 2));
    proc(k1, blk_of(j + 1));
  }
  if (blk_of(j) < nblk) proc(k0, blk_of(j));

  if (!EMIT) {  // this wave's quarter: its maximum per row
#pragma unroll
    for (int rb2 = 0; rb2 < 2; ++rb2) {
      const float mx = fmaxf(m[rb2], __shfl_xor(m[rb2], 32));
      if (have[rb2] && g == 0) p.qmax[(row0 + rb2 * 32 + ln) * nq + sp * 4 + wave] = mx;
    }
  }
}

// Per row: replace each quarter's maximum by the running maximum of the
// group's earlier quarters (-inf where a group starts).  One thread per row.
__global__ __launch_bounds__(256) void k_tiled_carry(SelParams p) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= p.rows) return;
  const int i = static_cast<int>(r % p.Np);
  const int L = eligible(i, p.P, p.N, p.causal);
  const int rq = p.split / 4;
  const int nq = 4 * p.nsplit;
  const int used = (L + rq - 1) / rq;  // quarters holding eligible keys of this row
  float run = kNegInf;
  for (int q = 0; q < used; ++q) {
    if ((static_cast<int64_t>(q) * rq) % p.tiled_gs == 0) run = kNegInf;
    const float x = p.qmax[r * nq + q];
    p.qmax[r * nq + q] = run;
    run = fmaxf(run, x);
  }
}

// Row state the compact step reads, for cross-tile minS launches.
__global__ __launch_bounds__(256) void k_tiled_init(SelParams p) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= p.rows) return;
  RowState& s = p.st[r];
  s.L = eligible(static_cast<int>(r % p.Np), p.P, p.N, p.causal);
  s.tie_partial = 0;
  s.k_eq = 0;
  s.phase = PH_EMIT;
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves (no LDS):
// shifts by 1, 2, 4, 8 inside each 16-lane row, then row 0's total into row 1
// and row 2's into row 3 (broadcast of lane 15), and rows 0-1's total into
// rows 2-3 (broadcast of lane 31).  Lanes without a source add 0.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// ---------------------------------------------------------------------------
// Resolve after a HIST pass: one wave per row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_resolve_hist(SelParams p, int level) {
  if (level > 0 && p.nact[level] == 0u) return;
  const int64_t r = blockIdx.x;
  RowState& s = p.st[r];
  if (s.phase != PH_HIST || s.level != level) return;
  __shared__ uint32_t hs[kBins];
  __shared__ double hm[kBins];
  const int lane = threadIdx.x;
  const int nb = kBins;
  for (int t = lane; t < nb; t += 64) {
    hs[t] = p.hist[r * kBins + t];
    p.hist[r * kBins + t] = 0u;  // ready for the next level
    if (s.topp) {
      hm[t] = static_cast<double>(p.hmass[r * kBins + t]) * kMassUnit;
      p.hmass[r * kBins + t] = 0ull;
    }
  }
  __syncthreads();
  // Sum the per-split statistics in split order (every lane alike).
  const int i = static_cast<int>(r % p.Np);
  const int rb = i / kRowsWG;
  const int i_last = min(p.Np, (rb + 1) * kRowsWG) - 1;
  const int Ltile = eligible(i_last, p.P, p.N, p.causal);
  const int ns = (Ltile + p.split - 1) / p.split;
  // (The mass above the interval of topP rows is carried in the row state.)
  uint32_t nab = 0;
  double z = 0.0;
  for (int q = 0; q < ns; ++q) {
    nab += p.n_above[r * p.nsplit + q];
    if (level == 0) z += p.zpart[r * p.nsplit + q];
  }
  // Count cut (topK, and minS rows over cap) across the wave: lane l holds
  // bins nb - 1 - 2 l - j (j < 2, descending), and the scan counts the keys in
  // every bin from the top through them.  The cut bin is the highest bin whose
  // count from the top reaches the target rank (never an empty bin: the bin
  // above it fell short); `cut_above` counts the keys in the bins above it.
  static_assert(kBins == 2 * 64, "two bins per lane");
  constexpr int per = 2;
  int hb[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) hb[j] = static_cast<int>(hs[nb - 1 - per * lane - j]);
  const int lsum = hb[0] + hb[1];
  const int incl = wave_incl_scan(lsum);
  const int total_in = __builtin_amdgcn_readlane(incl, 63);
  int cut_bin = -1, cut_above = 0;
  if (!s.topp) {
    const bool over_cap = s.mins && static_cast<uint32_t>(total_in) + nab >
                                        static_cast<uint32_t>(p.cap);
    const int kt = over_cap ? static_cast<int>(p.cap) : s.k_target;
    const int want = max(kt - static_cast<int>(nab), 1);
    const uint64_t hit = __ballot(incl >= want);
    if (hit != 0ull) {
      const int src = __builtin_ctzll(hit);  // lowest lane: the highest bins
      int c = incl - lsum, jb = 1;  // in lane src: the first j whose count reaches `want`
      if (c + hb[0] >= want) jb = 0;
      else c += hb[0];
      cut_bin = __builtin_amdgcn_readlane(nb - 1 - per * lane - jb, src);
      cut_above = __builtin_amdgcn_readlane(c, src);
    } else {  // cannot happen unless the counts disagree: the lowest non-empty bin
      const uint64_t ne = __ballot(lsum > 0);
      if (ne != 0ull) {
        const int src = 63 - __builtin_clzll(ne);  // highest lane: the lowest bins
        const int jb = hb[1] != 0 ? 1 : 0;
        cut_bin = __builtin_amdgcn_readlane(nb - 1 - per * lane - jb, src);
        const int h_low = jb == 0 ? hb[0] : hb[1];
        cut_above = total_in - __builtin_amdgcn_readlane(h_low, src);
      }
    }
  }
  if (lane != 0) return;
  if (level == 0 && s.topp) {
    s.Z = z;
    s.pZ = row_param(p, r) * z;
  }
  const float lo = s.blo, inv = s.binv, add = s.badd;
  const float top = static_cast<float>(s.ref / static_cast<double>(p.tau));  // raw score bound
  int ba = -1, bb = -1;
  uint32_t above_bins = 0;  // keys in bins above bb (inside the interval)
  if (s.mins) {  // level 0 of a minS row: the histogram counts the keys it keeps
    s.mins = 0;
    const uint32_t tot = static_cast<uint32_t>(total_in) + nab;
    if (tot <= static_cast<uint32_t>(p.cap)) {
      s.tstar = s.s_lo;  // the emit pass keeps s > t* and, all ties kept, s == t*
      s.tie_partial = 0;
      s.tie_interval = 0;
      s.k_eq = 0;
      s.count = static_cast<int>(tot);
      s.level = level + 1;
      s.phase = PH_EMIT;
      atomicAdd(&p.nact[kEmitSlot], 1u);
      return;
    }
    s.k_target = static_cast<int>(p.cap);  // more than cap: keep the cap best
    s.clamped = 1;
  }
  if (!s.topp) {
    ba = bb = cut_bin;  // from the wave scan above (target: k_target, or cap for minS)
    above_bins = static_cast<uint32_t>(cut_above);
  } else {
    // Mass bounds per bin: from its score range (count times the mass at
    // each edge) and, at level 0, from its mass sum -- the terms exp(tau s -
    // ref) <= 1, each within a relative (2 + |x|) 2^-22 (exp2 and the rounding
    // of its argument x = (s - max) tau log2 e, |x| bounded by the bin's lower
    // edge), rounded to the 2^-31 grid (<= 2^-32 each) and summed exactly.
    // Later levels split one level-0 bin 128 ways, so that the edge bounds
    // of a bin differ by a factor of ~1.003 at most.  The mass above the
    // interval lies in [mab_lo, mab_hi].  The cut bin range runs from the
    // first bin the cut for T may lie in down to the last one the cut for
    // T - kTopPMassSlack * Z may lie in: usually one bin.
    const double T_lo = s.pZ - s.mab_hi;
    const double Trel = s.pZ - s.mab_lo - kTopPMassSlack * s.Z;
    const float k1 = p.tau * 1.4426950408889634f;
    const float w = 1.0f / inv;
    const float slop = fabsf(w) * 1e-3f + fabsf(lo) * 1e-6f;
    double before_lo = 0.0, before_hi = 0.0, cut_lo = 0.0, cut_hi = 0.0;
    int top_nonempty = -1;
    for (int bn = nb - 1; bn >= 0; --bn) {
      if (hs[bn] == 0) continue;
      if (top_nonempty < 0) top_nonempty = bn;
      float e_lo = lo + static_cast<float>(bn) * w - slop;
      float e_hi = lo + static_cast<float>(bn + 1) * w + slop;
      if (level == 0 && bn == 0) e_lo = -FLT_MAX;
      if (level == 0 && bn == nb - 1) e_hi = top;
      double mlo = hs[bn] * mass_term(e_lo, p.tau, s.ref);
      double mhi = hs[bn] * mass_term(fminf(e_hi, top), p.tau, s.ref);
      if (level == 0) {
        const double grid = static_cast<double>(hs[bn]) * 0x1p-32;
        const double xmax = (static_cast<double>(s.smax) - static_cast<double>(e_lo)) * k1;
        const double eps = fmin(1.0, (2.0 + xmax) * 0x1p-22);
        mlo = fmax(mlo, hm[bn] * (1.0 - eps) - grid);
        mhi = fmin(mhi, hm[bn] * (1.0 + eps) + grid);
      }
      if (bb < 0) {
        if (before_hi + mhi >= T_lo) {  // the mass through bn may reach T
          bb = ba = bn;
          cut_lo = before_lo;
          cut_hi = before_hi;
        }
      } else if (before_lo < Trel) {
        ba = bn;  // the mass above bn may still fall short of T - slack
      } else {
        break;
      }
      before_lo += mlo;
      before_hi += mhi;
      if (bb >= 0 && before_lo >= Trel) break;
    }
    if (bb < 0) {  // T <= 0 or rounding: the cut is at the top of the interval
      bb = ba = top_nonempty >= 0 ? top_nonempty : 0;
    }
    s.mab_lo += cut_lo;  // the bins above bb join the mass above the interval
    s.mab_hi += cut_hi;
  }
  uint32_t inside = 0;
  for (int bn = ba; bn <= bb; ++bn) inside += hs[bn];
  (void)above_bins;
  // New interval: the chosen bins of this level, as exact float bounds.
  narrow(s.s_lo, s.s_hi, inv, add, ba, bb, nb);
  const int nl = level + 1;
  s.level = nl;
  if (inside <= static_cast<uint32_t>(kCand) || nl >= kLevels) {
    s.phase = PH_COLLECT;
  } else {
    atomicAdd(&p.nact[nl], 1u);
    // An end bin also holds the scores beyond the bin range (level 0 of topK
    // rows bins a sampled bracket, not the whole range): the next level spans
    // the chosen bins' actual extent, within the Cauchy-Schwarz bound.
    const float nlo = ba == 0 ? fmaxf(s.s_lo, -top) : lo + static_cast<float>(ba) / inv;
    const float nhi = bb == nb - 1 ? fminf(s.s_hi, top) : lo + static_cast<float>(bb + 1) / inv;
    set_bins(s, nlo, static_cast<float>(nb) / fmaxf(nhi - nlo, FLT_MIN));
  }
}

// ---------------------------------------------------------------------------
// Resolve after COLLECT: sort the candidates (score desc, index asc) and fix
// the cut.  One workgroup of 256 threads per row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_resolve_cand(SelParams p) {
  const int64_t r = blockIdx.x;
  RowState& s = p.st[r];
  if (s.phase != PH_COLLECT) return;
  __shared__ uint64_t kin[kCand];  // candidates as collected
  __shared__ uint64_t key[kCand];  // sorted, descending
  __shared__ int res[4];
  const int tid = threadIdx.x;
  const uint32_t nc_raw = p.cand_n[r];
  const int nc = static_cast<int>(min(nc_raw, static_cast<uint32_t>(kCand)));
  for (int t = tid; t < nc; t += 256) kin[t] = p.cand[r * kCand + t];
  __syncthreads();
  // Counting sort: the keys (ordered score, complemented index) are distinct,
  // so a candidate's place is the number of larger ones.  The reads of kin[j]
  // are the same address across the workgroup (LDS broadcast).
  for (int t = tid; t < nc; t += 256) {
    const uint64_t mine = kin[t];
    int rank = 0;
#pragma unroll 4
    for (int j = 0; j < nc; ++j) rank += kin[j] > mine ? 1 : 0;
    key[rank] = mine;
  }
  __syncthreads();
  // statistics of the final interval
  const int64_t bh = r / p.Np;
  (void)bh;
  const int i = static_cast<int>(r % p.Np);
  const int rb = i / kRowsWG;
  const int i_last = min(p.Np, (rb + 1) * kRowsWG) - 1;
  const int Ltile = eligible(i_last, p.P, p.N, p.causal);
  const int ns = (Ltile + p.split - 1) / p.split;
  if (tid == 0) {
    uint32_t nab = 0;
    double mab = 0.0;
    for (int q = 0; q < ns; ++q) {
      nab += p.n_above[r * p.nsplit + q];
      mab += p.m_above[r * p.nsplit + q];
    }
    const bool overflow = nc_raw > static_cast<uint32_t>(kCand);
    const bool all_tied = p.cand_lohi[2 * r] == p.cand_lohi[2 * r + 1];
    int n_sel = 0;      // keys kept from the interval (the first n_sel in sorted order)
    int count = 0;
    if (!s.topp) {
      n_sel = s.k_target - static_cast<int>(nab);
    } else {
      const double T = s.pZ - mab;
      if (overflow && all_tied) {
        const double term = mass_term(ord_val(p.cand_lohi[2 * r]), p.tau, s.ref);
        double need = T > 0.0 ? ceil(T / term) : 1.0;
        n_sel = static_cast<int>(fmin(fmax(need, 1.0), static_cast<double>(nc_raw)));
      } else {
        double c = 0.0;
        n_sel = nc;
        for (int t = 0; t < nc; ++t) {
          c += mass_term(ord_val(static_cast<uint32_t>(key[t] >> 32)), p.tau, s.ref);
          if (c >= T) { n_sel = t + 1; break; }
        }
        if (T <= 0.0) n_sel = 1;
      }
    }
    count = static_cast<int>(nab) + n_sel;
    // threshold modes: clamp to cap (keep the cap best)
    if (s.topp && count > p.cap) {
      if (p.cap <= static_cast<int64_t>(nab)) {
        // the cap cut lies above this interval: rerun this row as topK(cap)
        s.topp = 0;
        s.k_target = static_cast<int>(p.cap);
        s.clamped = 1;
        s.phase = PH_IDLE;
        res[0] = -1;
      } else {
        n_sel = static_cast<int>(p.cap - nab);
        count = static_cast<int>(p.cap);
        s.clamped = 1;
      }
    }
    res[1] = -1;  // no candidate bits to clear unless set below
    if (s.phase == PH_COLLECT && !overflow) {
      // The collect pass set a bit for every key at or above the interval;
      // keep the first n_sel candidates (score desc, index asc), clear the rest.
      n_sel = min(max(n_sel, 0), nc);
      res[1] = n_sel;
      s.tie_partial = 0;
      s.k_eq = 0;
      s.tstar = n_sel > 0 ? ord_val(static_cast<uint32_t>(key[n_sel - 1] >> 32)) : FLT_MAX;
      s.count = count;
      s.phase = PH_DONE;
      if (s.clamped && p.n_clamped) atomicAdd(p.n_clamped, 1);
    }
    if (s.phase == PH_COLLECT) {  // too many candidates to store: the emit pass redoes the row
      n_sel = max(n_sel, 0);
      if (overflow && all_tied) {
        s.tstar = ord_val(p.cand_lohi[2 * r]);
        s.tie_partial = n_sel < static_cast<int>(nc_raw);
        s.k_eq = n_sel;
      } else {
        // More than kCand distinct scores are left in an interval narrower
        // than the refinement resolves (after kLevels levels: only for scores
        // a few ulps apart, or the nothing-kept case): its keys count as
        // tied at the cut and the first n_sel by index are kept.
        s.tstar = s.s_hi;
        s.tie_interval = 1;
        s.tie_partial = 1;
        s.k_eq = n_sel;
      }
      s.count = count;
      s.phase = PH_EMIT;
      atomicAdd(&p.nact[kEmitSlot], 1u);
      if (s.clamped && p.n_clamped) atomicAdd(p.n_clamped, 1);
    }
  }
  __syncthreads();
  const int keep = res[1];
  if (keep >= 0) {
    for (int t = keep + tid; t < nc; t += 256) {
      const uint32_t j = ~static_cast<uint32_t>(key[t] & 0xFFFFFFFFull);
      atomicAnd(&p.bsel[r * p.W + j / 32], ~(1u << (j % 32)));
    }
  }
}

// ---------------------------------------------------------------------------
// Bitmasks -> ascending index lists.  One wave per row; each lane expands one
// 32-key word per step into LDS at its prefix position, then the wave copies
// the staged indices out contiguously.
// ---------------------------------------------------------------------------
// Bitmask words (64 per chunk, one per lane) whose loads are in flight
// together: the row's chunks are processed strictly in order, but their
// loads do not wait for one another.
constexpr int kCompactBatch = 8;

// Orders this wave's LDS accesses on either side (a one-wave workgroup needs
// no barrier).  Unlike __syncthreads() it does not wait for the wave's
// global loads and stores: the prefetched bitmask words stay in flight and
// the stores of the lists are not waited for.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ __launch_bounds__(64) void k_compact(SelParams p) {
  const int64_t r = blockIdx.x;
  const RowState& s = p.st[r];
  __shared__ __align__(16) int32_t stage[64 * 32 + 4];
  const int lane = threadIdx.x;
  const int L = s.L;
  const int nw = (L + 31) / 32;
  const bool tiep = s.tie_partial;
  const int k_eq = s.k_eq;
  const uint32_t* bsel = p.bsel + r * p.W;
  const uint32_t* btie = p.btie + r * p.W;
  int base = 0;      // entries listed so far
  int ties_seen = 0; // tied keys met so far (ascending index)
  int32_t* out = p.idx + r * p.cap;
  // Rows that start on 16 bytes and cannot exceed cap are stored four entries
  // per lane; the last (< 4) entries of a chunk wait in stage[0, 4) for the
  // next one, and go out one by one after the last chunk.
  const bool quads = p.quad_rows;
  int done = 0;      // entries stored (quad path)
  // keep_diag: this block's own rows, [i P, min(N, (i + 1) P))
  const int diag_lo = p.keep_diag ? static_cast<int>(r % p.Np) * p.P : 0;
  const int diag_hi = p.keep_diag ? min(p.N, diag_lo + p.P) : 0;
  // The next batch's words are loaded while this batch is listed.  Every
  // load is issued (indices past the row's words are clamped to its last one
  // and their words dropped when used), so that the compiler can count the
  // loads in flight and wait for one batch only; rows with partial ties take
  // a copy of the loop that also loads the tie words.
  const int wlast = max(nw - 1, 0);
  auto run = [&](auto tie_tag) __attribute__((always_inline)) {
  constexpr bool TIEP = decltype(tie_tag)::value;
  uint32_t mb[kCompactBatch], tb[kCompactBatch], mn[kCompactBatch], tn[kCompactBatch];
  auto load_batch = [&](uint32_t (&m)[kCompactBatch], uint32_t (&t)[kCompactBatch], int c0)
      __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kCompactBatch; ++j) {
      const int wd = min(c0 + 64 * j + lane, wlast);
      m[j] = bsel[wd];
      t[j] = TIEP ? btie[wd] : 0u;
    }
  };
  load_batch(mb, tb, 0);
  for (int c0 = 0; c0 < nw; c0 += 64 * kCompactBatch) {
    load_batch(mn, tn, c0 + 64 * kCompactBatch);
#pragma unroll
    for (int j = 0; j < kCompactBatch; ++j) {
      const int wd = c0 + 64 * j + lane;
      if (c0 + 64 * j >= nw) break;  // uniform
      uint32_t m = wd < nw ? mb[j] : 0u;
      if (TIEP) {  // keep only the first k_eq tied keys
        const uint32_t tw = wd < nw ? tb[j] : 0u;
        const int nt = __builtin_popcount(tw);
        const int incl = wave_incl_scan(nt);
        int room = k_eq - (ties_seen + incl - nt);  // ties this lane may still keep
        uint32_t t2 = tw;
        while (t2 && room > 0) {
          const uint32_t bit = t2 & (~t2 + 1u);
          m |= bit;
          t2 ^= bit;
          --room;
        }
        ties_seen += __builtin_amdgcn_readlane(incl, 63);
      }
      if (p.keep_diag) {  // the keys of the block's own rows
        const int lo = max(diag_lo - 32 * wd, 0), hi = min(diag_hi - 32 * wd, 32);
        if (lo < hi) m |= (hi == 32 ? 0xFFFFFFFFu : (1u << hi) - 1u) & ~((1u << lo) - 1u);
      }
      if (wd < nw && L - 32 * wd < 32) m &= (1u << (L - 32 * wd)) - 1u;
      const int nb = __builtin_popcount(m);
      const int pre = wave_incl_scan(nb);
      const int total = __builtin_amdgcn_readlane(pre, 63);
      const int pend = base - done;  // quad path: entries waiting in stage[0, pend), < 4
      int pos = (quads ? pend : 0) + pre - nb;
      uint32_t mm = m;
      while (mm) {
        const int bit = __builtin_ctz(mm);
        mm &= mm - 1;
        stage[pos++] = 32 * wd + bit;
      }
      wave_sync();
      if (quads) {
        const int avail = pend + total;
        const int nq = avail / 4;
        int4* out4 = reinterpret_cast<int4*>(out + done);
        const int4* st4 = reinterpret_cast<const int4*>(stage);
        for (int t = lane; t < nq; t += 64) out4[t] = st4[t];
        const int rem = avail - 4 * nq;
        const int carry = lane < rem ? stage[4 * nq + lane] : 0;
        wave_sync();
        if (lane < rem) stage[lane] = carry;
        done += 4 * nq;
      } else {
        for (int t = lane; t < total; t += 64)
          if (base + t < p.cap) out[base + t] = stage[t];
        wave_sync();
      }
      base += total;
    }
#pragma unroll
    for (int j = 0; j < kCompactBatch; ++j) {
      mb[j] = mn[j];
      tb[j] = tn[j];
    }
  }
  };
  if (tiep) run(std::true_type{});
  else run(std::false_type{});
  if (quads) {  // the last entries, fewer than 4
    wave_sync();
    if (lane < base - done) out[done + lane] = stage[lane];
  }
  const int n = min(base, static_cast<int>(p.cap));
  if (!p.unpadded)
    for (int t = n + lane; t < p.cap; t += 64) out[t] = -1;
  if (lane == 0) p.counts[r] = n;
  // Cross-tile minS keeps a block's first cap keys (key order) and counts it.
  if (lane == 0 && p.mode_tiled && base > p.cap && p.n_clamped) atomicAdd(p.n_clamped, 1);
}

__global__ __launch_bounds__(256) void k_zero_u32(uint32_t* p, int64_t n) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t < n) p[t] = 0u;
}

// ---------------------------------------------------------------------------
// Workspace layout.
// ---------------------------------------------------------------------------
struct Layout {
  size_t qp, state, hist, hmass, nab, mab, zp, cand_n, cand_lohi, cand, bsel, btie, qnorm, kmax,
      qmax, kop, nact, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

Layout layout(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t D, int32_t P, int split,
              bool topp) {
  const int64_t Np = (N + P - 1) / P;
  const int64_t rows = B * Hq * Np;
  const int64_t nsplit = (N + split - 1) / split;
  const int64_t W = (N + 31) / 32;
  Layout l{};
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align256(o + bytes); return at; };
  l.qp = take(rows * D * 2);
  l.state = take(rows * sizeof(RowState));
  l.hist = take(rows * kBins * 4);
  l.hmass = take(topp ? rows * kBins * 8 : 0);
  l.nab = take(rows * nsplit * 4);
  l.mab = take(rows * nsplit * 8);
  l.zp = take(rows * nsplit * 8);
  l.cand_n = take(rows * 4);
  l.cand_lohi = take(rows * 8);
  l.cand = take(rows * kCand * 8);
  l.bsel = take(rows * W * 4);
  l.btie = take(rows * W * 4);
  l.qnorm = take(rows * 4);
  l.kmax = take(B * Hkv * 4);
  l.qmax = take(rows * nsplit * 4 * 4);
  l.kop = take(B * Hkv * ((N + 31) / 32) * 32 * D * 2);
  l.nact = take(kActiveSlots * 4);
  l.total = o;
  return l;
}

int choose_split(int64_t B, int64_t Hq, int64_t N, int32_t P) {
  // 4096 keys (1 MB of K at D = 128): the ~64 workgroups resident on an XCD
  // cover a few splits of one head, whose K then fits the XCD's 4 MB L2.
  (void)B;
  (void)Hq;
  (void)P;
  const int64_t s = 4096;
  return static_cast<int>(N < s ? ((N + 127) / 128) * 128 : s);
}

}  // namespace

size_t select_workspace_bytes(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t D,
                              int32_t block, int32_t mode, int64_t cap) {
  (void)mode;
  (void)cap;
  return layout(B, Hq, Hkv, N, D, block, choose_split(B, Hq, N, block), mode == 1).total;
}

template <int MODE>
void score_pass(int64_t D, bool topp, dim3 grid, const SelParams& p, hipStream_t stream) {
  if (D == 128) {
    if (topp) hipLaunchKernelGGL((k_score_pass<128, MODE, true>), grid, dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((k_score_pass<128, MODE, false>), grid, dim3(kThreads), 0, stream, p);
  } else {
    if (topp) hipLaunchKernelGGL((k_score_pass<64, MODE, true>), grid, dim3(kThreads), 0, stream, p);
    else hipLaunchKernelGGL((k_score_pass<64, MODE, false>), grid, dim3(kThreads), 0, stream, p);
  }
}

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t B = a.q.B, Hq = a.q.H, Hkv = a.k.H, N = a.q.N, D = a.q.D;
  const int32_t P = a.block;
  const int64_t Np = (N + P - 1) / P;
  const int64_t rows = B * Hq * Np;
  const int split = choose_split(B, Hq, N, P);
  const Layout l = layout(B, Hq, Hkv, N, D, P, split, a.mode == 1);
  if (a.workspace_bytes < l.total) return hipErrorInvalidValue;
  char* ws = static_cast<char*>(a.workspace);
  SelParams p{};
  p.qp = reinterpret_cast<const uint16_t*>(ws + l.qp);
  p.k = static_cast<const uint16_t*>(a.k.ptr);
  p.st = reinterpret_cast<RowState*>(ws + l.state);
  p.hist = reinterpret_cast<uint32_t*>(ws + l.hist);
  p.hmass = reinterpret_cast<uint64_t*>(ws + l.hmass);
  p.n_above = reinterpret_cast<uint32_t*>(ws + l.nab);
  p.m_above = reinterpret_cast<double*>(ws + l.mab);
  p.zpart = reinterpret_cast<double*>(ws + l.zp);
  p.cand_n = reinterpret_cast<uint32_t*>(ws + l.cand_n);
  p.cand_lohi = reinterpret_cast<uint32_t*>(ws + l.cand_lohi);
  p.cand = reinterpret_cast<uint64_t*>(ws + l.cand);
  p.bsel = reinterpret_cast<uint32_t*>(ws + l.bsel);
  p.btie = reinterpret_cast<uint32_t*>(ws + l.btie);
  p.qnorm = reinterpret_cast<float*>(ws + l.qnorm);
  p.kmax = reinterpret_cast<float*>(ws + l.kmax);
  p.idx = a.idx;
  p.counts = a.counts;
  p.n_clamped = a.n_clamped;
  p.cap = a.cap;
  p.rows = rows;
  p.B = static_cast<int>(B);
  p.Hq = static_cast<int>(Hq);
  p.Hkv = static_cast<int>(Hkv);
  p.group = static_cast<int>(Hq / Hkv);
  p.N = static_cast<int>(N);
  p.P = P;
  p.Np = static_cast<int>(Np);
  p.D = static_cast<int>(D);
  p.causal = a.causal;
  p.keep_diag = a.keep_diag;
  p.unpadded = a.unpadded;
  p.quad_rows = (a.cap % 4 == 0) && (reinterpret_cast<uintptr_t>(a.idx) % 16 == 0) && a.mode != 3;
  p.split = split;
  p.nsplit = static_cast<int>((N + split - 1) / split);
  p.W = static_cast<int>((N + 31) / 32);
  p.nrb = static_cast<int>((Np + kRowsWG - 1) / kRowsWG);
  p.mode_topp = a.mode == 1;
  p.mode_mins = a.mode == 2;
  p.mins_direct = p.mode_mins && a.cap >= N;
  p.mode_tiled = a.mode == 3;
  p.qmax = reinterpret_cast<float*>(ws + l.qmax);
  p.kop = reinterpret_cast<const u32x4*>(ws + l.kop);
  p.nact = reinterpret_cast<uint32_t*>(ws + l.nact);
  p.gate = -1;
  p.nkb = static_cast<int>((N + 31) / 32);
  p.param = a.param;
  p.per_head = a.head_params != nullptr;
  if (p.per_head)
    for (int64_t h = 0; h < Hq; ++h) p.head_param[h] = a.head_params[h];
  p.tau = 1.0f / sqrtf(static_cast<float>(D));

  // Pooled queries (Eq. 2) into the workspace, contiguous [rows][D].
  hipError_t e = launch_pool(a.q, P, const_cast<uint16_t*>(p.qp), Hq * Np * D, Np * D, D, stream);
  if (e != hipSuccess) return e;
  const dim3 rgrid(static_cast<unsigned>(rows));
  const dim3 igrid(static_cast<unsigned>((rows + 255) / 256));
  {  // K in operand order, and the largest key norm per head
    hipLaunchKernelGGL(k_kmax_init, dim3(static_cast<unsigned>((B * Hkv + 255) / 256)), dim3(256),
                       0, stream, p.kmax, static_cast<int>(B * Hkv));
    const int64_t nbt = B * Hkv * p.nkb;
    const dim3 kgrid(static_cast<unsigned>((nbt + 3) / 4));
    if (D == 128)
      hipLaunchKernelGGL(k_k_operand_order<128>, kgrid, dim3(256), 0, stream, p.k, a.k.sB, a.k.sH,
                         a.k.sN, static_cast<int>(Hkv), static_cast<int>(N), p.nkb, nbt,
                         const_cast<u32x4*>(p.kop), p.kmax);
    else
      hipLaunchKernelGGL(k_k_operand_order<64>, kgrid, dim3(256), 0, stream, p.k, a.k.sB, a.k.sH,
                         a.k.sN, static_cast<int>(Hkv), static_cast<int>(N), p.nkb, nbt,
                         const_cast<u32x4*>(p.kop), p.kmax);
  }

  if (p.mode_tiled) {
    // Cross-tile minS: one emitting pass (after a quarter-maximum pass when a
    // group of tiles spans more than a split), then the lists.  Splits hold
    // whole groups when groups are at most a split long.
    const int64_t gs = static_cast<int64_t>(a.tile) * a.group_tiles;  // a power of two
    int64_t st = N < 4096 ? ((N + 127) / 128) * 128 : 4096;
    if (gs <= st) {
      const int64_t unit = gs > 128 ? gs : 128;
      if (N < 4096) st = ((N + unit - 1) / unit) * unit;
      p.tiled_carry = 0;
      p.tiled_sb = static_cast<int>((gs > 32 ? gs : 32) / 32);
    } else {
      p.tiled_carry = 1;
      p.tiled_sb = static_cast<int>(st / 128);  // a quarter of the split
    }
    p.split = static_cast<int>(st);
    p.nsplit = static_cast<int>((N + st - 1) / st);
    p.tiled_tile = a.tile;
    p.tiled_gs = static_cast<int>(gs);
    p.sqrt_d = sqrt(static_cast<double>(D));
    p.items = B * Hq * static_cast<int64_t>(p.nsplit) * p.nrb;
    p.per_xcd = (p.items + 7) / 8;
    const dim3 tgrid(static_cast<unsigned>(p.per_xcd * 8));
    hipLaunchKernelGGL(k_tiled_init, igrid, dim3(256), 0, stream, p);
    if (D == 128) {
      if (p.tiled_carry) {
        hipLaunchKernelGGL((k_mins_tiled<128, false>), tgrid, dim3(kThreads), 0, stream, p);
        hipLaunchKernelGGL(k_tiled_carry, igrid, dim3(256), 0, stream, p);
      }
      hipLaunchKernelGGL((k_mins_tiled<128, true>), tgrid, dim3(kThreads), 0, stream, p);
    } else {
      if (p.tiled_carry) {
        hipLaunchKernelGGL((k_mins_tiled<64, false>), tgrid, dim3(kThreads), 0, stream, p);
        hipLaunchKernelGGL(k_tiled_carry, igrid, dim3(256), 0, stream, p);
      }
      hipLaunchKernelGGL((k_mins_tiled<64, true>), tgrid, dim3(kThreads), 0, stream, p);
    }
    hipLaunchKernelGGL(k_compact, rgrid, dim3(64), 0, stream, p);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_qnorm, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream,
                     p.qp, rows, static_cast<int>(D), p.qnorm);
  const int64_t nh = rows * kBins;
  hipLaunchKernelGGL(k_zero_u32, dim3(static_cast<unsigned>((nh + 255) / 256)), dim3(256), 0, stream,
                     p.hist, nh);
  if (p.mode_topp)  // the bin masses (64-bit): 2 words each
    hipLaunchKernelGGL(k_zero_u32, dim3(static_cast<unsigned>((2 * nh + 255) / 256)), dim3(256), 0,
                       stream, reinterpret_cast<uint32_t*>(p.hmass), 2 * nh);
  p.items = B * Hq * static_cast<int64_t>(p.nsplit) * p.nrb;
  p.per_xcd = (p.items + 7) / 8;
  const dim3 pgrid(static_cast<unsigned>(p.per_xcd * 8));
  // Only topP rows can be sent back for a second round (count above cap).
  const int rounds = p.mode_topp ? kRounds : 1;
  for (int round = 0; round < rounds; ++round) {
    hipLaunchKernelGGL(k_sel_init, igrid, dim3(256), 0, stream, p, round);
    if (p.mode_mins) {  // minS: the row maxima fix each row's threshold
      score_pass<MODE_MAX>(D, false, pgrid, p, stream);
      hipLaunchKernelGGL(k_mins, igrid, dim3(256), 0, stream, p);
    } else if (round == 0 && p.mode_topp) {  // topP: the row maxima are the mass references
      score_pass<MODE_MAX>(D, false, pgrid, p, stream);
      hipLaunchKernelGGL(k_topp_ref, igrid, dim3(256), 0, stream, p);
    } else if (round == 0 && !p.mode_topp) {
      SelParams ps = p;  // one work item per 64 pooled rows (no key splits)
      ps.items = B * Hq * static_cast<int64_t>(p.nrb);
      ps.per_xcd = (ps.items + 7) / 8;
      const dim3 sgrid(static_cast<unsigned>(ps.per_xcd * 8));
      if (D == 128)
        hipLaunchKernelGGL(k_sample_bracket<128>, sgrid, dim3(kThreads), 0, stream, ps);
      else
        hipLaunchKernelGGL(k_sample_bracket<64>, sgrid, dim3(kThreads), 0, stream, ps);
    }
    if (p.mins_direct) break;  // every row goes straight to the emit pass
    for (int lv = 0; lv < kLevels; ++lv) {
      // Level 0 bins every key, except for minS rows, which count [threshold, max].
      SelParams pl = p;
      pl.gate = lv > 0 ? lv : -1;
      if (lv == 0 && !p.mode_mins) score_pass<MODE_HIST0>(D, p.mode_topp != 0, pgrid, pl, stream);
      else score_pass<MODE_HIST>(D, p.mode_topp != 0, pgrid, pl, stream);
      hipLaunchKernelGGL(k_resolve_hist, rgrid, dim3(64), 0, stream, p, lv);
    }
    score_pass<MODE_COLLECT>(D, p.mode_topp != 0, pgrid, p, stream);
    hipLaunchKernelGGL(k_resolve_cand, rgrid, dim3(256), 0, stream, p);
  }
  {
    SelParams pe = p;
    pe.gate = kEmitSlot;
    score_pass<MODE_EMIT>(D, p.mode_topp != 0, pgrid, pe, stream);
  }
  hipLaunchKernelGGL(k_compact, rgrid, dim3(64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace vecattn
