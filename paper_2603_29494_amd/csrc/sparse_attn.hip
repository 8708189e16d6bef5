// Vector-sparse attention (paper Eq. 4, Sec. 3.2; appendix Algorithm 2) for gfx950.
//
// One workgroup owns up to 64 query rows (4 waves) or, for blocks of a
// multiple of 128 rows, up to 128 (8 waves) of one query block of one head and
// walks the block's index list I[b,h,i,0:C) in tiles of 64 keys
// (starting at the tile where the workgroups running on its XCD are, and
// wrapping around; see below).  Blocks are dealt to groups of XCDs sized so
// that the heads swept at once fit the last-level cache (xcd_group).
// The K and V rows of a tile are gathered straight from global memory into
// LDS (global_load_lds, 16 B per lane, no register staging) two tiles deep,
// stored row-major with an XOR swizzle of their 16-byte chunks so that both
// the row reads of K and the transposing reads of V (ds_read_b64_tr_b16) are
// free of bank conflicts.  The waves compute S^T = K_tile Q^T and
// O^T += V_tile^T P^T with v_mfma_f32_32x32x16_bf16 and keep the
// online-softmax state in registers.  Wave w = (rw, kw): rw picks 32 of the
// workgroup's query rows, kw picks 32 of the 64 keys of each tile; the two
// key halves are merged at the end.
//
// MFMA 32x32x16 lane layout (lane l, g = l / 32):
//   A (M x K): lane holds row l % 32, K-slots 8g .. 8g + 7
//   B (K x N): lane holds column l % 32, K-slots 8g .. 8g + 7
//   C (M x N): lane holds column l % 32, rows 8 * (v / 4) + 4g + v % 4, v < 16
// Only the pairing of K-slots between A and B matters for the product, so the
// keys of a K-step are ordered to match C's row order.
//
// ds_read_b64_tr_b16, per group of 16 lanes: lane 4p + c receives as element q
// the c-th 16-bit value at the address supplied by lane 4q + p.
#include <algorithm>

#include "device_common.h"
#include "launch.h"

namespace vecattn {
namespace {

constexpr int kTile = 64;     // keys per gathered tile
// Progress of this kernel's workgroups on each XCD since the library was
// loaded, in units of 1/kHerdUnit of a list (wraps at 2^32).  It paces the
// tile order below: a locality hint only, so concurrent calls sharing it
// affect speed, never results.
__device__ unsigned int g_herd[8];
constexpr int kHerdUnit = 4096;
// Tiles per update of that counter: updates to one address serialise in L2,
// so they must be rare next to the gathers.
constexpr int kHerdBatch = 16;

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))


// Chunk swizzle: 16-byte chunk c of row r lives at chunk c ^ swz(r).  LDS has
// 64 banks of 4 bytes; a 16-byte read serves 16 lanes per cycle, an 8-byte
// read 32.  K reads (16 lanes = 16 consecutive rows, one logical chunk) need
// swz to separate the rows that share banks: a bijection on r % 16 for
// 256-byte rows, on (r / 2) % 8 for 128-byte rows (two rows per bank line).
// Transposing V reads (32 lanes = 4 consecutive rows x 4 chunks x 2 halves)
// need the row's contribution to move whole groups of 4 chunks: r % 4 drives
// bits 2-3 (D = 128), or r / 2 % 2 drives bit 2 across the rows that share
// banks (D = 64).  Both read patterns are then free of bank conflicts.
template <int D>
__host__ __device__ __forceinline__ constexpr int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// 16-byte copy per lane from a buffer (byte offset voff) to LDS (destination:
// wave-uniform base + 16 * lane).  The 16-byte form exists only on gfx950;
// the host pass of the compiler rejects it, so it is compiled for the device
// side only.
__device__ __forceinline__ void gather16_to_lds(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                                void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, LDS_PTR(void, lds_base), 16, voff, 0, 0, 0);
#endif
}

// 4-byte copy per lane of a list entry to LDS through the list's buffer
// resource: offsets past the list read 0, so no index can leave the list.
__device__ __forceinline__ void ids_to_lds(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                           void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, LDS_PTR(void, lds_base), 4, voff, 0, 0, 0);
#endif
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// SAME_STRIDE: K and V rows have the same stride, so a gathered row's K and V
// offsets coincide.  ROWS: query rows per workgroup (64: 4 waves, or 128: 8
// waves, for blocks of a multiple of 128 rows, so that one gather of a tile
// serves all 128 rows of the block).
template <int D, bool SAME_STRIDE, int ROWS>
__global__ __launch_bounds__(4 * ROWS) void k_sparse_attn(
    const uint16_t* __restrict__ q, int64_t q_sB, int64_t q_sH, int64_t q_sN,
    const uint16_t* __restrict__ k, int64_t k_sB, int64_t k_sH, int64_t k_sN,
    const uint16_t* __restrict__ v, int64_t v_sB, int64_t v_sH, int64_t v_sN,
    uint16_t* __restrict__ o, int64_t o_sB, int64_t o_sH, int64_t o_sN, float* __restrict__ lse,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ order, int64_t cap, int32_t Hq,
    int32_t group, int32_t N, int32_t P, int32_t Np, int32_t chunks, int32_t causal,
    float scale_log2, int64_t total, int32_t xgroup, int32_t herd_slots) {
  constexpr int CH = D / 8;                 // 16-byte chunks per row
  constexpr int kThreads = 4 * ROWS;  // 2 key halves x ROWS / 32 row groups, 64 lanes each
  constexpr int RG = ROWS / 32;             // row groups (waves per key half)
  constexpr int U = kTile * CH / kThreads;  // direct-load instructions per wave per matrix
  constexpr int DS = D / 16;                // MFMA K-steps over the head dimension
  constexpr int DB = D / 32;                // 32-wide blocks of the head dimension
  constexpr int RB = 2 * D;                 // bytes per LDS row
  constexpr bool kPrio = ROWS == 64;         // raised priority for the MFMA bursts
  // Each pipeline stage is its own LDS object, so that the compiler can tell
  // that reads of one stage do not depend on the gathers in flight into the
  // other and does not make them wait for those.
  __shared__ __align__(16) uint16_t k_s0[kTile * D];
  __shared__ __align__(16) uint16_t k_s1[kTile * D];
  __shared__ __align__(16) uint16_t v_s0[kTile * D];
  __shared__ __align__(16) uint16_t v_s1[kTile * D];
  __shared__ __align__(16) int32_t id_s0[kTile];
  __shared__ __align__(16) int32_t id_s1[kTile];
  __shared__ float s_ml[RG][128];  // (m, l) of the kw = 1 waves for the merge
  // Stage selectors; always called with a constant stage, so they fold to a
  // direct reference to one LDS object.
  auto kbuf = [&](int st) __attribute__((always_inline)) { return st ? k_s1 : k_s0; };
  auto vbuf = [&](int st) __attribute__((always_inline)) { return st ? v_s1 : v_s0; };
  auto ibuf = [&](int st) __attribute__((always_inline)) { return st ? id_s1 : id_s0; };

  // Work item: head bh = b * Hq + h, position pos in the head (block
  // order[bh, pos], or pos) and 64- or 128-row chunk of the block; the chunks
  // of a block stay on one XCD (they gather the same list).  XCDs form
  // 8 / xgroup groups.  Each group owns `whole` = nheads / groups whole heads,
  // in order, so that few heads are swept at once (their K/V rows then compete
  // less for the chip-wide last-level cache); the nheads % groups heads left
  // over are shared by all groups, group g taking the positions p = g (mod
  // groups) of each, so that every group gets the same work whatever the
  // blocks' list lengths (a head split at a group boundary would leave one
  // side with its longest lists).  A group's sequence is dealt to its XCDs
  // one block at a time, and each XCD walks its share in order.  The grid
  // covers the longest sequence (group 0's); every item is taken once.
  const int ngroups = 8 / xgroup;
  const int64_t nheads = total / (static_cast<int64_t>(Np) * chunks);
  const int64_t whole = nheads / ngroups;
  const int grp = (blockIdx.x & 7) / xgroup;
  const int64_t slot = blockIdx.x >> 3;
  const int chunk = static_cast<int>(slot % chunks);
  const int64_t e = (slot / chunks) * xgroup + (blockIdx.x & 7) % xgroup;
  int64_t bh;
  int pos;
  if (e < whole * Np) {
    bh = grp * whole + e / Np;
    pos = static_cast<int>(e % Np);
  } else {
    const int64_t e2 = e - whole * Np;
    const int64_t ng = (Np - grp + ngroups - 1) / ngroups;  // positions = grp (mod groups)
    if (ng <= 0) return;
    bh = whole * ngroups + e2 / ng;
    if (bh >= nheads) return;
    pos = static_cast<int>((e2 % ng) * ngroups + grp);
  }
  const int i = order ? min(max(order[bh * Np + pos], 0), Np - 1) : pos;
  const int b = static_cast<int>(bh / Hq);
  const int h = static_cast<int>(bh % Hq);
  const int hk = h / group;

  const int row0 = i * P + chunk * ROWS;
  const int row_end = min(N, min(i * P + P, row0 + ROWS));
  // A valid list holds distinct keys of [0, N), so at most N of them; the
  // clamp keeps the tile arithmetic below in range for any counts.
  const int count = __builtin_amdgcn_readfirstlane(static_cast<int>(
      min<int64_t>(min<int64_t>(max(counts[bh * Np + i], 0), cap), N)));
  const int32_t* list = idx + (bh * Np + i) * cap;
  const int ntiles = (count + kTile - 1) / kTile;
  // Tile order.  A block's keys are random rows of the head's K/V, far more
  // than an XCD's L2 holds; the workgroups running together on an XCD share
  // L2 hits only if they gather from the same key range at the same time.
  // Lists are ascending, so the fraction of its list a workgroup has walked
  // is a position in key space (the same for lists of different lengths).
  // Every workgroup adds its progress, in 1/kHerdUnit of its list, to its
  // XCD's counter; that sum over the XCD's workgroup slots is the mean
  // position of the workgroups running there, and a new workgroup starts at
  // the tile at that fraction of its own list (then wraps around), so the
  // workgroups on an XCD sweep the keys together at their actual pace.  The
  // order of the tiles changes only the order of the softmax sums (results
  // can differ between runs within fp32 rounding).  Causal lists are walked
  // from their first tile instead: block i's list lies in [0, (i + 1) P), so a
  // fraction of it is a different key position for every block, while the
  // walks from key 0 of lists of like length (taken together by the block
  // order) stay together.
  const int xcd = blockIdx.x & 7;  // the hardware deals workgroup x to XCD x % 8
  const bool herd = !causal;
  __shared__ int s_rot;
  if (threadIdx.x == 0 && !herd) s_rot = 0;
  if (threadIdx.x == 0 && herd) {
    const unsigned int progress =
        __hip_atomic_load(&g_herd[xcd], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned int at = (progress / static_cast<unsigned int>(herd_slots)) % kHerdUnit;
    // ntiles <= 2^18 (count <= N < 2^24), so the product fits 32 bits.
    s_rot = static_cast<int>((at * static_cast<unsigned int>(ntiles)) / kHerdUnit);
  }
  __syncthreads();
  const int t_rot = __builtin_amdgcn_readfirstlane(s_rot);
  // Progress after t tiles, in 1/kHerdUnit of the list (a whole list adds up
  // to kHerdUnit exactly).
  auto herd_units = [&](int t) __attribute__((always_inline)) {
    return static_cast<unsigned int>((kHerdUnit * t) / ntiles);
  };
  auto tile_of = [&](int t) __attribute__((always_inline)) {  // t-th tile processed
    if (t >= ntiles) return t;  // past the list (reads 0)
    const int x = t + t_rot;
    return x >= ntiles ? x - ntiles : x;
  };
  // The list entries of tile t as a buffer resource (scalar work only, so
  // that per-lane offsets stay loop-invariant); reads past the list return 0.
  auto tile_rsrc = [&](int t) __attribute__((always_inline)) {
    const int e0 = tile_of(t) * kTile;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(list) + e0, 0,
                                             max(count - e0, 0) * 4, 0x00020000);
  };

  // K and V of this head as buffer resources: gathers use 32-bit byte offsets
  // (row * row_bytes + 16 * chunk, the product in 24 bits); the host rejects
  // heads with N >= 2^24, a row stride of 2^24 bytes or more, or rows spanning
  // 2^31 bytes or more, so every offset here is exact.
  const uint16_t* kh = k + b * k_sB + hk * k_sH;
  const uint16_t* vh = v + b * v_sB + hk * v_sH;
  const uint32_t k_rowb = static_cast<uint32_t>(k_sN) * 2u;
  const uint32_t v_rowb = static_cast<uint32_t>(v_sN) * 2u;
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(kh), 0, static_cast<int>((N - 1) * k_rowb + RB), 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vh), 0, static_cast<int>((N - 1) * v_rowb + RB), 0x00020000);

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int g = lane >> 5;
  const int ln = lane & 31;
  const int rw = wave % RG;
  const int kw = wave / RG;

  // Q^T operand: this lane's query row, head-dim slots 16s + 8g .. +7.
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
    // Retire the Q loads here, so that the compiler's wait analysis does not
    // make the first MFMA of every tile wait for the gathers in flight.
    wait_vmcnt<0>();
  }

  // Gather mapping: direct-load instruction u of this wave covers LDS chunks
  // [(wave*U + u)*64, +64) of a tile; lane -> (row r, physical chunk x), and
  // it fetches logical chunk x ^ swz(r) of key row ids[r].
  auto grow = [&](int u) __attribute__((always_inline)) { return ((wave * U + u) * 64 + lane) / CH; };
  auto gcol = [&](int u) __attribute__((always_inline)) {
    const int L = (wave * U + u) * 64 + lane;
    return (L % CH) ^ swz<D>(L / CH);
  };
  int nid[U];  // key ids of the next tile to issue (raw; clamped when used)

  auto load_ids = [&](int t) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(t);
#pragma unroll
    for (int u = 0; u < U; ++u) nid[u] = __builtin_amdgcn_raw_buffer_load_b32(rs, grow(u) * 4, 0, 0);
  };
  auto issue_tile = [&](int t, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // Valid ids are below N < 2^24 and row strides below 2^24 bytes, as
      // __umul24 needs; an invalid id reads some row of this head or zeros,
      // never outside it (buffer range check).
      const uint32_t r = static_cast<uint32_t>(nid[u]);
      uint16_t* kd = kbuf(st) + (wave * U + u) * 64 * 8;
      uint16_t* vd = vbuf(st) + (wave * U + u) * 64 * 8;
      const uint32_t ko = __umul24(r, k_rowb) + 16u * gcol(u);
      gather16_to_lds(krs, ko, kd);
      gather16_to_lds(vrs, SAME_STRIDE ? ko : __umul24(r, v_rowb) + 16u * gcol(u), vd);
    }
    if (wave == 0)  // the tile's key ids (past count: 0, and masked)
      ids_to_lds(tile_rsrc(t), static_cast<uint32_t>(lane) * 4u, ibuf(st));
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = kNegInf;  // reference max (log2 units) this lane's row is scaled against
  float l_run = 0.0f;     // this lane's partial normaliser

  if (ntiles > 0) {
    load_ids(0);
    issue_tile(0, 0);
    load_ids(1);
  }

  // Per-lane constants of the LDS reads.
  const int krow = 32 * kw + ln;
  const int ksw = swz<D>(krow);
  const int j16 = lane & 15;
  const int tq = j16 >> 2, tp = j16 & 3;
  const int vhalf = (lane >> 4) & 1;

  auto step = [&](const int t, const int st) __attribute__((always_inline)) {
    // Tile t has landed, and the ids of tile t+1 (issued right after it) too;
    // the barrier (no fence: all LDS traffic here is waited for explicitly)
    // also guarantees every wave is done reading the other stage.
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (herd && wave == 0 && lane == 0 && (t % kHerdBatch) == kHerdBatch - 1)
      __hip_atomic_fetch_add(&g_herd[xcd], herd_units(t + 1) - herd_units(t + 1 - kHerdBatch),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (t + 1 < ntiles) issue_tile(t + 1, st ^ 1);
    load_ids(t + 2);  // past the list these read 0

    // S^T = K_tile Q^T for this wave's 32 keys x 32 rows.
    f32x16 sacc = f32x16{};
    const char* kb = reinterpret_cast<const char*>(kbuf(st)) + krow * RB;
    // In 64-row workgroups the MFMA bursts run at raised wave priority, so that
    // a wave issuing them is not held back by the softmax work of the other
    // wave on its SIMD (which belongs to the other workgroup, at another point
    // of its step).  The two waves a SIMD holds of an 8-wave workgroup are at
    // the same point of the same step, and run faster without it.
    if (kPrio) __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int s2 = 0; s2 < DS; ++s2) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(kb + 16 * ((2 * s2 + g) ^ ksw));
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), qf[s2], sacc,
                                                     0, 0, 0);
    }
    if (kPrio) __builtin_amdgcn_s_setprio(0);
    // The V^T operands (transposing LDS reads) are fetched now, so that their
    // latency hides behind the score MFMAs and the softmax.
    const char* vb = reinterpret_cast<const char*>(vbuf(st));
    i16x8 vfrag[DB][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int d = 32 * db + 16 * vhalf + 4 * tp;  // first of the 4 head-dim values addressed
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int k0 = 32 * kw + 16 * ks + 4 * g + tq;  // key row this lane addresses
        const int k1 = k0 + 8;
        const char* a0 = vb + k0 * RB + 16 * ((d >> 3) ^ swz<D>(k0)) + 8 * ((d >> 2) & 1);
        const char* a1 = vb + k1 * RB + 16 * ((d >> 3) ^ swz<D>(k1)) + 8 * ((d >> 2) & 1);
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(i16x4, a0));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(i16x4, a1));
        vfrag[db][ks] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }

    // Masks are needed only on the list's last tile and, when causal, on tiles
    // reaching past this wave's first row (lists are ascending).
    const int tbase = tile_of(t) * kTile;
    const int nvalid = min(kTile, count - tbase);
    const int32_t* ids = ibuf(st);
    const bool need_mask = nvalid < kTile || (causal && ids[nvalid - 1] > row0 + 32 * rw);
    if (need_mask) {
#pragma unroll
      for (int m4 = 0; m4 < 4; ++m4) {
        const int kl = 32 * kw + 8 * m4 + 4 * g;
        const int lim = nvalid - kl;  // entries e < lim of this group are in the list
        const int4 jj = *reinterpret_cast<const int4*>(ids + kl);
        const int js[4] = {jj.x, jj.y, jj.z, jj.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = (e < lim) && (!causal || js[e] <= my_row);
          sacc[4 * m4 + e] = ok ? sacc[4 * m4 + e] : kNegInf;
        }
      }
    }
    // Lazy rescaling: x = s * scale - m_run (log2 units) is what exp2 needs
    // anyway, and the weights 2^x are computed first.  Their tile sum (of the
    // fp32 weights, before the bf16 rounding of the ones that enter P V, so
    // that the normaliser and the LSE carry no bf16 error) bounds every
    // weight, so a sum <= 256 on all lanes shows that no weight exceeds 256
    // (harmless in bf16 / fp32) and the reference m_run stays.  Otherwise (a new maximum, or
    // m_run = -inf: nothing seen yet) the rows whose maximum grew by more than
    // 8 move their reference, O and l are rescaled, and the weights are
    // recomputed.
    float x[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) x[e] = __builtin_fmaf(sacc[e], scale_log2, -m_run);
    bf16x8 pb0, pb1;
    auto weights = [&]() __attribute__((always_inline)) {
      f32x8 pf[2];
#pragma unroll
      for (int e = 0; e < 16; ++e) pf[e >> 3][e & 7] = __builtin_amdgcn_exp2f(x[e]);
      pb0 = __builtin_convertvector(pf[0], bf16x8);
      pb1 = __builtin_convertvector(pf[1], bf16x8);
      // a tree of fp32 adds (short dependency chains)
      float s4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) s4[i] = (pf[0][i] + pf[0][i + 4]) + (pf[1][i] + pf[1][i + 4]);
      return (s4[0] + s4[1]) + (s4[2] + s4[3]);
    };
    float tsum = weights();
    if (__any(!(tsum <= 256.0f))) {
      float tmax = kNegInf;
#pragma unroll
      for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, sacc[e]);
      tmax = wave_max_xor32(tmax);
      const float m_new = fmaxf(m_run, tmax * scale_log2);
      const float m_ref = (m_new > m_run + 8.0f) ? m_new : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - (m_ref == kNegInf ? 0.0f : m_ref));
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
      m_run = m_ref;
      const float m_sub = m_run == kNegInf ? 0.0f : m_run;
#pragma unroll
      for (int e = 0; e < 16; ++e) x[e] = __builtin_fmaf(sacc[e], scale_log2, -m_sub);
      tsum = weights();
    }
    l_run += tsum;

    // O^T += V_tile^T P^T.
    if (kPrio) __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vfrag[db][ks]),
                                                           ks ? pb1 : pb0, oacc[db], 0, 0, 0);
    if (kPrio) __builtin_amdgcn_s_setprio(0);
  };
  for (int t = 0; t < ntiles; t += 2) {
    step(t, 0);
    if (t + 1 < ntiles) step(t + 1, 1);
  }

  if (herd && wave == 0 && lane == 0 && ntiles % kHerdBatch != 0)
    __hip_atomic_fetch_add(&g_herd[xcd], kHerdUnit - herd_units(ntiles - ntiles % kHerdBatch),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // Merge the two key halves (kw = 1 hands its state to kw = 0 through LDS).
  l_run += __shfl_xor(l_run, 32);
  wait_vmcnt<0>();  // no gather may still be landing in the buffers reused below
  __syncthreads();
  // Reuse the tile buffers (each holds one row group's 32 x D fp32 O).
  float* red_o = reinterpret_cast<float*>(rw == 0 ? k_s0 : rw == 1 ? v_s0 : rw == 2 ? k_s1 : v_s1);
  float* red_ml = s_ml[rw];
  if (kw == 1) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) red_o[(db * 16 + e) * 64 + lane] = oacc[db][e];
    red_ml[lane] = m_run;
    red_ml[64 + lane] = l_run;
  }
  __syncthreads();
  if (kw == 1) return;

  const float m1 = red_ml[lane];
  const float l1 = red_ml[64 + lane];
  const float m = fmaxf(m_run, m1);
  float a0 = 0.0f, a1 = 0.0f, inv = 0.0f, l = 0.0f;
  if (m != kNegInf) {
    a0 = __builtin_amdgcn_exp2f(m_run - m);
    a1 = __builtin_amdgcn_exp2f(m1 - m);
    l = a0 * l_run + a1 * l1;
    inv = l > 0.0f ? 1.0f / l : 0.0f;
  }
  if (my_row >= row_end) return;
  if (lse && g == 0)
    lse[bh * N + my_row] = l > 0.0f ? (m + __builtin_log2f(l)) * 0.69314718055994531f : kNegInf;
  uint16_t* orow = o + b * o_sB + h * o_sH + static_cast<int64_t>(my_row) * o_sN;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      f32x4 r;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ee = 4 * vq + e;
        r[e] = (a0 * oacc[db][ee] + a1 * red_o[(db * 16 + ee) * 64 + lane]) * inv;
      }
      *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * vq + 4 * g) = __builtin_convertvector(r, bf16x4);
    }
  }
}

}  // namespace

// XCDs per group in the work mapping (1, 2, 4 or 8): the smallest group for
// which the K/V rows of the heads swept at once stay within ~160 MB, well inside
// the 256 MB last-level cache (the rest holds the Q, O and list streams).  One
// KV head's rows are N * D * 4 bytes (K and V, bf16), half of that under
// causal masking (a block's list spans the keys up to its own rows); the 8 / G
// groups sweep at most B * Hkv distinct KV heads.  Measured (attention alone):
// 75k-token DiT, 38.7 MB per head: 22.8 / 22.1 / 22.2 / 22.8 ms at G = 1 / 2 /
// 4 / 8; 119k-token DiT, 60.8 MB: 140.4 / 136.7 / 125 / 127 ms; causal VLM
// prefill at 131k tokens: G = 1 best by ~2%.
static int32_t xcd_group(int64_t N, int64_t D, int64_t Hkv, int64_t B, int32_t causal) {
  const double head_bytes = static_cast<double>(N) * static_cast<double>(D) * 4.0 *
                            (causal ? 0.5 : 1.0);
  const double budget = 160.0 * 1024.0 * 1024.0;
  for (int32_t g = 1; g < 8; g *= 2) {
    const double swept = static_cast<double>(std::min<int64_t>(8 / g, B * Hkv)) * head_bytes;
    if (swept <= budget) return g;
  }
  return 8;
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream) {
  const int64_t B = a.q.B, Hq = a.q.H, N = a.q.N, D = a.q.D;
  const int32_t P = a.block;
  const int32_t Np = static_cast<int32_t>((N + P - 1) / P);
  // 128 rows per workgroup when blocks come in multiples of 128 rows (one
  // gather of a tile then serves the whole block), else 64.
  const int32_t rows = P % 128 == 0 ? 128 : 64;
  const int32_t chunks = (P + rows - 1) / rows;
  const int64_t nheads = B * Hq;
  const int64_t total = nheads * Np * chunks;
  if (total == 0) return hipSuccess;
  const int32_t xgroup = xcd_group(a.k.N, a.k.D, a.k.H, B, a.causal);
  // Group 0's sequence (the longest): its whole heads and its share of the
  // heads left over; each of its XCDs takes every xgroup-th block of it.
  const int64_t ngroups = 8 / xgroup, whole = nheads / ngroups;
  const int64_t seq0 = whole * Np + (nheads - whole * ngroups) * ((Np + ngroups - 1) / ngroups);
  const int64_t per_xcd = (seq0 + xgroup - 1) / xgroup * chunks;
  const dim3 grid(static_cast<unsigned>(per_xcd * 8));
  const float scale = a.scale != 0.0f ? a.scale : 1.0f / sqrtf(static_cast<float>(D));
  const float scale_log2 = scale * 1.4426950408889634f;
  const int32_t group = static_cast<int32_t>(Hq / a.k.H);
  const uint16_t* q = static_cast<const uint16_t*>(a.q.ptr);
  const uint16_t* k = static_cast<const uint16_t*>(a.k.ptr);
  const uint16_t* v = static_cast<const uint16_t*>(a.v.ptr);
  uint16_t* o = static_cast<uint16_t*>(a.o);
  const bool same = a.k.sN == a.v.sN;
  auto launch = [&](auto kernel) -> hipError_t {
    // Workgroup slots per XCD (resident workgroups per CU x CUs per XCD).
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int threads = 4 * rows;
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0);
    if (e != hipSuccess) return e;
    const int32_t slots = max(1, per_cu * cus / 8);
    hipLaunchKernelGGL(kernel, grid, dim3(threads), 0, stream, q, a.q.sB, a.q.sH, a.q.sN, k,
                       a.k.sB, a.k.sH, a.k.sN, v, a.v.sB, a.v.sH, a.v.sN, o, a.o_sB, a.o_sH,
                       a.o_sN, a.lse, a.idx, a.counts, a.order, a.cap, static_cast<int32_t>(Hq), group,
                       static_cast<int32_t>(N), P, Np, chunks, a.causal, scale_log2, total,
                       xgroup, slots);
    return hipGetLastError();
  };
  if (rows == 128) {
    if (D == 128) return same ? launch(k_sparse_attn<128, true, 128>) : launch(k_sparse_attn<128, false, 128>);
    return same ? launch(k_sparse_attn<64, true, 128>) : launch(k_sparse_attn<64, false, 128>);
  }
  if (D == 128) return same ? launch(k_sparse_attn<128, true, 64>) : launch(k_sparse_attn<128, false, 64>);
  return same ? launch(k_sparse_attn<64, true, 64>) : launch(k_sparse_attn<64, false, 64>);
}

}  // namespace vecattn
