// ql_gemm.hip -- 8-bit matrix products of Section 3.1 (eq. 1) on gfx950 MFMA.
//
// C[m][n] = sum_k X'[m][k] W'[n][k] with both operands K-contiguous.  Codes
// are stored as signed bytes s = V' - 128 so the signed int8 MFMA
// (v_mfma_i32_32x32x32_i8) applies directly; the exact zero-point terms of
// eq. 1 are added in the epilogue from per-row / per-column code sums, and the
// product is recovered to fp32 there (Fig. 1: R(Mult(.)) + B).
//
// Tiling: a workgroup of WM x WN wavefronts computes a BM x BN tile; each
// wavefront owns a (BM/WM) x (BN/WN) sub-tile built from 32x32 MFMA blocks.
// K advances in steps of BK bytes through two LDS stages (global -> VGPR ->
// LDS, one barrier per step); LDS rows are padded by 16 bytes so the 16-byte
// fragment reads of 32 consecutive rows spread over all banks.
#include "ql_device.h"
#include "ql_launch.h"

namespace ql {

enum { EPI_RECOVER = 0, EPI_RAW = 1, EPI_SMAX_STATS = 2, EPI_SMAX_OUT = 3 };

struct EpiArgs {
  // row (X) side
  const int32_t *x_zero;
  const float *x_inv_q;
  const int32_t *x_sums;
  // column (W) side
  const int32_t *w_zero;
  const float *w_inv_q;
  const int32_t *w_sums;
  int64_t w_rpb;
  const float *bias;
  // outputs
  float *Y;
  int32_t *acc;
  float *logits;
  float2 *stats;  // [M][ntn] (max, sum exp) per column tile
  int ntn;
  const float2 *rowstat;  // [M] (max, 1 / sum exp) per row
};

template <int BM, int BN, int BK, int WM, int WN>
struct Cfg {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int LDSS = BK + 16;  // padded LDS row stride in bytes
  static constexpr int STAGE = (BM + BN) * LDSS;
  static constexpr int LDS = 2 * STAGE;
  static constexpr int CPR = BK / 16;   // 16-byte chunks per row
  static constexpr int LA = BM * CPR / NT, LB = BN * CPR / NT;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile/threads mismatch");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be a multiple of 32");
};

template <int BM, int BN, int BK, int WM, int WN>
__device__ __forceinline__ void gemm_tile(const int8_t *__restrict__ A, int64_t lda,
                                          const int8_t *__restrict__ B, int64_t ldb, int64_t M,
                                          int64_t N, int64_t Kp, int64_t m0, int64_t n0,
                                          char *smem, v16i (&acc)[Cfg<BM, BN, BK, WM, WN>::FM]
                                                                 [Cfg<BM, BN, BK, WM, WN>::FN]) {
  using C = Cfg<BM, BN, BK, WM, WN>;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = v16i{};

  // global source offsets and LDS destinations of this thread's 16-byte chunks
  int64_t oa[C::LA], ob[C::LB];
  int sa[C::LA], sb[C::LB];
#pragma unroll
  for (int i = 0; i < C::LA; ++i) {
    const int c = tid + i * C::NT, r = c / C::CPR, kc = c % C::CPR;
    int64_t gr = m0 + r;
    gr = gr < M ? gr : M - 1;
    oa[i] = gr * lda + kc * 16;
    sa[i] = r * C::LDSS + kc * 16;
  }
#pragma unroll
  for (int i = 0; i < C::LB; ++i) {
    const int c = tid + i * C::NT, r = c / C::CPR, kc = c % C::CPR;
    int64_t gr = n0 + r;
    gr = gr < N ? gr : N - 1;
    ob[i] = gr * ldb + kc * 16;
    sb[i] = BM * C::LDSS + r * C::LDSS + kc * 16;
  }
  const int nk = (int)(Kp / BK);
  v4i ra[C::LA], rb[C::LB];
  if (nk > 0) {
#pragma unroll
    for (int i = 0; i < C::LA; ++i) ra[i] = *reinterpret_cast<const v4i *>(A + oa[i]);
#pragma unroll
    for (int i = 0; i < C::LB; ++i) rb[i] = *reinterpret_cast<const v4i *>(B + ob[i]);
#pragma unroll
    for (int i = 0; i < C::LA; ++i) *reinterpret_cast<v4i *>(smem + sa[i]) = ra[i];
#pragma unroll
    for (int i = 0; i < C::LB; ++i) *reinterpret_cast<v4i *>(smem + sb[i]) = rb[i];
  }
  __syncthreads();
  const int frow = lane & 31, fk = (lane >> 5) * 16;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t ko = (int64_t)(kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < C::LA; ++i) ra[i] = *reinterpret_cast<const v4i *>(A + oa[i] + ko);
#pragma unroll
      for (int i = 0; i < C::LB; ++i) rb[i] = *reinterpret_cast<const v4i *>(B + ob[i] + ko);
    }
    const char *base = smem + (kt & 1) * C::STAGE;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      v4i af[C::FM], bf[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
        af[i] = *reinterpret_cast<const v4i *>(base + (wm * C::TM + i * 32 + frow) * C::LDSS +
                                               ks * 32 + fk);
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        bf[j] = *reinterpret_cast<const v4i *>(base + BM * C::LDSS +
                                               (wn * C::TN + j * 32 + frow) * C::LDSS + ks * 32 +
                                               fk);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      char *nb = smem + ((kt + 1) & 1) * C::STAGE;
#pragma unroll
      for (int i = 0; i < C::LA; ++i) *reinterpret_cast<v4i *>(nb + sa[i]) = ra[i];
#pragma unroll
      for (int i = 0; i < C::LB; ++i) *reinterpret_cast<v4i *>(nb + sb[i]) = rb[i];
    }
    __syncthreads();
  }
}

// Deeper pipeline for large tiles: K advances ROW bytes (64 or 128) per step
// through NS LDS stages filled by direct global->LDS loads (no VGPR
// staging).  Chunk c (16 bytes) of row r of a stage sits in slot
// c ^ swz(r), which keeps the 16-byte fragment reads of 32 consecutive rows
// free of bank conflicts (any 8 aligned rows, and the even and the odd rows
// of any 16 aligned rows, take distinct slots).  swz uses only bits 0..4 of
// the row, so a fragment's swizzle follows from lane & 31 alone.
typedef __attribute__((address_space(3))) void lds_void;

// One 16-byte direct global->LDS load (each lane's 16 bytes land at
// consecutive 16-byte slots from the wave's LDS base).  A plain function so
// that every kernel instantiation shares one declaration of the builtin call.
__device__ __forceinline__ void load_lds16(const int8_t *g, char *l) {
  __builtin_amdgcn_global_load_lds(g, (lds_void *)l, 16, 0, 0);
}

template <int ROW>
__device__ __forceinline__ int swz(int r) {
  if constexpr (ROW == 64) return ((r >> 1) ^ (r >> 2)) & 3;
  else return (r & 7) ^ ((r >> 3) & 1);
}

// s_waitcnt with only the vector-memory count limited (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at maximum)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));
}

template <int BM, int BN, int WM, int WN, int ROW, int NS>
struct CfgDma {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TBM = BM, TBN = BN;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int CPR = ROW / 16;           // 16-byte chunks per row
  static constexpr int STAGE = (BM + BN) * ROW;
  static constexpr int LDS = NS * STAGE;
  static constexpr int LA = BM * CPR / NT, LB = BN * CPR / NT;  // loads per thread
  static_assert(ROW == 64 || ROW == 128, "row of 64 or 128 bytes");
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile/threads mismatch");
  static_assert(NS >= 2, "pipeline needs two stages");
};

template <int BM, int BN, int WM, int WN, int ROW, int NS>
__device__ __forceinline__ void gemm_tile_dma(
    const int8_t *__restrict__ A, int64_t lda, const int8_t *__restrict__ B, int64_t ldb, int64_t M,
    int64_t N, int64_t Kp, int64_t m0, int64_t n0, char *smem,
    v16i (&acc)[CfgDma<BM, BN, WM, WN, ROW, NS>::FM][CfgDma<BM, BN, WM, WN, ROW, NS>::FN]) {
  using C = CfgDma<BM, BN, WM, WN, ROW, NS>;
  constexpr int CPR = C::CPR, Q = ROW / 32;  // Q sub-steps of 32 bytes of K
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = v16i{};

  // Load i of this thread fills LDS slot p = i * NT + tid of the A (or B)
  // region: row p / CPR, slot p % CPR, holding global chunk
  // (p % CPR) ^ swz(row).  Each wave's load instruction covers 1 KB of
  // consecutive slots.
  const int8_t *ga[C::LA], *gb[C::LB];
#pragma unroll
  for (int i = 0; i < C::LA; ++i) {
    const int p = i * C::NT + tid, r = p / CPR, c = (p % CPR) ^ swz<ROW>(r);
    int64_t gr = m0 + r;
    gr = gr < M ? gr : M - 1;
    ga[i] = A + gr * lda + c * 16;
  }
#pragma unroll
  for (int i = 0; i < C::LB; ++i) {
    const int p = i * C::NT + tid, r = p / CPR, c = (p % CPR) ^ swz<ROW>(r);
    int64_t gr = n0 + r;
    gr = gr < N ? gr : N - 1;
    gb[i] = B + gr * ldb + c * 16;
  }
  const int nk = (int)(Kp / ROW);
  // Load i (of LA + LB) of step `ks` into its stage; steps past the end
  // reload the last step into a stage that is never read again, so every
  // step has the same number of loads in flight.
  auto load_one = [&](int ks, int i) {
    const int64_t ko = (int64_t)(ks < nk ? ks : nk - 1) * ROW;
    char *st = smem + (ks % NS) * C::STAGE + wave * 1024;
    if (i < C::LA)
      load_lds16(ga[i] + ko, st + i * C::NT * 16);
    else
      load_lds16(gb[i - C::LA] + ko, st + BM * ROW + (i - C::LA) * C::NT * 16);
  };
  if (nk == 0) return;

  // Fragment q of a sub-step: A fragments 0..FM-1, then B fragments.  A
  // fragment i of sub-step h is rows wm*TM + i*32 + (lane & 31), chunk
  // 2*h + (lane >> 5); swz depends only on lane & 31 here.
  const int fr = lane & 31, fsw = swz<ROW>(fr), fhi = lane >> 5;
  const int offa = (wm * C::TM + fr) * ROW, offb = BM * ROW + (wn * C::TN + fr) * ROW;
  constexpr int NMF = C::FM * C::FN, NRD = C::FM + C::FN, NLD = C::LA + C::LB;
  constexpr int SLOTS = NMF - NRD;  // load slots per sub-step
  static_assert(Q % 2 == 0, "sub-steps alternate between two fragment sets");
  static_assert(SLOTS > 0 && NLD <= Q * SLOTS, "not enough MFMAs to cover the memory ops");
  v4i f0[NRD], f1[NRD];
  auto read_one = [&](int ks, int h, int q, v4i &dst) {
    const char *st = smem + (ks % NS) * C::STAGE + ((2 * h + fhi) ^ fsw) * 16;
    dst = *reinterpret_cast<const v4i *>(st + (q < C::FM ? offa + q * 32 * ROW
                                                         : offb + (q - C::FM) * 32 * ROW));
  };
  auto mfma_one = [&](const v4i(&f)[NRD], int q) {
    const int i = q / C::FN, j = q % C::FN;
    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f[i], f[C::FM + j], acc[i][j], 0, 0, 0);
  };
  // One sub-step: the MFMAs on `cur`, with the next sub-step's fragment
  // reads into `nxt` and loads [l0, l0 + SLOTS) of step `lks` threaded one
  // per MFMA; the scheduling barriers hold that order so the matrix pipe
  // never waits on a memory instruction.
  auto substep = [&](const v4i(&cur)[NRD], v4i(&nxt)[NRD], int rks, int rh, int lks, int l0) {
#pragma unroll
    for (int q = 0; q < NMF; ++q) {
      mfma_one(cur, q);
      if (q < NRD) read_one(rks, rh, q, nxt[q]);
      else if (lks >= 0 && l0 + q - NRD < NLD) load_one(lks, l0 + q - NRD);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  for (int ks = 0; ks < NS; ++ks)
#pragma unroll
    for (int i = 0; i < NLD; ++i) load_one(ks, i);
  wait_vmcnt<(NS - 1) * NLD>();
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NRD; ++q) read_one(0, 0, q, f0[q]);
  wait_lgkmcnt0();
  // Step kt+NS-1 is loaded from the last sub-step of step kt-1 on (the
  // prologue loaded steps 0..NS-1).
  for (int kt = 0; kt < nk; ++kt) {
    const int lprev = kt > 0 ? kt + NS - 1 : -1;
#pragma unroll
    for (int h = 0; h < Q - 1; ++h) {
      if (h % 2 == 0) substep(f0, f1, kt, h + 1, lprev, (h + 1) * SLOTS);
      else substep(f1, f0, kt, h + 1, lprev, (h + 1) * SLOTS);
    }
    // Stage kt is fully read into registers and step kt+1 has landed (steps
    // up to kt+NS-1 were issued): after the barrier stage kt's buffer takes
    // step kt+NS.
    wait_vmcnt<(NS - 2) * NLD>();
    __syncthreads();
    substep(f1, f0, kt + 1, 0, kt + NS, 0);
    // the fragments just read landed while the MFMAs above issued; saying so
    // keeps the LDS counter (15 at most) from forcing a full wait on the
    // next sub-step's reads
    wait_lgkmcnt0();
  }
  wait_vmcnt<0>();
  __syncthreads();
}

// Tile of this (1-D) workgroup.  Workgroups are dealt round-robin to the 8
// XCDs; when the tile count allows, XCD x is given the x-th contiguous eighth
// of the tile order, and that order walks groups of 8 tile rows column by
// column, so the workgroups sharing an L2 also share A and B panels.
__device__ __forceinline__ void tile_of_block(int64_t M, int64_t N, int BM, int BN, int *tm, int *tn) {
  const int ntm = (int)((M + BM - 1) / BM), ntn = (int)((N + BN - 1) / BN);
  const int ntiles = ntm * ntn;
  int bid = blockIdx.x;
  if (ntiles % 8 == 0) bid = (bid % 8) * (ntiles / 8) + bid / 8;
  constexpr int kGroup = 8;
  const int group = bid / (kGroup * ntn);
  const int first = group * kGroup;
  const int gsize = ntm - first < kGroup ? ntm - first : kGroup;
  const int in_group = bid % (kGroup * ntn);
  *tm = first + in_group % gsize;
  *tn = in_group / gsize;
}

// Row/column of element r of a 32x32 MFMA block held by `lane`.
__device__ __forceinline__ int frag_row(int r, int lane) { return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3); }
__device__ __forceinline__ int frag_col(int lane) { return lane & 31; }

// Integer accumulators through LDS: each wave turns 32 rows of its
// accumulators at a time into V'-domain sums (eq. 1 with the code sums) and
// parks them row-major in its own LDS slab (row stride 136 words: the two
// half-waves of a store land on disjoint banks), then stores whole rows with
// 16-byte writes.  The tile's row sums are staged once.  The K loop has left
// LDS idle (its last barrier follows the final wait for loads).
template <class C>
__device__ __forceinline__ void raw_epilogue_lds(const EpiArgs &e, int64_t M, int64_t N, int64_t K,
                                                 int64_t m0, int64_t n0, int wm, int wn, int lane,
                                                 char *smem, v16i (&acc)[C::FM][C::FN]) {
  constexpr int TM = C::TM, TN = C::TN, RS = TN + 8;  // row stride in words
  static_assert(TN % 4 == 0 && (RS * 4) % 16 == 0, "16-byte rows");
  static_assert(C::TBM * 4 <= 4096 && 4096 + (C::NT / 64) * 32 * RS * 4 <= C::LDS, "LDS slabs");
  uint32_t *rterm = reinterpret_cast<uint32_t *>(smem);  // [BM]: 128 * sigma_x
  const int wave = threadIdx.x >> 6;
  uint32_t *slab = reinterpret_cast<uint32_t *>(smem + 4096) + wave * 32 * RS;
  for (int r = threadIdx.x; r < C::TBM; r += C::NT) {
    const int64_t m = m0 + r;
    rterm[r] = m < M ? 128u * (uint32_t)(e.x_sums[m] - 128 * (int32_t)K) : 0u;
  }
  uint32_t cterm[C::FN];
#pragma unroll
  for (int j = 0; j < C::FN; ++j) {
    int64_t n = n0 + wn * TN + j * 32 + (lane & 31);
    n = n < N ? n : N - 1;
    cterm[j] = 128u * (uint32_t)(e.w_sums[n] - 128 * (int32_t)K) + 16384u * (uint32_t)K;
  }
  __syncthreads();
  const bool vec = (N & 3) == 0;
#pragma unroll
  for (int i = 0; i < C::FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = frag_row(r, lane);
      const uint32_t rt = rterm[wm * TM + i * 32 + row];
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        slab[row * RS + j * 32 + (lane & 31)] = (uint32_t)acc[i][j][r] + cterm[j] + rt;
    }
    // the slab is this wave's own: LDS keeps one wave's accesses in order
#pragma unroll
    for (int it = 0; it < 32 * TN / 256; ++it) {
      const int q = it * 64 + lane, row = q / (TN / 4), c4 = (q % (TN / 4)) * 4;
      const v4i v = *reinterpret_cast<const v4i *>(slab + row * RS + c4);
      const int64_t m = m0 + wm * TM + i * 32 + row, n = n0 + wn * TN + c4;
      if (m < M) {
        int32_t *dst = e.acc + m * N + n;
        if (vec && n + 3 < N) {
          *reinterpret_cast<v4i *>(dst) = v;
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t)
            if (n + t < N) dst[t] = v[t];
        }
      }
    }
  }
}

// Calls f(integral_constant<int, I>) for I in [B, E).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// N independent reductions (max or sum) over each group of L lanes (32: a
// half-wave, 16: one DPP row): rotations within 16-lane rows, then for 32
// the exchange of the two rows.
template <bool MAX, int L, int N>
__device__ __forceinline__ void row_reduce(float (&v)[N]) {
  static_assert(L == 16 || L == 32, "16 or 32 lanes");
  auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : a + b; };
  auto ror = [](float x, auto ctrl) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), decltype(ctrl)::value,
                                                      0xf, 0xf, false));
  };
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = op(v[k], ror(v[k], std::integral_constant<int, 0x128>{}));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = op(v[k], ror(v[k], std::integral_constant<int, 0x124>{}));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = op(v[k], ror(v[k], std::integral_constant<int, 0x122>{}));
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = op(v[k], ror(v[k], std::integral_constant<int, 0x121>{}));
  if constexpr (L == 32) {
#pragma unroll
    for (int k = 0; k < N; ++k) v[k] = op(v[k], __shfl_xor(v[k], 16, 64));
  }
}

// Recovering epilogues (eq. 1 recovery plus bias; softmax statistics or
// output) through LDS: each wave parks 32 rows of raw signed sums at a time in
// its own slab (as above), then walks them row-major with every lane owning
// the same 4 consecutive columns of each row, so the per-column terms stay in
// registers and every store is a 16-byte write.  The tile's per-row terms are
// staged once.  Softmax statistics are reduced per wave over its TN columns
// (max, then sum of exp(y - max)) and the WN partials of a row are merged
// with the usual rescaling.
template <class C, int EPI>
__device__ __forceinline__ void recover_epilogue_lds(const EpiArgs &e, int64_t M, int64_t N,
                                                     int64_t K, int64_t m0, int64_t n0, int tn,
                                                     int wm, int wn, int lane, char *smem,
                                                     const float *rowmax, const float *rowinv,
                                                     v16i (&acc)[C::FM][C::FN]) {
  constexpr int BM = C::TBM, TM = C::TM, TN = C::TN, RS = TN + 8, WN = C::TBN / C::TN;
  // LPR lanes cover one row of the wave's TN columns, 4 columns each; a wave
  // covers RPI rows per iteration, NIT iterations per 32-row chunk
  constexpr int LPR = TN / 4, RPI = 64 / LPR, NIT = 32 / RPI;
  static_assert(TN == 128 || TN == 64, "32 or 16 lanes per row");
  constexpr int kSlab = (3 * BM * 4 + WN * BM * 8 + 4095) / 4096 * 4096;
  static_assert(kSlab + (C::NT / 64) * 32 * RS * 4 <= C::LDS, "LDS slabs");
  int32_t *rsig = reinterpret_cast<int32_t *>(smem);  // [BM] sigma_x
  int32_t *rzt = rsig + BM;                            // [BM] z~x
  float *riq = reinterpret_cast<float *>(rzt + BM);    // [BM] 1/Qx
  float2 *red = reinterpret_cast<float2 *>(smem + 3 * BM * 4);  // [WN][BM] (max, sum)
  const int wave = threadIdx.x >> 6;
  uint32_t *slab = reinterpret_cast<uint32_t *>(smem + kSlab) + wave * 32 * RS;
  bool fast = true;  // every row and column of the tile on recover()'s fast path
  for (int r = threadIdx.x; r < BM; r += C::NT) {
    int64_t m = m0 + r;
    m = m < M ? m : M - 1;
    rsig[r] = e.x_sums[m] - 128 * (int32_t)K;
    rzt[r] = e.x_zero[m] + 128;
    riq[r] = e.x_inv_q[m];
    fast = fast && fast_row(rzt[r]);
  }
  // this lane's columns: n0 + wn*TN + 4*(lane % LPR) + t
  const int64_t nc = n0 + wn * TN + 4 * (lane % LPR);
  int32_t ztw[4], sigw[4];
  int64_t colterm[4];
  float iqw[4], bn[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int64_t nn = nc + t < N ? nc + t : N - 1;
    const int64_t blk = nn / e.w_rpb;
    ztw[t] = e.w_zero[blk] + 128;
    sigw[t] = e.w_sums[nn] - 128 * (int32_t)K;
    colterm[t] = (int64_t)sigw[t] + K * (int64_t)ztw[t];
    iqw[t] = e.w_inv_q[blk];
    bn[t] = e.bias ? e.bias[nn] : 0.0f;
    fast = fast && fast_col(ztw[t], colterm[t]);
  }
  fast = __syncthreads_and(fast);
  int32_t colt32[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) colt32[t] = (int32_t)colterm[t];
  const bool vec = (N & 3) == 0 && nc + 3 < N;
  // chunks expanded at compile time: acc is only ever indexed by constants
  static_for<0, C::FM>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = frag_row(r, lane);
#pragma unroll
      for (int j = 0; j < C::FN; ++j) slab[row * RS + j * 32 + (lane & 31)] = (uint32_t)acc[i][j][r];
    }
    // the slab is this wave's own: LDS keeps one wave's accesses in order
    // row `it` of this half-wave: recover, store, and hand back y
    auto row_step = [&](int it, float (&y)[4]) {
      const int row = RPI * it + lane / LPR, lr = wm * TM + i * 32 + row;
      const int64_t m = m0 + lr;
      const v4i v = *reinterpret_cast<const v4i *>(slab + row * RS + 4 * (lane % LPR));
      const int32_t sigx = rsig[lr], ztx = rzt[lr];
      const float iqx = riq[lr];
      if (fast) {
#pragma unroll
        for (int t = 0; t < 4; ++t) y[t] = recover_fast(v[t], colt32[t], ztw[t], ztx, sigx, iqw[t], iqx) + bn[t];
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) y[t] = recover(v[t], colterm[t], ztw[t], ztx, sigx, iqw[t], iqx) + bn[t];
      }
      const int64_t off = m * N + nc;
      if (EPI == EPI_RECOVER || EPI == EPI_SMAX_OUT) {
        if (EPI == EPI_SMAX_OUT) {
          const float mx = rowmax[lr], inv = rowinv[lr];
#pragma unroll
          for (int t = 0; t < 4; ++t) y[t] = __expf(y[t] - mx) * inv;
        }
        if (m < M) {
          if (vec) {
            *reinterpret_cast<float4 *>(e.Y + off) = make_float4(y[0], y[1], y[2], y[3]);
          } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              if (nc + t < N) e.Y[off + t] = y[t];
          }
        }
      } else if (m < M && e.logits) {  // EPI_SMAX_STATS
        if (vec) {
          *reinterpret_cast<float4 *>(e.logits + off) = make_float4(y[0], y[1], y[2], y[3]);
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t)
            if (nc + t < N) e.logits[off + t] = y[t];
        }
      }
      if (EPI != EPI_SMAX_OUT && m < M && e.acc) {
        int32_t a[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) a[t] = acc_u8(v[t], sigw[t], sigx, K);
        if (vec) {
          *reinterpret_cast<v4i *>(e.acc + off) = v4i{a[0], a[1], a[2], a[3]};
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t)
            if (nc + t < N) e.acc[off + t] = a[t];
        }
      }
    };
    if constexpr (EPI != EPI_SMAX_STATS) {
#pragma unroll 2
      for (int it = 0; it < NIT; ++it) {
        float y[4];
        row_step(it, y);
      }
    } else {
      float ys[NIT][4];
#pragma unroll
      for (int it = 0; it < NIT; ++it) row_step(it, ys[it]);
      // per row (one per LPR lanes and iteration): max over the wave's TN
      // columns, then sum exp(y - max); NIT rows reduced together so the
      // steps overlap
      float mx[NIT], sm[NIT];
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        mx[it] = -INFINITY;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (nc + t < N) mx[it] = fmaxf(mx[it], ys[it][t]);
      }
      row_reduce<true, LPR>(mx);
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        sm[it] = 0.0f;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (nc + t < N) sm[it] += __expf(ys[it][t] - mx[it]);
      }
      row_reduce<false, LPR>(sm);
      if (lane % LPR == 0) {
#pragma unroll
        for (int it = 0; it < NIT; ++it)
          red[wn * BM + wm * TM + i * 32 + RPI * it + lane / LPR] = make_float2(mx[it], sm[it]);
      }
    }
  });
  if constexpr (EPI == EPI_SMAX_STATS) {
    __syncthreads();
    for (int r = threadIdx.x; r < BM; r += C::NT) {
      const int64_t m = m0 + r;
      if (m >= M) continue;
      float mx = -INFINITY;
#pragma unroll
      for (int w = 0; w < WN; ++w) mx = fmaxf(mx, red[w * BM + r].x);
      float sm = 0.0f;
#pragma unroll
      for (int w = 0; w < WN; ++w) {
        const float2 p = red[w * BM + r];
        if (p.y > 0.0f) sm += p.y * __expf(p.x - mx);
      }
      e.stats[m * e.ntn + tn] = make_float2(mx, sm);
    }
  }
}

// NS = 0: register-staged two-stage tile; NS >= 2: direct-load pipeline of
// NS stages with BK-byte rows.
template <int BM, int BN, int BK, int WM, int WN, int NS>
using GemmCfg = std::conditional_t<(NS >= 2), CfgDma<BM, BN, WM, WN, BK, (NS >= 2 ? NS : 2)>,
                                   Cfg<BM, BN, BK, WM, WN>>;

template <int BM, int BN, int BK, int WM, int WN, int NS, int EPI>
__global__ __launch_bounds__(64 * WM *WN) void k_gemm(const int8_t *__restrict__ A, int64_t lda,
                                                       const int8_t *__restrict__ B, int64_t ldb,
                                                       int64_t M, int64_t N, int64_t K,
                                                       int64_t Kp, EpiArgs e) {
  using C = GemmCfg<BM, BN, BK, WM, WN, NS>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int tm, tn;
  tile_of_block(M, N, BM, BN, &tm, &tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // softmax output pass: combine the per-tile statistics of this tile's rows
  float *rowmax = reinterpret_cast<float *>(smem + C::LDS);
  float *rowinv = rowmax + BM;
  if (EPI == EPI_SMAX_OUT) {
    for (int r = threadIdx.x; r < BM; r += C::NT) {
      const int64_t m = m0 + r;
      const float2 st = e.rowstat[m < M ? m : M - 1];
      rowmax[r] = st.x;
      rowinv[r] = st.y;
    }
  }

  v16i acc[C::FM][C::FN];
  if constexpr (NS >= 2)
    gemm_tile_dma<BM, BN, WM, WN, BK, NS>(A, lda, B, ldb, M, N, Kp, m0, n0, smem, acc);
  else
    gemm_tile<BM, BN, BK, WM, WN>(A, lda, B, ldb, M, N, Kp, m0, n0, smem, acc);

  if constexpr (NS >= 2) {
    if constexpr (EPI == EPI_RAW)
      raw_epilogue_lds<C>(e, M, N, K, m0, n0, wm, wn, lane, smem, acc);
    else
      recover_epilogue_lds<C, EPI>(e, M, N, K, m0, n0, tn, wm, wn, lane, smem, rowmax, rowinv, acc);
    return;
  }

  // per-column terms
  int32_t ztw[C::FN], sigw[C::FN];
  int64_t colterm[C::FN];
  float iqw[C::FN], bn[C::FN];
  int64_t ncol[C::FN];
#pragma unroll
  for (int j = 0; j < C::FN; ++j) {
    int64_t n = n0 + wn * C::TN + j * 32 + frag_col(lane);
    ncol[j] = n;
    const int64_t nn = n < N ? n : N - 1;
    if (EPI == EPI_RAW) {
      sigw[j] = e.w_sums[nn] - 128 * (int32_t)K;
      ztw[j] = 0;
      colterm[j] = 0;
      iqw[j] = 0.0f;
      bn[j] = 0.0f;
    } else {
      const int64_t blk = nn / e.w_rpb;
      ztw[j] = e.w_zero[blk] + 128;
      sigw[j] = e.w_sums[nn] - 128 * (int32_t)K;
      colterm[j] = (int64_t)sigw[j] + K * (int64_t)ztw[j];
      iqw[j] = e.w_inv_q[blk];
      bn[j] = e.bias ? e.bias[nn] : 0.0f;
    }
  }

  if (EPI == EPI_RECOVER || EPI == EPI_RAW || EPI == EPI_SMAX_OUT) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = wm * C::TM + i * 32 + frag_row(r, lane);
        const int64_t m = m0 + lr;
        if (m >= M) continue;
        const int32_t sigx = e.x_sums[m] - 128 * (int32_t)K;
        int32_t ztx = 0;
        float iqx = 0.0f;
        if (EPI != EPI_RAW) {
          ztx = e.x_zero[m] + 128;
          iqx = e.x_inv_q[m];
        }
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
          const int64_t n = ncol[j];
          if (n >= N) continue;
          const int32_t S = acc[i][j][r];
          if (EPI == EPI_RAW) {
            e.acc[m * N + n] = acc_u8(S, sigw[j], sigx, K);
          } else {
            const float y = recover(S, colterm[j], ztw[j], ztx, sigx, iqw[j], iqx) + bn[j];
            if (EPI == EPI_RECOVER) {
              e.Y[m * N + n] = y;
              if (e.acc) e.acc[m * N + n] = acc_u8(S, sigw[j], sigx, K);
            } else {
              e.Y[m * N + n] = __expf(y - rowmax[lr]) * rowinv[lr];
            }
          }
        }
      }
  } else {  // EPI_SMAX_STATS: per-row (max, sum exp) over this tile's columns
    float *red = reinterpret_cast<float *>(smem);  // [WN][BM] scratch (stages are free now)
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = wm * C::TM + i * 32 + frag_row(r, lane);
        const int64_t m = m0 + lr;
        const int64_t mm = m < M ? m : M - 1;
        const int32_t sigx = e.x_sums[mm] - 128 * (int32_t)K;
        const int32_t ztx = e.x_zero[mm] + 128;
        const float iqx = e.x_inv_q[mm];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
          const int64_t n = ncol[j];
          const float y = recover(acc[i][j][r], colterm[j], ztw[j], ztx, sigx, iqw[j], iqx) + bn[j];
          if (n < N) {
            mx = fmaxf(mx, y);
            if (m < M) {
              if (e.logits) e.logits[m * N + n] = y;
              if (e.acc) e.acc[m * N + n] = acc_u8(acc[i][j][r], sigw[j], sigx, K);
            }
          }
          // stash y in the accumulator register as float bits for the sum pass
          acc[i][j][r] = __float_as_int(y);
        }
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        if ((lane & 31) == 0) red[wn * BM + lr] = mx;
      }
    __syncthreads();
    float *tmax = red + WN * BM;  // [BM]
    for (int r = threadIdx.x; r < BM; r += C::NT) {
      float mx = -INFINITY;
      for (int w = 0; w < WN; ++w) mx = fmaxf(mx, red[w * BM + r]);
      tmax[r] = mx;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = wm * C::TM + i * 32 + frag_row(r, lane);
        const float mx = tmax[lr];
        float sm = 0.0f;
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
          if (ncol[j] < N) sm += __expf(__int_as_float(acc[i][j][r]) - mx);
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) sm += __shfl_xor(sm, o, 64);
        if ((lane & 31) == 0) red[wn * BM + lr] = sm;
      }
    __syncthreads();
    for (int r = threadIdx.x; r < BM; r += C::NT) {
      const int64_t m = m0 + r;
      if (m >= M) continue;
      float sm = 0.0f;
      for (int w = 0; w < WN; ++w) sm += red[w * BM + r];
      e.stats[m * e.ntn + tn] = make_float2(tmax[r], sm);
    }
  }
}

// ------------------------------------------------------------------ launch
template <int BM, int BN, int BK, int WM, int WN, int NS, int EPI>
static hipError_t run(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb, int64_t M,
                      int64_t N, int64_t K, const EpiArgs &e, hipStream_t s) {
  using C = GemmCfg<BM, BN, BK, WM, WN, NS>;
  const int64_t Kp = round_up(K, BK);
  size_t lds = (size_t)C::LDS;
  if (EPI == EPI_SMAX_OUT) lds += 2 * BM * sizeof(float);
  if (EPI == EPI_SMAX_STATS) {
    const size_t need = (size_t)(WN + 1) * BM * sizeof(float);
    lds = lds > need ? lds : need;
  }
  auto kern = k_gemm<BM, BN, BK, WM, WN, NS, EPI>;
  static bool attr_set = false;  // per instantiation; idempotent
  if (!attr_set) {
    const hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  dim3 grid((unsigned)(((N + BN - 1) / BN) * ((M + BM - 1) / BM)));
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), lds, s, A, lda, B, ldb, M, N, K, Kp, e);
  return hipGetLastError();
}

// Kp must stay within the padded leading dimensions: with ld a multiple of 64
// and BK = 64 this always holds; BK = 128 is used when both ld allow it.
// Column width of the tiles a product of M x N uses: 256 once there are
// enough 256x256 tiles to fill the chip, else 128.
static int big_tile_n(int64_t M, int64_t N) {
  return ((M + 255) / 256) * ((N + 255) / 256) >= 256 ? 256 : 128;
}

template <int EPI>
static hipError_t dispatch(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb, int64_t M,
                           int64_t N, int64_t K, const EpiArgs &e, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  const bool k128 = round_up(K, 128) <= lda && round_up(K, 128) <= ldb;
  // 256x256 tiles (128x128 per wave) once there are enough of them to fill
  // the chip; otherwise 128x128 tiles (64x64 per wave)
  if (big_tile_n(M, N) == 256) {
    if constexpr (EPI != EPI_RAW) {
      // recovering epilogues: 8 waves of 128x64 (two per SIMD, so one wave's
      // epilogue stalls hide behind the other's work)
      if (k128) return run<256, 256, 128, 2, 4, 2, EPI>(A, lda, B, ldb, M, N, K, e, s);
      return run<256, 256, 64, 2, 4, 4, EPI>(A, lda, B, ldb, M, N, K, e, s);
    }
    if (k128) return run<256, 256, 128, 2, 2, 2, EPI>(A, lda, B, ldb, M, N, K, e, s);
    return run<256, 256, 64, 2, 2, 4, EPI>(A, lda, B, ldb, M, N, K, e, s);
  }
  if (k128) return run<128, 128, 128, 2, 2, 0, EPI>(A, lda, B, ldb, M, N, K, e, s);
  return run<128, 128, 64, 2, 2, 0, EPI>(A, lda, B, ldb, M, N, K, e, s);
}

static EpiArgs make_epi(const ActRows &X, const WeightMat &W, const float *bias) {
  EpiArgs e{};
  e.x_zero = X.zero;
  e.x_inv_q = X.inv_q;
  e.x_sums = X.sums;
  e.w_zero = W.zero;
  e.w_inv_q = W.inv_q;
  e.w_sums = W.row_sums;
  e.w_rpb = W.rows_per_block;
  e.bias = bias;
  return e;
}

hipError_t launch_gemm_recover(const ActRows &X, const WeightMat &W, int64_t M, int64_t N,
                               int64_t K, const float *bias, float *Y, int32_t *acc,
                               hipStream_t s) {
  EpiArgs e = make_epi(X, W, bias);
  e.Y = Y;
  e.acc = acc;
  return dispatch<EPI_RECOVER>(X.codes, X.ld, W.codes, W.ld, M, N, K, e, s);
}

hipError_t launch_gemm_raw(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                           int32_t *C, int64_t M, int64_t N, int64_t K, const int32_t *a_sums,
                           const int32_t *b_sums, hipStream_t s) {
  EpiArgs e{};
  e.x_sums = a_sums;
  e.w_sums = b_sums;
  e.acc = C;
  return dispatch<EPI_RAW>(A, lda, B, ldb, M, N, K, e, s);
}

// Per-tile statistics [M][ntn] (ntn of 128-column tiles is the most any
// launch uses), then the per-row (max, 1 / sum) [M].
static size_t smax_stats_bytes(int64_t M, int64_t N) {
  return align_up((size_t)M * (size_t)((N + 127) / 128) * sizeof(float2), 256);
}
size_t softmax_ws(int64_t M, int64_t N) {
  return smax_stats_bytes(M, N) + align_up((size_t)M * sizeof(float2), 256);
}

// Softmax normaliser of each row from its column tiles' (max, sum exp):
// max over the tiles, sum of sum_t exp(max_t - max), stored as (max, 1/sum).
__global__ __launch_bounds__(256) void k_smax_combine(const float2 *__restrict__ stats, int ntn,
                                                      int64_t M, float2 *__restrict__ rowstat) {
  const int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (m >= M) return;
  const float2 *s = stats + m * ntn;
  float mx = -INFINITY;
  for (int t = 0; t < ntn; ++t) mx = fmaxf(mx, s[t].x);
  float sm = 0.0f;
  for (int t = 0; t < ntn; ++t) {
    const float2 st = s[t];
    sm += st.y * __expf(st.x - mx);
  }
  rowstat[m] = make_float2(mx, 1.0f / sm);
}

hipError_t launch_softmax_layer(const ActRows &X, const WeightMat &W, int64_t M, int64_t N,
                                int64_t K, const float *bias, float *post, int32_t *acc,
                                float *logits, void *ws, hipStream_t s) {
  EpiArgs e = make_epi(X, W, bias);
  e.stats = static_cast<float2 *>(ws);
  const int tn = big_tile_n(M, N);
  e.ntn = (int)((N + tn - 1) / tn);
  e.acc = acc;
  e.logits = logits;
  hipError_t err = dispatch<EPI_SMAX_STATS>(X.codes, X.ld, W.codes, W.ld, M, N, K, e, s);
  if (err != hipSuccess || M == 0) return err;
  float2 *rowstat = reinterpret_cast<float2 *>(static_cast<char *>(ws) + smax_stats_bytes(M, N));
  hipLaunchKernelGGL(k_smax_combine, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s,
                     e.stats, e.ntn, M, rowstat);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  e.rowstat = rowstat;
  e.acc = nullptr;
  e.logits = nullptr;
  e.Y = post;
  return dispatch<EPI_SMAX_OUT>(X.codes, X.ld, W.codes, W.ld, M, N, K, e, s);
}

}  // namespace ql
