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
};

template <int BM, int BN, int BK, int WM, int WN>
struct Cfg {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int LDSS = BK + 16;  // padded LDS row stride in bytes
  static constexpr int STAGE = (BM + BN) * LDSS;
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

// Row/column of element r of a 32x32 MFMA block held by `lane`.
__device__ __forceinline__ int frag_row(int r, int lane) { return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3); }
__device__ __forceinline__ int frag_col(int lane) { return lane & 31; }

template <int BM, int BN, int BK, int WM, int WN, int EPI>
__global__ __launch_bounds__(64 * WM *WN) void k_gemm(const int8_t *__restrict__ A, int64_t lda,
                                                       const int8_t *__restrict__ B, int64_t ldb,
                                                       int64_t M, int64_t N, int64_t K,
                                                       int64_t Kp, EpiArgs e) {
  using C = Cfg<BM, BN, BK, WM, WN>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // softmax output pass: combine the per-tile statistics of this tile's rows
  float *rowmax = reinterpret_cast<float *>(smem + 2 * C::STAGE);
  float *rowinv = rowmax + BM;
  if (EPI == EPI_SMAX_OUT) {
    for (int r = threadIdx.x; r < BM; r += C::NT) {
      const int64_t m = m0 + r;
      float mx = -INFINITY, sm = 0.0f;
      if (m < M) {
        for (int t = 0; t < e.ntn; ++t) mx = fmaxf(mx, e.stats[m * e.ntn + t].x);
        for (int t = 0; t < e.ntn; ++t) {
          const float2 st = e.stats[m * e.ntn + t];
          sm += st.y * __expf(st.x - mx);
        }
      }
      rowmax[r] = mx;
      rowinv[r] = 1.0f / sm;
    }
  }

  v16i acc[C::FM][C::FN];
  gemm_tile<BM, BN, BK, WM, WN>(A, lda, B, ldb, M, N, Kp, m0, n0, smem, acc);

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
      e.stats[m * e.ntn + blockIdx.x] = make_float2(tmax[r], sm);
    }
  }
}

// ------------------------------------------------------------------ launch
template <int BM, int BN, int BK, int WM, int WN, int EPI>
static hipError_t run(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb, int64_t M,
                      int64_t N, int64_t K, const EpiArgs &e, hipStream_t s) {
  using C = Cfg<BM, BN, BK, WM, WN>;
  const int64_t Kp = round_up(K, BK);
  size_t lds = 2 * (size_t)C::STAGE;
  if (EPI == EPI_SMAX_OUT) lds += 2 * BM * sizeof(float);
  if (EPI == EPI_SMAX_STATS) {
    const size_t need = (size_t)(WN + 1) * BM * sizeof(float);
    lds = lds > need ? lds : need;
  }
  auto kern = k_gemm<BM, BN, BK, WM, WN, EPI>;
  static bool attr_set = false;  // per instantiation; idempotent
  if (!attr_set) {
    hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr_set = true;
  }
  dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), lds, s, A, lda, B, ldb, M, N, K, Kp, e);
  return hipGetLastError();
}

// Kp must stay within the padded leading dimensions: with ld a multiple of 64
// and BK = 64 this always holds; BK = 128 is used when both ld allow it.
template <int EPI>
static hipError_t dispatch(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb, int64_t M,
                           int64_t N, int64_t K, const EpiArgs &e, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  if (round_up(K, 128) <= lda && round_up(K, 128) <= ldb)
    return run<128, 128, 128, 2, 2, EPI>(A, lda, B, ldb, M, N, K, e, s);
  return run<128, 128, 64, 2, 2, EPI>(A, lda, B, ldb, M, N, K, e, s);
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

size_t softmax_ws(int64_t M, int64_t N) {
  return align_up((size_t)M * (size_t)((N + 127) / 128) * sizeof(float2), 256);
}

hipError_t launch_softmax_layer(const ActRows &X, const WeightMat &W, int64_t M, int64_t N,
                                int64_t K, const float *bias, float *post, int32_t *acc,
                                float *logits, void *ws, hipStream_t s) {
  EpiArgs e = make_epi(X, W, bias);
  e.stats = static_cast<float2 *>(ws);
  e.ntn = (int)((N + 127) / 128);
  e.acc = acc;
  e.logits = logits;
  hipError_t err = dispatch<EPI_SMAX_STATS>(X.codes, X.ld, W.codes, W.ld, M, N, K, e, s);
  if (err != hipSuccess) return err;
  e.acc = nullptr;
  e.logits = nullptr;
  e.Y = post;
  return dispatch<EPI_SMAX_OUT>(X.codes, X.ld, W.codes, W.ld, M, N, K, e, s);
}

}  // namespace ql
