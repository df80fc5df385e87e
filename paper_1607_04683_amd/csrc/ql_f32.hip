// ql_f32.hip -- the unquantized fp32 model on gfx950: the float baseline the
// 8-bit model is compared with (the 'match' condition of Section 5).
//
// Same structure as the 8-bit path, float arithmetic throughout:
//   * input products hoisted over all T*B frames into one GEMM per layer
//     (v_mfma_f32_32x32x2f32, fp32 accumulation, bias in the epilogue);
//   * one persistent cooperative launch per layer for the recurrence, with
//     the layer's W_h slice resident in LDS where it fits (read from L2
//     otherwise), h_t / m_t passed between workgroups through device-coherent
//     stores and per-batch-slice arrival counters (ql_exchange.h);
//   * the output layer as a GEMM into the posterior buffer followed by an
//     in-place row softmax.
// Gate functions are the same own-exp sigmoid / tanh as the 8-bit path.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"

#include <algorithm>

namespace ql {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// GEMM  C[m][n] = sum_k A(m, k) B(n, k) (+ bias[n]).  An operand is stored
// either row-major [rows][ld] with k contiguous (A(m, k) = A[m*lda + k]) or,
// transposed (TA / TB), [K][ld] with its rows contiguous (A(m, k) =
// A[k*lda + m]); the training step's gradient products need both.
// 128x128 tiles, 2x2 waves of 64x64 (2x2 blocks of 32x32 MFMA), K in steps
// of 32 floats through two register-staged LDS stages; LDS rows hold 33
// floats so the column reads of 32 consecutive rows use 32 banks.  A grid
// with gridDim.y > 1 splits K: split s sums k in [s*klen, (s+1)*klen) into
// C + s*split_stride (partial sums, no bias), reduced afterwards in split
// order.
// ---------------------------------------------------------------------------
constexpr int kFB = 128, kFK = 32, kFLD = kFK + 1, kFThreads = 256;
constexpr size_t kFStage = (size_t)2 * kFB * kFLD;  // floats per stage (A and B)

// rows r0.., k in [k0, kend): 128 x 32 elements, 4 vectors of 4 per thread
template <bool TR>
__device__ __forceinline__ void f_load(const float *X, int64_t ld, int64_t nrows, int64_t kend,
                                       int64_t r0, int64_t k0, bool vec, v4f (&st)[4]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v4f x = {0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (!TR) {  // 4 consecutive k of row gr
      const int64_t gr = r0 + i * 32 + (tid >> 3), gk = k0 + 4 * (tid & 7);
      if (gr < nrows) {
        const float *p = X + gr * ld + gk;
        if (vec && gk + 3 < kend) {
          x = *reinterpret_cast<const v4f *>(p);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gk + e < kend) x[e] = p[e];
        }
      }
    } else {  // 4 consecutive rows at one k
      const int64_t gk = k0 + (tid >> 3), gr = r0 + 4 * ((tid & 7) + 8 * i);
      if (gk < kend) {
        const float *p = X + gk * ld + gr;
        if (vec && gr + 3 < nrows) {
          x = *reinterpret_cast<const v4f *>(p);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gr + e < nrows) x[e] = p[e];
        }
      }
    }
    st[i] = x;
  }
}

template <bool TR>
__device__ __forceinline__ void f_store(float *lds, const v4f (&st)[4]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (!TR)
        lds[(i * 32 + (tid >> 3)) * kFLD + 4 * (tid & 7) + e] = st[i][e];
      else
        lds[(4 * ((tid & 7) + 8 * i) + e) * kFLD + (tid >> 3)] = st[i][e];
    }
}

template <bool TA, bool TB>
__global__ __launch_bounds__(kFThreads) void k_sgemm(const float *__restrict__ A, int64_t lda,
                                                     const float *__restrict__ Bm, int64_t ldb,
                                                     int64_t M, int64_t N, int64_t K,
                                                     const float *__restrict__ bias,
                                                     float *__restrict__ C, int64_t ldc,
                                                     int64_t klen, int64_t split_stride) {
  extern __shared__ __attribute__((aligned(16))) float fsm[];
  const int ntn = (int)((N + kFB - 1) / kFB);
  const int64_t m0 = (int64_t)(blockIdx.x / ntn) * kFB, n0 = (int64_t)(blockIdx.x % ntn) * kFB;
  const int64_t kbeg = (int64_t)blockIdx.y * klen, kend = std::min<int64_t>(K, kbeg + klen);
  if (gridDim.y > 1) C += (int64_t)blockIdx.y * split_stride;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave >> 1, wn = wave & 1;
  const bool va = (lda & 3) == 0 && (reinterpret_cast<uintptr_t>(A) & 15) == 0;
  const bool vb = (ldb & 3) == 0 && (reinterpret_cast<uintptr_t>(Bm) & 15) == 0;
  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16f{};
  const int nk = kend > kbeg ? (int)((kend - kbeg + kFK - 1) / kFK) : 0;
  v4f sa[4], sb[4];
  if (nk > 0) {
    f_load<TA>(A, lda, M, kend, m0, kbeg, va, sa);
    f_load<TB>(Bm, ldb, N, kend, n0, kbeg, vb, sb);
    f_store<TA>(fsm, sa);
    f_store<TB>(fsm + kFB * kFLD, sb);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      f_load<TA>(A, lda, M, kend, m0, kbeg + (int64_t)(kt + 1) * kFK, va, sa);
      f_load<TB>(Bm, ldb, N, kend, n0, kbeg + (int64_t)(kt + 1) * kFK, vb, sb);
    }
    const float *as = fsm + (kt & 1) * kFStage, *bs = as + kFB * kFLD;
#pragma unroll 4
    for (int kk = 0; kk < kFK / 2; ++kk) {
      const int k = 2 * kk + (lane >> 5);
      float af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = as[(wm * 64 + i * 32 + (lane & 31)) * kFLD + k];
#pragma unroll
      for (int j = 0; j < 2; ++j) bf[j] = bs[(wn * 64 + j * 32 + (lane & 31)) * kFLD + k];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      float *nb = fsm + ((kt + 1) & 1) * kFStage;
      f_store<TA>(nb, sa);
      f_store<TB>(nb + kFB * kFLD, sb);
    }
    __syncthreads();
  }
  // element r of a 32x32 block: row ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3), column lane & 31
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t n = n0 + wn * 64 + j * 32 + (lane & 31);
      if (n >= N) continue;
      const float bn = bias && gridDim.y == 1 ? bias[n] : 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * 64 + i * 32 + ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3);
        if (m < M) C[m * ldc + n] = acc[i][j][r] + bn;
      }
    }
}

// C[m][n] = sum_s part[s][m][n] over the splits in order (+ bias[n]).
__global__ void k_sum_splits(const float *part, int splits, int64_t M, int64_t N,
                             const float *bias, float *C, int64_t ldc) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M * N) return;
  const int64_t m = i / N, n = i % N;
  float v = part[i];
  for (int sp = 1; sp < splits; ++sp) v += part[(int64_t)sp * M * N + i];
  C[m * ldc + n] = bias ? v + bias[n] : v;
}

template <bool TA, bool TB>
static hipError_t sgemm_set_attr() {
  static bool attr_set = false;
  if (attr_set) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_sgemm<TA, TB>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)(2 * kFStage * sizeof(float)));
  if (e == hipSuccess) attr_set = true;
  return e;
}

hipError_t launch_sgemm_ex(bool ta, bool tb, const float *A, int64_t lda, const float *B,
                           int64_t ldb, int64_t M, int64_t N, int64_t K, const float *bias,
                           float *C, int64_t ldc, int splits, float *part, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  const size_t lds = 2 * kFStage * sizeof(float);
  hipError_t e = ta ? (tb ? sgemm_set_attr<true, true>() : sgemm_set_attr<true, false>())
                    : (tb ? sgemm_set_attr<false, true>() : sgemm_set_attr<false, false>());
  if (e != hipSuccess) return e;
  const int64_t tiles = ((M + kFB - 1) / kFB) * ((N + kFB - 1) / kFB);
  if (splits < 1 || !part) splits = 1;
  const int64_t klen = splits > 1 ? round_up((K + splits - 1) / splits, kFK) : std::max<int64_t>(K, 1);
  if (splits > 1) splits = (int)((K + klen - 1) / klen);
  float *out = splits > 1 ? part : C;
  const int64_t ldo = splits > 1 ? N : ldc;
  const dim3 grid((unsigned)tiles, (unsigned)splits);
  const float *biasp = splits > 1 ? nullptr : bias;
  const int64_t stride = M * N;
#define QL_SGEMM(TA_, TB_)                                                                    \
  hipLaunchKernelGGL((k_sgemm<TA_, TB_>), grid, dim3(kFThreads), lds, s, A, lda, B, ldb, M, N, \
                     K, biasp, out, ldo, klen, stride)
  if (ta && tb) QL_SGEMM(true, true);
  else if (ta) QL_SGEMM(true, false);
  else if (tb) QL_SGEMM(false, true);
  else QL_SGEMM(false, false);
#undef QL_SGEMM
  e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t n = M * N;
  hipLaunchKernelGGL(k_sum_splits, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     (const float *)part, splits, M, N, bias, C, ldc);
  return hipGetLastError();
}

hipError_t launch_sgemm(const float *A, int64_t lda, const float *B, int64_t ldb, int64_t M,
                        int64_t N, int64_t K, const float *bias, float *C, int64_t ldc,
                        hipStream_t s) {
  return launch_sgemm_ex(false, false, A, lda, B, ldb, M, N, K, bias, C, ldc, 1, nullptr, s);
}

// ---------------------------------------------------------------------------
// Row softmax in place: p = exp(x - max) / sum exp(x - max), one workgroup per row.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block_reduce(float v, bool is_max, float *red) {
  for (int o = 32; o > 0; o >>= 1) {
    const float w = __shfl_xor(v, o, 64);
    v = is_max ? fmaxf(v, w) : v + w;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  v = red[0];
  for (int w = 1; w < nw; ++w) v = is_max ? fmaxf(v, red[w]) : v + red[w];
  return v;
}

__global__ __launch_bounds__(256) void k_softmax_rows(float *x, int64_t S) {
  __shared__ float red[4];
  float *row = x + (int64_t)blockIdx.x * S;
  float mx = -INFINITY;
  for (int64_t k = threadIdx.x; k < S; k += blockDim.x) mx = fmaxf(mx, row[k]);
  mx = block_reduce(mx, true, red);
  float sm = 0.0f;
  for (int64_t k = threadIdx.x; k < S; k += blockDim.x) sm += __expf(row[k] - mx);
  sm = block_reduce(sm, false, red);
  const float inv = 1.0f / sm;
  for (int64_t k = threadIdx.x; k < S; k += blockDim.x) row[k] = __expf(row[k] - mx) * inv;
}

hipError_t launch_softmax_rows(float *x, int64_t rows, int64_t S, hipStream_t s) {
  if (rows == 0 || S == 0) return hipSuccess;
  hipLaunchKernelGGL(k_softmax_rows, dim3((unsigned)rows), dim3(256), 0, s, x, S);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Persistent fp32 recurrence.  Tiles of bB batch rows x u hidden units (phase
// A: gates, cell, m_t) and, with a projection, bB2 batch rows x p2 outputs
// (phase B: h_t = W_r m_t).  Products: one batch row per tile (bB = 1) on
// the VALU, a wave per output row; 16 batch rows per tile on
// v_mfma_f32_16x16x4f32, the K range split over waves when there are fewer
// 16x16 output tiles than waves.
// ---------------------------------------------------------------------------
constexpr int kF32Threads = 512;

struct F32Tiling {
  int bB, u, nbt, nut;
  int bB2, p2, nbt2, npt;
  int grid, ldx, ldx2, w_lds, ksplit, ksplit2;
  size_t off_c, off_w, off_x, off_s, off_p, off_x2, off_s2, off_p2, lds_bytes;
};

// S[lb][n] = sum_{k < K} x[lb][k] w_n[k] for lb < 16 (MFMA) and n < nrows (a
// multiple of 16), with w_n = wrow(n).  x rows are zero beyond K up to a
// multiple of 4; w rows are read only below K.
template <class RowFn>
__device__ __forceinline__ void f_products_mfma(const float *x, int ldx, RowFn wrow, int nrows,
                                                int K, int ksplit, float *S, int ldS, float *part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int nt = nrows / 16, ntask = nt * ksplit;
  const int kchunk = ((K + 3) / 4 + ksplit - 1) / ksplit * 4;
  for (int task = wave; task < ntask; task += nw) {
    const int tj = task % nt, ks = task / nt;
    const int klo = ks * kchunk, khi = klo + kchunk < K ? klo + kchunk : K;
    const float *xr = x + (lane & 15) * ldx + (lane >> 4);
    const float *wr = wrow(tj * 16 + (lane & 15)) + (lane >> 4);
    v4f acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int k = klo; k < khi; k += 4) {
      const float av = xr[k];
      const float bv = k + (lane >> 4) < K ? wr[k] : 0.0f;
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
    }
    float *dst = ksplit == 1 ? S : part + ks * 16 * ldS;
#pragma unroll
    for (int r = 0; r < 4; ++r) dst[((lane >> 4) * 4 + r) * ldS + tj * 16 + (lane & 15)] = acc[r];
  }
  if (ksplit > 1) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < 16 * nrows; idx += blockDim.x) {
      const int lb = idx / nrows, n = idx % nrows;
      float v = 0.0f;
      for (int ks = 0; ks < ksplit; ++ks) v += part[ks * 16 * ldS + lb * ldS + n];
      S[lb * ldS + n] = v;
    }
  }
}

// One batch row: a wave per output row, lanes over K.
template <class RowFn>
__device__ __forceinline__ void f_products_valu(const float *x, RowFn wrow, int nrows, int K,
                                                float *S) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int n = wave; n < nrows; n += nw) {
    const float *wr = wrow(n);
    float acc = 0.0f;
    for (int k = lane; k < K; k += 64) acc += x[k] * wr[k];
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) S[n] = acc;
  }
}

__global__ __launch_bounds__(kF32Threads) void k_recurrent_f32(F32RecArgs a, F32Tiling tl) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float *cst = reinterpret_cast<float *>(smem + tl.off_c);
  float *wsl = reinterpret_cast<float *>(smem + tl.off_w);
  float *xs = reinterpret_cast<float *>(smem + tl.off_x);
  float *S = reinterpret_cast<float *>(smem + tl.off_s);
  float *part = reinterpret_cast<float *>(smem + tl.off_p);
  float *xs2 = reinterpret_cast<float *>(smem + tl.off_x2);
  float *S2 = reinterpret_cast<float *>(smem + tl.off_s2);
  float *part2 = reinterpret_cast<float *>(smem + tl.off_p2);
  __shared__ int s_abort;

  const int64_t T = a.T, B = a.B, H = a.H, P = a.P, R = a.R;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  unsigned *cnt = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
  auto counter = [&](int kind, int64_t par, int slice) {
    return cnt + ((kind * 2 + (int)par) * kMaxSlices + slice) * 16;
  };
  float *xhf = reinterpret_cast<float *>(static_cast<char *>(a.ws) + kHeaderBytes + kCounterBytes);
  float *xmf = xhf + 2 * B * R;

  const int tid = threadIdx.x;
  const bool mf = tl.bB > 1;
  const bool activeA = (int)blockIdx.x < tl.nbt * tl.nut;
  const int tb = activeA ? blockIdx.x / tl.nut : 0, tu = activeA ? blockIdx.x % tl.nut : 0;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = activeA ? (int)(B - b0 < tl.bB ? B - b0 : tl.bB) : 0;
  const int nu = activeA ? (int)(H - j0 < tl.u ? H - j0 : tl.u) : 0;
  const int nrows = 4 * tl.u;  // gate-major: row g*u + jj is W_h row g*H + j0 + jj
  const bool activeB = P > 0 && (int)blockIdx.x < tl.nbt2 * tl.npt;
  const int tb2 = activeB ? blockIdx.x / tl.npt : 0, tp = activeB ? blockIdx.x % tl.npt : 0;
  const int64_t c0 = (int64_t)tb2 * tl.bB2, p0 = (int64_t)tp * tl.p2;
  const int nb2 = activeB ? (int)(B - c0 < tl.bB2 ? B - c0 : tl.bB2) : 0;
  const int np2 = activeB ? (int)(P - p0 < tl.p2 ? P - p0 : tl.p2) : 0;
  const int tbB = activeB ? (int)(c0 / tl.bB) : 0;
  const unsigned prod_h =
      P == 0 ? (unsigned)tl.nut : (unsigned)(((nb + tl.bB2 - 1) / tl.bB2) * tl.npt);
  const unsigned prod_m = (unsigned)tl.nut;
  if (tid == 0) s_abort = 0;

  // row n of this tile's W_h slice (gate-major, n = g*u + jj): the LDS copy,
  // or W_h row g*H + j0 + jj in global memory (units past H read the last one)
  auto wh_row = [&](int n) -> const float * {
    if (tl.w_lds) return wsl + n * tl.ldx;
    const int g = n / tl.u, jj = n % tl.u;
    return a.Wh + (g * H + j0 + (jj < nu ? jj : nu - 1)) * R;
  };
  if (activeA) {
    if (tl.w_lds)
      for (int idx = tid; idx < nrows * tl.ldx; idx += blockDim.x) {
        const int r = idx / tl.ldx, k = idx % tl.ldx;
        const int g = r / tl.u, jj = r % tl.u;
        wsl[idx] = jj < nu && k < R ? a.Wh[(g * H + j0 + jj) * R + k] : 0.0f;
      }
    for (int idx = tid; idx < tl.bB * tl.u; idx += blockDim.x) {
      const int lb = idx / tl.u, jj = idx % tl.u;
      cst[idx] = lb < nb && jj < nu && a.c0 ? a.c0[(b0 + lb) * H + j0 + jj] : 0.0f;
    }
  }
  __syncthreads();

  for (int64_t t = 0; t < T; ++t) {
    const int64_t hcur = (t & 1) * B * R, mcur = (t & 1) * B * H;
    if (activeA) {
      // h_{t-1} rows of this batch slice (rows past B and columns past R are 0)
      const float *prev = nullptr;
      if (t > 0) {
        if (!wait_count(counter(0, (t - 1) & 1, tb), (unsigned)(((t - 1) >> 1) + 1) * prod_h, flag))
          s_abort = 1;
        __syncthreads();
        if (s_abort) return;
        prev = xhf + ((t - 1) & 1) * B * R;
      }
      for (int idx = tid; idx < tl.bB * tl.ldx; idx += blockDim.x) {
        const int lb = idx / tl.ldx, k = idx % tl.ldx;
        float v = 0.0f;
        if (lb < nb && k < R) {
          if (prev) v = ld_coherent(prev + (b0 + lb) * R + k);
          else if (a.h0) v = a.h0[(b0 + lb) * R + k];
        }
        xs[idx] = v;
      }
      __syncthreads();
      if (mf)
        f_products_mfma(xs, tl.ldx, wh_row, nrows, (int)R, tl.ksplit, S, nrows, part);
      else
        f_products_valu(xs, wh_row, nrows, (int)R, S);
      __syncthreads();
      const int pairs = nb * nu;
      for (int idx = tid; idx < pairs * 4; idx += blockDim.x) {
        const int pr = idx >> 2, gg = idx & 3;
        const int lb = pr / nu, jj = pr % nu;
        const int64_t b = b0 + lb, j = j0 + jj;
        const float av = a.gx[(t * B + b) * 4 * H + gg * H + j] + S[lb * nrows + gg * tl.u + jj];
        const float sg = sigmoid_cw(gg == 2 ? 2.0f * av : av);
        const float act = gg == 2 ? 2.0f * sg - 1.0f : sg;
        const int base = (threadIdx.x & 63) & ~3;
        const float ig = __shfl(act, base + 0, 64);
        const float fg = __shfl(act, base + 1, 64);
        const float gv = __shfl(act, base + 2, 64);
        const float og = __shfl(act, base + 3, 64);
        if (gg == 0) {
          const float cn = (fg * cst[lb * tl.u + jj]) + (ig * gv);
          cst[lb * tl.u + jj] = cn;
          const float m = og * tanh_cw(cn);
          if (P == 0) {
            st_coherent(&xhf[hcur + b * R + j], m);
            a.h[(t * B + b) * R + j] = m;
            if (t == T - 1 && a.hT) a.hT[b * R + j] = m;
          } else {
            st_coherent(&xmf[mcur + b * H + j], m);
          }
          if (t == T - 1 && a.cT) a.cT[b * H + j] = cn;
        }
      }
      arrive(counter(P == 0 ? 0 : 1, t & 1, tb));
    }
    if (P > 0 && activeB) {
      __syncthreads();
      if (!wait_count(counter(1, t & 1, tbB), (unsigned)((t >> 1) + 1) * prod_m, flag)) s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      const float *mrows = xmf + mcur;
      for (int idx = tid; idx < tl.bB2 * tl.ldx2; idx += blockDim.x) {
        const int lb = idx / tl.ldx2, k = idx % tl.ldx2;
        xs2[idx] = lb < nb2 && k < H ? ld_coherent(mrows + (c0 + lb) * H + k) : 0.0f;
      }
      __syncthreads();
      auto wr_row = [&](int n) -> const float * {
        return a.Wr + (p0 + (n < np2 ? n : np2 - 1)) * H;
      };
      if (tl.bB2 > 1)
        f_products_mfma(xs2, tl.ldx2, wr_row, tl.p2, (int)H, tl.ksplit2, S2, tl.p2, part2);
      else
        f_products_valu(xs2, wr_row, tl.p2, (int)H, S2);
      __syncthreads();
      for (int idx = tid; idx < nb2 * np2; idx += blockDim.x) {
        const int lb = idx / np2, pp = idx % np2;
        const int64_t b = c0 + lb, p = p0 + pp;
        const float hv = S2[lb * tl.p2 + pp];
        st_coherent(&xhf[hcur + b * P + p], hv);
        a.h[(t * B + b) * P + p] = hv;
        if (t == T - 1 && a.hT) a.hT[b * P + p] = hv;
      }
      arrive(counter(0, t & 1, tbB));
    }
    __syncthreads();
  }
}

size_t recurrent_f32_ws(int64_t B, int64_t H, int64_t P) {
  const int64_t R = P > 0 ? P : H;
  return kHeaderBytes + kCounterBytes + align_up((size_t)(2 * B * R + 2 * B * H) * sizeof(float), 256);
}

static bool plan_f32(const F32RecArgs &a, int G, int lds_max, F32Tiling *out) {
  F32Tiling tl{};
  const int64_t B = a.B, H = a.H, P = a.P, R = a.R;
  if (B < 16) {
    tl.bB = 1;
    tl.nbt = (int)B;
    const int nut = G / (int)B;
    if (nut < 1) return false;
    tl.u = (int)((H + nut - 1) / nut);
  } else {
    tl.bB = 16;
    tl.nbt = (int)((B + 15) / 16);
    if (tl.nbt > G) return false;
    const int nut = G / tl.nbt;
    tl.u = (int)((H + nut - 1) / nut);
    tl.u = (tl.u + 3) / 4 * 4;  // 4u a multiple of 16
  }
  tl.nut = (int)((H + tl.u - 1) / tl.u);
  if (tl.nbt > kMaxSlices) return false;
  const int nrows = 4 * tl.u;
  tl.ldx = (int)round_up(R, 32) + 2;  // rows 2 words off a bank multiple
  tl.ldx2 = (int)round_up(H, 32) + 2;
  if (P > 0) {
    if (B < 16) {
      tl.bB2 = 1;
      tl.nbt2 = (int)B;
      const int npt = G / (int)B;
      tl.p2 = (int)((P + npt - 1) / npt);
    } else {
      tl.bB2 = 16;
      tl.nbt2 = (int)((B + 15) / 16);
      const int npt = G / tl.nbt2;
      tl.p2 = (int)((P + npt - 1) / npt);
      tl.p2 = (tl.p2 + 15) / 16 * 16;
    }
    tl.npt = (int)((P + tl.p2 - 1) / tl.p2);
    tl.ksplit2 = tl.bB2 > 1 ? std::max(1, 8 / std::max(1, tl.p2 / 16)) : 1;
  }
  tl.grid = std::max(tl.nbt * tl.nut, P > 0 ? tl.nbt2 * tl.npt : 0);
  if (tl.grid > G) return false;
  // LDS: cell state; W_h slice (when it fits); phase A and phase B scratch
  // share one region (phase B starts after a barrier).
  auto layout = [&](bool wl) {
    size_t off = 0;
    tl.off_c = off;
    off = align_up(off + (size_t)tl.bB * tl.u * 4, 16);
    tl.off_w = off;
    if (wl) off = align_up(off + (size_t)nrows * tl.ldx * 4, 16);
    const size_t ua = off;
    // K split of the MFMA products: enough tasks for the 8 waves
    const int ks = tl.bB > 1 ? std::max(1, 8 / std::max(1, nrows / 16)) : 1;
    tl.ksplit = ks;
    tl.off_x = ua;
    size_t oa = align_up(ua + (size_t)tl.bB * tl.ldx * 4, 16);
    tl.off_s = oa;
    oa = align_up(oa + (size_t)tl.bB * nrows * 4, 16);
    tl.off_p = oa;
    oa = align_up(oa + (ks > 1 ? (size_t)ks * 16 * nrows * 4 : 0), 16);
    size_t ob = ua;
    if (P > 0) {
      tl.off_x2 = ob;
      ob = align_up(ob + (size_t)tl.bB2 * tl.ldx2 * 4, 16);
      tl.off_s2 = ob;
      ob = align_up(ob + (size_t)tl.bB2 * tl.p2 * 4, 16);
      tl.off_p2 = ob;
      ob = align_up(ob + (tl.ksplit2 > 1 ? (size_t)tl.ksplit2 * 16 * tl.p2 * 4 : 0), 16);
    }
    tl.lds_bytes = std::max(oa, ob);
    return tl.lds_bytes + 64 <= (size_t)lds_max;
  };
  tl.w_lds = 1;
  if (!layout(true)) {
    tl.w_lds = 0;
    if (!layout(false)) return false;
  }
  *out = tl;
  return true;
}

hipError_t launch_recurrent_f32(const F32RecArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0 || a.B == 0) return hipSuccess;
  int dev = 0, cus = 0, lds_max = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  F32Tiling tl;
  if (!plan_f32(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_recurrent_f32),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_recurrent_f32, kF32Threads,
                                                   tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  e = clear_exchange(a.ws, kCounterBytes / 8, s);
  if (e != hipSuccess) return e;
  F32RecArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(k_recurrent_f32), dim3(tl.grid),
                                    dim3(kF32Threads), kargs, (unsigned)tl.lds_bytes, s);
}

hipError_t set_wait_bound_f32(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
