// ql_recurrent.hip -- the serial part of a quantized LSTM layer (Section 4) on gfx950.
//
// One cooperative, persistent launch runs all T steps of a layer.  The grid is
// split into tiles of (bB batch rows) x (u hidden units); a workgroup owns one
// tile for the whole sequence, keeps the 4u gate rows of W_h' it needs
// resident in LDS, and keeps its cell state c in LDS.  Each step:
//   1. (before waiting) prefetch its slice of the precomputed W_x x_t + b;
//   2. grid barrier: h_{t-1} is complete;
//   3. quantize h_{t-1} per vector for its batch rows (eq. 2) into LDS
//      (redundantly in every unit tile: no extra barrier is needed);
//   4. Mult: signed 8-bit products against the resident W_h' slice
//      (v_dot4 for one batch row, v_mfma_i32_16x16x64_i8 for 16+ rows);
//   5. R(.) of eq. 1/3, + (W_x x + b), sigmoid/tanh gates, c and m update;
//   6. with a projection: grid barrier, quantize m per vector, W_r' product,
//      recover h_t.
// The workgroup whose unit tile is 0 also stores the codes of h_{t-1} (the
// next layer's / output layer's input) so they are never recomputed.
//
// The grid barrier is a monotone counter.  Its wait is bounded: if it ever
// expires, a flag in the workspace is raised and every workgroup returns at
// its next barrier, so the grid always drains.
#include "ql_device.h"
#include "ql_launch.h"

namespace ql {

constexpr long kSpinLimit = 1l << 22;

struct RecTiling {
  int bB, u;        // phase A tile: batch rows x units
  int nbt, nut;     // tile counts
  int bB2, p2;      // phase B (projection) tile: batch rows x outputs
  int nbt2, npt;
  int grid;
  int mfmaA, mfmaB; // use MFMA for the phase A / B products
  int ldR, ldH;     // padded widths of h and m codes
  int ldsW;         // LDS row stride of the W_h' slice
  int ldsX;         // LDS row stride of activation codes
  size_t off_w, off_x, off_s, off_c, off_col, off_row, lds_bytes;
};

struct ColParam {
  int64_t colterm;  // sum s_w + K (z_w + 128)
  int32_t ztw;      // z_w + 128
  int32_t sigw;     // sum s_w
  float iqw;
  int32_t pad;
};
struct RowParam {
  int32_t ztx, sigx;
  float iqx;
  int32_t z;
};

// Grid barrier.  The workgroup's own barrier orders every wave's stores before
// thread 0's release (agent scope) on the counter; thread 0's acquire after
// the wait orders the workgroup's later loads after every other workgroup's
// release.  One release and one acquire per workgroup per barrier.
__device__ __forceinline__ bool grid_sync(unsigned *ctr, int *flag, unsigned target) {
  __syncthreads();
  __shared__ int s_to;
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    int to = 0;
    long it = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        to = 1;
        break;
      }
      if (++it > kSpinLimit) {
        __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        to = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    s_to = to;
  }
  __syncthreads();
  return s_to != 0;
}

// Quantize one vector of K floats (src null = zeros) into LDS codes; one wave.
// Two passes over src (used when a row does not fit the register path).
__device__ __forceinline__ RowParam quantize_vec_wave(const float *src, int64_t K, int8_t *dst,
                                                      int ldpad, int lane, int32_t *sum_out) {
  float lo = INFINITY, hi = -INFINITY;
  if (src) {
    for (int64_t i = lane; i < K; i += kWave) {
      const float v = src[i];
      lo = fminf(lo, v);
      hi = fmaxf(hi, v);
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
  }
  if (!src || K == 0) lo = hi = 0.0f;
  const QParams p = make_qparams(lo, hi);
  int sum = 0;
  for (int64_t i = lane; i < ldpad; i += kWave) {
    int8_t b = 0;
    if (i < K) {
      const int c = encode(src ? src[i] : 0.0f, p.q, p.z);
      sum += c;
      b = (int8_t)(c ^ 0x80);
    }
    dst[i] = b;
  }
  sum = wave_sum(sum);
  *sum_out = sum;
  RowParam r;
  r.z = p.z;
  r.ztx = p.z + 128;
  r.sigx = sum - 128 * (int32_t)K;
  r.iqx = p.inv_q;
  return r;
}

// Quantize RB vectors of K <= 64*NV floats at once: every value is loaded
// exactly once into registers (all RB rows' loads in flight together), then
// min/max, params and codes come from registers.  srcs[r] null = zero vector.
template <int NV, int RB>
__device__ __forceinline__ void quantize_rows_regs(const float *const (&srcs)[RB], int K,
                                                   int8_t *const (&dst)[RB], int ldpad, int lane,
                                                   RowParam (&rp)[RB], int32_t (&sums)[RB]) {
  float v[RB][NV];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = i * kWave + lane;
      v[r][i] = (srcs[r] && k < K) ? srcs[r][k] : 0.0f;
    }
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (i * kWave + lane < K) {
        lo = fminf(lo, v[r][i]);
        hi = fmaxf(hi, v[r][i]);
      }
    lo = wave_min(lo);
    hi = wave_max(hi);
    if (!srcs[r] || K == 0) lo = hi = 0.0f;
    const QParams p = make_qparams(lo, hi);
    int sum = 0;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = i * kWave + lane;
      int8_t b = 0;
      if (k < K) {
        const int c = encode(v[r][i], p.q, p.z);
        sum += c;
        b = (int8_t)(c ^ 0x80);
      }
      if (k < ldpad) dst[r][k] = b;
    }
    for (int k = NV * kWave + lane; k < ldpad; k += kWave) dst[r][k] = 0;
    sum = wave_sum(sum);
    sums[r] = sum;
    rp[r].z = p.z;
    rp[r].ztx = p.z + 128;
    rp[r].sigx = sum - 128 * K;
    rp[r].iqx = p.inv_q;
  }
}

// Quantize rows [0, nrows) of a tile, rows handed round-robin to the waves;
// row lb reads src_of(lb) (null = zeros) with K values, codes to
// dst + lb * ldx.  Calls done(lb, param, sum) for every row (lane-uniform).
template <class Src, class Done>
__device__ __forceinline__ void quantize_tile_rows(int nrows, int K, int8_t *dst, int ldx,
                                                   int ldpad, Src src_of, Done done) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwave = blockDim.x >> 6;
  if (K <= 8 * kWave) {
    constexpr int RB = 4;
    for (int lb0 = wave * RB; lb0 < nrows; lb0 += nwave * RB) {
      const float *srcs[RB];
      int8_t *dsts[RB];
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int lb = lb0 + r < nrows ? lb0 + r : nrows - 1;
        srcs[r] = src_of(lb);
        dsts[r] = dst + lb * ldx;
      }
      RowParam rp[RB];
      int32_t sums[RB];
      quantize_rows_regs<8, RB>(srcs, K, dsts, ldpad, lane, rp, sums);
#pragma unroll
      for (int r = 0; r < RB; ++r)
        if (lb0 + r < nrows) done(lb0 + r, rp[r], sums[r]);
    }
  } else if (K <= 32 * kWave) {
    for (int lb = wave; lb < nrows; lb += nwave) {
      const float *srcs[1] = {src_of(lb)};
      int8_t *dsts[1] = {dst + lb * ldx};
      RowParam rp[1];
      int32_t sums[1];
      quantize_rows_regs<32, 1>(srcs, K, dsts, ldpad, lane, rp, sums);
      done(lb, rp[0], sums[0]);
    }
  } else {
    for (int lb = wave; lb < nrows; lb += nwave) {
      int32_t sum;
      const RowParam r = quantize_vec_wave(src_of(lb), K, dst + lb * ldx, ldpad, lane, &sum);
      done(lb, r, sum);
    }
  }
}

// S[lb][n] = sum_k x[lb][k] w[n][k] over K bytes (multiple of 64), signed.
// VALU path: groups of 16 lanes per (row, n) task, v_dot4 on 16-byte chunks.
__device__ __forceinline__ void products_valu(const int8_t *x, int ldx, int nb, const int8_t *w,
                                              int64_t ldw, int nrows, int wrows, int K, int32_t *S,
                                              int ldS) {
  const int tid = threadIdx.x, grp = tid >> 4, gl = tid & 15;
  const int ntask = nb * nrows, ngrp = blockDim.x >> 4;
  for (int task = grp; task < ntask; task += ngrp) {
    const int lb = task / nrows, n = task % nrows;
    const int8_t *xr = x + lb * ldx;
    const int8_t *wr = w + (int64_t)(n < wrows ? n : wrows - 1) * ldw;
    int acc = 0;
    for (int k = gl * 16; k < K; k += 16 * 16) {
      const v4i a = *reinterpret_cast<const v4i *>(xr + k);
      const v4i b = *reinterpret_cast<const v4i *>(wr + k);
      acc = __builtin_amdgcn_sdot4(a.x, b.x, acc, false);
      acc = __builtin_amdgcn_sdot4(a.y, b.y, acc, false);
      acc = __builtin_amdgcn_sdot4(a.z, b.z, acc, false);
      acc = __builtin_amdgcn_sdot4(a.w, b.w, acc, false);
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (gl == 0) S[lb * ldS + n] = acc;
  }
}

// MFMA path: nb (multiple of 16) rows x nrows (multiple of 16) outputs.
__device__ __forceinline__ void products_mfma(const int8_t *x, int ldx, int nb, const int8_t *w,
                                              int64_t ldw, int nrows, int wrows, int K, int32_t *S,
                                              int ldS) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int mt = nb / 16, nt = nrows / 16;
  for (int tile = wave; tile < mt * nt; tile += nw) {
    const int ti = tile / nt, tj = tile % nt;
    const int8_t *xr = x + (ti * 16 + (lane & 15)) * ldx + (lane >> 4) * 16;
    const int wrow = tj * 16 + (lane & 15);
    const int8_t *wr = w + (int64_t)(wrow < wrows ? wrow : wrows - 1) * ldw + (lane >> 4) * 16;
    v4i acc = v4i{};
    for (int k = 0; k < K; k += 64) {
      const v4i a = *reinterpret_cast<const v4i *>(xr + k);
      const v4i b = *reinterpret_cast<const v4i *>(wr + k);
      acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      S[(ti * 16 + (lane >> 4) * 4 + r) * ldS + tj * 16 + (lane & 15)] = acc[r];
  }
}

__global__ __launch_bounds__(256) void k_recurrent(RecurrentArgs a, RecTiling tl) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int8_t *wsl = reinterpret_cast<int8_t *>(smem + tl.off_w);
  int8_t *xc = reinterpret_cast<int8_t *>(smem + tl.off_x);
  int32_t *S = reinterpret_cast<int32_t *>(smem + tl.off_s);
  float *cst = reinterpret_cast<float *>(smem + tl.off_c);
  ColParam *cp = reinterpret_cast<ColParam *>(smem + tl.off_col);
  RowParam *rp = reinterpret_cast<RowParam *>(smem + tl.off_row);

  unsigned *ctr = static_cast<unsigned *>(a.ws);
  int *flag = reinterpret_cast<int *>(static_cast<char *>(a.ws) + 64);
  float *mbuf = reinterpret_cast<float *>(static_cast<char *>(a.ws) + 256);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nwave = blockDim.x >> 6;
  const int64_t T = a.T, B = a.B, H = a.H, P = a.P, R = a.R;
  const int G = gridDim.x;
  const bool activeA = (int)blockIdx.x < tl.nbt * tl.nut;
  const int tb = activeA ? blockIdx.x / tl.nut : 0, tu = activeA ? blockIdx.x % tl.nut : 0;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = activeA ? (int)(B - b0 < tl.bB ? B - b0 : tl.bB) : 0;
  const int nu = activeA ? (int)(H - j0 < tl.u ? H - j0 : tl.u) : 0;
  const int nrows = 4 * tl.u;  // slice rows, gate-major: row g*u + jj
  const int ldS = nrows;

  // ---- prologue: resident W_h' slice, column params, initial c
  if (activeA) {
    for (int idx = tid; idx < nrows * (tl.ldR / 16); idx += blockDim.x) {
      const int r = idx / (tl.ldR / 16), kc = idx % (tl.ldR / 16);
      const int g = r / tl.u, jj = r % tl.u;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (jj < nu) v = *reinterpret_cast<const uint4 *>(a.Wh.codes + (g * H + j0 + jj) * a.Wh.ld + kc * 16);
      *reinterpret_cast<uint4 *>(wsl + r * tl.ldsW + kc * 16) = v;
    }
    for (int r = tid; r < nrows; r += blockDim.x) {
      const int g = r / tl.u, jj = r % tl.u;
      const int64_t n = g * H + j0 + (jj < nu ? jj : 0);
      const int64_t blk = n / a.Wh.rows_per_block;
      ColParam c;
      c.ztw = a.Wh.zero[blk] + 128;
      c.sigw = a.Wh.row_sums[n] - 128 * (int32_t)R;
      c.colterm = (int64_t)c.sigw + R * (int64_t)c.ztw;
      c.iqw = a.Wh.inv_q[blk];
      c.pad = 0;
      cp[r] = c;
    }
    for (int idx = tid; idx < tl.bB * tl.u; idx += blockDim.x) {
      const int lb = idx / tl.u, jj = idx % tl.u;
      float c0 = 0.0f;
      if (lb < nb && jj < nu && a.c0) c0 = a.c0[(b0 + lb) * H + j0 + jj];
      cst[idx] = c0;
    }
  }
  __syncthreads();

  unsigned nsync = 0;
  const int pairs = nb * nu;
  const int ppt = (tl.bB * tl.u + blockDim.x - 1) / blockDim.x;  // pairs per thread (max)

  for (int64_t t = 0; t <= T; ++t) {
    // prefetch W_x x_t + b for this thread's (b, j) pairs
    float gxv[8][4];
    if (t < T && activeA) {
      for (int q = 0; q < ppt; ++q) {
        const int idx = tid + q * blockDim.x;
        if (idx < pairs) {
          const int lb = idx / nu, jj = idx % nu;
          const float *g = a.gx + ((t * B + b0 + lb) * 4 * H) + j0 + jj;
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) gxv[q][gg] = g[gg * H];
        }
      }
    }
    if (t > 0 && grid_sync(ctr, flag, (++nsync) * (unsigned)G)) return;

    if (activeA) {
      // ---- 3. quantize h_{t-1} rows of this batch slice
      auto src_h = [&](int lb) -> const float * {
        if (lb >= nb) return nullptr;
        return t == 0 ? (a.h0 ? a.h0 + (b0 + lb) * R : nullptr) : a.h + ((t - 1) * B + b0 + lb) * R;
      };
      auto done_h = [&](int lb, const RowParam &r, int32_t sum) {
        if (lane == 0) rp[lb] = r;
        if (t > 0 && tu == 0 && lb < nb) {  // codes of h_{t-1} for the next consumer
          const int64_t row = (t - 1) * B + b0 + lb;
          int8_t *oc = a.out_codes + row * a.ld_out;
          for (int64_t i = lane; i < a.ld_out; i += kWave) oc[i] = i < tl.ldR ? xc[lb * tl.ldsX + i] : 0;
          if (a.tap_codes)
            for (int64_t i = lane; i < R; i += kWave) a.tap_codes[row * R + i] = xc[lb * tl.ldsX + i];
          if (lane == 0) {
            a.out_zero[row] = r.z;
            a.out_inv_q[row] = r.iqx;
            a.out_sums[row] = sum;
            if (a.tap_zero) a.tap_zero[row] = r.z;
            if (a.tap_inv_q) a.tap_inv_q[row] = r.iqx;
          }
        }
      };
      quantize_tile_rows(tl.bB, (int)R, xc, tl.ldsX, tl.ldR, src_h, done_h);
      if (t < T) {
        __syncthreads();
        // ---- 4. Mult against the resident slice
        if (tl.mfmaA)
          products_mfma(xc, tl.ldsX, tl.bB, wsl, tl.ldsW, nrows, nrows, tl.ldR, S, ldS);
        else
          products_valu(xc, tl.ldsX, nb, wsl, tl.ldsW, nrows, nrows, tl.ldR, S, ldS);
        __syncthreads();
        // ---- 5. recover, gates, cell update
        for (int q = 0; q < ppt; ++q) {
          const int idx = tid + q * blockDim.x;
          if (idx >= pairs) break;
          const int lb = idx / nu, jj = idx % nu;
          const RowParam r = rp[lb];
          const int64_t b = b0 + lb, j = j0 + jj;
          float av[4];
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) {
            const int n = gg * tl.u + jj;
            const ColParam c = cp[n];
            const int32_t sv = S[lb * ldS + n];
            const float yh = recover(sv, c.colterm, c.ztw, r.ztx, r.sigx, c.iqw, r.iqx);
            av[gg] = gxv[q][gg] + yh;
            if (a.acc_h) a.acc_h[(t * B + b) * 4 * H + gg * H + j] = acc_u8(sv, c.sigw, r.sigx, R);
          }
          const float ig = sigmoid_cw(av[0]);
          const float fg = sigmoid_cw(av[1]);
          const float gv = tanh_cw(av[2]);
          const float og = sigmoid_cw(av[3]);
          const float cn = (fg * cst[lb * tl.u + jj]) + (ig * gv);
          cst[lb * tl.u + jj] = cn;
          const float m = og * tanh_cw(cn);
          if (P == 0) {
            a.h[(t * B + b) * R + j] = m;
            if (t == T - 1 && a.hT) a.hT[b * R + j] = m;
          } else {
            mbuf[b * H + j] = m;
          }
          if (t == T - 1 && a.cT) a.cT[b * H + j] = cn;
        }
      }
    }
    if (t == T) break;
    if (P == 0) continue;

    // ---- 6. projection h_t = R(Mult(Q(m_t), W_r'))
    if (grid_sync(ctr, flag, (++nsync) * (unsigned)G)) return;
    if ((int)blockIdx.x < tl.nbt2 * tl.npt) {
      const int tb2 = blockIdx.x / tl.npt, tp = blockIdx.x % tl.npt;
      const int64_t c0 = (int64_t)tb2 * tl.bB2, p0 = (int64_t)tp * tl.p2;
      const int nb2 = (int)(B - c0 < tl.bB2 ? B - c0 : tl.bB2);
      const int np2 = (int)(P - p0 < tl.p2 ? P - p0 : tl.p2);
      const int ldx2 = tl.ldH + 16;
      auto src_m = [&](int lb) -> const float * { return lb < nb2 ? mbuf + (c0 + lb) * H : nullptr; };
      auto done_m = [&](int lb, const RowParam &r, int32_t) {
        if (lane == 0) rp[lb] = r;
      };
      quantize_tile_rows(tl.bB2, (int)H, xc, ldx2, tl.ldH, src_m, done_m);
      __syncthreads();
      // W_r' rows p0 .. p0 + np2 - 1, read from global memory (L2 resident)
      const int8_t *wr = a.Wr.codes + p0 * a.Wr.ld;
      if (tl.mfmaB)
        products_mfma(xc, ldx2, tl.bB2, wr, a.Wr.ld, tl.p2, np2, tl.ldH, S, tl.p2);
      else
        products_valu(xc, ldx2, nb2, wr, a.Wr.ld, tl.p2, np2, tl.ldH, S, tl.p2);
      __syncthreads();
      const int32_t ztw = a.Wr.zero[0] + 128;  // W_r is quantized per matrix
      const float iqw = a.Wr.inv_q[0];
      for (int idx = tid; idx < nb2 * np2; idx += blockDim.x) {
        const int lb = idx / np2, pp = idx % np2;
        const int64_t b = c0 + lb, p = p0 + pp;
        const RowParam r = rp[lb];
        const int32_t sigw = a.Wr.row_sums[p] - 128 * (int32_t)H;
        const int64_t colterm = (int64_t)sigw + H * (int64_t)ztw;
        const int32_t sv = S[lb * tl.p2 + pp];
        const float hv = recover(sv, colterm, ztw, r.ztx, r.sigx, iqw, r.iqx);
        a.h[(t * B + b) * P + p] = hv;
        if (t == T - 1 && a.hT) a.hT[b * P + p] = hv;
        if (a.acc_r) a.acc_r[(t * B + b) * P + p] = acc_u8(sv, sigw, r.sigx, H);
      }
      __syncthreads();
    }
  }
}

// Clears the first `words` 32-bit words of the header: 16 = the barrier
// counter only, 32 = counter and timeout flag.
__global__ void k_zero_header(unsigned *p, int words) {
  if ((int)threadIdx.x < words) p[threadIdx.x] = 0u;
}

hipError_t reset_recurrent_flag(void *ws, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_header, dim3(1), dim3(64), 0, s, static_cast<unsigned *>(ws), 32);
  return hipGetLastError();
}

// ------------------------------------------------------------------ host side
size_t recurrent_ws(int64_t B, int64_t H, int64_t P) {
  return 256 + align_up((size_t)(P > 0 ? B * H : 0) * sizeof(float), 256);
}

static int device_cus(int *lds_max) {
  int dev = 0, cus = 0;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  hipDeviceGetAttribute(lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  return cus;
}

static bool plan(const RecurrentArgs &a, int cus, int lds_max, RecTiling *out) {
  RecTiling tl{};
  const int64_t B = a.B, H = a.H, P = a.P;
  tl.ldR = (int)round_up(a.R, 64);
  tl.ldH = (int)round_up(H, 64);
  tl.ldsW = tl.ldR + 16;
  const int G = cus;
  // phase A tile
  bool ok = false;
  if (B < 16) {
    tl.bB = 1;
    tl.mfmaA = 0;
    tl.nbt = (int)B;
    int nut = G / (int)B;
    if (nut < 1) return false;
    tl.u = (int)((H + nut - 1) / nut);
    tl.nut = (int)((H + tl.u - 1) / tl.u);
    ok = true;
  } else {
    for (int bB = 16; bB <= 256 && !ok; bB *= 2) {
      const int nbt = (int)((B + bB - 1) / bB);
      if (nbt > G) continue;
      const int nut = G / nbt;
      int u = (int)((H + nut - 1) / nut);
      u = (u + 3) / 4 * 4;
      if ((size_t)4 * u * (tl.ldR + 16) > (size_t)lds_max / 2) continue;
      tl.bB = bB;
      tl.nbt = nbt;
      tl.u = u;
      tl.nut = (int)((H + u - 1) / u);
      tl.mfmaA = 1;
      ok = true;
    }
  }
  if (!ok) return false;
  // phase B tile
  if (P > 0) {
    if (B < 16) {
      tl.bB2 = 1;
      tl.mfmaB = 0;
      tl.nbt2 = (int)B;
      const int npt = G / (int)B;
      tl.p2 = (int)((P + npt - 1) / npt);
      tl.p2 = (tl.p2 + 15) / 16 * 16;
      tl.npt = (int)((P + tl.p2 - 1) / tl.p2);
    } else {
      tl.bB2 = 16;
      tl.mfmaB = 1;
      tl.nbt2 = (int)((B + 15) / 16);
      if (tl.nbt2 > G) return false;
      const int npt = G / tl.nbt2;
      tl.p2 = (int)((P + npt - 1) / npt);
      tl.p2 = (tl.p2 + 15) / 16 * 16;
      tl.npt = (int)((P + tl.p2 - 1) / tl.p2);
    }
    // W_r rows read in 16-row groups must stay inside the matrix
    if (a.Wr.ld < tl.ldH) return false;
  }
  tl.grid = tl.nbt * tl.nut;
  if (P > 0 && tl.nbt2 * tl.npt > tl.grid) tl.grid = tl.nbt2 * tl.npt;
  if (tl.grid > G) return false;
  // LDS layout
  const int nrows = 4 * tl.u;
  tl.ldsX = tl.ldR + 16;
  size_t xbytes = (size_t)tl.bB * tl.ldsX;
  if (P > 0) {
    const size_t xb2 = (size_t)tl.bB2 * (tl.ldH + 16);
    xbytes = xbytes > xb2 ? xbytes : xb2;
  }
  size_t sbytes = (size_t)tl.bB * nrows * 4;
  if (P > 0) {
    const size_t sb2 = (size_t)tl.bB2 * tl.p2 * 4;
    sbytes = sbytes > sb2 ? sbytes : sb2;
  }
  size_t off = 0;
  tl.off_w = off;
  off = align_up(off + (size_t)nrows * tl.ldsW, 16);
  tl.off_x = off;
  off = align_up(off + xbytes, 16);
  tl.off_s = off;
  off = align_up(off + sbytes, 16);
  tl.off_c = off;
  off = align_up(off + (size_t)tl.bB * tl.u * 4, 16);
  tl.off_col = off;
  off = align_up(off + (size_t)nrows * sizeof(ColParam), 16);
  const int rows_rp = tl.bB > tl.bB2 ? tl.bB : tl.bB2;
  tl.off_row = off;
  off = align_up(off + (size_t)rows_rp * sizeof(RowParam), 16);
  tl.lds_bytes = off;
  if (tl.lds_bytes + 64 > (size_t)lds_max) return false;  // + static shared (barrier flag)
  // the per-thread gx prefetch holds up to 8 (b, j) pairs
  if ((tl.bB * tl.u + 255) / 256 > 8) return false;
  *out = tl;
  return true;
}

hipError_t launch_recurrent(const RecurrentArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0 || a.B == 0) return hipSuccess;
  int lds_max = 0;
  const int cus = device_cus(&lds_max);
  RecTiling tl;
  if (!plan(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_recurrent),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_recurrent, 256, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  hipLaunchKernelGGL(k_zero_header, dim3(1), dim3(64), 0, s, static_cast<unsigned *>(a.ws), 16);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  RecurrentArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(k_recurrent), dim3(tl.grid),
                                    dim3(256), kargs, (unsigned)tl.lds_bytes, s);
}

hipError_t recurrent_timed_out(const void *ws, hipStream_t s, bool *timed_out) {
  int flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, static_cast<const char *>(ws) + 64, sizeof(int),
                                hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  *timed_out = flag != 0;
  return e;
}

}  // namespace ql
