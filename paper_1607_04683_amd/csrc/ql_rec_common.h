// ql_rec_common.h -- pieces shared by the persistent recurrent kernels:
// per-vector quantization of activation rows into LDS (eq. 2) and the signed
// 8-bit products against LDS-resident weight slices.
#pragma once
#include "ql_device.h"
#include "ql_exchange.h"

namespace ql {

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
  int32_t sum;      // code sum (0..255 domain)
  int32_t pad[3];
};
// Row params of a row of codes (zero point z, recovery factor iq, code sum
// over K elements) as the products need them.
__device__ __forceinline__ RowParam row_param(int32_t z, float iq, int32_t sum, int K) {
  RowParam q;
  q.z = z;
  q.ztx = z + 128;
  q.sigx = sum - 128 * K;
  q.iqx = iq;
  q.sum = sum;
  q.pad[0] = q.pad[1] = q.pad[2] = 0;
  return q;
}

// ---------------------------------------------------------------------------
// Per-vector quantization (eq. 2) of RB consecutive rows by one wave.
// Rows [0, nvalid) are read from `src` (row stride `stride` elements): as
// published words carrying `tag` (kSrcTagged: re-read until every tag
// matches), as floats through device-coherent loads (kSrcCoherent: their
// availability was already established), or as plain floats (kSrcPlain;
// src null = zeros).  Rows [nvalid, ntotal) are zero vectors.  Lane l holds
// the 4-element chunks starting at k = 4 (c*64 + l), c < NV/4, so all of a
// group's loads are in flight together and four codes pack into one LDS
// word; min/max, params, codes and the code sum come from registers.  Codes
// go to dst + r*ldx (ldpad bytes, ldpad a multiple of 4), row params to
// rp[r].  Returns false if the wait expired.
// ---------------------------------------------------------------------------
enum { kSrcPlain = 0, kSrcTagged = 1, kSrcCoherent = 2 };

template <int NV, int RB, int MODE>
__device__ __forceinline__ bool quant_rows(const void *src, int64_t stride, int nvalid,
                                           int ntotal, uint32_t tag, int K, int8_t *dst,
                                           int ldx, int ldpad, int *flag, RowParam *rp) {
  constexpr int NC = NV / 4;
  const int lane = threadIdx.x & 63;
  float v[RB][NV];
  if (MODE == kSrcTagged) {
    // a word is re-read only until its tag has matched once (bit r*NV + i
    // of `got`), so later polls touch only what is still missing
    static_assert(RB * NV <= 32, "one bit per value of the lane");
    const uint64_t *base = static_cast<const uint64_t *>(src);
    uint32_t got = 0;
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int i = 0; i < NV; ++i) v[r][i] = 0.0f;
    long it = 0;
    for (;;) {
      uint32_t bad = 0;
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int k = 4 * (c * kWave + lane) + e;
            const uint32_t bit = 1u << (r * NV + 4 * c + e);
            if (r < nvalid && k < K && !(got & bit)) {
              const uint64_t w = ld_tagged(base + r * stride + k);
              if ((uint32_t)(w >> 32) == tag) {
                got |= bit;
                v[r][4 * c + e] = __uint_as_float((uint32_t)w);
              } else {
                bad = 1;
              }
            }
          }
      if (!__any(bad != 0)) break;
      if (wait_expired(flag, it)) return false;
    }
  } else {
    const float *base = static_cast<const float *>(src);
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = 4 * (c * kWave + lane) + e;
          float x = 0.0f;
          if (base && r < nvalid && k < K)
            x = MODE == kSrcCoherent ? ld_coherent(base + r * stride + k) : base[r * stride + k];
          v[r][4 * c + e] = x;
        }
  }
  // order-preserving keys: min over keys, max as ~min(~key); 2*RB reductions together
  int mm[2 * RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    int lo = 0x7fffffff, hi = 0x7fffffff;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = 4 * (c * kWave + lane) + e < K;
        const int key = float_key(v[r][4 * c + e]);
        lo = ok ? min(lo, key) : lo;
        hi = ok ? min(hi, ~key) : hi;
      }
    mm[r] = lo;
    mm[RB + r] = hi;
  }
  wave_min_n<2 * RB>(mm);
  int sums[RB];
  QParams prm[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    float lo = key_float(mm[r]), hi = key_float(~mm[RB + r]);
    if (r >= nvalid || !src || K == 0) lo = hi = 0.0f;
    prm[r] = make_qparams(lo, hi);
    int sum = 0;
    uint32_t *d = reinterpret_cast<uint32_t *>(dst + r * ldx);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int k0 = 4 * (c * kWave + lane);
      uint32_t word = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = k0 + e < K;
        const int code = encode(v[r][4 * c + e], prm[r].q, prm[r].z);
        sum += ok ? code : 0;
        word |= (ok ? (uint32_t)((code ^ 0x80) & 0xff) : 0u) << (8 * e);
      }
      if (r < ntotal && k0 < ldpad) d[k0 / 4] = word;
    }
    if (r < ntotal)
      for (int k0 = 4 * (NC * kWave + lane); k0 < ldpad; k0 += 4 * kWave) d[k0 / 4] = 0u;
    sums[r] = sum;
  }
  wave_add_n<RB>(sums);
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      if (r >= ntotal) break;
      RowParam q;
      q.z = prm[r].z;
      q.ztx = prm[r].z + 128;
      q.sigx = sums[r] - 128 * K;
      q.iqx = prm[r].inv_q;
      q.sum = sums[r];
      rp[r] = q;
    }
  }
  return true;
}

// All rows [0, ntotal) of a tile, RB-row groups handed round-robin to waves;
// rows [0, nvalid) are real.  row_src(lb) gives the source of row lb.
template <int NV, int RB, int MODE, class RowSrcFn>
__device__ __forceinline__ bool quant_tile(int nvalid, int ntotal, int64_t stride, uint32_t tag,
                                           int K, int8_t *dst, int ldx, int ldpad, int *flag,
                                           RowParam *rp, RowSrcFn row_src) {
  const int wave = threadIdx.x >> 6, nwave = blockDim.x >> 6;
  for (int lb0 = wave * RB; lb0 < ntotal; lb0 += nwave * RB) {
    const int nv = nvalid - lb0 < 0 ? 0 : (nvalid - lb0 < RB ? nvalid - lb0 : RB);
    const int nt = ntotal - lb0 < RB ? ntotal - lb0 : RB;
    if (!quant_rows<NV, RB, MODE>(row_src(lb0), stride, nv, nt, tag, K, dst + lb0 * ldx, ldx,
                                    ldpad, flag, rp + lb0))
      return false;
  }
  return true;
}

// One row of K <= 512 published values (tagged words of step tag `tag`)
// quantized per vector (eq. 2) by waves w0 and w0 + 1 together: wave w polls
// and encodes half w of the row (lane l: elements 4 (w*64 + l) .. +3), and the
// halves' min/max, then their code sums, meet in LDS slots xch[w*8 ..] (data,
// then a flag holding the tag, released after the data).  The codes go to
// dst (ldpad <= 512 bytes), the row params to *rp.  False if a wait expired.
__device__ __forceinline__ bool quant_row_2w(const uint64_t *src, uint32_t tag, int K,
                                             int8_t *dst, int ldpad, int *flag, RowParam *rp,
                                             int *xch, int w0 = 0) {
  const int lane = threadIdx.x & 63, w = (int)(threadIdx.x >> 6) - w0, o = 1 - w;
  const int kb = 4 * (w * kWave + lane);
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  uint32_t got = 0;
  long it = 0;
  for (;;) {
    uint32_t bad = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (kb + e < K && !(got & (1u << e))) {
        const uint64_t wd = ld_tagged(src + kb + e);
        if ((uint32_t)(wd >> 32) == tag) {
          got |= 1u << e;
          v[e] = __uint_as_float((uint32_t)wd);
        } else {
          bad = 1;
        }
      }
    if (!__any(bad != 0)) break;
    if (wait_expired(flag, it)) return false;
  }
  int mm[2] = {0x7fffffff, 0x7fffffff};
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (kb + e < K) {
      const int key = float_key(v[e]);
      mm[0] = min(mm[0], key);
      mm[1] = min(mm[1], ~key);
    }
  wave_min_n<2>(mm);
  if (lane == 0) {
    xch[w * 8 + 0] = mm[0];
    xch[w * 8 + 1] = mm[1];
    __hip_atomic_store(&xch[w * 8 + 2], (int)tag, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  it = 0;
  while (__hip_atomic_load(&xch[o * 8 + 2], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != (int)tag)
    if (wait_expired(flag, it)) return false;
  const int lo = min(mm[0], xch[o * 8 + 0]), hi = min(mm[1], xch[o * 8 + 1]);
  const QParams prm = make_qparams(key_float(lo), key_float(~hi));
  int sum = 0;
  uint32_t word = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ok = kb + e < K;
    const int code = encode(v[e], prm.q, prm.z);
    sum += ok ? code : 0;
    word |= (ok ? (uint32_t)((code ^ 0x80) & 0xff) : 0u) << (8 * e);
  }
  if (kb < ldpad) reinterpret_cast<uint32_t *>(dst)[kb / 4] = word;
  int s1[1] = {sum};
  wave_add_n<1>(s1);
  if (w == 1) {
    if (lane == 0) {
      xch[8 + 3] = s1[0];
      __hip_atomic_store(&xch[8 + 4], (int)tag, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    return true;
  }
  it = 0;
  while (__hip_atomic_load(&xch[8 + 4], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != (int)tag)
    if (wait_expired(flag, it)) return false;
  if (lane == 0) *rp = row_param(prm.z, prm.inv_q, s1[0] + xch[8 + 3], K);
  return true;
}

// ---------------------------------------------------------------------------
// Products S[lb][n] = sum_k x[lb][k] w[n][k] over K bytes (a multiple of 64).
// ---------------------------------------------------------------------------
// VALU: groups of 16 lanes per (row, n) task, v_dot4 on 16-byte chunks.
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
    if (K == 512) {
      // two 16-byte chunks per lane, both loaded first
      const v4i a0 = *reinterpret_cast<const v4i *>(xr + gl * 16);
      const v4i b0 = *reinterpret_cast<const v4i *>(wr + gl * 16);
      const v4i a1 = *reinterpret_cast<const v4i *>(xr + gl * 16 + 256);
      const v4i b1 = *reinterpret_cast<const v4i *>(wr + gl * 16 + 256);
      acc = __builtin_amdgcn_sdot4(a0.x, b0.x, acc, false);
      acc = __builtin_amdgcn_sdot4(a0.y, b0.y, acc, false);
      acc = __builtin_amdgcn_sdot4(a0.z, b0.z, acc, false);
      acc = __builtin_amdgcn_sdot4(a0.w, b0.w, acc, false);
      acc = __builtin_amdgcn_sdot4(a1.x, b1.x, acc, false);
      acc = __builtin_amdgcn_sdot4(a1.y, b1.y, acc, false);
      acc = __builtin_amdgcn_sdot4(a1.z, b1.z, acc, false);
      acc = __builtin_amdgcn_sdot4(a1.w, b1.w, acc, false);
    } else {
      for (int k = gl * 16; k < K; k += 16 * 16) {
        const v4i a = *reinterpret_cast<const v4i *>(xr + k);
        const v4i b = *reinterpret_cast<const v4i *>(wr + k);
        acc = __builtin_amdgcn_sdot4(a.x, b.x, acc, false);
        acc = __builtin_amdgcn_sdot4(a.y, b.y, acc, false);
        acc = __builtin_amdgcn_sdot4(a.z, b.z, acc, false);
        acc = __builtin_amdgcn_sdot4(a.w, b.w, acc, false);
      }
    }
    // sum over the group's 16 lanes (one DPP row): rotations by 1, 2, 4, 8
    acc += __builtin_amdgcn_update_dpp(0, acc, 0x121, 0xf, 0xf, false);
    acc += __builtin_amdgcn_update_dpp(0, acc, 0x122, 0xf, 0xf, false);
    acc += __builtin_amdgcn_update_dpp(0, acc, 0x124, 0xf, 0xf, false);
    acc += __builtin_amdgcn_update_dpp(0, acc, 0x128, 0xf, 0xf, false);
    if (gl == 0) S[lb * ldS + n] = acc;
  }
}

// MFMA: nb (multiple of 16) rows x nrows (multiple of 16) outputs.
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
    if (K % 512 == 0) {
      // whole 512-byte blocks of K: each block's fragments are loaded before its MFMAs
      for (int k0 = 0; k0 < K; k0 += 512) {
        v4i a[8], b[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          a[c] = *reinterpret_cast<const v4i *>(xr + k0 + c * 64);
          b[c] = *reinterpret_cast<const v4i *>(wr + k0 + c * 64);
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[c], b[c], acc, 0, 0, 0);
      }
    } else {
      for (int k = 0; k < K; k += 64) {
        const v4i a = *reinterpret_cast<const v4i *>(xr + k);
        const v4i b = *reinterpret_cast<const v4i *>(wr + k);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc, 0, 0, 0);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      S[(ti * 16 + (lane >> 4) * 4 + r) * ldS + tj * 16 + (lane & 15)] = acc[r];
  }
}

// Fragments of 16-row block `blk` of a weight slice in LDS (rows of ldw
// bytes, K codes) as the B operand of v_mfma_i32_16x16x64_i8: lane l holds row
// l % 16, bytes 16 (l / 16) .. +15 of every 64-byte chunk of K; chunks past K
// are zero.  Loaded once and kept in registers across a launch.
__device__ __forceinline__ void load_wfrag(v4i (&b)[8], const int8_t *w, int ldw, int blk, int K) {
  const int lane = threadIdx.x & 63;
  const int8_t *wr = w + (blk * 16 + (lane & 15)) * ldw + (lane >> 4) * 16;
#pragma unroll
  for (int c = 0; c < 8; ++c)
    b[c] = c * 64 < K ? *reinterpret_cast<const v4i *>(wr + c * 64) : v4i{};
}

// The products of every 16-row block of x (nb rows, a multiple of 16, in LDS)
// against the register fragments b of weight block blk (K <= 512 codes):
// S[row][blk * 16 + col].  One wave; two row blocks go through the MFMA
// pipeline side by side.
__device__ __forceinline__ void products_mfma_reg(const int8_t *x, int ldx, int nb,
                                                  const v4i (&b)[8], int blk, int K, int32_t *S,
                                                  int ldS) {
  const int lane = threadIdx.x & 63;
  const int mt = nb / 16;
  auto put = [&](int ti, const v4i &acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      S[(ti * 16 + (lane >> 4) * 4 + r) * ldS + blk * 16 + (lane & 15)] = acc[r];
  };
  int ti = 0;
  for (; ti + 1 < mt; ti += 2) {
    const int8_t *x0 = x + (ti * 16 + (lane & 15)) * ldx + (lane >> 4) * 16;
    const int8_t *x1 = x0 + 16 * ldx;
    v4i acc0 = v4i{}, acc1 = v4i{};
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (c * 64 < K) {
        const v4i a0 = *reinterpret_cast<const v4i *>(x0 + c * 64);
        const v4i a1 = *reinterpret_cast<const v4i *>(x1 + c * 64);
        acc0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0, b[c], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1, b[c], acc1, 0, 0, 0);
      }
    put(ti, acc0);
    put(ti + 1, acc1);
  }
  if (ti < mt) {
    const int8_t *x0 = x + (ti * 16 + (lane & 15)) * ldx + (lane >> 4) * 16;
    v4i acc = v4i{};
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (c * 64 < K)
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(*reinterpret_cast<const v4i *>(x0 + c * 64),
                                                   b[c], acc, 0, 0, 0);
    put(ti, acc);
  }
}

}  // namespace ql
