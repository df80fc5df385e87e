// ql_device.h -- device-side building blocks shared by the gfx950 kernels.
//
// The arithmetic here follows the numerical conventions stated in
// include/qlstm.h.  Every float operation is an IEEE fp32/fp64 + - * / or,
// where written out (the reduction and polynomial of e^x), a fused
// multiply-add; nothing is contracted implicitly (the library is compiled
// with -ffp-contract=off, and the pragma below pins it for this header), so
// the gate functions give the same bits as any other IEEE implementation of
// the same formulas.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace ql {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr double kScale = 255.0;  // S, the 8-bit scale (Section 3)
constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// e^x: Cody & Waite ("Software Manual for the Elementary Functions", 1980)
// range reduction x = n ln2 + r with ln2 split into a 15-bit head (so n * head
// is exact for |n| <= 127) and a tail; e^r by the Taylor series of exp to
// degree 7 in Horner form, each step of the reduction and of Horner's scheme
// one fused multiply-add; the result scaled by 2^n through its exponent
// field.  x is clamped to [-87, 87] so results and 1 / (1 + e^x) are normal.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float exp_cw(float x_in) {
  // the clamp as one median-of-three; a NaN input is passed through by the
  // select at the end (no branch)
  const float x = __builtin_amdgcn_fmed3f(x_in, -87.0f, 87.0f);
  const float n = floorf(__builtin_fmaf(x, 1.44269504088896340736f, 0.5f));
  float r = __builtin_fmaf(-n, 0.693145751953125f, x);
  r = __builtin_fmaf(-n, 1.42860682030941723212e-6f, r);
  float p = 1.0f / 5040.0f;
  p = __builtin_fmaf(p, r, 1.0f / 720.0f);
  p = __builtin_fmaf(p, r, 1.0f / 120.0f);
  p = __builtin_fmaf(p, r, 1.0f / 24.0f);
  p = __builtin_fmaf(p, r, 1.0f / 6.0f);
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  const float scale = __int_as_float(((int)n + 127) << 23);
  return x_in != x_in ? x_in : p * scale;
}
// 1 / d for d in [1, 2^126) (every denominator 1 + e^-x of the gate
// functions), correctly rounded: v_rcp_f32 refined by two Newton steps whose
// residual and update are each one fused multiply-add (Markstein's reciprocal,
// IBM J. Res. Dev. 34(1), 1990).  Equal bit for bit to IEEE division 1.0f / d
// (checked over every float in [1, 6.1e37]), in 5 instructions instead of the
// 11 of the general division sequence.
__device__ __forceinline__ float recip_ge1(float d) {
  float r = __builtin_amdgcn_rcpf(d);
  float e = __builtin_fmaf(-d, r, 1.0f);
  r = __builtin_fmaf(e, r, r);
  e = __builtin_fmaf(-d, r, 1.0f);
  return __builtin_fmaf(e, r, r);
}
__device__ __forceinline__ float sigmoid_cw(float x) { return recip_ge1(1.0f + exp_cw(-x)); }
__device__ __forceinline__ float tanh_cw(float x) { return 2.0f * sigmoid_cw(2.0f * x) - 1.0f; }

// ---------------------------------------------------------------------------
// Quantizer of Section 3 with the rounding of eq. 2.
// ---------------------------------------------------------------------------
// round(): half up.  floor is exact and the tie test x - floor(x) >= 0.5 is
// decided exactly for every double.
__device__ __forceinline__ double round_half_up(double x) {
  double r = floor(x);
  return (x - r >= 0.5) ? r + 1.0 : r;
}

struct QParams {
  double q;     // Q = S / R (1 for an all-zero set)
  int32_t z;    // round(Q Vmin)
  float inv_q;  // (float)(R / S)
  double range; // R
};

// Range rule: R = Vmax - Vmin in fp64; a zero range, or one so narrow that
// Q max|V| would exceed 2^24, is widened to include 0.
__device__ __forceinline__ QParams make_qparams(float vmin_f, float vmax_f) {
  double lo = (double)vmin_f, hi = (double)vmax_f;
  double R = hi - lo;
  const double alo = lo < 0.0 ? -lo : lo, ahi = hi < 0.0 ? -hi : hi;
  const double amax = alo > ahi ? alo : ahi;
  if (R == 0.0 || kScale * amax > 16777216.0 * R) {
    if (lo > 0.0) lo = 0.0;
    if (hi < 0.0) hi = 0.0;
    R = hi - lo;
  }
  QParams p;
  p.range = R;
  if (R == 0.0) {
    p.q = 1.0;
    p.z = 0;
    p.inv_q = 1.0f;
  } else {
    p.q = kScale / R;
    p.z = (int32_t)round_half_up(p.q * lo);
    p.inv_q = (float)(R / kScale);
  }
  return p;
}

// eq. 2: V' = round(Q V) - round(Q Vmin), kept in [0, 255].  round() is
// floor(x) + (x - floor(x) >= 0.5); floor(x) is integral with |x| <= 2^24
// (the range rule bounds Q max|V|), so its int conversion is exact.
__device__ __forceinline__ int encode(float v, double q, int32_t z) {
  const double x = q * (double)v;
  const double r = floor(x);
  int c = (int)r - z + ((x - r) >= 0.5 ? 1 : 0);
  c = c < 0 ? 0 : c;
  return c > 255 ? 255 : c;
}

// Pack four codes (0..255) into the device layout (V' - 128 per byte).
__device__ __forceinline__ uint32_t pack4_s8(int c0, int c1, int c2, int c3) {
  return ((uint32_t)(c0 ^ 0x80) & 0xffu) | (((uint32_t)(c1 ^ 0x80) & 0xffu) << 8) |
         (((uint32_t)(c2 ^ 0x80) & 0xffu) << 16) | (((uint32_t)(c3 ^ 0x80) & 0xffu) << 24);
}

// ---------------------------------------------------------------------------
// Recovery of eq. 1 / eq. 3.  With device codes s = V' - 128, shifted zero
// points zt = z + 128 and signed sums sig = sum s, the numerator of eq. 1 is
//   T = sum_k (sw + ztw)(sx + ztx) = S + ztx * sigw + ztw * sigx + K ztw ztx
// where S = sum_k sw sx is what the signed 8-bit MFMA/dot products return.
// ---------------------------------------------------------------------------
// Low 32 bits of the product of two signed 24-bit values (v_mul_i32_i24,
// full rate; a 32-bit v_mul_lo_u32 runs at a quarter of it).  Written out
// because the compiler, having proved the range, would fold the 24-bit
// extension of __mul24 away and fall back to the 32-bit multiply.
__device__ __forceinline__ int32_t mul_i24(int32_t a, int32_t b) {
  int32_t r;
  asm("v_mul_i32_i24 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// T in 32 bits with 24-bit multiplies; only valid where recover() below
// takes its fast path (both shifted zero points in [-127, 128] and
// |colterm| < 2^23): callers check that once for a whole tile.
__device__ __forceinline__ float recover_fast(int32_t S, int32_t colterm, int32_t ztw, int32_t ztx,
                                              int32_t sigx, float iqw, float iqx) {
  const uint32_t t = (uint32_t)S + (uint32_t)mul_i24(ztx, colterm) + (uint32_t)mul_i24(ztw, sigx);
  return ((float)(int32_t)t * iqw) * iqx;
}
// The fast-path condition for one row (ztx) or one column (ztw, colterm).
__device__ __forceinline__ bool fast_row(int32_t ztx) { return (uint32_t)(ztx + 127) <= 255u; }
__device__ __forceinline__ bool fast_col(int32_t ztw, int64_t colterm) {
  return (uint32_t)(ztw + 127) <= 255u && (uint64_t)(colterm + (1 << 23)) < (uint64_t)(1 << 24);
}

__device__ __forceinline__ float recover(int32_t S, int64_t colterm /* sigw + K ztw */,
                                         int32_t ztw, int32_t ztx, int32_t sigx,
                                         float iqw, float iqx) {
  // When both zero points lie in [-255, 0] (every set whose range contains 0),
  // V'' = V' + z lies in [-255, 255], so |T| <= K * 255^2 < 2^31 for K <= 33025
  // and the wrapping 32-bit evaluation is T exactly (z~ = z + 128 in [-127, 128]).
  // Every factor then fits 24 signed bits (|sigx| <= 128 K; colterm is checked,
  // it does for K < 32768), so the full-rate 24-bit multiplies, which return
  // the low 32 bits of the exact product, serve.
  if ((uint32_t)(ztx + 127) <= 255u && (uint32_t)(ztw + 127) <= 255u &&
      (uint64_t)(colterm + (1 << 23)) < (uint64_t)(1 << 24)) {
    const uint32_t t = (uint32_t)S + (uint32_t)mul_i24(ztx, (int32_t)colterm) +
                       (uint32_t)mul_i24(ztw, sigx);
    return ((float)(int32_t)t * iqw) * iqx;
  }
  const int64_t t = (int64_t)S + (int64_t)ztx * colterm + (int64_t)ztw * (int64_t)sigx;
  return ((float)t * iqw) * iqx;
}
// Raw 0..255-domain accumulator sum_k V'w V'x from the signed one.
__device__ __forceinline__ int32_t acc_u8(int32_t S, int32_t sigw, int32_t sigx, int64_t K) {
  return (int32_t)((int64_t)S + 128 * (int64_t)sigw + 128 * (int64_t)sigx + 16384 * K);
}

// ---------------------------------------------------------------------------
// Wavefront (64-lane) reductions with DPP: shifts within 16-lane rows, then
// row broadcasts; the result is read from lane 63 and is the same in every
// lane.  min/max are exact in any order, integer sums too.
// ---------------------------------------------------------------------------
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_i(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWS, 0xf, false);
}
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;

template <class Op>
__device__ __forceinline__ int wave_reduce_i(int v, int identity, Op op) {
  v = op(v, dpp_i<kRowShr1, 0xf>(identity, v));
  v = op(v, dpp_i<kRowShr2, 0xf>(identity, v));
  v = op(v, dpp_i<kRowShr4, 0xf>(identity, v));
  v = op(v, dpp_i<kRowShr8, 0xf>(identity, v));
  v = op(v, dpp_i<kRowBcast15, 0xa>(v, v));
  v = op(v, dpp_i<kRowBcast31, 0xc>(v, v));
  return __builtin_amdgcn_readlane(v, 63);
}
// N independent reductions at once: each DPP step is applied to all N values
// before the next, so their latencies overlap.
template <int N, class Op>
__device__ __forceinline__ void wave_reduce_n(int (&v)[N], int identity, Op op) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowShr1, 0xf>(identity, v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowShr2, 0xf>(identity, v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowShr4, 0xf>(identity, v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowShr8, 0xf>(identity, v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowBcast15, 0xa>(v[i], v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = op(v[i], dpp_i<kRowBcast31, 0xc>(v[i], v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = __builtin_amdgcn_readlane(v[i], 63);
}
// All-lane reductions built from rotations inside 16-lane rows (every lane
// has a valid source, so the compiler folds the DPP into the min/add itself),
// then the four row results combined from lanes 0, 16, 32, 48.  N
// independent values step together so their latencies overlap.
template <int N>
__device__ __forceinline__ void wave_min_n(int (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = min(v[i], __builtin_amdgcn_update_dpp(0, v[i], 0x121, 0xf, 0xf, false));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = min(v[i], __builtin_amdgcn_update_dpp(0, v[i], 0x122, 0xf, 0xf, false));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = min(v[i], __builtin_amdgcn_update_dpp(0, v[i], 0x124, 0xf, 0xf, false));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = min(v[i], __builtin_amdgcn_update_dpp(0, v[i], 0x128, 0xf, 0xf, false));
#pragma unroll
  for (int i = 0; i < N; ++i)
    v[i] = min(min(__builtin_amdgcn_readlane(v[i], 0), __builtin_amdgcn_readlane(v[i], 16)),
               min(__builtin_amdgcn_readlane(v[i], 32), __builtin_amdgcn_readlane(v[i], 48)));
}
template <int N>
__device__ __forceinline__ void wave_add_n(int (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += __builtin_amdgcn_update_dpp(0, v[i], 0x121, 0xf, 0xf, false);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += __builtin_amdgcn_update_dpp(0, v[i], 0x122, 0xf, 0xf, false);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += __builtin_amdgcn_update_dpp(0, v[i], 0x124, 0xf, 0xf, false);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] += __builtin_amdgcn_update_dpp(0, v[i], 0x128, 0xf, 0xf, false);
#pragma unroll
  for (int i = 0; i < N; ++i)
    v[i] = (__builtin_amdgcn_readlane(v[i], 0) + __builtin_amdgcn_readlane(v[i], 16)) +
           (__builtin_amdgcn_readlane(v[i], 32) + __builtin_amdgcn_readlane(v[i], 48));
}
// The value lane (lane & ~3) + K of this lane's group of four holds
// (DPP quad_perm broadcast; all four lanes of the group must be active).
template <int K>
__device__ __forceinline__ float quad_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), K * 0x55, 0xf, 0xf, false));
}

// Order-preserving map of a (non-NaN) float to int and back.
__device__ __forceinline__ int float_key(float f) {
  const int u = __float_as_int(f);
  return u ^ ((u >> 31) & 0x7fffffff);
}
__device__ __forceinline__ float key_float(int k) { return __int_as_float(k ^ ((k >> 31) & 0x7fffffff)); }

struct OpMinF {
  __device__ int operator()(int a, int b) const {
    return __float_as_int(fminf(__int_as_float(a), __int_as_float(b)));
  }
};
struct OpMaxF {
  __device__ int operator()(int a, int b) const {
    return __float_as_int(fmaxf(__int_as_float(a), __int_as_float(b)));
  }
};
struct OpAddI {
  __device__ int operator()(int a, int b) const { return a + b; }
};

__device__ __forceinline__ float wave_min(float v) {
  return __int_as_float(wave_reduce_i(__float_as_int(v), __float_as_int(INFINITY), [](int a, int b) {
    return __float_as_int(fminf(__int_as_float(a), __int_as_float(b)));
  }));
}
__device__ __forceinline__ float wave_max(float v) {
  return __int_as_float(wave_reduce_i(__float_as_int(v), __float_as_int(-INFINITY), [](int a, int b) {
    return __float_as_int(fmaxf(__int_as_float(a), __int_as_float(b)));
  }));
}
__device__ __forceinline__ int wave_sum(int v) {
  return wave_reduce_i(v, 0, [](int a, int b) { return a + b; });
}

}  // namespace ql
