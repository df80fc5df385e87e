// ql_quantize.hip -- the quantizer of Section 3 / eq. 2 on gfx950.
//
//  * k_quantize_rows: the on-the-fly activation quantizer (Section 3.1: inputs
//    are quantized on the fly).  One wavefront per vector: fused min/max
//    wavefront reduction -> (R, Q, round(Q Vmin), Q^-1) -> packed codes and the
//    code sum, in one pass over HBM (4 bytes read + 1 byte written per value).
//  * k_quantize_stacked: the same quantizer reading the network's input straight
//    from the frontend's base frames (Section 4: 8 consecutive frames stacked,
//    every third stacked frame presented), so the stacked copy is never written.
//  * k_set_*: quantization of larger sets (a weight matrix or one of its gate
//    blocks; a whole activation tensor): partial min/max over many blocks,
//    a finalize step, then the row encoder.
//  * k_dequantize: recovery of eq. 3.
#include "ql_device.h"
#include "ql_launch.h"

namespace ql {

// Row accessors of the on-the-fly quantizer: value i of one input vector.
// A row of a dense [m][ldx] matrix.
struct DenseRow {
  const float *x;
  __device__ bool vec4(int64_t K) const { return (K & 3) == 0 && (((uintptr_t)x) & 15) == 0; }
  __device__ float4 load4(int64_t q) const { return reinterpret_cast<const float4 *>(x)[q]; }
  __device__ float load1(int64_t i) const { return x[i]; }
};
// One presented input of the frontend (Section 4): `stack` consecutive base
// frames of one utterance, `dim` values each, laid end to end.  f points at the
// first of them; consecutive base frames of the utterance lie `fstride` floats
// apart (B * dim in a time-major [frames][B][dim] array).  K = stack * dim < 2^31.
struct StackedRow {
  const float *f;
  int dim;
  int64_t fstride;
  __device__ bool vec4(int64_t) const {
    return (dim & 3) == 0 && (fstride & 3) == 0 && (((uintptr_t)f) & 15) == 0;
  }
  __device__ float4 load4(int64_t q) const {  // dim % 4 == 0: a float4 never straddles frames
    const int i = 4 * (int)q, j = i / dim;
    return *reinterpret_cast<const float4 *>(f + j * fstride + (i - j * dim));
  }
  __device__ float load1(int64_t i) const {
    const int j = (int)i / dim;
    return f[j * fstride + ((int)i - j * dim)];
  }
};

// min and max of the K values of row x, reduced over the wave (every lane).
template <class Row>
__device__ __forceinline__ float2 row_minmax_wave(const Row &x, int64_t K, int lane) {
  float lo = INFINITY, hi = -INFINITY;
  if (x.vec4(K)) {
    for (int64_t i = lane; i < K / 4; i += kWave) {
      const float4 v = x.load4(i);
      lo = fminf(fminf(lo, v.x), fminf(v.y, fminf(v.z, v.w)));
      hi = fmaxf(fmaxf(hi, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
    }
  } else {
    for (int64_t i = lane; i < K; i += kWave) {
      const float v = x.load1(i);
      lo = fminf(lo, v);
      hi = fmaxf(hi, v);
    }
  }
  return make_float2(wave_min(lo), wave_max(hi));
}

// Encode the K values of row x with params (q, z) into out[0, ld);
// returns the code sum (0..255 domain) in every lane of the wave.
template <class Row>
__device__ __forceinline__ int encode_row_wave(const Row &x, int64_t K, int8_t *__restrict__ out,
                                               int64_t ld, double q, int32_t z, int lane) {
  int sum = 0;
  if (x.vec4(K)) {
    uint32_t *o4 = reinterpret_cast<uint32_t *>(out);
    for (int64_t i = lane; i < K / 4; i += kWave) {
      const float4 v = x.load4(i);
      const int c0 = encode(v.x, q, z), c1 = encode(v.y, q, z), c2 = encode(v.z, q, z),
                c3 = encode(v.w, q, z);
      sum += c0 + c1 + c2 + c3;
      o4[i] = pack4_s8(c0, c1, c2, c3);
    }
  } else {
    for (int64_t i = lane; i < K; i += kWave) {
      const int c = encode(x.load1(i), q, z);
      sum += c;
      out[i] = (int8_t)(c ^ 0x80);
    }
  }
  // zero padding [K, ld) in the signed layout (V' - 128 = 0 contributes 0)
  for (int64_t i = K + lane; i < ld; i += kWave) out[i] = 0;
  return wave_sum(sum);
}

// One wave quantizes one vector: min/max, params, codes, code sum.
template <class Row>
__device__ __forceinline__ void quantize_row_wave(const Row &x, int64_t K, int64_t row,
                                                  int8_t *__restrict__ codes, int64_t ld,
                                                  int32_t *__restrict__ zero,
                                                  float *__restrict__ inv_q,
                                                  int32_t *__restrict__ sums, int lane) {
  float2 mm = row_minmax_wave(x, K, lane);
  if (K == 0) mm = make_float2(0.0f, 0.0f);
  const QParams p = make_qparams(mm.x, mm.y);
  const int s = encode_row_wave(x, K, codes + row * ld, ld, p.q, p.z, lane);
  if (lane == 0) {
    if (zero) zero[row] = p.z;
    if (inv_q) inv_q[row] = p.inv_q;
    if (sums) sums[row] = s;
  }
}

__global__ __launch_bounds__(256) void k_quantize_rows(const float *__restrict__ X, int64_t ldx,
                                                       int64_t m, int64_t K,
                                                       int8_t *__restrict__ codes, int64_t ld,
                                                       int32_t *__restrict__ zero,
                                                       float *__restrict__ inv_q,
                                                       int32_t *__restrict__ sums) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x >> 6);
  if (row >= m) return;
  quantize_row_wave(DenseRow{X + row * ldx}, K, row, codes, ld, zero, inv_q, sums, lane);
}

// Frontend fused into the input quantizer: presented input t of utterance b
// (row t * B + b of the output) is base frames skip*t .. skip*t + stack - 1 of
// that utterance, frames [nframes][B][dim]; the caller guarantees
// skip * (T - 1) + stack <= nframes.
__global__ __launch_bounds__(256) void k_quantize_stacked(const float *__restrict__ frames,
                                                          int64_t B, int dim, int stack,
                                                          int skip, int64_t m,
                                                          int8_t *__restrict__ codes, int64_t ld,
                                                          int32_t *__restrict__ zero,
                                                          float *__restrict__ inv_q,
                                                          int32_t *__restrict__ sums) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x >> 6);
  if (row >= m) return;
  const int64_t t = row / B, b = row - t * B;
  const StackedRow x{frames + ((int64_t)skip * t * B + b) * dim, dim, B * (int64_t)dim};
  quantize_row_wave(x, (int64_t)stack * dim, row, codes, ld, zero, inv_q, sums, lane);
}

// Partial min/max: set s = rows [s*rps, (s+1)*rps) of a [rows][cols] matrix
// with leading dimension ldx; part p covers a contiguous slice of the set.
__global__ __launch_bounds__(256) void k_set_minmax(const float *__restrict__ X, int64_t ldx,
                                                    int64_t rps, int64_t cols, int nparts,
                                                    float2 *__restrict__ part) {
  const int s = blockIdx.y, p = blockIdx.x;
  const int64_t n = rps * cols;
  const int64_t per = (n + nparts - 1) / nparts;
  const int64_t b = (int64_t)p * per, e = b + per < n ? b + per : n;
  float lo = INFINITY, hi = -INFINITY;
  for (int64_t i = b + threadIdx.x; i < e; i += blockDim.x) {
    const int64_t r = i / cols, c = i - r * cols;
    const float v = X[(s * rps + r) * ldx + c];
    lo = fminf(lo, v);
    hi = fmaxf(hi, v);
  }
  lo = wave_min(lo);
  hi = wave_max(hi);
  __shared__ float slo[4], shi[4];
  if ((threadIdx.x & 63) == 0) {
    slo[threadIdx.x >> 6] = lo;
    shi[threadIdx.x >> 6] = hi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
      lo = fminf(lo, slo[w]);
      hi = fmaxf(hi, shi[w]);
    }
    part[(int64_t)s * nparts + p] = make_float2(lo, hi);
  }
}

__global__ void k_set_params(const float2 *__restrict__ part, int nsets, int nparts,
                             int64_t setsize, double *__restrict__ q_out,
                             int32_t *__restrict__ z_out, float *__restrict__ iq_out,
                             double *__restrict__ range, int32_t *__restrict__ zero,
                             float *__restrict__ inv_q) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= nsets) return;
  float lo = INFINITY, hi = -INFINITY;
  for (int p = 0; p < nparts; ++p) {
    lo = fminf(lo, part[(int64_t)s * nparts + p].x);
    hi = fmaxf(hi, part[(int64_t)s * nparts + p].y);
  }
  if (setsize == 0) lo = hi = 0.0f;
  const QParams p = make_qparams(lo, hi);
  q_out[s] = p.q;
  z_out[s] = p.z;
  iq_out[s] = p.inv_q;
  if (range) range[s] = p.range;
  if (zero) zero[s] = p.z;
  if (inv_q) inv_q[s] = p.inv_q;
}

// Encode every row with its set's params; row sums; optional per-row copies of
// the set's zero point / recovery factor.
__global__ __launch_bounds__(256) void k_set_encode(
    const float *__restrict__ X, int64_t ldx, int64_t rows, int64_t cols, int64_t rps,
    const double *__restrict__ q, const int32_t *__restrict__ zero,
    const float *__restrict__ inv_q, int8_t *__restrict__ codes, int64_t ld,
    int32_t *__restrict__ row_sums, int32_t *__restrict__ row_zero,
    float *__restrict__ row_inv_q) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t s = row / rps;
  const int sum =
      encode_row_wave(DenseRow{X + row * ldx}, cols, codes + row * ld, ld, q[s], zero[s], lane);
  if (lane == 0) {
    if (row_sums) row_sums[row] = sum;
    if (row_zero) row_zero[row] = zero[s];
    if (row_inv_q) row_inv_q[row] = inv_q[s];
  }
}

__global__ void k_dequantize(const int8_t *__restrict__ codes, int64_t ld, int64_t rows,
                             int64_t cols, int64_t rpb, const int32_t *__restrict__ zero,
                             const float *__restrict__ inv_q, float *__restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int64_t r = i / cols, c = i - r * cols;
  const int64_t b = r / rpb;
  const int v = (int)codes[r * ld + c] + 128;  // V'
  dst[i] = (float)(v + zero[b]) * inv_q[b];
}

// Row sums of 0..255 codes stored in the signed layout.
__global__ __launch_bounds__(256) void k_code_row_sums(const int8_t *__restrict__ codes,
                                                       int64_t ld, int64_t rows, int64_t K,
                                                       int32_t *__restrict__ sums) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int8_t *c = codes + row * ld;
  int s = 0;
  for (int64_t i = lane; i < K; i += kWave) s += (int)c[i] + 128;
  s = wave_sum(s);
  if (lane == 0) sums[row] = s;
}

__global__ void k_gate_fn(int fn, const float *__restrict__ x, float *__restrict__ y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float v = x[i];
  y[i] = fn == 0 ? exp_cw(v) : fn == 1 ? sigmoid_cw(v) : fn == 2 ? tanh_cw(v) : recip_ge1(v);
}

// ---------------------------------------------------------------- launchers
static inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

hipError_t launch_quantize_rows(const float *X, int64_t ldx, int64_t m, int64_t K, int8_t *codes,
                                int64_t ld, int32_t *zero, float *inv_q, int32_t *sums,
                                hipStream_t s) {
  if (m == 0) return hipSuccess;
  hipLaunchKernelGGL(k_quantize_rows, dim3(blocks_for(m, 4)), dim3(256), 0, s, X, ldx, m, K,
                     codes, ld, zero, inv_q, sums);
  return hipGetLastError();
}

hipError_t launch_quantize_stacked(const float *frames, int64_t B, int dim, int stack, int skip,
                                   int64_t T, int8_t *codes, int64_t ld, int32_t *zero,
                                   float *inv_q, int32_t *sums, hipStream_t s) {
  const int64_t m = T * B;
  if (m == 0) return hipSuccess;
  hipLaunchKernelGGL(k_quantize_stacked, dim3(blocks_for(m, 4)), dim3(256), 0, s, frames, B, dim,
                     stack, skip, m, codes, ld, zero, inv_q, sums);
  return hipGetLastError();
}

size_t set_quantize_ws(int nsets) {
  return align_up((size_t)nsets * kSetParts * sizeof(float2), 256) +
         3 * align_up((size_t)nsets * sizeof(double), 256);
}

hipError_t launch_set_quantize(const float *X, int64_t ldx, int64_t rows, int64_t cols,
                               int nsets, int8_t *codes, int64_t ld, double *range,
                               int32_t *zero, float *inv_q, int32_t *row_sums,
                               int32_t *row_zero, float *row_inv_q, void *ws, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  char *w = static_cast<char *>(ws);
  float2 *part = reinterpret_cast<float2 *>(w);
  w += align_up((size_t)nsets * kSetParts * sizeof(float2), 256);
  double *q = reinterpret_cast<double *>(w);
  w += align_up((size_t)nsets * sizeof(double), 256);
  int32_t *zs = reinterpret_cast<int32_t *>(w);
  w += align_up((size_t)nsets * sizeof(double), 256);
  float *iqs = reinterpret_cast<float *>(w);
  const int64_t rps = rows / nsets;
  hipLaunchKernelGGL(k_set_minmax, dim3(kSetParts, nsets), dim3(256), 0, s, X, ldx, rps, cols,
                     kSetParts, part);
  hipLaunchKernelGGL(k_set_params, dim3(blocks_for(nsets, 64)), dim3(64), 0, s, part, nsets,
                     kSetParts, rps * cols, q, zs, iqs, range, zero, inv_q);
  hipLaunchKernelGGL(k_set_encode, dim3(blocks_for(rows, 4)), dim3(256), 0, s, X, ldx, rows,
                     cols, rps, q, zs, iqs, codes, ld, row_sums, row_zero, row_inv_q);
  return hipGetLastError();
}

hipError_t launch_dequantize(const int8_t *codes, int64_t ld, int64_t rows, int64_t cols,
                             int nblocks, const int32_t *zero, const float *inv_q, float *dst,
                             hipStream_t s) {
  if (rows * cols == 0) return hipSuccess;
  hipLaunchKernelGGL(k_dequantize, dim3(blocks_for(rows * cols, 256)), dim3(256), 0, s, codes,
                     ld, rows, cols, rows / nblocks, zero, inv_q, dst);
  return hipGetLastError();
}

hipError_t launch_code_row_sums(const int8_t *codes, int64_t ld, int64_t rows, int64_t K,
                                int32_t *sums, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(k_code_row_sums, dim3(blocks_for(rows, 4)), dim3(256), 0, s, codes, ld,
                     rows, K, sums);
  return hipGetLastError();
}

hipError_t launch_gate_fn(int fn, const float *x, float *y, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gate_fn, dim3(blocks_for(n, 256)), dim3(256), 0, s, fn, x, y, n);
  return hipGetLastError();
}

}  // namespace ql
