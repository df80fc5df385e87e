// ql_train.hip -- kernels of the quantization-aware training step (Section
// 3.2, Algorithm 1): the forward pass is the inference path of this library
// on freshly quantized copies of the float parameters; what follows here is
// ordinary floating-point backpropagation with the float parameters,
// evaluated at the activations that quantized forward pass produced:
//   * the output error of frame-level cross-entropy on the posteriors;
//   * backpropagation through time of one LSTM layer (k_bptt): the serial
//     part, dC/da_t for every step, in one persistent launch;
//   * column sums (bias gradients) and the SGD update.
// The gradient products themselves are fp32 GEMMs (ql_f32.hip).
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"

#include <algorithm>

namespace ql {

// ---------------------------------------------------------------------------
// Cross-entropy of one frame's posteriors p against target y, averaged over
// the N frames: the row's loss term -log p[y], and dC/dz = (p - onehot(y)) / N
// written over p (one workgroup per row).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_xent_grad(float *p, const int32_t *targets, int64_t S,
                                                   float n_frames, float *row_loss) {
  const int64_t r = blockIdx.x;
  const int32_t y = targets[r];
  float *row = p + r * S;
  for (int64_t s = threadIdx.x; s < S; s += blockDim.x) {
    const float v = row[s];
    if (s == y) row_loss[r] = -logf(v);
    row[s] = (v - (s == y ? 1.0f : 0.0f)) / n_frames;
  }
}

// loss = (sum of the row terms) / N, summed in fp64 in a fixed order.
__global__ __launch_bounds__(256) void k_mean(const float *v, int64_t n, float *out) {
  __shared__ double part[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) s += (double)v[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = n > 0 ? (float)(part[0] / (double)n) : 0.0f;
}

// Column sums out[n] = sum_m X[m][n]: chunk c of the rows into part[c][n],
// then the chunks in order.
constexpr int kColChunks = 64;
__global__ __launch_bounds__(256) void k_colsum_part(const float *X, int64_t M, int64_t N,
                                                     int64_t rows_per_chunk, float *part) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const int64_t m0 = (int64_t)blockIdx.y * rows_per_chunk;
  const int64_t m1 = std::min<int64_t>(M, m0 + rows_per_chunk);
  float s = 0.0f;
  for (int64_t m = m0; m < m1; ++m) s += X[m * N + n];
  part[(int64_t)blockIdx.y * N + n] = s;
}
__global__ __launch_bounds__(256) void k_colsum_final(const float *part, int chunks, int64_t N,
                                                      float *out) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float s = part[n];
  for (int c = 1; c < chunks; ++c) s += part[(int64_t)c * N + n];
  out[n] = s;
}

// w <- w - lr g (fp32, no contraction)
__global__ __launch_bounds__(256) void k_sgd(float *w, const float *g, int64_t n, float lr) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    w[i] = w[i] - lr * g[i];
}

hipError_t launch_xent_grad(float *post, const int32_t *targets, int64_t N, int64_t S,
                            float *row_loss, float *loss, hipStream_t s) {
  if (N == 0) {
    if (loss) hipLaunchKernelGGL(k_mean, dim3(1), dim3(256), 0, s, row_loss, (int64_t)0, loss);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_xent_grad, dim3((unsigned)N), dim3(256), 0, s, post, targets, S, (float)N,
                     row_loss);
  if (loss) hipLaunchKernelGGL(k_mean, dim3(1), dim3(256), 0, s, (const float *)row_loss, N, loss);
  return hipGetLastError();
}

size_t colsum_ws(int64_t N) { return (size_t)kColChunks * (size_t)N * sizeof(float); }

hipError_t launch_colsum(const float *X, int64_t M, int64_t N, float *out, float *part,
                         hipStream_t s) {
  if (N == 0) return hipSuccess;
  const int64_t rpc = std::max<int64_t>(1, (M + kColChunks - 1) / kColChunks);
  const int chunks = (int)std::max<int64_t>(1, (M + rpc - 1) / rpc);
  hipLaunchKernelGGL(k_colsum_part, dim3((unsigned)((N + 255) / 256), (unsigned)chunks), dim3(256),
                     0, s, X, M, N, rpc, part);
  hipLaunchKernelGGL(k_colsum_final, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s,
                     (const float *)part, chunks, N, out);
  return hipGetLastError();
}

hipError_t launch_sgd(float *w, const float *g, int64_t n, float lr, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>(4096, (n + 255) / 256);
  hipLaunchKernelGGL(k_sgd, dim3(blocks), dim3(256), 0, s, w, g, n, lr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backpropagation through time of one LSTM layer without projection (gate
// order i, f, g, o; c = f c + i g; h = m = o tanh(c); zero initial state),
// serial over t = T-1 .. 0:
//   dh_t   = dy_t + W_h^T da_{t+1}                (dy: dC/dh from above)
//   dc_t   = dh_t o (1 - tanh^2 c_t) + f_{t+1} dc_{t+1}
//   da_t   = (dc_t g i (1 - i), dc_t c_{t-1} f (1 - f), dc_t i (1 - g^2),
//             dh_t tanh(c_t) o (1 - o))            (dC/d pre-activation)
// A tile owns (bB batch rows) x (u cells): the 4u rows of W_h^T it needs
// (columns j of W_h) stay in LDS for the launch.  Per step it waits until
// every tile of its batch slice has published da_{t+1} (device-coherent
// stores, then an arrival on the slice's counter of that step), stages those
// rows' da_{t+1} through LDS in chunks, forms W_h^T da_{t+1} for its cells
// (each (row, cell) pair's sum split over several lanes, the partial sums
// added in a fixed order), runs the cell's backward step and publishes its
// part of da_t.  Counters are per step, so nothing is reused in a launch.
// ---------------------------------------------------------------------------
constexpr int kBpttThreads = 512;

struct BpttTiling {
  int bB, u, nbt, nut, grid, chunk, ns;  // ns lanes per (row, cell) pair
  int ldw, ldc;                          // LDS row strides (floats) of W_h^T and the da chunk
  size_t off_w, off_d, off_p, off_dc, lds_bytes;
};

__global__ __launch_bounds__(kBpttThreads) void k_bptt(BpttArgs a, BpttTiling tl) {
  extern __shared__ __attribute__((aligned(16))) float bsm[];
  float *wT = bsm + tl.off_w / 4;    // [u][ldw]: W_h[n][j0 + jj] at wT[jj * ldw + n]
  float *dS = bsm + tl.off_d / 4;    // [bB][ldc]: staged da_{t+1} chunk
  float *part = bsm + tl.off_p / 4;  // [ns][bB * u]
  float *dcn = bsm + tl.off_dc / 4;  // [bB * u]: dC/dc carried to the step before
  __shared__ int s_abort;
  const int tid = threadIdx.x;
  const int64_t T = a.T, B = a.B, H = a.H, G4 = 4 * a.H;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  unsigned *cnt0 = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
  auto counter = [&](int64_t t, int tb) { return cnt0 + (t * tl.nbt + tb) * 16; };

  const int tb = blockIdx.x / tl.nut, tu = blockIdx.x % tl.nut;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = (int)std::min<int64_t>(tl.bB, B - b0);
  const int nu = (int)std::min<int64_t>(tl.u, H - j0);
  const int npr = tl.bB * tl.u;  // pair p = lb * u + jj

  for (int idx = tid; idx < tl.u * G4; idx += blockDim.x) {
    const int jj = idx / (int)G4;
    const int64_t n = idx % G4;
    wT[jj * tl.ldw + n] = jj < nu ? a.Wh[n * H + j0 + jj] : 0.0f;
  }
  for (int p = tid; p < npr; p += blockDim.x) dcn[p] = 0.0f;
  if (tid == 0) s_abort = 0;
  __syncthreads();

  const int p = tid % npr, q = tid / npr;  // this lane: pair p, share q of each chunk
  const bool dot_lane = q < tl.ns;
  const int lb = p / tl.u, jj = p % tl.u;
  for (int64_t t = T - 1; t >= 0; --t) {
    // ---- W_h^T da_{t+1} for this tile's (row, cell) pairs
    float acc = 0.0f;
    if (t + 1 < T) {
      if (!wait_count(counter(t + 1, tb), (unsigned)tl.nut, flag)) s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      const float *src = a.da + ((t + 1) * B + b0) * G4;
      for (int64_t c0 = 0; c0 < G4; c0 += tl.chunk) {
        const int cl = (int)std::min<int64_t>(tl.chunk, G4 - c0);
        for (int idx = tid; idx < nb * cl; idx += blockDim.x) {
          const int r = idx / cl, nn = idx % cl;
          dS[r * tl.ldc + nn] = ld_coherent(src + r * G4 + c0 + nn);
        }
        __syncthreads();
        if (dot_lane && lb < nb) {
          const float *w = wT + jj * tl.ldw + c0;
          const float *d = dS + lb * tl.ldc;
          for (int nn = q; nn < cl; nn += tl.ns) acc += w[nn] * d[nn];
        }
        __syncthreads();
      }
    }
    if (dot_lane) part[q * npr + p] = acc;
    __syncthreads();

    // ---- the cell's backward step and da_t
    if (tid < npr && lb < nb && jj < nu) {
      float dhrec = 0.0f;
      for (int k = 0; k < tl.ns; ++k) dhrec += part[k * npr + tid];
      const int64_t row = t * B + b0 + lb, j = j0 + jj;
      const float *gt = a.gates + row * G4;
      const float ig = gt[j], fg = gt[H + j], gg = gt[2 * H + j], og = gt[3 * H + j];
      const float ct = a.c[row * H + j];
      const float cp = t > 0 ? a.c[(row - B) * H + j] : 0.0f;
      const float dh = a.dy[row * H + j] + dhrec;
      const float tc = tanh_cw(ct);
      const float d_o = dh * tc;
      const float d_c = dh * og * (1.0f - tc * tc) + dcn[tid];
      const float d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * cp;
      dcn[tid] = d_c * fg;
      float *dst = a.da + row * G4 + j;
      st_coherent(dst, d_i * ig * (1.0f - ig));
      st_coherent(dst + H, d_f * fg * (1.0f - fg));
      st_coherent(dst + 2 * H, d_g * (1.0f - gg * gg));
      st_coherent(dst + 3 * H, d_o * og * (1.0f - og));
    }
    if (t > 0) arrive(counter(t, tb));  // (no tile waits on step 0's arrivals)
  }
}

static bool plan_bptt(const BpttArgs &a, int cus, int lds_max, BpttTiling *out) {
  BpttTiling tl{};
  const int64_t G4 = 4 * a.H;
  tl.bB = (int)std::min<int64_t>(a.B, 16);
  tl.nbt = (int)((a.B + tl.bB - 1) / tl.bB);
  if (tl.nbt > cus) return false;
  tl.ldw = (int)G4 + 1;
  // W_h^T rows in LDS: at most 96 KB of them
  const int umax = (int)std::min<int64_t>(kBpttThreads / tl.bB, (96 * 1024) / (4 * tl.ldw));
  if (umax < 1) return false;
  const int nut0 = std::max(1, cus / tl.nbt);
  tl.u = (int)std::min<int64_t>(umax, std::max<int64_t>(1, (a.H + nut0 - 1) / nut0));
  tl.nut = (int)((a.H + tl.u - 1) / tl.u);
  tl.grid = tl.nbt * tl.nut;
  if (tl.grid > cus) return false;
  const int npr = tl.bB * tl.u;
  tl.ns = std::max(1, kBpttThreads / npr);
  tl.chunk = (int)std::min<int64_t>(G4, std::max<int64_t>(64, (16 * 1024) / tl.bB));
  tl.ldc = tl.chunk + 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 16);
    return o;
  };
  tl.off_w = take((size_t)tl.u * tl.ldw * 4);
  tl.off_d = take((size_t)tl.bB * tl.ldc * 4);
  tl.off_p = take((size_t)tl.ns * npr * 4);
  tl.off_dc = take((size_t)npr * 4);
  tl.lds_bytes = off;
  if ((int64_t)tl.lds_bytes + 64 > lds_max) return false;
  *out = tl;
  return true;
}

size_t bptt_ws(int64_t T, int64_t B) {
  // per-step, per-slice arrival counters (64 bytes each) after the header
  return kHeaderBytes + (size_t)std::max<int64_t>(T, 1) * (size_t)((B + 15) / 16) * 64;
}

hipError_t launch_bptt(const BpttArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0 || a.B == 0) return hipSuccess;
  int dev = 0, cus = 0, lds_max = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  BpttTiling tl;
  if (!plan_bptt(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_bptt),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_bptt, kBpttThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  e = clear_exchange(a.ws, (int64_t)((bptt_ws(a.T, a.B) - kHeaderBytes) / 8), s);
  if (e != hipSuccess) return e;
  BpttArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(k_bptt), dim3(tl.grid),
                                    dim3(kBpttThreads), kargs, (unsigned)tl.lds_bytes, s);
}

}  // namespace ql
