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
  // eight rows loaded before they are added (in row order), so eight loads
  // are in flight per thread
  constexpr int kU = 8;
  float s = 0.0f;
  int64_t m = m0;
  for (; m + kU <= m1; m += kU) {
    float v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = X[(m + u) * N + n];
#pragma unroll
    for (int u = 0; u < kU; ++u) s += v[u];
  }
  for (; m < m1; ++m) s += X[m * N + n];
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
// A tile owns (bB <= 16 batch rows) x (u <= 16 cells).  Per step it waits
// until every tile of its batch slice has published da_{t+1} (device-coherent
// stores, then an arrival on the slice's counter of that step) and forms
// W_h^T da_{t+1} for its (row, cell) pairs on fp32 MFMA (one 16 x 16 block,
// K = 4H split over the eight waves, 256 k each): the W_h columns of its
// cells stay in LDS for the launch (transposed, one padded row of k per
// cell), and the da values go from memory straight into registers, lane
// (row r, group q) reading 16 consecutive k of row r per 64-k block and the
// same 16 k of its cell's W_h column from LDS; an MFMA then sums
// k = base + 16 q + j over q for one j, so A and B take the same order of k.  The waves' partial blocks are
// added in wave order (the result does not depend on timing); then the
// cell's backward step and its part of da_t.  Counters are per step, so
// nothing is reused in a launch.
// On the whole chip (8 XCDs of 32 CUs) with at most 8 batch slices of at most
// 32 tiles, every CU gets a workgroup, which reads its XCC_ID and takes the
// next free slot of its XCD: tile `slot` of slice `XCC_ID`.  A slice's tiles
// then share one L2 for the da_{t+1} they all read.  da_t still goes out with
// device-coherent stores: the gradient products launched after this kernel
// read it from every XCD.
// ---------------------------------------------------------------------------
constexpr int kBpttThreads = 512;
constexpr int kBpttWaves = kBpttThreads / 64;
constexpr int kBpttKBlocks = 4;  // 64-k blocks per wave: 8 x 4 x 64 = 2048 >= 4H

constexpr int kBpttLdw = kBpttWaves * kBpttKBlocks * 64 + 4;  // padded row of W_h^T (floats)

constexpr int kBpttXcds = 8, kBpttXcdCus = 32;
constexpr int kBpttSlotBytes = kBpttXcds * 64;  // per-XCD slot counters after the header

struct BpttTiling {
  int bB, u, nbt, nut, grid, xcd;
  size_t off_w, off_p, off_dc, lds_bytes;
};

typedef float v4f_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kBpttThreads) void k_bptt(BpttArgs a, BpttTiling tl) {
  extern __shared__ __attribute__((aligned(16))) float bsm[];
  float *wT = bsm + tl.off_w / 4;    // [16 cells][kBpttLdw]: W_h[k][j0 + c] at wT[c * ldw + k]
  float *part = bsm + tl.off_p / 4;  // [waves][16 rows][16 cells] partial blocks
  float *dcn = bsm + tl.off_dc / 4;  // [bB * u]: dC/dc carried to the step before
  __shared__ int s_abort;
  const int tid = threadIdx.x;
  const int64_t T = a.T, B = a.B, H = a.H, G4 = 4 * a.H;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  unsigned *slots = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
  unsigned *cnt0 = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes +
                                                kBpttSlotBytes);
  auto counter = [&](int64_t t, int tb) { return cnt0 + (t * tl.nbt + tb) * 16; };

  int blk = (int)blockIdx.x;
  if (tl.xcd) {
    __shared__ int s_role;
    if (tid == 0) {
      const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
      s_role = -1;
      if (xcc < tl.nbt) {
        const unsigned k = __hip_atomic_fetch_add(slots + xcc * 16, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        if (k < (unsigned)tl.nut) s_role = xcc * tl.nut + (int)k;
      }
    }
    __syncthreads();
    if (s_role < 0) return;
    blk = s_role;
  }
  const int tb = blk / tl.nut, tu = blk % tl.nut;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = (int)std::min<int64_t>(tl.bB, B - b0);
  const int nu = (int)std::min<int64_t>(tl.u, H - j0);
  const int npr = tl.bB * tl.u;  // pair p = lb * u + jj
  const int lane = tid & 63, wave = tid >> 6, fr = lane & 15, fq = lane >> 4;

  // k of element j of block kb of this lane (rows / cells fr, group fq)
  auto kof = [&](int kb, int j) {
    return (int64_t)wave * (64 * kBpttKBlocks) + kb * 64 + fq * 16 + j;
  };
  // the W_h column block of the tile's cells, transposed into LDS (zeros past
  // the cells and past 4H)
  for (int idx = tid; idx < 16 * kBpttWaves * kBpttKBlocks * 64; idx += blockDim.x) {
    const int c = idx / (kBpttWaves * kBpttKBlocks * 64);
    const int64_t k = idx % (kBpttWaves * kBpttKBlocks * 64);
    wT[c * kBpttLdw + k] = c < nu && k < G4 ? a.Wh[k * H + j0 + c] : 0.0f;
  }
  for (int q = tid; q < npr; q += blockDim.x) dcn[q] = 0.0f;
  if (tid == 0) s_abort = 0;
  __syncthreads();

  const int lb = tid / tl.u, jj = tid % tl.u;  // cell lanes: pair (row lb, cell jj)
  const bool cell_lane = tid < npr && lb < nb && jj < nu;
  // this lane's cell operands of a step (the forward pass's gates, c_t,
  // c_{t-1} and dC/dh from above): loaded a step ahead, right after the
  // step's arrival
  float ig = 0.0f, fg = 0.0f, gg = 0.0f, og = 0.0f, ct = 0.0f, cp = 0.0f, dyv = 0.0f;
  auto load_cell = [&](int64_t t) {
    if (!cell_lane || t < 0) return;
    const int64_t row = t * B + b0 + lb, j = j0 + jj;
    const float *gt = a.gates + row * G4;
    ig = gt[j], fg = gt[H + j], gg = gt[2 * H + j], og = gt[3 * H + j];
    ct = a.c[row * H + j];
    cp = t > 0 ? a.c[(row - B) * H + j] : 0.0f;
    dyv = a.dy[row * H + j];
  };
  load_cell(T - 1);
  for (int64_t t = T - 1; t >= 0; --t) {
    // ---- W_h^T da_{t+1} for this tile's (row, cell) pairs
    v4f_t acc = v4f_t{0.0f, 0.0f, 0.0f, 0.0f};
    if (t + 1 < T) {
      if (!wait_count(counter(t + 1, tb), (unsigned)tl.nut, flag)) s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      // 16 consecutive k of row fr per block, as 8-byte words, all in flight,
      // issued block by block so that each block's products wait only for its
      // own loads.  Every lane loads: a row past the slice reads the slice's
      // row 0 (its products land in output rows nobody reads), and k past 4H
      // reads k = 0 (a finite value, times the zero columns of W_h^T in LDS).
      const float *src = a.da + ((t + 1) * B + b0 + (fr < nb ? fr : 0)) * G4;
      uint64_t dv[kBpttKBlocks][8];
#pragma unroll
      for (int kb = 0; kb < kBpttKBlocks; ++kb) {
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const int64_t k = kof(kb, 2 * w);
          dv[kb][w] = ld_coherent64(reinterpret_cast<const uint64_t *>(src + (k < G4 ? k : 0)));
        }
        __builtin_amdgcn_sched_barrier(0);  // issue order: block by block
      }
#pragma unroll
      for (int kb = 0; kb < kBpttKBlocks; ++kb) {
        const v4f_t *wr = reinterpret_cast<const v4f_t *>(wT + fr * kBpttLdw + kof(kb, 0));
        const v4f_t w4[4] = {wr[0], wr[1], wr[2], wr[3]};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const uint32_t bits = (uint32_t)(dv[kb][j / 2] >> (32 * (j & 1)));
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bits), w4[j / 4][j % 4], acc,
                                                     0, 0, 0);
        }
      }
    }
    // An XDL result needs a pass-count-dependent number of wait states before
    // an LDS store may read it, and nothing checks that in hardware.  The
    // compiler's spacing was found missing here (the stores of acc[0..1] two
    // instructions after the last MFMA, on the path that falls through from
    // the products): those rows then took a value from before the final
    // pass, at random.  The statement below reads and writes acc, so it sits
    // between the last MFMA and the stores whatever the schedule, and gives
    // 24 wait states (a 16-pass XDL result needs at most 19).
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc));
    // partial blocks to LDS: part[wave][row][cell]
#pragma unroll
    for (int i = 0; i < 4; ++i) part[(wave * 16 + 4 * fq + i) * 16 + fr] = acc[i];
    __syncthreads();

    // ---- the cell's backward step and da_t
    if (cell_lane) {
      float dhrec = 0.0f;
      for (int w = 0; w < kBpttWaves; ++w) dhrec += part[(w * 16 + lb) * 16 + jj];
      const int64_t row = t * B + b0 + lb, j = j0 + jj;
      const float dh = dyv + dhrec;
      const float tc = tanh_cw(ct);
      const float d_o = dh * tc;
      const float d_c = dh * og * (1.0f - tc * tc) + dcn[tid];
      const float d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * cp;
      dcn[tid] = d_c * fg;
      float *dst = a.da + row * G4 + j;
      const float v0 = d_i * ig * (1.0f - ig), v1 = d_f * fg * (1.0f - fg);
      const float v2 = d_g * (1.0f - gg * gg), v3 = d_o * og * (1.0f - og);
      st_coherent(dst, v0);
      st_coherent(dst + H, v1);
      st_coherent(dst + 2 * H, v2);
      st_coherent(dst + 3 * H, v3);
    }
    if (t > 0) arrive(counter(t, tb));  // (no tile waits on step 0's arrivals)
    else __syncthreads();               // part is rewritten only by a next launch
    // the next step's cell operands, issued after the arrival so that its
    // wait for the stores of da_t does not also wait for these loads
    load_cell(t - 1);
  }
}

static bool plan_bptt(const BpttArgs &a, int cus, int lds_max, BpttTiling *out) {
  BpttTiling tl{};
  // K = 4H in registers: eight waves of four 64-k blocks
  if (4 * a.H > (int64_t)kBpttWaves * kBpttKBlocks * 64) return false;
  // 16 cells per tile (one MFMA column block): every tile of a slice reads all
  // of the slice's da_{t+1}, so fewer, wider tiles move fewer bytes a step
  tl.u = (int)std::min<int64_t>(16, a.H);
  tl.nut = (int)((a.H + tl.u - 1) / tl.u);
  // a slice per XCD when the chip is whole and a slice's tiles fit one XCD
  // (the batch spread over all eight), else slices of 16 rows
  tl.xcd = 0;
  if (cus == kBpttXcds * kBpttXcdCus && tl.nut <= kBpttXcdCus) {
    tl.bB = (int)std::min<int64_t>(16, (a.B + kBpttXcds - 1) / kBpttXcds);
    tl.nbt = (int)((a.B + tl.bB - 1) / tl.bB);
    tl.xcd = tl.nbt <= kBpttXcds;
  }
  if (!tl.xcd) {
    tl.bB = (int)std::min<int64_t>(a.B, 16);
    tl.nbt = (int)((a.B + tl.bB - 1) / tl.bB);
  }
  tl.grid = tl.xcd ? cus : tl.nbt * tl.nut;
  if (tl.grid > cus) return false;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 16);
    return o;
  };
  tl.off_w = take((size_t)16 * kBpttLdw * 4);
  tl.off_p = take((size_t)kBpttWaves * 256 * 4);
  tl.off_dc = take((size_t)tl.bB * tl.u * 4);
  tl.lds_bytes = off;
  if ((int64_t)tl.lds_bytes + 64 > lds_max) return false;
  *out = tl;
  return true;
}

size_t bptt_ws(int64_t T, int64_t B) {
  // per-XCD slot counters, then per-step, per-slice arrival counters (64
  // bytes each; at most max(8, B / 16 rounded up) slices) after the header
  const int64_t slices = std::max<int64_t>(8, (B + 15) / 16);
  return kHeaderBytes + kBpttSlotBytes + (size_t)std::max<int64_t>(T, 1) * (size_t)slices * 64;
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

hipError_t set_wait_bound_train(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
