// ql_pstack.hip -- stacked LSTM layers with a linear projection after each
// (Section 4: 5 x 500 cells with P = 100 .. 400 projection units) at one batch
// row, all in one persistent launch run as a wavefront: while layer l works on
// frame t, layer l-1 is already on a later frame.
//
// A tile owns u cells of one layer (the 4u gate rows of W_x' and W_h', resident
// in LDS) and v rows of the layer's projection W_r' (also resident).  Per
// frame t it
//   1. quantizes h_{t-1} (eq. 2, per vector) from the layer's tagged words and
//      forms the recurrent product W_h' h'_{t-1} for its gate rows (MFMA, the
//      vector as row 0 of a 16-row block);
//   2. recovers both products (eq. 1 / eq. 3), (W_x x + b) + W_h h, runs the
//      gates and the cell update, and publishes its cells of m_t;
//   3. quantizes m_t (per vector) from the tagged words of all the layer's
//      tiles and forms its rows of the projection h_t = recover(W_r' m'_t),
//      which it publishes;
// and, beside step 1 on two other waves, takes x_t: the launch's first layer
// reads its codes, a later layer quantizes layer l-1's published h_t itself
// (one vector, one quantization: the same codes layer l-1 makes of it).
// Every value exchanged goes into a full-length [T] buffer of 64-bit tagged
// words (step tag + fp32 value), so no slot is ever reused inside a launch and
// a layer may run any number of frames ahead of the next.  Every wait is
// bounded (timeout flag in the workspace header, see ql_exchange.h).
//
// Layout: when the chip is whole (256 CUs, 8 XCDs of 32) and a layer needs at
// most 32 tiles, the launch has one workgroup per CU; each reads its XCC_ID and
// takes the next free slot of its XCD, playing tile `slot` of layer `XCC_ID`.
// A layer's tiles then share one L2, and m_t, read only by the own layer, goes
// out with plain stores that stay in that L2.  h_t goes out twice: with plain
// stores for the own layer's tiles, and with device-coherent stores into a
// second buffer for the next layer (another XCD).
// Otherwise workgroup i plays tile i % G of layer i / G.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"
#include "ql_rec_common.h"

#include <algorithm>

namespace ql {

constexpr int kPThreads = 512;
constexpr int kPXcds = 8, kPXcdCus = 32;
constexpr int kPSlotBytes = kPXcds * 64;  // per-XCD slot counters after the header

struct PStackTiling {
  int G, u, v;      // tiles per layer, cells per tile, projection rows per tile
  int grid, xcd;
  int ldXmax, ldHmax, ldPmax;
  size_t off_wx, off_wh, off_wr, off_xc, off_hc, off_mc, off_sx, off_sh, off_sr, off_cpx, off_cph,
      off_cpr, off_bias, off_c, off_rp, lds_bytes;
  size_t layer_off[kMaxStack];  // byte offset of layer l's m and h words in the workspace
};

__device__ __forceinline__ ColParam col_param(const WeightMat &W, int64_t n, int64_t K) {
  const int64_t blk = n / W.rows_per_block;
  ColParam c;
  c.ztw = W.zero[blk] + 128;
  c.sigw = W.row_sums[n] - 128 * (int32_t)K;
  c.colterm = (int64_t)c.sigw + K * (int64_t)c.ztw;
  c.iqw = W.inv_q[blk];
  c.pad = 0;
  return c;
}

// TP: the launch writes sums, gate or cell taps or a final state (the variant
// without them carries none of their per-step code).
template <bool TP>
__global__ __launch_bounds__(kPThreads) void k_pstack(PStackArgs a, PStackTiling tl) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int s_abort;
  __shared__ int s_role;
  __shared__ int xch_x[16], xch_h[16], xch_m[16];  // the two quantizing waves' exchange slots

  const int64_t T = a.T;
  const int tid = threadIdx.x;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  char *wsb = static_cast<char *>(a.ws);

  int blk = (int)blockIdx.x;
  if (tl.xcd) {
    if (tid == 0) {
      const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
      unsigned *slots = reinterpret_cast<unsigned *>(wsb + kHeaderBytes);
      s_role = -1;
      if (xcc < a.nl) {  // a.nl <= 8: the slot counter exists
        const unsigned k = __hip_atomic_fetch_add(slots + xcc * 16, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        if (k < (unsigned)tl.G) s_role = xcc * tl.G + (int)k;
      }
    }
    __syncthreads();
    if (s_role < 0) return;
    blk = s_role;
  }
  const int l = blk / tl.G, g = blk % tl.G;
  const PStackLayer &Ly = a.L[l];
  const int64_t H = Ly.H, P = Ly.P, IN = Ly.in;
  const int ldX = (int)((IN + 63) / 64 * 64), ldH = (int)((H + 63) / 64 * 64);
  const int ldP = (int)((P + 63) / 64 * 64);
  const int u = tl.u, v = tl.v, nrows = 4 * u;
  const int64_t j0 = (int64_t)g * u, p0 = (int64_t)g * v;
  const int nu = (int)std::max<int64_t>(0, std::min<int64_t>(u, H - j0));
  const int nv = (int)std::max<int64_t>(0, std::min<int64_t>(v, P - p0));

  int8_t *wx = reinterpret_cast<int8_t *>(smem + tl.off_wx);
  int8_t *wh = reinterpret_cast<int8_t *>(smem + tl.off_wh);
  int8_t *wr = reinterpret_cast<int8_t *>(smem + tl.off_wr);
  int8_t *xc = reinterpret_cast<int8_t *>(smem + tl.off_xc);
  int8_t *hc = reinterpret_cast<int8_t *>(smem + tl.off_hc);
  int8_t *mc = reinterpret_cast<int8_t *>(smem + tl.off_mc);
  int32_t *Sx = reinterpret_cast<int32_t *>(smem + tl.off_sx);
  int32_t *Sh = reinterpret_cast<int32_t *>(smem + tl.off_sh);
  int32_t *Sr = reinterpret_cast<int32_t *>(smem + tl.off_sr);
  ColParam *cpx = reinterpret_cast<ColParam *>(smem + tl.off_cpx);
  ColParam *cph = reinterpret_cast<ColParam *>(smem + tl.off_cph);
  ColParam *cpr = reinterpret_cast<ColParam *>(smem + tl.off_cpr);
  float *bsl = reinterpret_cast<float *>(smem + tl.off_bias);
  float *cst = reinterpret_cast<float *>(smem + tl.off_c);
  RowParam *rp = reinterpret_cast<RowParam *>(smem + tl.off_rp);  // [0] x, [1] h, [2] m
  const int ldsX = tl.ldXmax, ldsH = tl.ldHmax, ldsP = tl.ldPmax;

  // tagged words of layer k: m [T][H], h for the next layer [T][P], then (XCD
  // layout) h for the own layer [T][P]
  auto mwords = [&](int k) { return reinterpret_cast<uint64_t *>(wsb + tl.layer_off[k]); };
  auto hwords = [&](int k) {
    return reinterpret_cast<uint64_t *>(wsb + tl.layer_off[k]) + T * a.L[k].H;
  };
  uint64_t *mw = mwords(l), *hw = hwords(l);
  uint64_t *hown = tl.xcd ? hw + T * P : hw;

  // ---- prologue: weight slices, column params, bias, c = 0
  for (int idx = tid; idx < nrows * (ldX / 16); idx += blockDim.x) {
    const int r = idx / (ldX / 16), kc = idx % (ldX / 16), gt = r / u, jj = r % u;
    uint4 w = make_uint4(0, 0, 0, 0);
    if (jj < nu) w = *reinterpret_cast<const uint4 *>(Ly.Wx.codes + (gt * H + j0 + jj) * Ly.Wx.ld + kc * 16);
    *reinterpret_cast<uint4 *>(wx + r * ldsX + kc * 16) = w;
  }
  for (int idx = tid; idx < nrows * (ldP / 16); idx += blockDim.x) {
    const int r = idx / (ldP / 16), kc = idx % (ldP / 16), gt = r / u, jj = r % u;
    uint4 w = make_uint4(0, 0, 0, 0);
    if (jj < nu) w = *reinterpret_cast<const uint4 *>(Ly.Wh.codes + (gt * H + j0 + jj) * Ly.Wh.ld + kc * 16);
    *reinterpret_cast<uint4 *>(wh + r * ldsP + kc * 16) = w;
  }
  for (int idx = tid; idx < v * (ldH / 16); idx += blockDim.x) {
    const int r = idx / (ldH / 16), kc = idx % (ldH / 16);
    uint4 w = make_uint4(0, 0, 0, 0);
    if (r < nv) w = *reinterpret_cast<const uint4 *>(Ly.Wr.codes + (p0 + r) * Ly.Wr.ld + kc * 16);
    *reinterpret_cast<uint4 *>(wr + r * ldsH + kc * 16) = w;
  }
  for (int r = tid; r < nrows; r += blockDim.x) {
    const int gt = r / u, jj = r % u;
    // rows past the layer's cells (zero weights, results unused) take the
    // params of a real row; a tile without cells takes cell 0's
    const int64_t n = gt * H + (nu > 0 ? j0 + (jj < nu ? jj : 0) : 0);
    cph[r] = col_param(Ly.Wh, n, P);
    cpx[r] = col_param(Ly.Wx, n, IN);
    bsl[r] = Ly.bias[n];
  }
  for (int r = tid; r < v; r += blockDim.x)
    cpr[r] = col_param(Ly.Wr, nv > 0 ? p0 + (r < nv ? r : 0) : 0, H);
  for (int j = tid; j < u; j += blockDim.x) cst[j] = Ly.c0 && j < nu ? Ly.c0[j0 + j] : 0.0f;
  if (tid == 0) s_abort = 0;
  for (int i = tid; i < 16; i += blockDim.x) xch_x[i] = xch_h[i] = xch_m[i] = 0;
  // the codes of x_t and h_{t-1} are row 0 of 16-row blocks whose other rows
  // stay zero, so the gate-row products run on MFMA (rows 1..15 give 0)
  for (int k = tid; k < 16 * ldsX; k += blockDim.x) xc[k] = 0;
  for (int k = tid; k < 16 * ldsP; k += blockDim.x) hc[k] = 0;
  __syncthreads();

  // Codes of row t of this layer's h (quantized here, in hc) to the layer's
  // output rows; this tile's share of the code words, tile 0 the row params.
  auto store_out = [&](int64_t t) {
    const int owords = (int)(Ly.out.ld / 4), share = (owords + tl.G - 1) / tl.G;
    for (int k = g * share + tid; k < std::min(owords, (g + 1) * share); k += blockDim.x) {
      const uint32_t w = k < ldP / 4 ? reinterpret_cast<const uint32_t *>(hc)[k] : 0u;
      reinterpret_cast<uint32_t *>(Ly.out.codes + t * Ly.out.ld)[k] = w;
    }
    if (g == 0 && tid == 0) {
      const RowParam r = rp[1];
      Ly.out.zero[t] = r.z;
      Ly.out.inv_q[t] = r.iqx;
      Ly.out.sums[t] = r.sum;
      if (Ly.tap_zero) Ly.tap_zero[t] = r.z;
      if (Ly.tap_inv_q) Ly.tap_inv_q[t] = r.iqx;
    }
    if (Ly.tap_codes)
      for (int k = g * (int)P / tl.G + tid; k < (g + 1) * (int)P / tl.G; k += blockDim.x)
        Ly.tap_codes[t * P + k] = hc[k];
  };

  for (int64_t t = 0; t < T; ++t) {
    // 1. codes of h_{t-1} (waves 0, 1) and of x_t (waves 2, 3 for a later
    //    layer, which quantizes layer l-1's h_t; waves 2 .. 7 copy the input
    //    codes for the first layer) side by side.  An all-zero h_{-1} quantizes to
    //    Q = 1, zero point 0, codes V' = 0 (stored -128): W_h h is exactly 0.
    if (tid < 2 * kWave) {
      if (t == 0 && Ly.h0) {
        // h_{-1} = h0 (plain floats), quantized per vector by wave 0
        if (tid < kWave)
          quant_rows<8, 1, kSrcPlain>(Ly.h0, P, 1, 1, 0u, (int)P, hc, ldsP, ldP, flag, &rp[1]);
      } else if (t == 0) {
        for (int k = tid; k < ldP; k += 2 * kWave) hc[k] = k < P ? (int8_t)-128 : (int8_t)0;
        if (tid == 0) rp[1] = row_param(0, 1.0f, 0, (int)P);
      } else if (!quant_row_2w(hown + (t - 1) * P, (uint32_t)t, (int)P, hc, ldP, flag, &rp[1],
                               xch_h)) {
        s_abort = 1;
      }
    } else if (l > 0) {
      if (tid < 4 * kWave &&
          !quant_row_2w(hwords(l - 1) + t * IN, (uint32_t)(t + 1), (int)IN, xc, ldX, flag, &rp[0],
                        xch_x, 2))
        s_abort = 1;
    } else {
      const int8_t *src = Ly.xin.codes + t * Ly.xin.ld;
      for (int k = tid - 2 * kWave; k < ldX / 4; k += (int)blockDim.x - 2 * kWave)
        reinterpret_cast<uint32_t *>(xc)[k] = reinterpret_cast<const uint32_t *>(src)[k];
      if (tid == 2 * kWave)
        rp[0] = row_param(Ly.xin.zero[t], Ly.xin.inv_q[t], Ly.xin.sums[t], (int)IN);
    }
    __syncthreads();
    if (s_abort) return;
    products_mfma(hc, ldsP, 16, wh, ldsP, nrows, nrows, ldP, Sh, nrows);
    products_mfma(xc, ldsX, 16, wx, ldsX, nrows, nrows, ldX, Sx, nrows);
    __syncthreads();
    if (TP && (Ly.acc_x || Ly.acc_h))  // sums of step t (row 0 of S) to the taps [T][4H], 0..255 domain
      for (int n = tid; n < nrows; n += blockDim.x) {
        const int gt = n / u, jj = n % u;
        if (jj >= nu) continue;
        const int64_t o = (t * 4 + gt) * H + j0 + jj;
        if (Ly.acc_x) Ly.acc_x[o] = acc_u8(Sx[n], cpx[n].sigw, rp[0].sigx, IN);
        if (Ly.acc_h) Ly.acc_h[o] = acc_u8(Sh[n], cph[n].sigw, rp[1].sigx, P);
      }

    // 2. gates: lane 4 jj + gt computes gate gt of cell jj (i, f, g, o)
    if (tid < 4 * u) {
      const int jj = tid >> 2, gt = tid & 3, n = gt * u + jj;
      const RowParam rx = rp[0], rh = rp[1];
      const ColParam cx = cpx[n], ch = cph[n];
      const float gx = recover(Sx[n], cx.colterm, cx.ztw, rx.ztx, rx.sigx, cx.iqw, rx.iqx) + bsl[n];
      const float av = gx + recover(Sh[n], ch.colterm, ch.ztw, rh.ztx, rh.sigx, ch.iqw, rh.iqx);
      const float sg = sigmoid_cw(gt == 2 ? 2.0f * av : av);
      const float act = gt == 2 ? 2.0f * sg - 1.0f : sg;
      const float ig = quad_bcast<0>(act), fg = quad_bcast<1>(act);
      const float gv = quad_bcast<2>(act), og = quad_bcast<3>(act);
      if (TP && Ly.tap_gates && jj < nu) Ly.tap_gates[(t * 4 + gt) * H + j0 + jj] = act;
      if (gt == 0 && jj < nu) {
        const float cn = (fg * cst[jj]) + (ig * gv);
        cst[jj] = cn;
        const float m = og * tanh_cw(cn);
        if (tl.xcd) publish_local(&mw[t * H + j0 + jj], (uint32_t)(t + 1), m);
        else publish(&mw[t * H + j0 + jj], (uint32_t)(t + 1), m);
        if constexpr (TP) {
          if (Ly.tap_c) Ly.tap_c[t * H + j0 + jj] = cn;
          if (Ly.tap_m) Ly.tap_m[t * H + j0 + jj] = m;
          if (Ly.cT && t == T - 1) Ly.cT[j0 + jj] = cn;
        }
      }
    }
    // the output codes of h_{t-1} (in hc) leave while m_t travels
    if (t > 0) store_out(t - 1);

    // 3. codes of m_t, projection rows of h_t
    if (tid < 2 * kWave) {
      if (!quant_row_2w(mw + t * H, (uint32_t)(t + 1), (int)H, mc, ldH, flag, &rp[2], xch_m))
        s_abort = 1;
    }
    __syncthreads();
    if (s_abort) return;
    if (nv > 0) products_valu(mc, ldsH, 1, wr, ldsH, v, nv, ldH, Sr, v);
    __syncthreads();
    if (tid < nv) {
      const RowParam rm = rp[2];
      const ColParam cr = cpr[tid];
      const float hv = recover(Sr[tid], cr.colterm, cr.ztw, rm.ztx, rm.sigx, cr.iqw, rm.iqx);
      if (tl.xcd) publish_local(&hown[t * P + p0 + tid], (uint32_t)(t + 1), hv);
      publish(&hw[t * P + p0 + tid], (uint32_t)(t + 1), hv);
      if (Ly.h) Ly.h[t * P + p0 + tid] = hv;
      if constexpr (TP) {
        if (Ly.acc_r) Ly.acc_r[t * P + p0 + tid] = acc_u8(Sr[tid], cr.sigw, rm.sigx, H);
        if (Ly.hT && t == T - 1) Ly.hT[p0 + tid] = hv;
      }
    }
    // the next step's first phase writes only hc, xc, rp[0], rp[1]: none of
    // them is read after the last barrier
  }
  // codes of the last h
  if (tid < 2 * kWave) {
    if (!quant_row_2w(hown + (T - 1) * P, (uint32_t)T, (int)P, hc, ldP, flag, &rp[1], xch_h))
      s_abort = 1;
  }
  __syncthreads();
  if (s_abort) return;
  store_out(T - 1);
}

// ------------------------------------------------------------------ host side
static bool plan_pstack(const PStackArgs &a, int cus, int lds_max, PStackTiling *out) {
  PStackTiling tl{};
  int64_t maxH = 0, maxP = 0, maxIn = 0;
  for (int l = 0; l < a.nl; ++l) {
    const PStackLayer &L = a.L[l];
    if (L.H <= 0 || L.P <= 0 || L.H > 512 || L.P > 512 || L.in > 512 || L.in <= 0) return false;
    if (l > 0 && L.in != a.L[l - 1].P) return false;
    maxH = std::max(maxH, L.H);
    maxP = std::max(maxP, L.P);
    maxIn = std::max(maxIn, L.in);
  }
  // tiles of at least 20 cells (wider tiles publish more per step, but fewer
  // tiles poll every word), and at most the layer's share of the CUs
  const int share = cus / a.nl;
  if (share < 1) return false;
  tl.u = (int)std::max<int64_t>(20, (maxH + share - 1) / share);
  tl.u = (tl.u + 3) / 4 * 4;  // 4u gate rows in whole 16-row MFMA tiles
  tl.G = (int)((maxH + tl.u - 1) / tl.u);
  tl.v = (int)((maxP + tl.G - 1) / tl.G);
  if (4 * tl.u > kPThreads || tl.v > kPThreads) return false;
  tl.ldXmax = (int)round_up(maxIn, 64);
  tl.ldHmax = (int)round_up(maxH, 64);
  tl.ldPmax = (int)round_up(maxP, 64);
  const int nrows = 4 * tl.u;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 16);
    return o;
  };
  tl.off_wx = take((size_t)nrows * tl.ldXmax);
  tl.off_wh = take((size_t)nrows * tl.ldPmax);
  tl.off_wr = take((size_t)tl.v * tl.ldHmax);
  tl.off_xc = take((size_t)16 * tl.ldXmax);
  tl.off_hc = take((size_t)16 * tl.ldPmax);
  tl.off_mc = take(tl.ldHmax);
  tl.off_sx = take((size_t)16 * nrows * 4);
  tl.off_sh = take((size_t)16 * nrows * 4);
  tl.off_sr = take((size_t)tl.v * 4);
  tl.off_cpx = take((size_t)nrows * sizeof(ColParam));
  tl.off_cph = take((size_t)nrows * sizeof(ColParam));
  tl.off_cpr = take((size_t)tl.v * sizeof(ColParam));
  tl.off_bias = take((size_t)nrows * 4);
  tl.off_c = take((size_t)tl.u * 4);
  tl.off_rp = take(3 * sizeof(RowParam));
  tl.lds_bytes = off;
  if ((int64_t)tl.lds_bytes > lds_max) return false;
  tl.xcd = cus == kPXcds * kPXcdCus && a.nl <= kPXcds && tl.G <= kPXcdCus;
  tl.grid = tl.xcd ? cus : a.nl * tl.G;
  if (tl.grid > cus) return false;  // one workgroup per CU at most is planned for
  size_t woff = kHeaderBytes + kPSlotBytes;
  for (int l = 0; l < a.nl; ++l) {
    tl.layer_off[l] = woff;
    woff += align_up((size_t)a.T * (a.L[l].H + 2 * a.L[l].P) * 8, 256);
  }
  *out = tl;
  return true;
}

size_t pstack_ws(const int64_t *H, const int64_t *P, int nl, int64_t T) {
  size_t n = kHeaderBytes + kPSlotBytes;
  for (int l = 0; l < nl; ++l) n += align_up((size_t)T * (H[l] + 2 * P[l]) * 8, 256);
  return n;
}

static int device_props(int *cus, int *lds_max) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return 0;
  return 1;
}

hipError_t launch_pstack(const PStackArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0) return hipSuccess;
  if (a.nl < 1 || a.nl > kMaxStack) {
    *unsupported = true;
    return hipSuccess;
  }
  int cus = 0, lds_max = 0;
  if (!device_props(&cus, &lds_max)) return hipErrorInvalidDevice;
  PStackTiling tl;
  if (!plan_pstack(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  bool tp = false;  // any tap or final state asked for
  for (int l = 0; l < a.nl; ++l) {
    const PStackLayer &L = a.L[l];
    tp = tp || L.acc_x || L.acc_h || L.acc_r || L.tap_gates || L.tap_c || L.tap_m || L.hT || L.cT;
  }
  auto kern = tp ? k_pstack<true> : k_pstack<false>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kPThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  // slot counters and every tagged word start at 0 (tags count from 1)
  const size_t used = tl.layer_off[a.nl - 1] +
                      align_up((size_t)a.T * (a.L[a.nl - 1].H + 2 * a.L[a.nl - 1].P) * 8, 256);
  e = clear_exchange(a.ws, (int64_t)((used - kHeaderBytes) / 8), s);
  if (e != hipSuccess) return e;
  PStackArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(kern), dim3(tl.grid),
                                    dim3(kPThreads), kargs, (unsigned)tl.lds_bytes, s);
}

int pstack_layers_per_launch(const PStackArgs &a) {
  int cus = 0, lds_max = 0;
  if (!device_props(&cus, &lds_max)) return 1;
  for (int nl = std::min(a.nl, kMaxStack); nl >= 2; --nl) {
    PStackArgs b = a;
    b.nl = nl;
    PStackTiling tl;
    if (plan_pstack(b, cus, lds_max, &tl)) return nl;
  }
  return 1;
}

hipError_t set_wait_bound_pstack(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
