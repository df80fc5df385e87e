// ql_stack.hip -- several stacked LSTM layers (Section 4) in one persistent
// launch, run as a wavefront: while layer l works on frame t, layer l-1 is
// already on frame t+1 or later, so a launch of n layers takes about T + n
// steps instead of n * T.
//
// A unit tile owns (bB batch rows) x (u hidden units) of one layer and keeps
// both of the layer's weight slices resident in LDS: the 4u gate rows of W_x'
// and of W_h'.  Per step it
//   1. takes the codes of x_t: the launch's first layer reads them from the
//      already quantized input, a later layer reads the codes layer l-1
//      produced for its h_t, which are the same codes layer l-1 used itself
//      (one vector, one quantization; no re-quantization), and forms the
//      input-side product; none of this depends on h_{t-1}, so it is done
//      while h_{t-1} is still travelling between the workgroups;
//   2. takes the codes of h_{t-1} (quantized per vector, eq. 2);
//   3. forms the recurrent 8-bit product, recovers both products (eq. 1 /
//      eq. 3), adds the bias as the hoisted path does, (W_x x + b) + W_h h,
//      and runs the gates and the cell update;
//   4. publishes h_t as tagged words (step tag + value).
// Who quantizes h_t: with one batch row per tile, every unit tile quantizes
// its row itself from the tagged words (one wave does it while the others
// store the tile's share of the previous codes and form the next input
// side); the codes for the next layer travel as tagged words too.  With 16+
// batch rows, a few quantizing workgroups per batch slice (8 rows each, one
// per wave; they own no units, so no gate work waits behind them) re-read
// the tagged h words until every tag matches, quantize, store the codes with
// device-coherent stores and then bump the slice's arrival counter, which
// the unit tiles and the next layer wait on.
// Between layers nothing is reused: codes go to full-length [T*B] buffers,
// so a layer may run any number of steps ahead of the next one; a layer
// never waits on a later layer.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"
#include "ql_rec_common.h"

#include <algorithm>

namespace ql {

constexpr int kStackThreads = 512;
constexpr int kXcds = 8;  // accelerator complex dies (XCDs) of the MI355X, each with its own L2
constexpr int kXcdCus = 32;  // CUs of one XCD
// Replicas of the tagged h words at one batch row (readers spread over them).
constexpr int kMaxReph = 2;

// Per-layer arrival counters of the codes of h: [parity][slice], 64 bytes apart.
constexpr size_t kStackCounterBytes = (size_t)2 * kMaxSlices * 64;

struct StackTiling {
  int bB, u, nbt, nut, gl;  // tile shape and counts; gl workgroups per layer
  int nq;                   // quantizing workgroups per batch slice (batched tiles)
  int grid, mfma;
  int ldH;                  // padded width of h codes (and W_h' rows)
  int ldXmax;               // largest padded input width over the launch
  int ldsW, ldsWx, ldsX, ldsXx;
  int reph;                 // replicas of the tagged h buffer (one batch row per tile)
  int xcd;                  // one-row tiles: every layer's tiles on one XCD of its own
  int64_t strideh;          // 64-bit words between replicas
  int nw;                   // tagged code words per row: ldH / 4 codes + 3 params
  size_t hx_bytes, cx_bytes, layer_bytes;  // exchange bytes per layer
  size_t off_xh2, off_rowh2;  // second buffer of the codes of h (one-row tiles)
  size_t off_wh, off_wx, off_xh, off_xx, off_sh, off_sx, off_c, off_colh, off_colx, off_rowh,
      off_rowx, off_bias, lds_bytes;
};



// RBA: rows one wave quantizes together (2 for batched tiles, 1 at one row).
// TP: the launch writes sums, gate or cell taps or a final state (the
// variant without them carries none of their per-step code).
template <int NVA, bool MFA, int RBA, bool TP>
__global__ __launch_bounds__(kStackThreads) void k_stack(StackArgs a, StackTiling tl) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int8_t *wh = reinterpret_cast<int8_t *>(smem + tl.off_wh);
  int8_t *wx = reinterpret_cast<int8_t *>(smem + tl.off_wx);
  int8_t *xh = reinterpret_cast<int8_t *>(smem + tl.off_xh);
  int8_t *xx = reinterpret_cast<int8_t *>(smem + tl.off_xx);
  int32_t *Sh = reinterpret_cast<int32_t *>(smem + tl.off_sh);
  int32_t *Sx = reinterpret_cast<int32_t *>(smem + tl.off_sx);
  float *cst = reinterpret_cast<float *>(smem + tl.off_c);
  ColParam *cph = reinterpret_cast<ColParam *>(smem + tl.off_colh);
  ColParam *cpx = reinterpret_cast<ColParam *>(smem + tl.off_colx);
  RowParam *rph = reinterpret_cast<RowParam *>(smem + tl.off_rowh);
  RowParam *rpx = reinterpret_cast<RowParam *>(smem + tl.off_rowx);
  float *bsl = reinterpret_cast<float *>(smem + tl.off_bias);
  __shared__ int s_abort;
  __shared__ int s_xch[16];  // one-row tiles: the two quantizing waves' exchange
  constexpr bool CNT = MFA;  // batched tiles: counters + coherent data; else tagged words

  const int64_t T = a.T, B = a.B, H = a.H;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  unsigned *cnt0 = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
  // XCD-local layout: the launch has a workgroup for every CU; each takes the
  // next free slot of the XCD it runs on (XCC_ID) and plays tile `slot` of
  // layer `xcc`, so a layer's tiles share one L2 (the per-layer counters,
  // unused at one batch row, hand out the slots); the rest leave at once.
  int blk = (int)blockIdx.x;
  if (tl.xcd) {
    __shared__ int s_role;
    if (threadIdx.x == 0) {
      const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
      const unsigned k = __hip_atomic_fetch_add(cnt0 + xcc * 16, 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      s_role = xcc < a.nl && k < (unsigned)tl.gl ? xcc * tl.gl + (int)k : -1;
    }
    __syncthreads();
    if (s_role < 0) return;
    blk = s_role;
  }
  const int l = blk / tl.gl, wgi = blk % tl.gl;
  const StackLayer &Ly = a.L[l];
  const int64_t IN = Ly.in;
  const int ldXl = (int)((IN + 63) / 64 * 64);
  auto ctr = [&](int layer, int64_t par, int slice) {
    return cnt0 + ((layer * 2 + (int)par) * kMaxSlices + slice) * 16;
  };
  char *xbase = static_cast<char *>(a.ws) + kHeaderBytes + (size_t)a.nl * kStackCounterBytes;
  auto xdata = [&](int layer) { return xbase + (size_t)layer * tl.layer_bytes; };
  // own layer's h exchange: tagged words, replicas of [2][B][H] (one replica
  // for batched tiles, whose h is read by the designated tiles only)
  uint64_t *xht = reinterpret_cast<uint64_t *>(xdata(l));
  const uint64_t *xht_mine = xht + (blk % tl.reph) * tl.strideh;
  // tagged codes of every h_t of a layer: [T*B][nw] words after its h exchange
  auto ctag = [&](int layer) {
    return reinterpret_cast<uint64_t *>(xdata(layer) + tl.hx_bytes);
  };

  const int tid = threadIdx.x;
  // a batch slice: nut unit tiles, then (batched tiles) nq quantizing workgroups
  const int tb = wgi / (tl.nut + tl.nq), tw = wgi % (tl.nut + tl.nq);
  const bool quantizer = tw >= tl.nut;
  const int tu = quantizer ? 0 : tw;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = (int)(B - b0 < tl.bB ? B - b0 : tl.bB);
  const int nu = (int)(H - j0 < tl.u ? H - j0 : tl.u);
  const int nrows = 4 * tl.u;  // gate-major: row g*u + jj
  const int rowsA = MFA ? tl.bB : nb;
  if (tid == 0) s_abort = 0;
  __syncthreads();

  if (CNT && quantizer) {
    // Quantizing workgroup of a batched slice: per step, the codes of
    // h_{t-1} for 8 rows of the slice (one per wave, re-reading the row's
    // tagged words until every tag matches), stored with device-coherent
    // stores, then an arrival on the slice's codes counter.
    const int q0 = (tw - tl.nut) * 8;
    // a ragged last slice may leave a quantizing workgroup without rows: it
    // must not arrive either (an arrival that waited for nothing could stand
    // in for a missing one of a later step)
    if (q0 >= nb) return;
    const int nq = nb - q0 < 8 ? nb - q0 : 8;
    const int hwords = tl.ldH / 8;
    for (int64_t t = 1; t <= T; ++t) {
      const int64_t par = (t - 1) & 1;
      const uint64_t *prev = xht + par * B * H;
      const bool ok = quant_tile<NVA, 1, kSrcTagged>(nq, nq, H, (uint32_t)t, (int)H, xh, tl.ldsX,
                                                     tl.ldH, flag, rph,
                                                     [&](int lb) -> const void * {
                                                       return prev + (b0 + q0 + lb) * H;
                                                     });
      if (!ok) s_abort = 1;
      // each wave stores the row it quantized (its own LDS writes are in order)
      const int lb = tid >> 6, lane = tid & 63;
      if (ok && lb < nq) {
        const int64_t row = (t - 1) * B + b0 + q0 + lb;
        const int owords = (int)(Ly.out.ld / 8);
        for (int wd = lane; wd < owords; wd += kWave) {
          uint64_t v = 0;
          if (wd < hwords) v = *reinterpret_cast<const uint64_t *>(xh + lb * tl.ldsX + wd * 8);
          st_coherent64(reinterpret_cast<uint64_t *>(Ly.out.codes + row * Ly.out.ld) + wd, v);
        }
        if (lane == 0) {
          const RowParam r = rph[lb];
          st_coherent_i(&Ly.out.zero[row], r.z);
          st_coherent(&Ly.out.inv_q[row], r.iqx);
          st_coherent_i(&Ly.out.sums[row], r.sum);
          if (Ly.tap_zero) Ly.tap_zero[row] = r.z;
          if (Ly.tap_inv_q) Ly.tap_inv_q[row] = r.iqx;
        }
        if (Ly.tap_codes)
          for (int k = lane; k < (int)H; k += kWave) Ly.tap_codes[row * H + k] = xh[lb * tl.ldsX + k];
      }
      // arrival once every wave's stores have completed (none after a failed wait)
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (s_abort) return;
      if (tid == 0)
        __hip_atomic_fetch_add(ctr(l, par, tb), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }

  // ---- prologue: W_x' and W_h' slices, column params, bias, c = 0
  for (int idx = tid; idx < nrows * (tl.ldH / 16); idx += blockDim.x) {
    const int r = idx / (tl.ldH / 16), kc = idx % (tl.ldH / 16);
    const int g = r / tl.u, jj = r % tl.u;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (jj < nu) v = *reinterpret_cast<const uint4 *>(Ly.Wh.codes + (g * H + j0 + jj) * Ly.Wh.ld + kc * 16);
    *reinterpret_cast<uint4 *>(wh + r * tl.ldsW + kc * 16) = v;
  }
  for (int idx = tid; idx < nrows * (ldXl / 16); idx += blockDim.x) {
    const int r = idx / (ldXl / 16), kc = idx % (ldXl / 16);
    const int g = r / tl.u, jj = r % tl.u;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (jj < nu) v = *reinterpret_cast<const uint4 *>(Ly.Wx.codes + (g * H + j0 + jj) * Ly.Wx.ld + kc * 16);
    *reinterpret_cast<uint4 *>(wx + r * tl.ldsWx + kc * 16) = v;
  }
  for (int r = tid; r < nrows; r += blockDim.x) {
    const int g = r / tl.u, jj = r % tl.u;
    const int64_t n = g * H + j0 + (jj < nu ? jj : 0);
    {
      const int64_t blk = n / Ly.Wh.rows_per_block;
      ColParam c;
      c.ztw = Ly.Wh.zero[blk] + 128;
      c.sigw = Ly.Wh.row_sums[n] - 128 * (int32_t)H;
      c.colterm = (int64_t)c.sigw + H * (int64_t)c.ztw;
      c.iqw = Ly.Wh.inv_q[blk];
      c.pad = 0;
      cph[r] = c;
    }
    {
      const int64_t blk = n / Ly.Wx.rows_per_block;
      ColParam c;
      c.ztw = Ly.Wx.zero[blk] + 128;
      c.sigw = Ly.Wx.row_sums[n] - 128 * (int32_t)IN;
      c.colterm = (int64_t)c.sigw + IN * (int64_t)c.ztw;
      c.iqw = Ly.Wx.inv_q[blk];
      c.pad = 0;
      cpx[r] = c;
    }
    bsl[r] = Ly.bias[n];
  }
  for (int idx = tid; idx < tl.bB * tl.u; idx += blockDim.x) {
    const int lb = idx / tl.u, jj = idx % tl.u;
    cst[idx] = Ly.c0 && lb < nb && jj < nu ? Ly.c0[(b0 + lb) * H + j0 + jj] : 0.0f;
  }
  if constexpr (!MFA) {  // rows 1..15 of the one-row code blocks stay zero
    int8_t *xh2 = reinterpret_cast<int8_t *>(smem + tl.off_xh2);
    for (int k = tid; k < 16 * tl.ldsX; k += blockDim.x) xh[k] = xh2[k] = 0;
    for (int k = tid; k < 16 * tl.ldsXx; k += blockDim.x) xx[k] = 0;
  }
  __syncthreads();

  // Sums of step t (signed-code sums S[lb][n], gate-major n = g u + jj) to a
  // tap [T][B][4H] in the 0..255 code domain; only when the caller asked.
  auto tap_acc = [&](int32_t *dst, const int32_t *S, const ColParam *cp, const RowParam *rp,
                     int64_t K, int64_t t) {
    for (int idx = tid; idx < nb * nrows; idx += blockDim.x) {
      const int lb = idx / nrows, n = idx % nrows, g = n / tl.u, jj = n % tl.u;
      if (jj < nu)
        dst[((t * B + b0 + lb) * 4 + g) * H + j0 + jj] = acc_u8(S[idx], cp[n].sigw, rp[lb].sigx, K);
    }
  };
  // Initial state h_{-1}: rows of h0 (plain floats), or zeros.
  auto h0_row = [&](int lb) -> const void * { return Ly.h0 ? Ly.h0 + (b0 + lb) * H : nullptr; };

  // Counter mode: the codes of x_t (the input, or layer l-1's h_t) are loaded
  // into registers before h_{t-1} is quantized, and parked in LDS afterwards
  // (kXPre words per thread cover 32 rows of up to 512 codes).
  constexpr int kXPre = 4;
  uint64_t xpre[kXPre];
  int32_t xpz = 0, xps = 0;
  float xpq = 0.0f;
  const int xwords = ldXl / 8;
  auto prefetch_x = [&](int64_t t) {
    const int64_t xrow0 = t * B + b0;
#pragma unroll
    for (int i = 0; i < kXPre; ++i) {
      const int idx = tid + i * kStackThreads, lb = idx / xwords, wd = idx % xwords;
      uint64_t v = 0;
      if (lb < nb && idx < rowsA * xwords)
        v = ld_coherent64(reinterpret_cast<const uint64_t *>(Ly.xin.codes + (xrow0 + lb) * Ly.xin.ld) + wd);
      xpre[i] = v;
    }
    if (tid < nb) {
      xpz = ld_coherent_i(&Ly.xin.zero[xrow0 + tid]);
      xpq = ld_coherent(&Ly.xin.inv_q[xrow0 + tid]);
      xps = ld_coherent_i(&Ly.xin.sums[xrow0 + tid]);
    }
  };

  // Batched tiles: input side of the pre-activations, (W_x x + b) recovered in
  // place in Sx (float bits) for rows [0, nr), off the recurrence's critical
  // path.  (One-row tiles recover it in the gates: there the gates are not
  // the long pole and the extra pass would delay the next step.)
  auto x_preact = [&](int64_t t, int nr) {
    __syncthreads();  // Sx complete
    if (TP && Ly.acc_x) tap_acc(Ly.acc_x, Sx, cpx, rpx, IN, t);  // each lane reads its own sums first
    for (int idx = tid; idx < nr * nrows; idx += blockDim.x) {
      const int lb = idx / nrows, n = idx % nrows;
      const RowParam rx = rpx[lb];
      const ColParam cx = cpx[n];
      const float g = recover(Sx[idx], cx.colterm, cx.ztw, rx.ztx, rx.sigx, cx.iqw, rx.iqx) + bsl[n];
      Sx[idx] = __float_as_int(g);
    }
  };

  // Gates, cell update; publish h_t (step t).  Pairs (batch row, cell) are
  // dealt one per lane in full rounds of the workgroup; the remainder is
  // spread over 2 or 4 lanes per pair (lane g computes gates g of the pair's
  // gate set) when that fits, so no lane does much more than its share.
  auto gates = [&](int64_t t, int64_t hcur) {
    const int pairs = nb * nu, nt = (int)blockDim.x;
    auto preact = [&](int lb, int n) {
      const RowParam rh = rph[lb];
      const ColParam ch = cph[n];
      const float yh = recover(Sh[lb * nrows + n], ch.colterm, ch.ztw, rh.ztx, rh.sigx, ch.iqw, rh.iqx);
      if constexpr (CNT) return __int_as_float(Sx[lb * nrows + n]) + yh;
      const RowParam rx = rpx[lb];
      const ColParam cx = cpx[n];
      const float gxv = recover(Sx[lb * nrows + n], cx.colterm, cx.ztw, rx.ztx, rx.sigx, cx.iqw, rx.iqx) + bsl[n];
      return gxv + yh;
    };
    // activation of gate g of pair (lb, jj): sigmoid for i, f, o and
    // tanh(x) = 2 sigmoid(2x) - 1 for g
    auto act = [&](int lb, int jj, int g) {
      const float av = preact(lb, g * tl.u + jj);
      const float sg = sigmoid_cw(g == 2 ? 2.0f * av : av);
      return g == 2 ? 2.0f * sg - 1.0f : sg;
    };
    auto finish = [&](int lb, int jj, float ig, float fg, float gv, float og) {
      const int64_t b = b0 + lb, j = j0 + jj;
      const float cn = (fg * cst[lb * tl.u + jj]) + (ig * gv);
      cst[lb * tl.u + jj] = cn;
      const float m = og * tanh_cw(cn);
      for (int c2 = 0; c2 < tl.reph; ++c2) {
        if (tl.xcd) publish_local(&xht[c2 * tl.strideh + hcur + b * H + j], (uint32_t)(t + 1), m);
        else publish(&xht[c2 * tl.strideh + hcur + b * H + j], (uint32_t)(t + 1), m);
      }
      if (Ly.h) Ly.h[(t * B + b) * H + j] = m;
      if constexpr (TP) {
        if (Ly.tap_gates) {
          float *gp = Ly.tap_gates + (t * B + b) * 4 * H + j;
          gp[0] = ig, gp[H] = fg, gp[2 * H] = gv, gp[3 * H] = og;
        }
        if (Ly.tap_c) Ly.tap_c[(t * B + b) * H + j] = cn;
        if (Ly.tap_m) Ly.tap_m[(t * B + b) * H + j] = m;
        if (t == T - 1) {
          if (Ly.hT) Ly.hT[b * H + j] = m;
          if (Ly.cT) Ly.cT[b * H + j] = cn;
        }
      }
    };
    const int full = pairs / nt, rem = pairs % nt;
    for (int k = 0; k < full; ++k) {
      const int pr = k * nt + tid, lb = pr / nu, jj = pr % nu;
      finish(lb, jj, act(lb, jj, 0), act(lb, jj, 1), act(lb, jj, 2), act(lb, jj, 3));
    }
    if (rem == 0) return;
    const int p0 = full * nt;
    if (4 * rem <= nt) {
      // four lanes per pair (whole quads active: 4 * rem lanes from lane 0)
      if (tid < 4 * rem) {
        const int pr = p0 + (tid >> 2), lb = pr / nu, jj = pr % nu;
        const float a = act(lb, jj, tid & 3);
        const float ig = quad_bcast<0>(a), fg = quad_bcast<1>(a);
        const float gv = quad_bcast<2>(a), og = quad_bcast<3>(a);
        if ((tid & 3) == 0) finish(lb, jj, ig, fg, gv, og);
      }
    } else if (2 * rem <= nt) {
      // two lanes per pair: the even lane takes i and f, the odd one g and o
      if (tid < 2 * rem) {
        const int pr = p0 + (tid >> 1), lb = pr / nu, jj = pr % nu, h = tid & 1;
        const float a0 = act(lb, jj, 2 * h), a1 = act(lb, jj, 2 * h + 1);
        // swap with the other lane of the pair (quad_perm 1,0,3,2)
        const float b0v = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a0), 0xB1, 0xf, 0xf, false));
        const float b1v = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a1), 0xB1, 0xf, 0xf, false));
        if (h == 0) finish(lb, jj, a0, a1, b0v, b1v);
      }
    } else if (tid < rem) {
      const int pr = p0 + tid, lb = pr / nu, jj = pr % nu;
      finish(lb, jj, act(lb, jj, 0), act(lb, jj, 1), act(lb, jj, 2), act(lb, jj, 3));
    }
  };

  if constexpr (CNT) {
    // Batched unit tiles: the codes of h_{t-1} are made once per slice by its
    // quantizing workgroups that have rows (Qn of them); every tile loads all
    // rows' codes once their arrivals are in, as it loads x_t.
    const int Qn = (nb + 7) / 8 < tl.nq ? (nb + 7) / 8 : tl.nq;
    const int hwords = tl.ldH / 8;
    uint64_t hpre[kXPre];

    // With at most one 16-row block of gate rows per wave, wave w keeps the
    // fragments of block w of W_h' in registers for the launch: the recurrent
    // product (on the critical path) then reads only the activation
    // fragments from LDS.
    const int wave = tid >> 6, nblk = nrows / 16;
    const bool wreg = nblk <= kStackThreads / 64;
    v4i fh[8];
    if (wreg && wave < nblk) load_wfrag(fh, wh, tl.ldsW, wave, tl.ldH);

    // Gate work of this lane, fixed for the launch: pair (row, cell) number
    // tid of every full round of nt pairs, then in the remainder one pair
    // over lpp lanes (gates g0 .. g0 + ng - 1 on this lane).  Index
    // arithmetic and the column params of the 24-bit recovery are made once
    // here instead of at every step.
    struct PairRec {
      int lb, jj, sidx, cidx;  // row and cell in the tile; Sh/Sx and c index of gate 0
      int64_t poff;            // b * H + j
      int32_t colt[4], ztw[4];
      float iqw[4];
      bool cfast, valid;       // every column of the lane fits the 24-bit recovery
    };
    const int nt = (int)blockDim.x, pairs = nb * nu;
    const int full = pairs / nt, rem = pairs % nt;
    const int lpp = 4 * rem <= nt ? 4 : 2 * rem <= nt ? 2 : 1;
    auto make_pair = [&](int pr, bool valid, int g0, int ng) {
      PairRec p;
      p.valid = valid;
      const int prc = valid ? pr : 0;
      p.lb = prc / nu;
      p.jj = prc % nu;
      p.sidx = p.lb * nrows + p.jj;
      p.cidx = p.lb * tl.u + p.jj;
      p.poff = (b0 + p.lb) * H + j0 + p.jj;
      p.cfast = true;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p.colt[i] = 0;
        p.ztw[i] = 0;
        p.iqw[i] = 0.0f;
        if (i < ng) {
          const ColParam c = cph[(g0 + i) * tl.u + p.jj];
          p.colt[i] = (int32_t)c.colterm;
          p.ztw[i] = c.ztw;
          p.iqw[i] = c.iqw;
          p.cfast = p.cfast && (uint32_t)(c.ztw + 127) <= 255u &&
                    (uint64_t)(c.colterm + (1 << 23)) < (uint64_t)(1 << 24);
        }
      }
      return p;
    };
    const PairRec pf = make_pair(tid, full > 0, 0, 4);
    const int rg0 = lpp == 4 ? (tid & 3) : lpp == 2 ? 2 * (tid & 1) : 0;
    const PairRec prm = make_pair(full * nt + tid / lpp, rem > 0 && tid < lpp * rem, rg0, 4 / lpp);
    // activation of gate g (slot i of the lane's columns) of pair p: the
    // recovered recurrent product plus the recovered input side in Sx
    auto act_b = [&](const PairRec &p, int i, int g, const RowParam &rh, bool fast) {
      const int n = g * tl.u;
      const int32_t S = Sh[p.sidx + n];
      float yh;
      if (fast) {
        const uint32_t tt = (uint32_t)S + (uint32_t)mul_i24(rh.ztx, p.colt[i]) +
                            (uint32_t)mul_i24(p.ztw[i], rh.sigx);
        yh = ((float)(int32_t)tt * p.iqw[i]) * rh.iqx;
      } else {
        const ColParam c = cph[n + p.jj];
        yh = recover(S, c.colterm, c.ztw, rh.ztx, rh.sigx, c.iqw, rh.iqx);
      }
      const float av = __int_as_float(Sx[p.sidx + n]) + yh;
      const float sg = sigmoid_cw(g == 2 ? 2.0f * av : av);
      return g == 2 ? 2.0f * sg - 1.0f : sg;
    };
    auto finish_b = [&](const PairRec &p, int64_t t, int64_t hcur, float ig, float fg, float gv,
                        float og) {
      const float cn = (fg * cst[p.cidx]) + (ig * gv);
      cst[p.cidx] = cn;
      const float m = og * tanh_cw(cn);
      for (int c2 = 0; c2 < tl.reph; ++c2)
        publish(&xht[c2 * tl.strideh + hcur + p.poff], (uint32_t)(t + 1), m);
      if (Ly.h) Ly.h[t * B * H + p.poff] = m;
      if constexpr (TP) {
        if (Ly.tap_gates) {
          float *gp = Ly.tap_gates + (t * B + b0 + p.lb) * 4 * H + j0 + p.jj;
          gp[0] = ig, gp[H] = fg, gp[2 * H] = gv, gp[3 * H] = og;
        }
        if (Ly.tap_c) Ly.tap_c[t * B * H + p.poff] = cn;
        if (Ly.tap_m) Ly.tap_m[t * B * H + p.poff] = m;
        if (t == T - 1) {
          if (Ly.hT) Ly.hT[p.poff] = m;
          if (Ly.cT) Ly.cT[p.poff] = cn;
        }
      }
    };
    auto row_fast = [](const RowParam &rh) { return (uint32_t)(rh.ztx + 127) <= 255u; };
    auto gates_b = [&](int64_t t, int64_t hcur) {
      auto one_lane = [&](const PairRec &p) {
        const RowParam rh = rph[p.lb];
        const bool fast = p.cfast && row_fast(rh);
        const float ig = act_b(p, 0, 0, rh, fast), fg = act_b(p, 1, 1, rh, fast);
        const float gv = act_b(p, 2, 2, rh, fast), og = act_b(p, 3, 3, rh, fast);
        finish_b(p, t, hcur, ig, fg, gv, og);
      };
      if (full > 0) one_lane(pf);
      for (int k = 1; k < full; ++k) one_lane(make_pair(k * nt + tid, true, 0, 4));
      if (!prm.valid) return;
      const RowParam rh = rph[prm.lb];
      const bool fast = prm.cfast && row_fast(rh);
      if (lpp == 4) {
        // whole quads are active (4 * rem lanes from lane 0)
        const float a = act_b(prm, 0, tid & 3, rh, fast);
        const float ig = quad_bcast<0>(a), fg = quad_bcast<1>(a);
        const float gv = quad_bcast<2>(a), og = quad_bcast<3>(a);
        if ((tid & 3) == 0) finish_b(prm, t, hcur, ig, fg, gv, og);
      } else if (lpp == 2) {
        // the even lane takes i and f, the odd one g and o; swap within the
        // pair of lanes (quad_perm 1,0,3,2)
        const int h2 = 2 * (tid & 1);
        const float a0 = act_b(prm, 0, h2, rh, fast), a1 = act_b(prm, 1, h2 + 1, rh, fast);
        const float b0v = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a0), 0xB1, 0xf, 0xf, false));
        const float b1v = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a1), 0xB1, 0xf, 0xf, false));
        if (h2 == 0) finish_b(prm, t, hcur, a0, a1, b0v, b1v);
      } else {
        const float ig = act_b(prm, 0, 0, rh, fast), fg = act_b(prm, 1, 1, rh, fast);
        const float gv = act_b(prm, 2, 2, rh, fast), og = act_b(prm, 3, 3, rh, fast);
        finish_b(prm, t, hcur, ig, fg, gv, og);
      }
    };

    for (int64_t t = 0; t < T; ++t) {
      const int64_t hcur = (t & 1) * B * H;
      const int64_t par = (t - 1) & 1;

      // ---- 1. the input side of step t, which does not depend on h_{t-1}:
      // codes of x_t and their product, done while the codes of h_{t-1} are
      // still being made
      if (l > 0 && !wait_count(ctr(l - 1, t & 1, tb), (unsigned)((t >> 1) + 1) * Qn, flag))
        s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      prefetch_x(t);
#pragma unroll
      for (int i = 0; i < kXPre; ++i) {
        const int idx = tid + i * kStackThreads, lb = idx / xwords, wd = idx % xwords;
        if (idx < rowsA * xwords) *reinterpret_cast<uint64_t *>(xx + lb * tl.ldsXx + wd * 8) = xpre[i];
      }
      if (tid < rowsA)
        rpx[tid] = tid < nb ? row_param(xpz, xpq, xps, (int)IN) : row_param(0, 0.0f, 0, (int)IN);
      __syncthreads();
      products_mfma(xx, tl.ldsXx, tl.bB, wx, tl.ldsWx, nrows, nrows, ldXl, Sx, nrows);
      x_preact(t, nb);

      // ---- 2. codes of h_{t-1}
      if (t > 0 && !wait_count(ctr(l, par, tb), (unsigned)(((t - 1) >> 1) + 1) * Qn, flag))
        s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      const int64_t hrow0 = (t - 1) * B + b0;
      int32_t hz = 0, hs = 0;
      float hq = 0.0f;
      if (t > 0) {
#pragma unroll
        for (int i = 0; i < kXPre; ++i) {
          const int idx = tid + i * kStackThreads, lb = idx / hwords, wd = idx % hwords;
          uint64_t v = 0;
          if (lb < nb && idx < rowsA * hwords)
            v = ld_coherent64(reinterpret_cast<const uint64_t *>(Ly.out.codes + (hrow0 + lb) * Ly.out.ld) + wd);
          hpre[i] = v;
        }
        if (tid < nb) {
          hz = ld_coherent_i(&Ly.out.zero[hrow0 + tid]);
          hq = ld_coherent(&Ly.out.inv_q[hrow0 + tid]);
          hs = ld_coherent_i(&Ly.out.sums[hrow0 + tid]);
        }
      }
      if (t == 0) {
        // h_{-1} (h0, or zeros): every tile quantizes those rows itself
        quant_tile<NVA, RBA, kSrcPlain>(nb, rowsA, H, 0u, (int)H, xh, tl.ldsX, tl.ldH, flag, rph,
                                        h0_row);
      } else {
#pragma unroll
        for (int i = 0; i < kXPre; ++i) {
          const int idx = tid + i * kStackThreads, lb = idx / hwords, wd = idx % hwords;
          if (idx < rowsA * hwords) *reinterpret_cast<uint64_t *>(xh + lb * tl.ldsX + wd * 8) = hpre[i];
        }
        if (tid < rowsA)
          rph[tid] = tid < nb ? row_param(hz, hq, hs, (int)H) : row_param(0, 0.0f, 0, (int)H);
      }
      __syncthreads();

      // ---- 3. the recurrent product against the resident W_h' slice
      if (!wreg)
        products_mfma(xh, tl.ldsX, tl.bB, wh, tl.ldsW, nrows, nrows, tl.ldH, Sh, nrows);
      else if (wave < nblk)
        products_mfma_reg(xh, tl.ldsX, tl.bB, fh, wave, tl.ldH, Sh, nrows);
      __syncthreads();
      if (TP && Ly.acc_h) tap_acc(Ly.acc_h, Sh, cph, rph, H, t);

      // ---- 4. recover, gates, cell; publish h_t
      gates_b(t, hcur);
      __syncthreads();  // LDS of this step is free before the next step
    }
    return;
  }

  // One batch row per tile: every tile quantizes its row of h_{t-1} from the
  // tagged words of its own layer, and takes x_t from the input (first layer)
  // or from layer l-1's tagged code words.
  // Codes of x_t (the input, or layer l-1's tagged words) and the input-side
  // product into Sx; false if a wait expired.
  auto input_side = [&](int64_t t) -> bool {
    const int64_t xrow0 = t * B + b0;
    if (l == 0) {
      const int chunks = ldXl / 16;
      for (int idx = tid; idx < rowsA * chunks; idx += blockDim.x) {
        const int lb = idx / chunks, ch = idx % chunks;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (lb < nb) v = *reinterpret_cast<const uint4 *>(Ly.xin.codes + (xrow0 + lb) * Ly.xin.ld + ch * 16);
        *reinterpret_cast<uint4 *>(xx + lb * tl.ldsXx + ch * 16) = v;
      }
      for (int lb = tid; lb < rowsA; lb += blockDim.x)
        rpx[lb] = lb < nb ? row_param(Ly.xin.zero[xrow0 + lb], Ly.xin.inv_q[xrow0 + lb],
                                      Ly.xin.sums[xrow0 + lb], (int)IN)
                          : row_param(0, 0.0f, 0, (int)IN);
    } else {
      // tagged words of layer l-1 for rows xrow0 .. xrow0 + nb - 1, tag t + 1
      const uint64_t *ct = ctag(l - 1);
      const int nwx = ldXl / 4 + 3;  // layer l-1's row: its ldH == ldXl here
      long it = 0;
      for (;;) {
        uint32_t bad = 0;
        for (int idx = tid; idx < nb * nwx; idx += blockDim.x) {
          const int lb = idx / nwx, wd = idx % nwx;
          const uint64_t wv = ld_tagged(ct + (xrow0 + lb) * nwx + wd);
          bad |= (uint32_t)(wv >> 32) ^ (uint32_t)(t + 1);
          const uint32_t pay = (uint32_t)wv;
          if (wd < ldXl / 4) *reinterpret_cast<uint32_t *>(xx + lb * tl.ldsXx + 4 * wd) = pay;
          else if (wd == ldXl / 4) rpx[lb].z = (int32_t)pay;
          else if (wd == ldXl / 4 + 1) rpx[lb].iqx = __uint_as_float(pay);
          else rpx[lb].sum = (int32_t)pay;
        }
        if (!__syncthreads_or(bad != 0)) break;
        if (tid == 0 && wait_expired(flag, it)) s_abort = 1;
        __syncthreads();
        if (s_abort) return false;
      }
      for (int lb = tid; lb < nb; lb += blockDim.x)
        rpx[lb] = row_param(rpx[lb].z, rpx[lb].iqx, rpx[lb].sum, (int)IN);
    }
    __syncthreads();

    products_mfma(xx, tl.ldsXx, 16, wx, tl.ldsWx, nrows, nrows, ldXl, Sx, nrows);
    __syncthreads();
    return true;
  };
  // Share of the codes of h_{t-1} (in xh / rph) by threads first, first +
  // stride, ...: this layer's output and, inside the launch, the next
  // layer's input (16-byte chunk c and tagged word w go to tile c % nut and
  // w % nut).
  const int chunks_out = (int)(Ly.out.ld / 16);
  const int mych = (chunks_out - tu + tl.nut - 1) / tl.nut;  // chunks tu, tu + nut, ...
  const int mywd = (tl.nw - tu + tl.nut - 1) / tl.nut;       // words tu, tu + nut, ...
  auto share_prev = [&](int64_t t, int first, int stride) {
    const int64_t row0 = (t - 1) * B + b0;
    const int me = tid - first;
    for (int idx = me; idx < nb * mych; idx += stride) {
      const int lb = idx / mych, ch = tu + (idx % mych) * tl.nut;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (ch * 16 < tl.ldH) v = *reinterpret_cast<const uint4 *>(xh + lb * tl.ldsX + ch * 16);
      *reinterpret_cast<uint4 *>(Ly.out.codes + (row0 + lb) * Ly.out.ld + ch * 16) = v;
    }
    if (tu == 0)
      for (int lb = me; lb < nb; lb += stride) {
        const int64_t row = row0 + lb;
        Ly.out.zero[row] = rph[lb].z;
        Ly.out.inv_q[row] = rph[lb].iqx;
        Ly.out.sums[row] = rph[lb].sum;
        if (Ly.tap_zero) Ly.tap_zero[row] = rph[lb].z;
        if (Ly.tap_inv_q) Ly.tap_inv_q[row] = rph[lb].iqx;
      }
    if (Ly.tap_codes && tu == 0)
      for (int idx = me; idx < nb * (int)H; idx += stride) {
        const int lb = idx / (int)H, k = idx % (int)H;
        Ly.tap_codes[(row0 + lb) * H + k] = xh[lb * tl.ldsX + k];
      }
    if (l + 1 < a.nl) {
      // tagged words for the next layer: 4 codes per word, then z, inv_q, sum
      uint64_t *ct = ctag(l);
      for (int idx = me; idx < nb * mywd; idx += stride) {
        const int lb = idx / mywd, wd = tu + (idx % mywd) * tl.nut;
        uint32_t pay;
        if (wd < tl.ldH / 4) pay = *reinterpret_cast<const uint32_t *>(xh + lb * tl.ldsX + 4 * wd);
        else if (wd == tl.ldH / 4) pay = (uint32_t)rph[lb].z;
        else if (wd == tl.ldH / 4 + 1) pay = __float_as_uint(rph[lb].iqx);
        else pay = (uint32_t)rph[lb].sum;
        __hip_atomic_store(ct + (row0 + lb) * tl.nw + wd, ((uint64_t)t << 32) | pay,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  };

  // Input side of step t for waves 2..: the codes of x_t straight into
  // registers (plain input, or layer l-1's tagged words re-read until their
  // tags match), their products against the resident W_x' slice into Sx,
  // and the row params into rpx; no workgroup barrier inside.  False if a
  // wait expired.  One batch row; its ld of at most 512 codes is two 16-byte
  // chunks per lane of a 16-lane group.
  auto input_side_async = [&](int64_t t) -> bool {
    const int gt = tid - 2 * kWave, grp = gt >> 4, gl = gt & 15;
    const int ngrp = ((int)blockDim.x - 2 * kWave) >> 4;
    const int64_t xrow = t * B + b0;
    v4i xa[2] = {v4i{}, v4i{}};
    bool ok = true;
    if (l == 0) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int k = gl * 16 + c * 256;
        if (k < ldXl) xa[c] = *reinterpret_cast<const v4i *>(Ly.xin.codes + xrow * Ly.xin.ld + k);
      }
      if (gt == 0)
        rpx[0] = row_param(Ly.xin.zero[xrow], Ly.xin.inv_q[xrow], Ly.xin.sums[xrow], (int)IN);
    } else {
      const int nwx = ldXl / 4 + 3;  // layer l-1's row: its ldH == ldXl here
      const uint64_t *ct = ctag(l - 1) + xrow * nwx;
      const uint32_t tag = (uint32_t)(t + 1);
      uint32_t pz = 0, pq = 0, ps = 0;
      long it = 0;
      for (;;) {
        uint32_t bad = 0;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int k = gl * 16 + c * 256;
          if (k < ldXl) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint64_t w = ld_tagged(ct + k / 4 + e);
              bad |= (uint32_t)(w >> 32) ^ tag;
              xa[c][e] = (int)(uint32_t)w;
            }
          }
        }
        if (gt == 0) {
          const uint64_t w0 = ld_tagged(ct + ldXl / 4), w1 = ld_tagged(ct + ldXl / 4 + 1),
                         w2 = ld_tagged(ct + ldXl / 4 + 2);
          bad |= ((uint32_t)(w0 >> 32) ^ tag) | ((uint32_t)(w1 >> 32) ^ tag) |
                 ((uint32_t)(w2 >> 32) ^ tag);
          pz = (uint32_t)w0;
          pq = (uint32_t)w1;
          ps = (uint32_t)w2;
        }
        if (bad == 0) break;
        if (wait_expired(flag, it)) {
          ok = false;
          break;
        }
      }
      if (gt == 0 && ok) rpx[0] = row_param((int32_t)pz, __uint_as_float(pq), (int32_t)ps, (int)IN);
    }
    for (int n = grp; n < nrows; n += ngrp) {
      const int8_t *wr = wx + n * tl.ldsWx;
      int acc = 0;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int k = gl * 16 + c * 256;
        if (k < ldXl) {
          const v4i b = *reinterpret_cast<const v4i *>(wr + k);
          acc = __builtin_amdgcn_sdot4(xa[c].x, b.x, acc, false);
          acc = __builtin_amdgcn_sdot4(xa[c].y, b.y, acc, false);
          acc = __builtin_amdgcn_sdot4(xa[c].z, b.z, acc, false);
          acc = __builtin_amdgcn_sdot4(xa[c].w, b.w, acc, false);
        }
      }
      // sum over the group's 16 lanes (one DPP row)
      acc += __builtin_amdgcn_update_dpp(0, acc, 0x121, 0xf, 0xf, false);
      acc += __builtin_amdgcn_update_dpp(0, acc, 0x122, 0xf, 0xf, false);
      acc += __builtin_amdgcn_update_dpp(0, acc, 0x124, 0xf, 0xf, false);
      acc += __builtin_amdgcn_update_dpp(0, acc, 0x128, 0xf, 0xf, false);
      if (gl == 0) Sx[n] = acc;
    }
    return ok;
  };

  // Per step: the recurrent product and the gates (all waves); then, while
  // h_t travels, waves 0 and 1 quantize h_t into the other buffer of codes
  // and the other waves share the codes of h_{t-1} and form the input side of
  // step t+1.
  int8_t *const xhb[2] = {xh, reinterpret_cast<int8_t *>(smem + tl.off_xh2)};
  RowParam *const rphb[2] = {rph, reinterpret_cast<RowParam *>(smem + tl.off_rowh2)};
  if (tid < 16) s_xch[tid] = 0;  // flags hold step tags, which start at 1
  if (T > 0 && !input_side(0)) return;
  if (!quant_tile<NVA, RBA, kSrcPlain>(nb, rowsA, H, 0u, (int)H, xh, tl.ldsX, tl.ldH, flag, rph,
                                       h0_row))
    return;
  __syncthreads();
  const int wave = tid >> 6;
  for (int64_t t = 0; t < T; ++t) {
    const int64_t hcur = (t & 1) * B * H;
    xh = xhb[t & 1];
    rph = rphb[t & 1];

    // ---- 1. the recurrent product (the input side's is already in Sx)
    products_mfma(xh, tl.ldsX, 16, wh, tl.ldsW, nrows, nrows, tl.ldH, Sh, nrows);
    __syncthreads();
    if (TP && Ly.acc_x) tap_acc(Ly.acc_x, Sx, cpx, rpx, IN, t);
    if (TP && Ly.acc_h) tap_acc(Ly.acc_h, Sh, cph, rph, H, t);

    // ---- 2. recover, gates, cell; publish h_t
    gates(t, hcur);
    __syncthreads();  // Sx and Sh are free

    // ---- 3. while h_t travels: its codes (waves 0, 1); the share of the codes
    // of h_{t-1} and the input side of step t+1 (the other waves)
    if (wave < 2) {
      const uint64_t *cur = xht_mine + (t & 1) * B * H;
      if (!quant_row_2w(cur + b0 * H, (uint32_t)(t + 1), (int)H, xhb[(t + 1) & 1], tl.ldH, flag,
                        rphb[(t + 1) & 1], s_xch))
        s_abort = 1;
    } else {
      if (t > 0) share_prev(t, 2 * kWave, (int)blockDim.x - 2 * kWave);
      if (t + 1 < T && !input_side_async(t + 1)) s_abort = 1;
    }
    __syncthreads();
    if (s_abort) return;
  }
  // the codes of h_{T-1}
  xh = xhb[T & 1];
  rph = rphb[T & 1];
  share_prev(T, 0, (int)blockDim.x);
}

// ------------------------------------------------------------------ host side
// bB: batch rows per tile (1, or a multiple of 16 for the MFMA products).
static bool plan_stack_bb(const StackArgs &a, int cus, int lds_max, int bB, StackTiling *out) {
  StackTiling tl{};
  const int64_t B = a.B, H = a.H;
  // workgroups per layer: at one row per tile, half of the CUs' share: the
  // per-step exchange costs less with fewer readers than the extra cells per
  // tile cost (with dot-product gate rows, every layer on an XCD of its own:
  // 20, 25, 28 and 32 tiles gave 5.05, 4.88, 4.97 and 4.97 us per frame;
  // spread over all XCDs, 40%, 50%, 60% and 100% of the share gave 5.80,
  // 5.59, 5.68 and 6.54).  With MFMA gate rows a single batch row takes the
  // 16-cell tiling below instead.
  const int G = bB == 1 ? cus / a.nl / 2 : cus / a.nl;
  tl.ldH = (int)round_up(H, 64);
  int64_t maxin = 0;
  for (int l = 0; l < a.nl; ++l) maxin = std::max(maxin, a.L[l].in);
  tl.ldXmax = (int)round_up(maxin, 64);
  tl.ldsW = tl.ldH + 16;
  tl.ldsWx = tl.ldXmax + 16;
  tl.ldsX = tl.ldH + 16;
  tl.ldsXx = tl.ldXmax + 16;
  tl.bB = bB;
  tl.mfma = bB > 1;
  tl.nbt = (int)((B + bB - 1) / bB);
  if (tl.nbt > G || tl.nbt > kMaxSlices) return false;
  tl.nq = tl.mfma ? bB / 8 : 0;  // batched: quantizing workgroups of 8 rows each
  {
    const int nut = G / tl.nbt - tl.nq;
    if (nut < 1) return false;
    tl.u = (int)((H + nut - 1) / nut);
  }
  // one row with MFMA products: tiles of at least 16 cells over up to a whole
  // XCD per layer (five 500-cell layers: 32 tiles of 16 cells 4.39 us a frame,
  // 25 of 20 4.47, 21 of 24 4.44, 42 of 12 4.77; five 300-cell layers: 19 of
  // 16 4.04, 25 of 12 4.08), when every batch row's tiles still fit the
  // layer's share of the CUs (otherwise the half-share tiling above stands,
  // so that at 2..15 rows no layer drops out of the launch)
  if (bB == 1) {
    const int64_t u16 = std::max<int64_t>(16, (H + kXcdCus - 1) / kXcdCus);
    if (tl.nbt * ((H + u16 - 1) / u16) <= cus / a.nl) tl.u = (int)u16;
  }
  tl.u = (tl.u + 3) / 4 * 4;  // 4u gate rows a multiple of 16 (MFMA tiles)
  tl.nut = (int)((H + tl.u - 1) / tl.u);
  // the x-code prefetch holds 4 words of 8 codes per thread
  if (tl.ldH > 512 || (size_t)(tl.mfma ? bB : 0) * (tl.ldXmax / 8) > 4 * (size_t)kStackThreads)
    return false;
  if (!tl.mfma && tl.ldXmax > 512) return false;  // one-row input side: two 16-byte chunks per lane
  tl.gl = tl.nbt * (tl.nut + tl.nq);
  tl.grid = a.nl * tl.gl;
  if (tl.grid > cus) return false;
  // one-row tiles: each layer on an XCD of its own when its tiles fit one
  // (the h exchange then stays in that XCD's L2); the grid covers every CU.
  // Only on the whole chip (all eight XCDs, XCC_IDs 0..7): a partition of it
  // keeps the spread layout.
  tl.xcd = 0;
  if (bB == 1 && cus == kXcds * kXcdCus && a.nl <= kXcds && tl.gl <= kXcdCus) {
    tl.xcd = 1;
    tl.grid = cus;
  }
  const int nrows = 4 * tl.u;
  // LDS layout
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 16);
    return o;
  };
  tl.off_wh = take((size_t)nrows * tl.ldsW);
  tl.off_wx = take((size_t)nrows * tl.ldsWx);
  // one-row tiles keep their row of codes as row 0 of a 16-row block whose
  // other rows stay zero, so their products run on MFMA too
  const int rowsB = tl.mfma ? tl.bB : 16;
  tl.off_xh = take((size_t)rowsB * tl.ldsX);
  tl.off_xx = take((size_t)rowsB * tl.ldsXx);
  // batched tiles: the codes of x_t are consumed (their product formed)
  // before the recurrent product is written, so Sh may share their space
  tl.off_sh = tl.mfma && (size_t)nrows * 4 <= (size_t)tl.ldsXx ? tl.off_xx
                                                               : take((size_t)rowsB * nrows * 4);
  tl.off_sx = take((size_t)rowsB * nrows * 4);
  tl.off_c = take((size_t)tl.bB * tl.u * 4);
  tl.off_colh = take((size_t)nrows * sizeof(ColParam));
  tl.off_colx = take((size_t)nrows * sizeof(ColParam));
  tl.off_rowh = take((size_t)tl.bB * sizeof(RowParam));
  tl.off_rowx = take((size_t)tl.bB * sizeof(RowParam));
  tl.off_bias = take((size_t)nrows * 4);
  // one-row tiles make the codes of h_t while h_{t-1}'s are still being shared
  tl.off_xh2 = tl.mfma ? tl.off_xh : take((size_t)rowsB * tl.ldsX);
  tl.off_rowh2 = tl.mfma ? tl.off_rowh : take((size_t)tl.bB * sizeof(RowParam));
  tl.lds_bytes = off;
  if (tl.lds_bytes + 64 > (size_t)lds_max) return false;
  // exchange per layer
  tl.nw = tl.ldH / 4 + 3;
  if (B < 16) {
    tl.reph = std::max(1, std::min(kMaxReph, 2048 / std::max(1, tl.u)));
    tl.strideh = round_up(2 * B * H, 8192) + 512;
    tl.hx_bytes = (size_t)tl.reph * tl.strideh * 8;
    tl.cx_bytes = (size_t)a.T * B * tl.nw * 8;
  } else {
    tl.reph = 1;
    tl.strideh = 2 * B * H;
    tl.hx_bytes = align_up((size_t)2 * B * H * 8, 256);
    tl.cx_bytes = 0;
  }
  tl.layer_bytes = align_up(tl.hx_bytes + tl.cx_bytes, 256);
  *out = tl;
  return true;
}

// One batch row per tile below 16 rows; otherwise 16-row tiles, or 32-row
// tiles when 16-row tiles of this many layers do not fit the chip's LDS (a
// tile quantizes twice the rows per step, but all layers share one launch).
static bool plan_stack(const StackArgs &a, int cus, int lds_max, StackTiling *out) {
  if (a.B < 16) return plan_stack_bb(a, cus, lds_max, 1, out);
  if (plan_stack_bb(a, cus, lds_max, 16, out)) return true;
  return a.B >= 32 && plan_stack_bb(a, cus, lds_max, 32, out);
}

size_t stack_ws(int nl, int64_t T, int64_t B, int64_t H) {
  // same sizing as plan_stack's exchange, for any tiling
  const int64_t ldH = round_up(H, 64);
  size_t per;
  if (B < 16) {
    const int64_t strideh = round_up(2 * B * H, 8192) + 512;
    per = align_up((size_t)kMaxReph * strideh * 8 + (size_t)T * B * (ldH / 4 + 3) * 8, 256);
  } else {
    per = align_up(align_up((size_t)2 * B * H * 8, 256), 256);
  }
  return std::max(kHeaderBytes + (size_t)nl * kStackCounterBytes + (size_t)nl * per, xstack_ws(nl));
}

using StackKernel = void (*)(StackArgs, StackTiling);

int stack_layout(const StackArgs &a) {
  int dev = 0, cus = 0, lds_max = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return xstack_applies(a, cus, lds_max) ? 1 : 0;
}

hipError_t launch_stack(const StackArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0 || a.B == 0) return hipSuccess;
  if (a.nl < 1 || a.nl > kMaxStack || a.H > 512) {
    *unsupported = true;
    return hipSuccess;
  }
  int dev = 0, cus = 0, lds_max = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  bool tp = false;  // any tap or final state asked for
  for (int l = 0; l < a.nl; ++l) {
    const StackLayer &L = a.L[l];
    tp = tp || L.acc_x || L.acc_h || L.tap_gates || L.tap_c || L.tap_m || L.hT || L.cT;
  }
  // batch 16 to 64 on the whole chip: one XCD per layer
  bool done = false;
  e = launch_xstack(a, cus, lds_max, tp, s, &done);
  if (e != hipSuccess || done) return e;
  StackTiling tl;
  if (!plan_stack(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  StackKernel kern = tl.bB == 1 ? (tp ? k_stack<8, false, 1, true> : k_stack<8, false, 1, false>)
                                : (tp ? k_stack<8, true, 2, true> : k_stack<8, true, 2, false>);
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kStackThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  const int64_t n64 =
      (int64_t)(((size_t)a.nl * kStackCounterBytes + (size_t)a.nl * tl.layer_bytes) / 8);
  e = clear_exchange(a.ws, n64, s);
  if (e != hipSuccess) return e;
  StackArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(kern), dim3(tl.grid),
                                    dim3(kStackThreads), kargs, (unsigned)tl.lds_bytes, s);
}

// Layers per launch for a stack of n layers of width H at batch B: the most
// that fit the chip together (at least 1; 1 means "use the one-layer path").
int stack_layers_per_launch(int n, int64_t T, int64_t B, int64_t H, int64_t in0, int64_t in1) {
  int dev = 0, cus = 0, lds_max = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 1;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return 1;
  if (H > 512) return 1;
  for (int nl = std::min(n, kMaxStack); nl >= 2; --nl) {
    StackArgs a{};
    a.nl = nl;
    a.T = T;
    a.B = B;
    a.H = H;
    for (int l = 0; l < nl; ++l) a.L[l].in = l == 0 ? in0 : in1;
    StackTiling tl;
    if (plan_stack(a, cus, lds_max, &tl)) return nl;
  }
  return 1;
}

hipError_t set_wait_bound_stack(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
