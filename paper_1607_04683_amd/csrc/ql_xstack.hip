// ql_xstack.hip -- stacked LSTM layers without a projection (Section 4) at
// batch 16 .. 64 in one persistent launch over the whole chip, one XCD per
// layer, run as a wavefront: layer l works on frame t while layer l-1 is
// already further on.
//
// XCD l runs layer l for the whole sequence and the whole batch; its 32
// workgroups (one per CU; each reads its XCC_ID and takes the next free slot
// s of its XCD) are 2 row groups (half of the batch each) x 16 cell tiles (32
// cells each).  Every hand-off inside a layer stays in that XCD's L2: plain
// stores, device-coherent loads that find them there.  A tile keeps the 128
// gate rows of its cells of both W_x' and W_h' in registers as MFMA
// fragments, four cells (their gates i f g o adjacent) per 16-row block, so
// an MFMA result gives a lane the four gate sums of one (cell, row) pair, and
// c stays in that lane's registers.  A step t, for the tile's rows:
//   1. the codes of x_t (the launch's input, or the codes layer l-1 made of
//      its h_t, published across XCDs with an arrival counter) and their
//      product with W_x', recovered (eq. 1 / eq. 3) plus the bias, exactly
//      as the hoisted input product does;
//   2. the codes of h_{t-1} from the row group's 16 tiles (each encoded its
//      own cells, below); this tile's part of them also goes out, with the
//      row's params, as the layer's quantized output (which layer l+1 reads);
//   3. the product with W_h', recovered, + (W_x x + b), gates, c and h_t;
//   4. E1: the per-row min/max of h_t over the tile's cells, published; every
//      tile of the row group reads all 16 parts and forms the quantizer of
//      each row (eq. 2, fp64 params);
//   5. E2: each tile encodes its own cells of h_t and publishes the codes and
//      their per-row sums, which step t+1 reads (2).
// The output of step t goes out at step t+1, once the tile holds the row's
// whole code sum; layer l+1 then lags one step more, which costs latency,
// not throughput.  Exchanged words are 64-bit (step tag << 32 | payload) in
// a double buffer by step parity; a tile can only reuse a half after every
// tile of its row group has read it, since each hand-off needs the previous
// one from all of them.  Every wait is bounded: on expiry a flag in the
// workspace is raised and every workgroup leaves at its next wait.  The
// arithmetic is that of k_stack and the one-layer path, so the results are
// bit-identical to them.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"
#include "ql_rec_common.h"
#include "ql_xcd.h"

#include <algorithm>
#include <cstddef>

namespace ql {

constexpr int kXsThreads = 512;
constexpr int kXsWaves = kXsThreads / 64;
constexpr int kXsXcds = 8;      // XCDs of the MI355X, each with its own L2
constexpr int kXsSlots = 32;    // CUs (workgroups) of one XCD
constexpr int kXsGroups = 2;    // row groups of a layer
constexpr int kXsTiles = 16;    // cell tiles of a row group
constexpr int kXsCells = 32;    // cells of a tile: one 4-cell block per wave
constexpr int kXsMaxW = 512;    // widths (cells, input) the layout is sized for
constexpr int kXsSlotBytes = kXsXcds * 64;
constexpr int kXsCounterBytes = kMaxStack * 2 * kXsGroups * 64;  // [layer][parity][group]

struct XsTiling {
  int rows;          // batch rows per row group (the second may hold fewer)
  size_t lds_bytes;  // (host) dynamic LDS of the instance
  int64_t xwords;    // (host) exchange words per layer
};

// LDS and exchange layout of an instance (rows per group up to 16 NT).
template <int NT>
struct XsLay {
  static constexpr int bX = 16 * NT, u = kXsCells, uw = u / 4;
  static constexpr int ldsX = kXsMaxW + 16;  // row stride of the codes of x and of h
  static constexpr size_t xxb = (size_t)bX * ldsX;                             // one x buffer
  static constexpr size_t xx = 0;                                              // 2 x [bX][ldsX]
  static constexpr size_t xh = xal16(xx + 2 * xxb);                            // [bX][ldsX]
  static constexpr size_t cph = xal16(xh + (size_t)bX * ldsX);                 // [u][4]
  static constexpr size_t cpx = xal16(cph + (size_t)4 * u * sizeof(ColParam)); // [u][4]
  static constexpr size_t cf = xal16(cpx + (size_t)4 * u * sizeof(ColParam));  // 6 x [u] x 16
  static constexpr size_t bias = xal16(cf + (size_t)6 * u * 16);               // [u] float4
  static constexpr size_t rph = xal16(bias + (size_t)u * 16);                  // [bX]
  static constexpr size_t rpx = xal16(rph + (size_t)bX * sizeof(RowParam));    // 2 x [bX]
  static constexpr size_t hp = xal16(rpx + (size_t)2 * bX * sizeof(RowParam)); // [bX]
  static constexpr size_t pm = xal16(hp + (size_t)bX * sizeof(XParam));        // [bX][32][2]
  static constexpr size_t mcs = xal16(pm + (size_t)bX * 32 * 2 * 4);           // [bX][u]
  static constexpr size_t sum = xal16(mcs + (size_t)bX * u);                   // [bX][16]
  static constexpr size_t bytes = xal16(sum + (size_t)bX * kXsTiles * 4);
  // exchange words of one row group, one parity:
  //   E1  [bX][16 tiles][2]   min / max keys of h_t
  //   E2c [bX][16 tiles][uw]  codes of h_t, E2s [bX][16 tiles] their sums
  static constexpr int64_t e1 = 0;
  static constexpr int64_t e2c = e1 + (int64_t)bX * kXsTiles * 2;
  static constexpr int64_t e2s = e2c + (int64_t)bX * kXsTiles * uw;
  static constexpr int64_t gwords = (e2s + (int64_t)bX * kXsTiles + 31) / 32 * 32;
  static constexpr int64_t lwords = 2 * kXsGroups * gwords;  // a layer: 2 parities x 2 groups
};

struct XsKArgs {
  StackArgs a;
  XsTiling tl;
};
typedef const __attribute__((address_space(4))) XsKArgs *XsKArgPtr;

// What a workgroup derives from the launch's scalars and its role: stated
// once for the kernel, and again (through the kernel-argument pointer) on the
// rare output path of the step.  What the step needs on every step (the x
// and output addresses) is held in vector registers instead, so that no
// scalar reload sits on the step's chain.
#define XS_SCALARS(a, tl, role)                                                                 \
  const int l = (role) / kXsSlots, s = (role) % kXsSlots;                                      \
  const int g = s / kXsTiles, ct = s % kXsTiles;                                               \
  auto &Ly = a.L[l];                                                                           \
  const int64_t T = a.T, B = a.B, H = a.H, IN = Ly.in;                                         \
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;                                        \
  const int64_t b0 = (int64_t)g * tl.rows;                                                     \
  const int nb = (int)std::min<int64_t>((int64_t)tl.rows, B - b0);                             \
  const int64_t j0 = (int64_t)ct * u;                                                          \
  const int ldX = (int)((IN + 63) / 64 * 64), ldH = (int)((H + 63) / 64 * 64);                 \
  unsigned *cnt0 = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes +     \
                                                kXsSlotBytes);                                 \
  auto ctr = [&](int layer, int64_t par, int grp) {                                            \
    return cnt0 + ((layer * 2 + (int)par) * kXsGroups + grp) * 16;                             \
  };                                                                                           \
  uint64_t *X = reinterpret_cast<uint64_t *>(static_cast<char *>(a.ws) + kHeaderBytes +        \
                                             kXsSlotBytes + kXsCounterBytes) +                 \
                (int64_t)l * L::lwords;                                                        \
  auto E = [&](int64_t tt_) { return X + ((tt_ & 1) * kXsGroups + g) * L::gwords; };          \
  (void)T, (void)flag, (void)ldX, (void)ldH, (void)ctr, (void)E, (void)IN

template <int NT, bool TP>
__global__ __launch_bounds__(kXsThreads) void k_xstack(StackArgs a, XsTiling tl) {
  static_assert(offsetof(XsKArgs, tl) == sizeof(StackArgs), "argument layout");
  using L = XsLay<NT>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int s_abort, s_role;
  constexpr int bX = L::bX, u = L::u, uw = L::uw, ldsX = L::ldsX;

  if (threadIdx.x == 0) {
    const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
    unsigned *slots = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
    s_role = -1;
    s_abort = 0;
    if (xcc < a.nl) {
      const unsigned k = __hip_atomic_fetch_add(slots + xcc * 16, 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      if (k < (unsigned)kXsSlots) s_role = xcc * kXsSlots + (int)k;
    }
  }
  __syncthreads();
  const int role = __builtin_amdgcn_readfirstlane(s_role);
  if (role < 0) return;
  int8_t *xx = reinterpret_cast<int8_t *>(smem + L::xx);          // codes of x_t, by step parity
  int8_t *xh = reinterpret_cast<int8_t *>(smem + L::xh);          // codes of h_{t-1}
  ColParam *cph = reinterpret_cast<ColParam *>(smem + L::cph);    // [u][4] W_h' rows
  ColParam *cpx = reinterpret_cast<ColParam *>(smem + L::cpx);    // [u][4] W_x' rows
  // the same for the 24-bit recovery, four gates of a cell per vector (low 32
  // bits of colterm, shifted zero point, 1/Q), h side then x side
  int4 *ctmh = reinterpret_cast<int4 *>(smem + L::cf);
  int4 *czth = ctmh + u;
  float4 *ciqh = reinterpret_cast<float4 *>(czth + u);
  int4 *ctmx = reinterpret_cast<int4 *>(ciqh + u);
  int4 *cztx = ctmx + u;
  float4 *ciqx = reinterpret_cast<float4 *>(cztx + u);
  float4 *bias4 = reinterpret_cast<float4 *>(smem + L::bias);      // [u] gates i f g o
  RowParam *rph = reinterpret_cast<RowParam *>(smem + L::rph);    // rows of h_{t-1}
  RowParam *rpx = reinterpret_cast<RowParam *>(smem + L::rpx);    // rows of x_t, by step parity
  XParam *hp = reinterpret_cast<XParam *>(smem + L::hp);          // quantizer of each row of h_t
  int *pm = reinterpret_cast<int *>(smem + L::pm);                // min/max parts of h_t
  uint8_t *mcs = reinterpret_cast<uint8_t *>(smem + L::mcs);      // own cells' codes of h_t
  int *ssum = reinterpret_cast<int *>(smem + L::sum);             // polled code sums

  XS_SCALARS(a, tl, role);

  // ---- prologue: W_x', W_h' fragments, column params, bias, c_0
  const int tid0 = threadIdx.x, wave0 = tid0 >> 6, fr0 = tid0 & 15, fq0 = (tid0 & 63) >> 4;
  // block of wave w: cells 4w .. 4w+3; lane row fr is gate fr & 3 of cell fr >> 2
  v4i wh[8], wx[8];
  {
    const int jj = 4 * wave0 + (fr0 >> 2);
    const bool ok = j0 + jj < H;
    const int64_t n = (int64_t)(fr0 & 3) * H + j0 + jj;
    const int8_t *sh = Ly.Wh.codes + n * Ly.Wh.ld + 16 * fq0;
    const int8_t *sx = Ly.Wx.codes + n * Ly.Wx.ld + 16 * fq0;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      wh[c] = ok && c * 64 < ldH ? *reinterpret_cast<const v4i *>(sh + c * 64) : v4i{};
      wx[c] = ok && c * 64 < ldX ? *reinterpret_cast<const v4i *>(sx + c * 64) : v4i{};
    }
  }
  for (int r = tid0; r < 4 * u; r += kXsThreads) {
    const int jj = r >> 2, gate = r & 3;
    const int64_t n = (int64_t)gate * H + std::min<int64_t>(j0 + jj, H - 1);
    {
      const int64_t blk = n / Ly.Wh.rows_per_block;
      ColParam c;
      c.ztw = Ly.Wh.zero[blk] + 128;
      c.sigw = Ly.Wh.row_sums[n] - 128 * (int32_t)H;
      c.colterm = (int64_t)c.sigw + H * (int64_t)c.ztw;
      c.iqw = Ly.Wh.inv_q[blk];
      c.pad = 0;
      cph[r] = c;
      reinterpret_cast<int *>(ctmh + jj)[gate] = (int32_t)c.colterm;
      reinterpret_cast<int *>(czth + jj)[gate] = c.ztw;
      reinterpret_cast<float *>(ciqh + jj)[gate] = c.iqw;
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
      reinterpret_cast<int *>(ctmx + jj)[gate] = (int32_t)c.colterm;
      reinterpret_cast<int *>(cztx + jj)[gate] = c.ztw;
      reinterpret_cast<float *>(ciqx + jj)[gate] = c.iqw;
    }
    reinterpret_cast<float *>(bias4 + jj)[gate] = Ly.bias[n];
  }
  // the lane's (cell, row) pairs: cell 4 wave + fq, row 16 tt + fr
  float cst[NT];
#pragma unroll
  for (int tt = 0; tt < NT; ++tt) {
    const int64_t j = j0 + 4 * wave0 + fq0;
    const int lb = 16 * tt + fr0;
    cst[tt] = Ly.c0 && j < H && lb < nb ? Ly.c0[(b0 + lb) * H + j] : 0.0f;
  }
  __syncthreads();
  // whether the lane's cell allows the 24-bit recovery on every gate: bit 0
  // the recurrent side, bit 1 the input side
  int cfm = 0;
  {
    bool fh = true, fx = true;
#pragma unroll
    for (int gate = 0; gate < 4; ++gate) {
      const ColParam ch = cph[(4 * wave0 + fq0) * 4 + gate], cx = cpx[(4 * wave0 + fq0) * 4 + gate];
      fh = fh && fast_col(ch.ztw, ch.colterm);
      fx = fx && fast_col(cx.ztw, cx.colterm);
    }
    cfm = (fh ? 1 : 0) | (fx ? 2 : 0);
  }

  XsKArgPtr kp = (XsKArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
  // The codes of x_t (the launch's input, or layer l-1's output, once its
  // arrival counter says step t is complete) and the row params, in
  // registers: word i of a thread is row 8 i + tid / 64, 8-byte word tid % 64
  // (a row has at most 64).  park_x puts them into LDS.  Each wave waits for
  // the counter itself (no barrier), starting from a value `seen` it read
  // earlier (0: none), so that a count already reached costs no round trip;
  // if the wait expires it raises the abort, which the next check after a
  // barrier acts on, and its loads read whatever is there.
  uint64_t xv[bX / 8];
  int32_t xz = 0, xs = 0;
  float xq = 0.0f;
  // What load_x and park_x need, computed once and held in vector registers
  // (no scalar reloads on the step's critical path): bit i of xmask says
  // whether word i of this thread is a real code word, xmeta whether the
  // thread reads a row's params.
  const int xr0 = tid0 >> 6, xwd = tid0 & 63;
  uint32_t xmask = 0;
#pragma unroll
  for (int i = 0; i < bX / 8; ++i)
    if (8 * i + xr0 < nb && xwd < ldX / 8) xmask |= 1u << i;
  const bool xmeta = tid0 < nb;
  const char *xsrc0 = reinterpret_cast<const char *>(Ly.xin.codes + (b0 + xr0) * Ly.xin.ld + 8 * xwd);
  const int32_t *xzp = Ly.xin.zero + b0 + tid0;
  const float *xqp = Ly.xin.inv_q + b0 + tid0;
  const int32_t *xsp = Ly.xin.sums + b0 + tid0;
  int64_t xrow8 = 8 * Ly.xin.ld, xstep = B * Ly.xin.ld, xB = B;
  int xin_k = (int)IN;
  asm volatile("" : "+v"(xrow8), "+v"(xstep), "+v"(xB), "+v"(xin_k));
  const unsigned *cprev = l > 0 ? ctr(l - 1, 0, g) : nullptr;  // parity 1: + kXsGroups * 16
  auto load_x = [&](int64_t tx, unsigned seen) {
    if (cprev) {
      const unsigned *c = cprev + (tx & 1) * (kXsGroups * 16);
      const unsigned target = (unsigned)((tx >> 1) + 1) * kXsTiles;
      long it = 0;
      while (seen < target) {
        if (wait_expired(flag, it)) {
          s_abort = 1;
          break;
        }
        seen = __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    const char *src = xsrc0 + tx * xstep;
#pragma unroll
    for (int i = 0; i < bX / 8; ++i)
      xv[i] = (xmask >> i) & 1u ? ld_coherent64(reinterpret_cast<const uint64_t *>(src + i * xrow8)) : 0;
    if (xmeta) {
      const int64_t o = tx * xB;
      xz = ld_coherent_i(xzp + o);
      xq = ld_coherent(xqp + o);
      xs = ld_coherent_i(xsp + o);
    }
  };
  // into the LDS buffer of step parity par
  auto park_x = [&](int par) {
    int8_t *xd = xx + par * L::xxb;
#pragma unroll
    for (int i = 0; i < bX / 8; ++i)
      if ((xmask >> i) & 1u) *reinterpret_cast<uint64_t *>(xd + (8 * i + xr0) * ldsX + 8 * xwd) = xv[i];
    if (threadIdx.x < bX)
      rpx[par * bX + threadIdx.x] = xmeta ? row_param(xz, xq, xs, xin_k) : row_param(0, 0.0f, 0, xin_k);
  };
  // This tile's part of the layer's quantized output of step tx (codes of
  // its cells, from the codes of h_tx in LDS; tile 0 also the rows' z, 1/Q
  // and code sums from their row params), with device-coherent stores, for
  // layer l+1 on another XCD; taps of the codes.
  // What publish_out needs on every step, held in vector registers like the
  // above: this thread's word of 4 codes (row tid / 8, word tid % 8 of the
  // tile's 32 cells) and, in tile 0, its row's params.
  const int orw = tid0 >> 3, oww = tid0 & 7;
  const bool ocode = orw < nb && j0 + 4 * oww < ldH;
  const int oxh = orw * ldsX + (int)j0 + 4 * oww;
  uint32_t *ocp = reinterpret_cast<uint32_t *>(Ly.out.codes + (b0 + orw) * Ly.out.ld + j0) + oww;
  int64_t ostep = B * Ly.out.ld / 4;  // 4-byte words from frame t to t + 1
  asm volatile("" : "+v"(ostep));
  const bool ometa = ct == 0 && tid0 < nb;
  int32_t *ozp = Ly.out.zero + b0 + tid0;
  float *oqp = Ly.out.inv_q + b0 + tid0;
  int32_t *osp = Ly.out.sums + b0 + tid0;
  // (the last tile zeroes the rows' padding up to the output's stride; taps)
  const bool orare = (ct == kXsTiles - 1 && Ly.out.ld > ldH) || Ly.tap_codes || Ly.tap_zero ||
                     Ly.tap_inv_q;
  // This tile's part of the layer's quantized output of step tx (codes of
  // its cells, from the codes of h_tx in LDS; tile 0 also the rows' z, 1/Q
  // and code sums from their row params), with device-coherent stores, for
  // layer l+1 on another XCD; taps of the codes.
  auto publish_out = [&](int64_t tx) {
    if (ometa) {
      const RowParam r = rph[threadIdx.x];
      const int64_t o = tx * xB;
      st_coherent_i(ozp + o, r.z);
      st_coherent(oqp + o, r.iqx);
      st_coherent_i(osp + o, r.sum);
    }
    if (ocode)
      __hip_atomic_store(ocp + tx * ostep, *reinterpret_cast<const uint32_t *>(xh + oxh),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (orare) {
      auto &a = kp->a;
      auto &tl = kp->tl;
      XS_SCALARS(a, tl, role);
      const int tid = threadIdx.x;
      const int64_t orow0 = tx * B + b0;
      if (ct == 0 && tid < nb) {
        const RowParam r = rph[tid];
        if (Ly.tap_zero) Ly.tap_zero[orow0 + tid] = r.z;
        if (Ly.tap_inv_q) Ly.tap_inv_q[orow0 + tid] = r.iqx;
      }
      if (ct == kXsTiles - 1)
        for (int idx = tid; idx < nb * (int)((Ly.out.ld - ldH) / 4); idx += kXsThreads) {
          const int nw = (int)((Ly.out.ld - ldH) / 4), r2 = idx / nw, w2 = idx % nw;
          __hip_atomic_store(reinterpret_cast<uint32_t *>(Ly.out.codes + (orow0 + r2) * Ly.out.ld + ldH) + w2,
                             0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      if (Ly.tap_codes)
        for (int idx = tid; idx < nb * u; idx += kXsThreads) {
          const int r2 = idx / u, k = idx % u;
          if (j0 + k < H) Ly.tap_codes[(orow0 + r2) * H + j0 + k] = xh[r2 * ldsX + j0 + k];
        }
    }
  };
  float *hout = Ly.h;
  asm volatile("" : "+v"(hout));
  // the weight fragments have landed before the loop (no wait for them in it);
  // x_0 goes to LDS, x_1 into registers
  wait_vmcnt0();
  load_x(0, 0u);
  park_x(0);
  if (T > 1) load_x(1, 0u);
  __syncthreads();
  for (int64_t t = 0;; ++t) {
    int tid = (int)threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = tid >> 6, fr = lane & 15, fq = lane >> 4;
    const int jjL = 4 * wave + fq;  // the lane's cell (tile-local)
    const int64_t jL = j0 + jjL;
    // ---- 0. the first round of the poll for the codes of h_{t-1} (E2 of step
    // t-1), issued now and examined after step 1: word i of a thread is row
    // 4 i + tid / 128, word tid % 128 (a row has at most 128); sums of (row
    // tid / 16, tile tid % 16)
    constexpr int CW = bX / 4;
    constexpr int rs4 = 4 * kXsTiles * uw, ls4 = 4 * ldsX;
    const uint64_t *e2 = E(t - 1);
    const uint64_t *e2c = e2 + L::e2c, *e2s = e2 + L::e2s;
    auto e2src = [&](int i, int th) -> const uint64_t * {
      return i < CW ? e2c + i * rs4 + (th >> 7) * (rs4 / 4) + (th & 127) : e2s + th;
    };
    auto e2dst = [&](int i, int th) -> uint32_t * {
      return reinterpret_cast<uint32_t *>(i < CW ? xh + i * ls4 + (th >> 7) * ldsX + 4 * (th & 127)
                                                 : (int8_t *)(ssum + th));
    };
    uint32_t need = 0;
    uint64_t w2[CW + 1];
    if (t > 0) {
      const int cw = ldH / 4;
#pragma unroll
      for (int k = 0; k < CW; ++k)
        if (4 * k + (tid >> 7) < nb && (tid & 127) < cw) need |= 1u << k;
      if (tid < nb * kXsTiles) need |= 1u << CW;
      poll_to_lds_issue<CW + 1>(need, e2src, w2);
    }

    // ---- 1. W_x' x_t, recovered (eq. 1 / eq. 3) plus the bias, as the
    // hoisted input product forms it.  x_t has been in LDS since the step
    // before, so this runs while the codes of h_{t-1} are on their way.  All
    // 8 chunks of 64 columns, without a branch, so that the LDS reads of a
    // chunk overlap the MFMAs of the one before: chunks past the padded
    // width multiply zero weight fragments with whatever their LDS bytes
    // hold, which adds exactly nothing to an integer sum.
    float xb[NT][4];
    if (t < T) {
      const int8_t *xxt = xx + (t & 1) * L::xxb;
      const RowParam *rpxt = rpx + (t & 1) * bX;
      v4i accx[NT];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) accx[tt] = v4i{};
#pragma unroll
      for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
          accx[tt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
              wx[c], *reinterpret_cast<const v4i *>(xxt + (16 * tt + fr) * ldsX + c * 64 + 16 * fq),
              accx[tt], 0, 0, 0);
      // the MFMA results are read by ordinary instructions below: at least 19
      // wait states after the last pass, which the hardware does not check
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(accx[0]), "+v"(accx[NT - 1]));
      const int4 cthx = ctmx[jjL], czx = cztx[jjL];
      const float4 cix = ciqx[jjL], b4 = bias4[jjL];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int lb = 16 * tt + fr;
        const RowParam rx = rpxt[lb];
        float yx[4];
        yx[0] = recover_fast(accx[tt][0], cthx.x, czx.x, rx.ztx, rx.sigx, cix.x, rx.iqx);
        yx[1] = recover_fast(accx[tt][1], cthx.y, czx.y, rx.ztx, rx.sigx, cix.y, rx.iqx);
        yx[2] = recover_fast(accx[tt][2], cthx.z, czx.z, rx.ztx, rx.sigx, cix.z, rx.iqx);
        yx[3] = recover_fast(accx[tt][3], cthx.w, czx.w, rx.ztx, rx.sigx, cix.w, rx.iqx);
        // the exact form where a zero point or column term rules the 24-bit
        // one out (rare), in a branch the wave takes only then
        const bool fastx = (cfm & 2) && fast_row(rx.ztx);
        if (__any(!fastx) && !fastx)
#pragma unroll
          for (int gate = 0; gate < 4; ++gate) {
            const ColParam c = cpx[jjL * 4 + gate];
            yx[gate] = recover(accx[tt][gate], c.colterm, c.ztw, rx.ztx, rx.sigx, c.iqw, rx.iqx);
          }
        xb[tt][0] = yx[0] + b4.x;
        xb[tt][1] = yx[1] + b4.y;
        xb[tt][2] = yx[2] + b4.z;
        xb[tt][3] = yx[3] + b4.w;
        if (TP && Ly.acc_x && jL < H && lb < nb)
#pragma unroll
          for (int gate = 0; gate < 4; ++gate)
            Ly.acc_x[((t * B + b0 + lb) * 4 + gate) * H + jL] =
                acc_u8(accx[tt][gate], cpx[jjL * 4 + gate].sigw, rx.sigx, IN);
      }
    }

    // ---- 2. the codes of h_{t-1} from the row group's 16 tiles
    if (t == 0) {
      if (!quant_tile<8, 2, kSrcPlain>(nb, bX, H, 0u, (int)H, xh, ldsX, ldH, flag, rph,
                                       [&](int lb) -> const void * {
                                         return Ly.h0 ? Ly.h0 + (b0 + lb) * H : nullptr;
                                       }))
        s_abort = 1;
    } else {
      if (!poll_to_lds_finish<CW + 1>(need, (uint32_t)t, w2, e2src, e2dst, flag)) s_abort = 1;
    }
    // (on both paths: nothing of the step's first round stays in flight)
    wait_vmcnt0();
    // the arrival count of x_{t+2}, read now so that it is in hand when its
    // loads are issued (step 8)
    unsigned seen = 0;
    if (l > 0 && t + 2 < T)
      seen = __hip_atomic_load(ctr(l - 1, (t + 2) & 1, g), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (s_abort) return;
    // the row params of h_{t-1}: the quantizer of step t-1 and the row's code
    // sum over the 16 tiles (formed while the MFMAs of step 3 run)
    auto build_rph = [&]() {
      const int row = tid >> 4, og = tid & 15;
      const int total = red16(row < nb ? ssum[row * kXsTiles + og] : 0, AddI{});
      if (row < nb && og == 0) {
        const XParam xp = hp[row];
        rph[row] = row_param(xp.z, xp.inv_q, total, (int)H);
      }
    };
    if (t == T) {
      build_rph();
      // the last step's output, and the arrival once its stores have completed
      __syncthreads();
      publish_out(t - 1);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0)
        __hip_atomic_fetch_add(ctr(l, (t - 1) & 1, g), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }

    // ---- 3. W_h' h_{t-1}
    v4i acch[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) acch[tt] = v4i{};
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
        acch[tt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
            wh[c], *reinterpret_cast<const v4i *>(xh + (16 * tt + fr) * ldsX + c * 64 + 16 * fq),
            acch[tt], 0, 0, 0);
    if (t > 0) build_rph();
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acch[0]), "+v"(acch[NT - 1]));
    __syncthreads();  // the row params of h_{t-1} are in LDS
    // this tile's part of the layer's quantized output of step t-1, across
    // XCDs: its stores complete while the gates are computed
    if (t > 0) publish_out(t - 1);

    // ---- 4. recovery of W_h' h_{t-1}, + (W_x x + b), gates, c and h_t
    float hv[NT];
    {
      const int4 cth = ctmh[jjL], czh = czth[jjL];
      const float4 cih = ciqh[jjL];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int lb = 16 * tt + fr;
        const int64_t brow = b0 + lb;
        const RowParam r = rph[lb];
        float y[4];
        y[0] = recover_fast(acch[tt][0], cth.x, czh.x, r.ztx, r.sigx, cih.x, r.iqx);
        y[1] = recover_fast(acch[tt][1], cth.y, czh.y, r.ztx, r.sigx, cih.y, r.iqx);
        y[2] = recover_fast(acch[tt][2], cth.z, czh.z, r.ztx, r.sigx, cih.z, r.iqx);
        y[3] = recover_fast(acch[tt][3], cth.w, czh.w, r.ztx, r.sigx, cih.w, r.iqx);
        const bool fasth = (cfm & 1) && fast_row(r.ztx);
        if (__any(!fasth) && !fasth)
#pragma unroll
          for (int gate = 0; gate < 4; ++gate) {
            const ColParam c = cph[jjL * 4 + gate];
            y[gate] = recover(acch[tt][gate], c.colterm, c.ztw, r.ztx, r.sigx, c.iqw, r.iqx);
          }
        float gv[4];
#pragma unroll
        for (int gate = 0; gate < 4; ++gate) {
          const float av = xb[tt][gate] + y[gate];
          const float sg = sigmoid_cw(gate == 2 ? 2.0f * av : av);
          gv[gate] = gate == 2 ? 2.0f * sg - 1.0f : sg;
        }
        const float cn = (gv[1] * cst[tt]) + (gv[0] * gv[2]);
        cst[tt] = cn;
        const float m = gv[3] * tanh_cw(cn);
        hv[tt] = m;
        if (jL < H && lb < nb) {
          if (hout) hout[(t * B + brow) * H + jL] = m;
          if (TP) {
            if (Ly.acc_h)
#pragma unroll
              for (int gate = 0; gate < 4; ++gate)
                Ly.acc_h[((t * B + brow) * 4 + gate) * H + jL] =
                    acc_u8(acch[tt][gate], cph[jjL * 4 + gate].sigw, r.sigx, H);
            if (Ly.tap_gates) {
              float *gp = Ly.tap_gates + (t * B + brow) * 4 * H + jL;
              gp[0] = gv[0], gp[H] = gv[1], gp[2 * H] = gv[2], gp[3 * H] = gv[3];
            }
            if (Ly.tap_c) Ly.tap_c[(t * B + brow) * H + jL] = cn;
            if (Ly.tap_m) Ly.tap_m[(t * B + brow) * H + jL] = m;
            if (t == T - 1) {
              if (Ly.hT) Ly.hT[brow * H + jL] = m;
              if (Ly.cT) Ly.cT[brow * H + jL] = cn;
            }
          }
        }
      }
    }

    // ---- 5. E1: min/max of h_t per row over the tile's cells
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      int lo = 0x7fffffff, hi = 0x7fffffff;
      if (jL < H) {
        const int key = float_key(hv[tt]);
        lo = key;
        hi = ~key;
      }
      int *d = pm + ((16 * tt + fr) * 32 + wave * 4 + fq) * 2;
      d[0] = lo;
      d[1] = hi;
    }
    __syncthreads();
    uint64_t *e = E(t);
    const uint32_t tag = (uint32_t)(t + 1);
    {
      // 16 lanes per row, two of the row's 32 (wave, lane group) parts each
      const int row = tid >> 4, j = tid & 15;
      int lo = 0x7fffffff, hi = 0x7fffffff;
      if (row < bX) {
        const int *q = pm + (row * 32 + 2 * j) * 2;
        lo = min(q[0], q[2]);
        hi = min(q[1], q[3]);
      }
      lo = red16(lo, MinI{});
      hi = red16(hi, MinI{});
      if (row < nb && j == 0) {
        put_word(e + L::e1 + (row * kXsTiles + ct) * 2, tag, (uint32_t)lo);
        put_word(e + L::e1 + (row * kXsTiles + ct) * 2 + 1, tag, (uint32_t)hi);
      }
    }
    {
      // every row's params from the 16 tiles' parts: 16 lanes per row, one
      // tile's (min, max) words each
      const int row = tid >> 4, j = tid & 15;
      uint32_t v[2] = {0u, 0u};
      const uint32_t need = row < nb ? 3u : 0u;
      const uint64_t *e1 = e + L::e1 + (row * kXsTiles + j) * 2;
      uint64_t w1[2] = {0, 0};
      if (need) {
        w1[0] = ld_tagged(e1);
        w1[1] = ld_tagged(e1 + 1);
      }
      // ---- 6. x_{t+1} (loaded a step ago) into the LDS buffer of the next
      // step, while these loads are in flight
      if (t + 1 < T) park_x((int)((t + 1) & 1));
      uint32_t left = need;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (((left >> i) & 1u) && (uint32_t)(w1[i] >> 32) == tag) {
          v[i] = (uint32_t)w1[i];
          left &= ~(1u << i);
        }
      bool ok = true;
      if (__any(left != 0))
        ok = poll_words<2>(left, tag, v, [&](int i) -> const uint64_t * { return e1 + i; }, flag);
      if (!ok) s_abort = 1;
      int lo = red16(need ? (int)v[0] : 0x7fffffff, MinI{});
      int hi = red16(need ? (int)v[1] : 0x7fffffff, MinI{});
      if (row < nb && j == 0 && ok) {
        const QParams prm = make_qparams(key_float(lo), key_float(~hi));
        XParam xp;
        xp.q = prm.q;
        xp.z = prm.z;
        xp.inv_q = prm.inv_q;
        hp[row] = xp;
      }
    }
    // every memory operation so far has completed (the output stores of step
    // t-1 among them)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (s_abort) return;

    // ---- 7. E2: the tile's cells of h_t encoded (eq. 2), with per-row sums
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      const int lb = 16 * tt + fr;
      if (lb < nb) {
        int code = 128;  // device byte 0: cells past H add nothing to a product
        if (jL < H) code = encode(hv[tt], hp[lb].q, hp[lb].z);
        mcs[lb * u + jjL] = (uint8_t)(code ^ 0x80);
      }
    }
    __syncthreads();
    {
      // 8 lanes per row (aligned), one word of four codes each
      const int row = tid >> 3, wd = tid & 7;
      int sum = 0;
      if (row < nb) {
        const uint32_t word = *reinterpret_cast<const uint32_t *>(mcs + row * u + 4 * wd);
        put_word(e + L::e2c + (int64_t)row * (kXsTiles * uw) + ct * uw + wd, tag, word);
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (j0 + 4 * wd + k < H) sum += (int)((word >> (8 * k)) & 0xffu) ^ 0x80;
      }
      sum = red8(sum, AddI{});
      if (row < nb && wd == 0) put_word(e + L::e2s + row * kXsTiles + ct, tag, (uint32_t)sum);
    }
    // ---- 8. the loads of x_{t+2} issued, to land during the next step; then
    // the arrival that tells layer l+1 step t-1 is out
    if (t + 2 < T) load_x(t + 2, seen);
    if (t > 0 && tid == 0)
      __hip_atomic_fetch_add(ctr(l, (t - 1) & 1, g), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ------------------------------------------------------------------ host side
size_t xstack_ws(int nl) {
  return kHeaderBytes + kXsSlotBytes + kXsCounterBytes + (size_t)nl * XsLay<2>::lwords * 8;
}

static bool plan_xstack(const StackArgs &a, int cus, int lds_max, XsTiling *out) {
  if (cus != kXsXcds * kXsSlots || a.nl < 2 || a.nl > kXsXcds) return false;
  if (a.B < 16 || a.B > kXsGroups * 32 || a.H > kXsTiles * kXsCells) return false;
  XsTiling tl{};
  tl.rows = (int)((a.B + kXsGroups - 1) / kXsGroups);
  const int64_t ldH = round_up(a.H, 64);
  for (int l = 0; l < a.nl; ++l) {
    const StackLayer &L = a.L[l];
    if (L.in > kXsMaxW || L.Wx.ld < round_up(L.in, 64) || L.Wh.ld < ldH) return false;
    if (L.out.ld < ldH || L.out.ld % 4) return false;
  }
  tl.lds_bytes = tl.rows <= 16 ? XsLay<1>::bytes : XsLay<2>::bytes;
  tl.xwords = XsLay<2>::lwords;
  if (tl.lds_bytes + 64 > (size_t)lds_max) return false;
  *out = tl;
  return true;
}

using XsKernel = void (*)(StackArgs, XsTiling);

bool xstack_applies(const StackArgs &a, int cus, int lds_max) {
  XsTiling tl;
  return plan_xstack(a, cus, lds_max, &tl);
}

hipError_t launch_xstack(const StackArgs &a, int cus, int lds_max, bool taps, hipStream_t s,
                         bool *done) {
  *done = false;
  XsTiling tl;
  if (!plan_xstack(a, cus, lds_max, &tl)) return hipSuccess;
  XsKernel kern = tl.rows <= 16 ? (taps ? k_xstack<1, true> : k_xstack<1, false>)
                                : (taps ? k_xstack<2, true> : k_xstack<2, false>);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kXsThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu < 1) return hipSuccess;
  e = clear_exchange(a.ws, (kXsSlotBytes + kXsCounterBytes) / 8 + (int64_t)a.nl * tl.xwords, s);
  if (e != hipSuccess) return e;
  StackArgs args = a;
  void *kargs[] = {&args, &tl};
  e = hipLaunchCooperativeKernel(reinterpret_cast<void *>(kern), dim3(cus), dim3(kXsThreads), kargs,
                                 (unsigned)tl.lds_bytes, s);
  if (e == hipSuccess) *done = true;
  return e;
}

hipError_t set_wait_bound_xstack(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
