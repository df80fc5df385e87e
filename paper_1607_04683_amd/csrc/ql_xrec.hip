// ql_xrec.hip -- a quantized LSTM layer with a projection (Section 4, the
// LSTMP layer: m_t = o tanh(c_t), h_t = W_r m_t) at batch 16 .. 256, one
// persistent launch over the whole chip laid out by XCD.
//
// The batch rows of a layer are independent of one another, so the batch is
// split over the eight XCDs: XCD x owns rows [x rows, (x + 1) rows) of the
// batch for the whole sequence, and its 32 workgroups (one per CU; each reads
// its XCC_ID and takes the next free slot s of its XCD) never exchange a value
// with another XCD.  Every hand-off of a step then stays in that XCD's L2:
// values go out with plain stores and are read with device-coherent loads,
// which find them there.  Slot s plays two tiles:
//   * a unit tile: cells [s u, (s + 1) u) of every row of the XCD.  Its 4u
//     gate rows of W_h' stay in registers as MFMA fragments for the launch,
//     four cells (their 16 gate rows, gates i f g o of a cell adjacent) per
//     fragment block, so an MFMA result gives a lane the four gates of one
//     (cell, row) pair and c stays in that lane's registers;
//   * a projection tile: outputs [o pw, (o + 1) pw) of row group g (half of
//     the XCD's rows), with (g, o) = (s / 16, s % 16); its rows of W_r' stay
//     in registers too, K split over the eight waves.
// A step t, for the XCD's rows:
//   1. the codes of h_{t-1} (quantized per vector, eq. 2) and their row
//      params, from the projection tiles (E4 below); at t = 0 every tile
//      quantizes h_0 itself;
//   2. Mult against W_h', R(.) of eq. 1 / eq. 3, + (W_x x + b) (the hoisted
//      input product, staged through LDS), gates, c and m;
//   3. E1: per-row min/max of m over the tile's cells, published; every tile
//      reads all of them and forms the quantizer params of every row of m;
//   4. E2: each unit tile encodes its own cells of m (eq. 2) and publishes the
//      codes with their per-row code sums; each projection tile reads the
//      codes of its rows;
//   5. Mult against W_r' and R(.) give h_t; E3: per-row min/max of h_t over
//      the tile's outputs, published; the row group's tiles read them and
//      form the params of h_t;
//   6. E4: each projection tile encodes its outputs of h_t and publishes the
//      codes, code sums and (output group 0) the row's zero point and
//      recovery factor; they are the layer's quantized output too.
// Every value a step needs from another tile of the XCD is one of these four
// hand-offs, each a single round trip through L2.  Exchanged words are 64-bit
// (step tag << 32 | 32-bit payload) in a double buffer indexed by step
// parity; a consumer re-reads the words it needs until every tag matches.
// A buffer half is reused two steps later, and a tile can only reach that
// point after every tile of its XCD has read the step in between (each hand-off
// needs the previous one from every tile of the XCD), so nothing is
// overwritten before it is read.  Every wait is bounded: on expiry a flag in
// the workspace is raised and every workgroup leaves at its next wait.
// The arithmetic (quantizer, recovery, gate functions, their operand order)
// is that of the other recurrent kernels, so the results are bit-identical.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"
#include "ql_rec_common.h"
#include "ql_xcd.h"

#include <algorithm>
#include <cstddef>

namespace ql {

constexpr int kXrecThreads = 512;
constexpr int kXrecWaves = kXrecThreads / 64;
constexpr int kXrecXcds = 8;     // XCDs of the MI355X, each with its own L2
constexpr int kXrecSlots = 32;   // CUs (workgroups) of one XCD
constexpr int kXrecGroups = 2;   // projection row groups per XCD
constexpr int kXrecOuts = 16;    // projection output groups per row group
constexpr int kXrecOutBlocks = 2;  // 16-output MFMA blocks of a projection tile (pw <= 32)
constexpr int kXrecSlotBytes = kXrecXcds * 64;  // slot counters after the header
// batches below this keep the spread layout of k_recurrent
constexpr int64_t kXrecMinBatch = 16;

struct XrecTiling {
  int rows;      // batch rows per XCD (the last XCDs may hold fewer)
  int bX;        // rows padded to MFMA tiles: 16 * NT
  int u;         // cells per unit tile: 32 * NBW
  int ldR, ldH;  // padded widths of the codes of h (K of W_h') and of m (K of W_r')
  int ksw;       // 64-byte K chunks of W_r' per wave
  size_t lds_bytes;  // (host) dynamic LDS of the instance
  int64_t xwords;    // (host) exchange words per XCD
};

// Widths the layout is sized for: h up to 512 values (16 projection tiles of
// 32 outputs), m up to 2048.
constexpr int kXrecMaxR = 512, kXrecMaxH = 2048, kXrecMaxPw = 32;

// The LDS and exchange layout of an instance, fixed at compile time (the
// widths of a layer only bound the loops): every offset is an immediate.
template <int NBW, int NT>
struct XLay {
  static constexpr int bX = 16 * NT, u = 32 * NBW, uw = u / 4, rg = bX / kXrecGroups;
  static constexpr int ldsX = kXrecMaxR + 16;    // row stride of the codes of h
  static constexpr int ldsM = kXrecMaxH + 16;    // row stride of the codes of m
  static constexpr int gxr = 4 * u + 4;          // row stride (floats) of W_x x + b
  static constexpr int e4rw = kXrecOuts * kXrecMaxPw / 4;  // code words of a row of h
  static constexpr int nsum = bX * kXrecOuts > rg * kXrecSlots ? bX * kXrecOuts : rg * kXrecSlots;
  // LDS byte offsets
  static constexpr size_t xc = 0;                                               // [bX][ldsX]
  static constexpr size_t gx = xal16(xc + (size_t)bX * ldsX);                   // [2][bX][gxr]
  static constexpr size_t cp = xal16(gx + (size_t)2 * bX * gxr * 4);            // [u][4]
  static constexpr size_t cf = xal16(cp + (size_t)4 * u * sizeof(ColParam));    // 3 x [u] x 16
  static constexpr size_t rp = xal16(cf + (size_t)3 * u * 16);                  // [bX]
  static constexpr size_t mp = xal16(rp + (size_t)bX * sizeof(RowParam));       // [bX]
  static constexpr size_t pm = xal16(mp + (size_t)bX * sizeof(XParam));         // [bX][32][2]
  static constexpr size_t mcs = xal16(pm + (size_t)bX * 32 * 2 * 4);            // [bX][u]
  static constexpr size_t mc = xal16(mcs + (size_t)bX * u);                     // [rg][ldsM]
  static constexpr size_t red = xal16(mc + (size_t)rg * ldsM);                  // [waves][pw][rg]
  static constexpr size_t rpp = xal16(red + (size_t)kXrecWaves * kXrecMaxPw * rg * 4);
  static constexpr size_t hp = xal16(rpp + (size_t)rg * sizeof(RowParam));      // [rg]
  static constexpr size_t hcs = xal16(hp + (size_t)rg * sizeof(XParam));        // [rg][pw]
  static constexpr size_t sum = xal16(hcs + (size_t)rg * kXrecMaxPw);           // [nsum]
  static constexpr size_t par = xal16(sum + (size_t)nsum * 4);                  // [bX][2]
  static constexpr size_t bytes = xal16(par + (size_t)bX * 2 * 4);
  // exchange word offsets inside one parity of an XCD's area:
  //   E1  [bX][32 tiles][2]   min / max keys of m_t
  //   E2c [bX][32 tiles][uw]  codes of m_t, E2s [bX][32 tiles] their sums
  //   E3  [bX][16 groups][2]  min / max keys of h_t
  //   E4c [bX][e4rw]          codes of h_t, E4s [bX][16 groups] their sums,
  //   E4p [bX][2]             zero point and recovery factor of h_t
  static constexpr int64_t e1 = 0;
  static constexpr int64_t e2c = e1 + (int64_t)bX * kXrecSlots * 2;
  static constexpr int64_t e2s = e2c + (int64_t)bX * kXrecSlots * uw;
  static constexpr int64_t e3 = e2s + (int64_t)bX * kXrecSlots;
  static constexpr int64_t e4c = e3 + (int64_t)bX * kXrecOuts * 2;
  static constexpr int64_t e4s = e4c + (int64_t)bX * e4rw;
  static constexpr int64_t e4p = e4s + (int64_t)bX * kXrecOuts;
  static constexpr int64_t pwords = (e4p + (int64_t)bX * 2 + 31) / 32 * 32;  // parities 256 B apart
  static constexpr int64_t xwords = 2 * pwords;
};


// NBW: fragment blocks (four cells each) per wave, u = 32 NBW cells a unit
// tile; NT: 16-row MFMA tiles of the XCD's rows; TP: the launch writes taps.
// What a workgroup derives from the launch's scalars and its role: its rows,
// cells, projection tile and exchange area.  The kernel states it once for
// the prologue and again at the top of every step, reading the arguments
// through a pointer the compiler cannot follow across steps, so that none of
// these values (nor anything computed from them) stays live across the loop:
// kept live, they overflow the scalar registers.
#define XREC_SCALARS(a, tl, role)                                                               \
  const int64_t T = a.T, B = a.B, H = a.H, P = a.P, R = a.R;                                   \
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;                                        \
  const int x = (role) / kXrecSlots, s = (role) % kXrecSlots;                                  \
  const int64_t xb0 = (int64_t)x * tl.rows; /* the XCD's first batch row */                    \
  const int nbx = (int)std::min<int64_t>((int64_t)tl.rows, B - xb0);                           \
  const int64_t j0 = (int64_t)s * u;                                                           \
  const int ldR = tl.ldR, ldH = tl.ldH;                                                        \
  constexpr int pw = kXrecMaxPw; /* outputs per projection tile */                             \
  const int g = s / kXrecOuts, o = s % kXrecOuts;                                              \
  const int prow0 = g * rg; /* the row group's first row (XCD-local) */                        \
  const int nrg = std::max(0, std::min(rg, nbx - prow0));                                      \
  const int64_t p0 = (int64_t)o * pw;                                                          \
  uint64_t *X = reinterpret_cast<uint64_t *>(static_cast<char *>(a.ws) + kHeaderBytes +        \
                                             kXrecSlotBytes) + (int64_t)x * L::xwords;         \
  auto E = [&](int64_t tt_) { return X + (tt_ & 1) * L::pwords; };                             \
  (void)T, (void)P, (void)R, (void)flag, (void)nbx, (void)ldR, (void)ldH, (void)nrg, (void)p0, \
      (void)E, (void)g, (void)o

// The kernel's arguments as laid out in its argument segment.
struct XrecKArgs {
  RecurrentArgs a;
  XrecTiling tl;
};
typedef const __attribute__((address_space(4))) XrecKArgs *KArgPtr;

template <int NBW, int NT, bool TP>
__global__ __launch_bounds__(kXrecThreads) void k_xrec(RecurrentArgs a, XrecTiling tl) {
  static_assert(offsetof(XrecKArgs, tl) == sizeof(RecurrentArgs), "argument layout");
  using L = XLay<NBW, NT>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int s_abort, s_role;
  constexpr int bX = 16 * NT, u = 32 * NBW, uw = u / 4;  // uw: code words of a row per unit tile

  if (threadIdx.x == 0) {
    const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
    unsigned *slots = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
    s_role = -1;
    s_abort = 0;
    if (xcc < kXrecXcds) {
      const unsigned k = __hip_atomic_fetch_add(slots + xcc * 16, 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      if (k < (unsigned)kXrecSlots) s_role = xcc * kXrecSlots + (int)k;
    }
  }
  __syncthreads();
  const int role = __builtin_amdgcn_readfirstlane(s_role);
  if (role < 0) return;
  int8_t *xc = reinterpret_cast<int8_t *>(smem + L::xc);        // codes of h_{t-1}
  float *gxs = reinterpret_cast<float *>(smem + L::gx);         // W_x x + b, [row][gate][u]
  ColParam *cp = reinterpret_cast<ColParam *>(smem + L::cp);    // [u][4] gate rows of W_h'
  // the same for the 24-bit recovery, four gates of a cell per vector:
  // low 32 bits of colterm, shifted zero point, 1/Q
  int4 *ctm = reinterpret_cast<int4 *>(smem + L::cf);
  int4 *czt = ctm + u;
  float4 *ciq = reinterpret_cast<float4 *>(czt + u);
  RowParam *rp = reinterpret_cast<RowParam *>(smem + L::rp);   // rows of h_{t-1}
  XParam *mp = reinterpret_cast<XParam *>(smem + L::mp);       // quantizer of each row of m_t
  int *pm = reinterpret_cast<int *>(smem + L::pm);             // min/max parts of m_t
  uint8_t *mcs = reinterpret_cast<uint8_t *>(smem + L::mcs);   // own cells' codes of m_t
  int8_t *mc = reinterpret_cast<int8_t *>(smem + L::mc);       // the row group's codes of m_t
  int32_t *red = reinterpret_cast<int32_t *>(smem + L::red);   // the waves' partial products
  RowParam *rpp = reinterpret_cast<RowParam *>(smem + L::rpp); // the row group's rows of m_t
  XParam *hp = reinterpret_cast<XParam *>(smem + L::hp);       // quantizer of h_t
  uint8_t *hcs = reinterpret_cast<uint8_t *>(smem + L::hcs);   // own outputs' codes of h_t
  int *ssum = reinterpret_cast<int *>(smem + L::sum);          // code sums of polled words
  int *spar = reinterpret_cast<int *>(smem + L::par);          // z, 1/Q of h_{t-1}
  constexpr int ldsX = L::ldsX, ldsM = L::ldsM;
  constexpr int rg = L::rg;
  XREC_SCALARS(a, tl, role);
  if (nbx <= 0) return;  // no rows: the whole XCD leaves

  // ---- prologue: W_h' and W_r' fragments, column params, c_0
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, fr = lane & 15, fq = lane >> 4;
  // W_h' block b of wave w (cells 4 (w NBW + b) .. +3): lane row fr is gate
  // fr & 3 of cell fr >> 2; 16 bytes 16 fq of each 64-byte chunk of K
  v4i wh[NBW][8];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const int jj = 4 * (wave * NBW + b) + (fr >> 2);
    const bool ok = j0 + jj < H;
    const int8_t *src = a.Wh.codes + ((int64_t)(fr & 3) * H + j0 + jj) * a.Wh.ld + 16 * fq;
#pragma unroll
    for (int c = 0; c < 8; ++c)
      wh[b][c] = ok && c * 64 < ldR ? *reinterpret_cast<const v4i *>(src + c * 64) : v4i{};
  }
  // W_r' output block nb of the tile: lane row fr is output p0 + 16 nb + fr;
  // this wave's K chunks wave * ksw + ks
  v4i wr[kXrecOutBlocks][4];
#pragma unroll
  for (int nb = 0; nb < kXrecOutBlocks; ++nb)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int64_t p = p0 + 16 * nb + fr;
      const int c = wave * tl.ksw + ks;
      wr[nb][ks] = v4i{};
      if (16 * nb < pw && ks < tl.ksw && p < P && c * 64 < ldH)
        wr[nb][ks] = *reinterpret_cast<const v4i *>(a.Wr.codes + p * a.Wr.ld + c * 64 + 16 * fq);
    }
  for (int r = tid; r < 4 * u; r += kXrecThreads) {
    const int jj = r >> 2, gate = r & 3;
    const int64_t n = (int64_t)gate * H + std::min<int64_t>(j0 + jj, H - 1);
    const int64_t blk = n / a.Wh.rows_per_block;
    ColParam c;
    c.ztw = a.Wh.zero[blk] + 128;
    c.sigw = a.Wh.row_sums[n] - 128 * (int32_t)R;
    c.colterm = (int64_t)c.sigw + R * (int64_t)c.ztw;
    c.iqw = a.Wh.inv_q[blk];
    c.pad = 0;
    cp[r] = c;
    reinterpret_cast<int *>(ctm + jj)[gate] = (int32_t)c.colterm;
    reinterpret_cast<int *>(czt + jj)[gate] = c.ztw;
    reinterpret_cast<float *>(ciq + jj)[gate] = c.iqw;
  }
  // the lane's (cell, row) pairs: block b, row tile tt -> cell
  // 4 (wave NBW + b) + fq, row 16 tt + fr
  float cst[NBW][NT];
#pragma unroll
  for (int b = 0; b < NBW; ++b)
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      const int64_t j = j0 + 4 * (wave * NBW + b) + fq, lb = 16 * tt + fr;
      cst[b][tt] = a.c0 && j < H && lb < nbx ? a.c0[(xb0 + lb) * H + j] : 0.0f;
    }
  // the projection lane (row tid / pw, output tid % pw): column params of its
  // W_r' row
  int32_t r_ztw = 0, r_sigw = 0;
  int64_t r_colterm = 0;
  float r_iqw = 0.0f;
  {
    const int64_t pc = std::min<int64_t>(p0 + tid % pw, P - 1);
    const int64_t blk = pc / a.Wr.rows_per_block;
    r_ztw = a.Wr.zero[blk] + 128;
    r_sigw = a.Wr.row_sums[pc] - 128 * (int32_t)H;
    r_colterm = (int64_t)r_sigw + H * (int64_t)r_ztw;
    r_iqw = a.Wr.inv_q[blk];
  }
  __syncthreads();
  // blocks b whose four gate rows of this lane's cell allow the 24-bit recovery
  int cfm = 0;
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    bool f = true;
#pragma unroll
    for (int gate = 0; gate < 4; ++gate) {
      const ColParam c = cp[(4 * (wave * NBW + b) + fq) * 4 + gate];
      f = f && fast_col(c.ztw, c.colterm);
    }
    cfm |= f ? 1 << b : 0;
  }

  // the arguments where the launch put them (the kernel argument segment:
  // scalar loads)
  KArgPtr kp = (KArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
  for (int64_t t = 0;; ++t) {
    // the launch's scalars and the per-thread indices re-derived every step
    // (an opaque argument pointer, an opaque thread id), so that the compiler
    // keeps none of them alive across the loop
    asm volatile("" : "+s"(kp));
    auto &a = kp->a;
    auto &tl = kp->tl;
    XREC_SCALARS(a, tl, role);
    int tid = (int)threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = tid >> 6, fr = lane & 15, fq = lane >> 4;
    auto jjOf = [&](int b) { return 4 * (wave * NBW + b) + fq; };
    auto rowOf = [&](int tt) { return 16 * tt + fr; };
    const int lr = tid / pw, pp = tid % pw;
    const int64_t pout = p0 + pp;
    const bool plane = lr < rg;
    // ---- W_x x + b of step tt straight into LDS buffer tt & 1, [row][gate][u]
    // with rows 4u + 4 floats apart: one 16-byte load per lane, one row (4
    // gates x u cells) per wave instruction (u = 32: the first 32 lanes).
    // Step t + 1's is issued as soon as step t's codes of h_{t-1} are in:
    // loads complete in order, so issued at the top of a step it would hold
    // up that step's first poll.  (Issued later in the step, before a poll
    // or before the gates, it measured slower: its latency, about 2 us under
    // this load, then falls on that phase.)
    auto load_gx = [&](int64_t tt) {
      if (tt < T && (u == 64 || lane < 32)) {
        const int gate = lane / uw, c4 = lane % uw;
        const int64_t jc = j0 + 4 * c4 < H ? j0 + 4 * c4 : 0;  // past H: any cell in bounds
        float *buf = gxs + (tt & 1) * (bX * L::gxr);
        for (int row = wave; row < nbx; row += kXrecWaves)
          __builtin_amdgcn_global_load_lds(a.gx + ((tt * B + xb0 + row) * 4 * H + gate * H + jc),
                                           (lds_ptr)(buf + row * L::gxr), 16, 0, 0);
      }
    };
    if (t == 0) load_gx(0);
    // ---- 1. the codes of h_{t-1} and their row params
    if (t == 0) {
      if (!quant_tile<8, 2, kSrcPlain>(nbx, bX, R, 0u, (int)R, xc, ldsX, ldR, flag, rp,
                                       [&](int lb) -> const void * {
                                         return a.h0 ? a.h0 + (xb0 + lb) * R : nullptr;
                                       }))
        s_abort = 1;
    } else {
      // E4 of step t - 1: code words into xc; per (row, output group) the code
      // sum, and the row's z and 1/Q, into LDS
      // word i of a thread: row 4 i + th / 128, word th % 128 of it (a row
      // has at most 128), no division; the bases once per step
      const uint64_t *e4 = E(t - 1);
      const uint64_t *e4c = e4 + L::e4c, *e4s = e4 + L::e4s, *e4p = e4 + L::e4p;
      const int cwr = ldR / 4;
      constexpr int rs4 = 4 * L::e4rw, ls4 = 4 * ldsX;
      constexpr int CW = bX / 4;
      uint32_t need = 0;
#pragma unroll
      for (int k = 0; k < CW; ++k)
        if (4 * k + (tid >> 7) < nbx && (tid & 127) < cwr) need |= 1u << k;
      if (tid < nbx * kXrecOuts) need |= 1u << CW;  // sum of (row tid / 16, group tid % 16)
      if (tid < nbx * 2) need |= 1u << (CW + 1);    // z (even tid) or 1/Q of row tid / 2
      if (!poll_to_lds<CW + 2>(
              need, (uint32_t)t,
              [&](int i, int th) -> const uint64_t * {
                if (i < CW) return e4c + i * rs4 + (th >> 7) * (rs4 / 4) + (th & 127);
                return (i == CW ? e4s : e4p) + th;
              },
              [&](int i, int th) -> uint32_t * {
                if (i < CW)
                  return reinterpret_cast<uint32_t *>(xc + i * ls4 + (th >> 7) * ldsX + 4 * (th & 127));
                return reinterpret_cast<uint32_t *>(i == CW ? ssum + th : spar + th);
              },
              flag))
        s_abort = 1;
    }
    wait_vmcnt0();  // the direct loads of W_x x + b have landed in LDS
    __syncthreads();
    if (s_abort) return;
    if (t > 0) {
      // the row's code sum over its 16 output groups: 16 lanes per row
      const int row = tid >> 4, og = tid & 15;
      const int total = red16(row < nbx ? ssum[row * kXrecOuts + og] : 0, AddI{});
      if (row < nbx && og == 0) {
        rp[row] = row_param(spar[2 * row], __int_as_float(spar[2 * row + 1]), total, (int)R);
        if (s == 0) a.out_sums[(t - 1) * B + xb0 + row] = total;
      }
    }
    if (t == T) break;  // step T only collects the last step's code sums
    // W_x x + b of the next step, into the other buffer
    load_gx(t + 1);

    // ---- 2. Mult against the resident W_h' fragments: block b, row tile tt
    v4i acc[NBW][NT];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) acc[b][tt] = v4i{};
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if (c * 64 >= ldR) break;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const v4i bx = *reinterpret_cast<const v4i *>(xc + rowOf(tt) * ldsX + c * 64 + 16 * fq);
#pragma unroll
        for (int b = 0; b < NBW; ++b)
          acc[b][tt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wh[b][c], bx, acc[b][tt], 0, 0, 0);
      }
    }
    // the MFMA results are read by ordinary instructions below: at least 19
    // wait states after the last pass, which the hardware does not check
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc[0][0]));
    __syncthreads();  // the row params of h_{t-1} are in LDS

    // ---- recover (eq. 1 / eq. 3), + W_x x + b, gates, c and m
    float mv[NBW][NT];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int jj = jjOf(b), lb = rowOf(tt);
        const int64_t j = j0 + jj, brow = xb0 + lb;
        const RowParam r = rp[lb];
        // recovery: the 24-bit form straight through; where a zero point or
        // column term rules it out (rare), the exact form, in a branch the
        // wave takes only then
        const int4 ct = ctm[jj], cz = czt[jj];
        const float4 ci = ciq[jj];
        float yh[4];
        yh[0] = recover_fast(acc[b][tt][0], ct.x, cz.x, r.ztx, r.sigx, ci.x, r.iqx);
        yh[1] = recover_fast(acc[b][tt][1], ct.y, cz.y, r.ztx, r.sigx, ci.y, r.iqx);
        yh[2] = recover_fast(acc[b][tt][2], ct.z, cz.z, r.ztx, r.sigx, ci.z, r.iqx);
        yh[3] = recover_fast(acc[b][tt][3], ct.w, cz.w, r.ztx, r.sigx, ci.w, r.iqx);
        const bool fast = ((cfm >> b) & 1) && fast_row(r.ztx);
        if (__any(!fast)) {
          if (!fast)
#pragma unroll
            for (int gate = 0; gate < 4; ++gate) {
              const ColParam c = cp[jj * 4 + gate];
              yh[gate] = recover(acc[b][tt][gate], c.colterm, c.ztw, r.ztx, r.sigx, c.iqw, r.iqx);
            }
        }
        float gv[4];
#pragma unroll
        for (int gate = 0; gate < 4; ++gate) {
          const float av = gxs[(t & 1) * (bX * L::gxr) + lb * L::gxr + gate * u + jj] + yh[gate];
          const float sg = sigmoid_cw(gate == 2 ? 2.0f * av : av);
          gv[gate] = gate == 2 ? 2.0f * sg - 1.0f : sg;
          if (TP && a.acc_h && j < H && lb < nbx)
            a.acc_h[(t * B + brow) * 4 * H + gate * H + j] =
                acc_u8(acc[b][tt][gate], cp[jj * 4 + gate].sigw, r.sigx, R);
        }
        const float cn = (gv[1] * cst[b][tt]) + (gv[0] * gv[2]);
        cst[b][tt] = cn;
        const float m = gv[3] * tanh_cw(cn);
        mv[b][tt] = m;
        if (j < H && lb < nbx) {
          if (TP) {
            if (a.tap_gates) {
              float *gp = a.tap_gates + (t * B + brow) * 4 * H + j;
              gp[0] = gv[0], gp[H] = gv[1], gp[2 * H] = gv[2], gp[3 * H] = gv[3];
            }
            if (a.tap_c) a.tap_c[(t * B + brow) * H + j] = cn;
            if (a.tap_m) a.tap_m[(t * B + brow) * H + j] = m;
          }
          if (t == T - 1 && a.cT) a.cT[brow * H + j] = cn;
        }
      }

    // ---- 3. E1: min/max of m per row over the tile's cells
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      int lo = 0x7fffffff, hi = 0x7fffffff;
#pragma unroll
      for (int b = 0; b < NBW; ++b)
        if (j0 + jjOf(b) < H) {
          const int key = float_key(mv[b][tt]);
          lo = min(lo, key);
          hi = min(hi, ~key);
        }
      int *d = pm + (rowOf(tt) * 32 + wave * 4 + fq) * 2;
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
      if (row < nbx && j == 0) {
        put_word(e + L::e1 + (row * kXrecSlots + s) * 2, tag, (uint32_t)lo);
        put_word(e + L::e1 + (row * kXrecSlots + s) * 2 + 1, tag, (uint32_t)hi);
      }
    }
    // every row's params from the 32 tiles' parts: 16 lanes per row, two
    // tiles' (min, max) words each
    {
      const int row = tid >> 4, j = tid & 15;
      uint32_t v[4];
      const uint32_t need = row < nbx ? 0xfu : 0u;
      const uint64_t *e1 = e + L::e1 + (row * kXrecSlots + 2 * j) * 2;  // 4 consecutive words
      const bool ok = poll_words<4>(need, tag, v, [&](int i) -> const uint64_t * { return e1 + i; },
                                    flag);
      if (!ok) s_abort = 1;
      int lo = need ? min((int)v[0], (int)v[2]) : 0x7fffffff;
      int hi = need ? min((int)v[1], (int)v[3]) : 0x7fffffff;
      lo = red16(lo, MinI{});
      hi = red16(hi, MinI{});
      if (row < nbx && j == 0 && ok) {
        const QParams prm = make_qparams(key_float(lo), key_float(~hi));
        XParam xp;
        xp.q = prm.q;
        xp.z = prm.z;
        xp.inv_q = prm.inv_q;
        mp[row] = xp;
      }
    }
    __syncthreads();
    if (s_abort) return;

    // ---- 4. E2: the tile's cells of m encoded (eq. 2), with per-row code sums
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int jj = jjOf(b), lb = rowOf(tt);
        if (lb < nbx) {
          int code = 128;  // device byte 0: cells past H add nothing to a product
          if (j0 + jj < H) code = encode(mv[b][tt], mp[lb].q, mp[lb].z);
          mcs[lb * u + jj] = (uint8_t)(code ^ 0x80);
        }
      }
    __syncthreads();
    {
      // uw lanes per row (8 or 16, aligned), one word of four codes each
      const int row = tid / uw, wd = tid % uw;
      int sum = 0;
      if (row < nbx) {
        const uint32_t word = *reinterpret_cast<const uint32_t *>(mcs + row * u + 4 * wd);
        put_word(e + L::e2c + (int64_t)row * (kXrecSlots * uw) + s * uw + wd, tag, word);
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (j0 + 4 * wd + k < H) sum += (int)((word >> (8 * k)) & 0xffu) ^ 0x80;
      }
      sum = uw == 16 ? red16(sum, AddI{}) : red8(sum, AddI{});
      if (row < nbx && wd == 0) put_word(e + L::e2s + row * kXrecSlots + s, tag, (uint32_t)sum);
    }

    // ---- 5. the projection tile: the codes of m_t of its rows, Mult against
    // W_r', recovery of h_t
    float hv = 0.0f;
    if (nrg > 0) {
      // word i of a thread: row i of the group, word th of it (a row has at
      // most 512), no division; the bases once per step
      const int cwm = ldH / 4;  // code words of a row of m
      constexpr int CW = bX / kXrecGroups;
      const uint64_t *e2c = e + L::e2c + (int64_t)prow0 * (kXrecSlots * uw);
      const uint64_t *e2s = e + L::e2s + prow0 * kXrecSlots;
      uint32_t need = 0;
#pragma unroll
      for (int k = 0; k < CW; ++k)
        if (k < nrg && tid < cwm) need |= 1u << k;
      if (tid < nrg * kXrecSlots) need |= 1u << CW;  // sum of (row tid / 32, tile tid % 32)
      if (!poll_to_lds<CW + 1>(
              need, tag,
              [&](int i, int th) -> const uint64_t * {
                return i < CW ? e2c + i * (kXrecSlots * uw) + th : e2s + th;
              },
              [&](int i, int th) -> uint32_t * {
                return reinterpret_cast<uint32_t *>(i < CW ? mc + i * ldsM + 4 * th : (int8_t *)(ssum + th));
              },
              flag))
        s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      {
        // the row's code sum over the 32 unit tiles: 16 lanes per row, two each
        const int row = tid >> 4, j = tid & 15;
        const int sum = red16(row < nrg ? ssum[row * kXrecSlots + 2 * j] +
                                              ssum[row * kXrecSlots + 2 * j + 1]
                                        : 0,
                              AddI{});
        if (row < nrg && j == 0) {
          const XParam xp = mp[prow0 + row];
          rpp[row] = row_param(xp.z, xp.inv_q, sum, (int)H);
        }
      }
      __syncthreads();
      // this wave's K chunks against every output block; rows past the group
      // read zeros
      v4i accp[kXrecOutBlocks] = {v4i{}, v4i{}};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = wave * tl.ksw + ks;
        if (ks >= tl.ksw || c * 64 >= ldH) break;
        const v4i bm = fr < nrg ? *reinterpret_cast<const v4i *>(mc + fr * ldsM + c * 64 + 16 * fq)
                                : v4i{};
#pragma unroll
        for (int nb = 0; nb < kXrecOutBlocks; ++nb)
          if (16 * nb < pw) accp[nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wr[nb][ks], bm, accp[nb], 0, 0, 0);
      }
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(accp[0]));
      if (fr < rg)
#pragma unroll
        for (int nb = 0; nb < kXrecOutBlocks; ++nb)
          if (16 * nb < pw)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              red[(wave * pw + 16 * nb + 4 * fq + r) * rg + fr] = accp[nb][r];
      __syncthreads();
      const bool valid = plane && lr < nrg && pout < P;
      if (plane) {
        int32_t pv[kXrecWaves];
#pragma unroll
        for (int w = 0; w < kXrecWaves; ++w) pv[w] = red[(w * pw + pp) * rg + lr];
        int32_t sv = 0;
#pragma unroll
        for (int w = 0; w < kXrecWaves; ++w) sv += pv[w];
        const RowParam r = rpp[lr < nrg ? lr : 0];
        hv = recover(sv, r_colterm, r_ztw, r.ztx, r.sigx, r_iqw, r.iqx);
        if (valid) {
          const int64_t brow = xb0 + prow0 + lr;
          a.h[(t * B + brow) * P + pout] = hv;
          if (t == T - 1 && a.hT) a.hT[brow * P + pout] = hv;
          if (TP && a.acc_r) a.acc_r[(t * B + brow) * P + pout] = acc_u8(sv, r_sigw, r.sigx, H);
        }
      }
      // E3: min/max of h_t per row over the tile's outputs
      int lo = 0x7fffffff, hi = 0x7fffffff;
      if (valid) {
        const int key = float_key(hv);
        lo = key;
        hi = ~key;
      }
      lo = red_w(lo, pw, MinI{});
      hi = red_w(hi, pw, MinI{});
      if (plane && lr < nrg && pp == 0) {
        put_word(e + L::e3 + ((prow0 + lr) * kXrecOuts + o) * 2, tag, (uint32_t)lo);
        put_word(e + L::e3 + ((prow0 + lr) * kXrecOuts + o) * 2 + 1, tag, (uint32_t)hi);
      }
      // ---- 6. the row group's params of h_t (16 lanes per row, one output
      // group's words each), then E4
      {
        const int row = tid >> 4, og = tid & 15;
        uint32_t w2[2];
        const uint32_t need3 = row < nrg ? 3u : 0u;
        const uint64_t *e3 = e + L::e3 + ((prow0 + row) * kXrecOuts + og) * 2;
        const bool ok3 = poll_words<2>(need3, tag, w2, [&](int i) -> const uint64_t * { return e3 + i; },
                                       flag);
        if (!ok3) s_abort = 1;
        const int l2 = red16(need3 ? (int)w2[0] : 0x7fffffff, MinI{});
        const int h2 = red16(need3 ? (int)w2[1] : 0x7fffffff, MinI{});
        if (row < nrg && og == 0 && ok3) {
          const QParams prm = make_qparams(key_float(l2), key_float(~h2));
          XParam xp;
          xp.q = prm.q;
          xp.z = prm.z;
          xp.inv_q = prm.inv_q;
          hp[row] = xp;
        }
      }
      __syncthreads();
      if (s_abort) return;
      int code = 0;
      if (plane && lr < nrg) {
        const XParam xp = hp[lr];
        code = valid ? encode(hv, xp.q, xp.z) : 128;  // outputs past P: device byte 0
        hcs[lr * pw + pp] = (uint8_t)(code ^ 0x80);
        const int64_t orow = t * B + xb0 + prow0 + lr;
        if (TP && a.tap_codes && valid) a.tap_codes[orow * R + pout] = (int8_t)(code ^ 0x80);
        if (pp == 0 && o == 0) {
          a.out_zero[orow] = xp.z;
          a.out_inv_q[orow] = xp.inv_q;
          if (TP && a.tap_zero) a.tap_zero[orow] = xp.z;
          if (TP && a.tap_inv_q) a.tap_inv_q[orow] = xp.inv_q;
        }
      }
      const int csum = red_w(valid ? code : 0, pw, AddI{});
      if (plane && lr < nrg && pp == 0) {
        const int row = prow0 + lr;
        put_word(e + L::e4s + row * kXrecOuts + o, tag, (uint32_t)csum);
        if (o == 0) {
          put_word(e + L::e4p + row * 2, tag, (uint32_t)hp[lr].z);
          put_word(e + L::e4p + row * 2 + 1, tag, __float_as_uint(hp[lr].inv_q));
        }
      }
      __syncthreads();
      {
        const int pw4 = pw / 4, row = tid / pw4, wd = tid % pw4;
        if (row < nrg) {
          const uint32_t word = *reinterpret_cast<const uint32_t *>(hcs + row * pw + 4 * wd);
          put_word(e + L::e4c + (int64_t)(prow0 + row) * L::e4rw + o * pw4 + wd, tag, word);
          const int64_t orow = t * B + xb0 + prow0 + row, k = p0 + 4 * wd;
          if (k < a.ld_out) *reinterpret_cast<uint32_t *>(a.out_codes + orow * a.ld_out + k) = word;
        }
        // the output rows' padding past the last group (wider layouts only)
        if (o == kXrecOuts - 1)
          for (int idx = tid; idx < nrg * (int)((a.ld_out - kXrecOuts * pw) / 4); idx += kXrecThreads) {
            const int nw = (int)((a.ld_out - kXrecOuts * pw) / 4), row = idx / nw, wd = idx % nw;
            *reinterpret_cast<uint32_t *>(a.out_codes + (t * B + xb0 + prow0 + row) * a.ld_out +
                                          kXrecOuts * pw + 4 * wd) = 0u;
          }
      }
    }
  }
}

// ------------------------------------------------------------------ host side
static bool plan_xrec(const RecurrentArgs &a, int cus, int lds_max, XrecTiling *out) {
  const int64_t B = a.B, H = a.H, P = a.P;
  if (P <= 0 || a.R != P || cus != kXrecXcds * kXrecSlots) return false;
  if (B < kXrecMinBatch || B > kXrecXcds * 32 || H > kXrecMaxH || H % 4 || P > kXrecMaxR)
    return false;
  XrecTiling tl{};
  tl.rows = (int)((B + kXrecXcds - 1) / kXrecXcds);
  tl.bX = tl.rows <= 16 ? 16 : 32;
  tl.u = H <= 1024 ? 32 : 64;
  tl.ldR = (int)round_up(P, 64);
  tl.ldH = (int)round_up(H, 64);
  tl.ksw = (tl.ldH / 64 + kXrecWaves - 1) / kXrecWaves;
  if (tl.ksw > 4 || tl.u * kXrecSlots < H) return false;
  if (a.Wh.ld < tl.ldR || a.Wr.ld < tl.ldH) return false;
  if (a.ld_out < tl.ldR || a.ld_out % 4) return false;
  const int nbw = tl.u / 32, nt = tl.bX / 16;
  tl.lds_bytes = nbw == 1 ? (nt == 1 ? XLay<1, 1>::bytes : XLay<1, 2>::bytes)
                          : (nt == 1 ? XLay<2, 1>::bytes : XLay<2, 2>::bytes);
  tl.xwords = nbw == 1 ? (nt == 1 ? XLay<1, 1>::xwords : XLay<1, 2>::xwords)
                       : (nt == 1 ? XLay<2, 1>::xwords : XLay<2, 2>::xwords);
  if (tl.lds_bytes + 64 > (size_t)lds_max) return false;
  *out = tl;
  return true;
}

size_t xrec_ws(int64_t B, int64_t H, int64_t P) {
  if (P <= 0) return 0;
  return kHeaderBytes + kXrecSlotBytes + (size_t)kXrecXcds * XLay<2, 2>::xwords * 8;  // the largest
}

using XrecKernel = void (*)(RecurrentArgs, XrecTiling);

static XrecKernel pick_xrec(const XrecTiling &tl, bool taps) {
  const int nbw = tl.u / 32, nt = tl.bX / 16;
  if (taps) {
    if (nbw == 1) return nt == 1 ? k_xrec<1, 1, true> : k_xrec<1, 2, true>;
    return nt == 1 ? k_xrec<2, 1, true> : k_xrec<2, 2, true>;
  }
  if (nbw == 1) return nt == 1 ? k_xrec<1, 1, false> : k_xrec<1, 2, false>;
  return nt == 1 ? k_xrec<2, 1, false> : k_xrec<2, 2, false>;
}

bool xrec_applies(const RecurrentArgs &a, int cus, int lds_max) {
  XrecTiling tl;
  return plan_xrec(a, cus, lds_max, &tl);
}

int recurrent_layout(const RecurrentArgs &a) {
  int dev = 0, cus = 0, lds_max = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return xrec_applies(a, cus, lds_max) ? 1 : 0;
}

hipError_t launch_xrec(const RecurrentArgs &a, int cus, int lds_max, hipStream_t s, bool *done) {
  *done = false;
  XrecTiling tl;
  if (!plan_xrec(a, cus, lds_max, &tl)) return hipSuccess;
  const bool taps = a.acc_h || a.acc_r || a.tap_codes || a.tap_zero || a.tap_inv_q ||
                    a.tap_gates || a.tap_c || a.tap_m;
  XrecKernel kern = pick_xrec(tl, taps);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kXrecThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu < 1) return hipSuccess;  // leave it to the spread layout
  e = clear_exchange(a.ws, kXrecSlotBytes / 8 + kXrecXcds * tl.xwords, s);
  if (e != hipSuccess) return e;
  RecurrentArgs args = a;
  void *kargs[] = {&args, &tl};
  e = hipLaunchCooperativeKernel(reinterpret_cast<void *>(kern), dim3(cus), dim3(kXrecThreads),
                                 kargs, (unsigned)tl.lds_bytes, s);
  if (e == hipSuccess) *done = true;
  return e;
}

hipError_t set_wait_bound_xrec(int polls) { return set_wait_bound_here(polls); }

}  // namespace ql
