// ql_recurrent.hip -- the serial part of a quantized LSTM layer (Section 4) on gfx950.
//
// One cooperative, persistent launch runs all T steps of a layer.  The grid is
// split into tiles of (bB batch rows) x (u hidden units); a workgroup owns one
// tile for the whole sequence, keeps the 4u gate rows of W_h' it needs
// resident in LDS, and keeps its cell state c in LDS.  Each step:
//   1. prefetch its slice of the precomputed W_x x_t + b;
//   2. the codes of h_{t-1} of its batch rows, quantized per vector (eq. 2):
//      one-row tiles quantize their row themselves; in batched tiles the
//      first ceil(rows / 8) unit tiles of a batch slice quantize 8 rows each
//      (one per wave) into the layer's output codes and signal a counter,
//      and every unit tile of the slice loads the codes from there;
//   3. Mult: signed 8-bit products against the resident W_h' slice
//      (v_dot4 for one batch row, v_mfma_i32_16x16x64_i8 for 16+ rows);
//   4. R(.) of eq. 1/3, + (W_x x + b), sigmoid/tanh gates, c and m update;
//   5. with a projection: wait for m_t of the batch rows of a projection
//      tile, quantize it per vector, W_r' product, recover h_t.
// Those codes are the layer's quantized output (the next layer's or the
// output layer's input), so they are never recomputed: with one row per tile
// the workgroup whose unit tile is 0 stores them.
//
// There is no grid barrier.  Values passed between workgroups inside the
// launch (h_t, and m_t with a projection) are published as 64-bit words
// (step tag << 32 | fp32 bits) with device-coherent atomic stores into a
// double buffer indexed by step parity; a consumer polls the words it needs
// until every tag equals the step it waits for.  One store and one poll per
// exchange, no counters.  Small buffers are written to several replicas a few
// KB apart and each consumer polls its own replica, so hundreds of
// workgroups polling one short vector do not all queue on one memory channel.  Reuse of a buffer half is safe because producing
// step t+2 requires every workgroup's step-t+1 values, which each workgroup
// only publishes after it has finished reading step t.  Tags start from 1 and
// the buffer is cleared before every launch.  Every wait is bounded: on expiry
// a flag in the workspace is raised, and all workgroups leave at their next
// wait, so the grid always drains.
#include "ql_device.h"
#include "ql_exchange.h"
#include "ql_launch.h"
#include "ql_rec_common.h"

#include <algorithm>

namespace ql {

// 8 wavefronts per workgroup (two per SIMD): more rows / gate quads in
// flight per step, and one wave's memory wait overlaps another's work.
constexpr int kRecThreads = 512;
// arrival counters [kind][parity][slice], one 64-byte line each; kinds: 0 the
// floats of h_t, 1 those of m_t, 2 the codes of h_t, 3 the codes of m_t
// (batched tiles)
constexpr int kRecCounterBytes = 4 * 2 * kMaxSlices * 64;
// W_r' fragments (16 bytes per lane each) a lane may hold for the projection:
// up to 2 output tiles of 16 x up to 4 K steps of 64 bytes
constexpr int kWrTiles = 2, kWrSteps = 4;

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
  int reph, repm;   // replicas of the published h / m double buffers
  int tc;           // steps of W_x x + b staged in LDS at a time (0: none)
  int wres;         // projection: W_r' fragments resident in registers, K split over the waves
  int64_t strideh, stridem;  // 64-bit words between replicas
  size_t off_w, off_x, off_s, off_c, off_col, off_row, off_gx, lds_bytes;
  size_t off_mc;    // workspace bytes before the codes of m_t (batched tiles, projection)
  size_t mc_zoff, mc_poff;  // from there: bytes to the zero points, between param arrays
};

// Store the codes of h_{t-1} (held in LDS) and their params as the layer's
// quantized output; the whole workgroup cooperates, 16 bytes per thread.
__device__ __forceinline__ void store_codes(const RecurrentArgs &a, const RecTiling &tl,
                                            const int8_t *xc, const RowParam *rp, int nb,
                                            int64_t row0) {
  const int chunks = (int)(a.ld_out / 16);
  for (int idx = threadIdx.x; idx < nb * chunks; idx += blockDim.x) {
    const int lb = idx / chunks, ch = idx % chunks;
    const int64_t row = row0 + lb;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (ch * 16 < tl.ldR) v = *reinterpret_cast<const uint4 *>(xc + lb * tl.ldsX + ch * 16);
    *reinterpret_cast<uint4 *>(a.out_codes + row * a.ld_out + ch * 16) = v;
    if (ch == 0) {
      a.out_zero[row] = rp[lb].z;
      a.out_inv_q[row] = rp[lb].iqx;
      a.out_sums[row] = rp[lb].sum;
      if (a.tap_zero) a.tap_zero[row] = rp[lb].z;
      if (a.tap_inv_q) a.tap_inv_q[row] = rp[lb].iqx;
    }
  }
  if (a.tap_codes)
    for (int idx = threadIdx.x; idx < nb * (int)a.R; idx += blockDim.x) {
      const int lb = idx / (int)a.R, k = idx % (int)a.R;
      a.tap_codes[(row0 + lb) * a.R + k] = xc[lb * tl.ldsX + k];
    }
}

// Quantizes one row of K <= 4 * blockDim floats (eq. 2) with the whole
// workgroup: thread i takes elements 4i .. 4i+3 (device-coherent loads), the
// min/max and the code sum are reduced within each wave and then across the
// waves through red (16 + waves ints of LDS).  The four codes of a thread go
// out as one device-coherent 32-bit store (device layout, zero from K up to
// ldk), the row params to zp / iqp / sump with device-coherent stores.
// Every thread calls it; it ends with a workgroup barrier.
__device__ __forceinline__ void quant_row_wg(const float *src, int K, int ldk, int8_t *dst,
                                             int32_t *zp, float *iqp, int32_t *sump, int *red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nwave = blockDim.x >> 6;
  const int k0 = 4 * tid;
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = k0 + e < K ? ld_coherent(src + k0 + e) : 0.0f;
  int mm[2] = {0x7fffffff, 0x7fffffff};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int key = float_key(v[e]);
    if (k0 + e < K) {
      mm[0] = min(mm[0], key);
      mm[1] = min(mm[1], ~key);
    }
  }
  wave_min_n<2>(mm);
  if (lane == 0) {
    red[2 * wave] = mm[0];
    red[2 * wave + 1] = mm[1];
  }
  __syncthreads();
  int lo = red[0], hi = red[1];
  for (int w = 1; w < nwave; ++w) {
    lo = min(lo, red[2 * w]);
    hi = min(hi, red[2 * w + 1]);
  }
  const QParams prm = make_qparams(key_float(lo), key_float(~hi));
  int sum = 0;
  uint32_t word = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ok = k0 + e < K;
    const int code = encode(v[e], prm.q, prm.z);
    sum += ok ? code : 0;
    word |= (ok ? (uint32_t)((code ^ 0x80) & 0xff) : 0u) << (8 * e);
  }
  for (int k = k0; k < ldk; k += 4 * (int)blockDim.x)
    __hip_atomic_store(reinterpret_cast<uint32_t *>(dst + k), k == k0 ? word : 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  int s1[1] = {sum};
  wave_add_n<1>(s1);
  if (lane == 0) red[16 + wave] = s1[0];
  __syncthreads();
  if (tid == 0) {
    int total = 0;
    for (int w = 0; w < nwave; ++w) total += red[16 + w];
    st_coherent_i(zp, prm.z);
    st_coherent(iqp, prm.inv_q);
    st_coherent_i(sump, total);
  }
}

// ---------------------------------------------------------------------------
// The persistent kernel.  NVA / NVB: values per lane of an h / m row (8 for
// widths <= 512, 32 for <= 2048; NVB = 0 without projection); MFA / MFB: MFMA
// (16+ batch rows per tile) or v_dot4 products.
// ---------------------------------------------------------------------------
template <int NVA, bool MFA, int NVB, bool MFB>
__global__ __launch_bounds__(kRecThreads) void k_recurrent(RecurrentArgs a, RecTiling tl) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int8_t *wsl = reinterpret_cast<int8_t *>(smem + tl.off_w);
  int8_t *xc = reinterpret_cast<int8_t *>(smem + tl.off_x);
  int32_t *S = reinterpret_cast<int32_t *>(smem + tl.off_s);
  float *cst = reinterpret_cast<float *>(smem + tl.off_c);
  ColParam *cp = reinterpret_cast<ColParam *>(smem + tl.off_col);
  RowParam *rp = reinterpret_cast<RowParam *>(smem + tl.off_row);
  float *gxs = reinterpret_cast<float *>(smem + tl.off_gx);  // [tc][pairs][4]
  __shared__ int s_abort;
  __shared__ int s_red[32];

  const int64_t T = a.T, B = a.B, H = a.H, P = a.P, R = a.R;
  int *flag = reinterpret_cast<int *>(a.ws) + kHdrFlag;
  constexpr bool CNT = MFA;  // batched tiles: counters + coherent floats; else tagged words
  // arrival counters: [kind h/m][parity][slice], 64 bytes apart
  unsigned *cnt = reinterpret_cast<unsigned *>(static_cast<char *>(a.ws) + kHeaderBytes);
  auto counter = [&](int kind, int64_t par, int slice) {
    return cnt + ((kind * 2 + (int)par) * kMaxSlices + slice) * 16;
  };
  char *xdata = static_cast<char *>(a.ws) + kHeaderBytes + kRecCounterBytes;
  // counter mode: h_t in xhf [2][B][R], m_t in xmf [2][B][H] (slot t & 1)
  float *xhf = reinterpret_cast<float *>(xdata);
  float *xmf = xhf + 2 * B * R;
  // tagged mode: replica c of h: xh + c * strideh, [2][B][R]; of m: xm + c * stridem
  uint64_t *xh = reinterpret_cast<uint64_t *>(xdata);
  uint64_t *xm = xh + tl.reph * tl.strideh;
  const uint64_t *xh_mine = xh + (blockIdx.x % tl.reph) * tl.strideh;
  const uint64_t *xm_mine = xm + (blockIdx.x % tl.repm) * tl.stridem;

  const int tid = threadIdx.x;
  const bool activeA = (int)blockIdx.x < tl.nbt * tl.nut;
  const int tb = activeA ? blockIdx.x / tl.nut : 0, tu = activeA ? blockIdx.x % tl.nut : 0;
  const int64_t b0 = (int64_t)tb * tl.bB, j0 = (int64_t)tu * tl.u;
  const int nb = activeA ? (int)(B - b0 < tl.bB ? B - b0 : tl.bB) : 0;
  const int nu = activeA ? (int)(H - j0 < tl.u ? H - j0 : tl.u) : 0;
  const int nrows = 4 * tl.u;  // slice rows, gate-major: row g*u + jj
  const int ldS = nrows;
  const int rowsA = MFA ? tl.bB : nb;  // rows quantized (MFMA tiles need zero padding rows)
  // rows per wave-level group: two rows of a batched tile share one set of
  // reductions (16 rows keep all 8 waves busy); one-row tiles use single rows
  constexpr int RBA = (MFA && NVA <= 8) ? 2 : 1;
  constexpr int RBB = (MFB && NVB <= 8) ? 2 : 1;
  const bool activeB = NVB > 0 && (int)blockIdx.x < tl.nbt2 * tl.npt;
  const int tb2 = activeB ? blockIdx.x / tl.npt : 0, tp = activeB ? blockIdx.x % tl.npt : 0;
  const int64_t c0 = (int64_t)tb2 * tl.bB2, p0 = (int64_t)tp * tl.p2;
  const int nb2 = activeB ? (int)(B - c0 < tl.bB2 ? B - c0 : tl.bB2) : 0;
  const int np2 = activeB ? (int)(P - p0 < tl.p2 ? P - p0 : tl.p2) : 0;
  const int tbB = activeB ? (int)(c0 / tl.bB) : 0;  // phase A slice holding these rows
  // producers per slot use: of h for this slice, of m for the projection's slice
  const unsigned prod_h =
      NVB == 0 ? (unsigned)tl.nut : (unsigned)(((nb + tl.bB2 - 1) / tl.bB2) * tl.npt);
  const unsigned prod_m = (unsigned)tl.nut;
  // batched tiles: the codes of h_{t-1} are made once, by the first Qn unit
  // tiles of the slice (groups of 8 rows, one row per wave), straight into
  // the layer's output codes; every tile of the slice then loads them
  const int Qn = (nb + 7) / 8 < tl.nut ? (nb + 7) / 8 : tl.nut;
  const int wave = tid >> 6, lane = tid & 63;
  if (tid == 0) s_abort = 0;

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
      float cv = 0.0f;
      if (lb < nb && jj < nu && a.c0) cv = a.c0[(b0 + lb) * H + j0 + jj];
      cst[idx] = cv;
    }
  }
  __syncthreads();

  // resident W_r' slice: fragment [tj][ks] of this wave covers output tile tj
  // and K step ks of the wave's share of K (ldH / 8 bytes)
  v4i wfr[kWrTiles][kWrSteps];
  const int ksw = tl.ldH / 512, ntw = tl.p2 / 16, kwave = (tid >> 6) * (tl.ldH / 8);
  if (NVB > 0 && MFB && activeB && tl.wres) {
#pragma unroll
    for (int tj = 0; tj < kWrTiles; ++tj)
#pragma unroll
      for (int ks = 0; ks < kWrSteps; ++ks) {
        wfr[tj][ks] = v4i{};
        if (tj < ntw && ks < ksw) {
          const int wrow = tj * 16 + (tid & 15);
          const int64_t rr = p0 + (wrow < np2 ? wrow : np2 - 1);
          wfr[tj][ks] = *reinterpret_cast<const v4i *>(a.Wr.codes + rr * a.Wr.ld + kwave + ks * 64 +
                                                       ((tid & 63) >> 4) * 16);
        }
      }
  }
  const int pairs = nb * nu;
  const int nthr = (int)blockDim.x, fullr = pairs / nthr;
  // Batched tiles whose cell count divides the workgroup: a lane's cell is
  // the same in every full round of pairs (rows lbL, lbL + dlb, ...), so the
  // column params of its four gates, and whether they allow the 24-bit
  // recovery, are read once here.
  const bool cfix = CNT && activeA && nu > 0 && nthr % nu == 0;
  const int jjL = cfix ? tid % nu : 0, lbL = cfix ? tid / nu : 0, dlb = cfix ? nthr / nu : 0;
  int32_t fcol[4] = {0, 0, 0, 0}, fztw[4] = {0, 0, 0, 0};
  float fiqw[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  bool fcf = cfix;
  if (cfix) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const ColParam c = cp[g * tl.u + jjL];
      fcol[g] = (int32_t)c.colterm;
      fztw[g] = c.ztw;
      fiqw[g] = c.iqw;
      fcf = fcf && (uint32_t)(c.ztw + 127) <= 255u &&
            (uint64_t)(c.colterm + (1 << 23)) < (uint64_t)(1 << 24);
    }
  }
  // Without room to stage W_x x + b in LDS, each lane's values of the first
  // kGxPre full rounds of pairs are loaded into registers at the top of the
  // step, so their latency passes while h_{t-1} is awaited.
  constexpr int kGxPre = 4;
  float gxr[kGxPre][4];
  for (int64_t t = 0; t <= T; ++t) {
    const int64_t hcur = (t & 1) * B * R;  // h_t is published here with tag t+1
    if (CNT && activeA && tl.tc == 0 && t < T) {
#pragma unroll
      for (int k = 0; k < kGxPre; ++k) {
        const int pr = k * nthr + tid, lb = pr / nu, jj = pr % nu;
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
          gxr[k][gg] = k < fullr ? a.gx[(t * B + b0 + lb) * 4 * H + gg * H + j0 + jj] : 0.0f;
      }
    }
    if (activeA) {
      // ---- 1. every tc steps, stage W_x x + b of the next tc steps in LDS
      if (tl.tc > 0 && t < T && t % tl.tc == 0) {
        const int steps = (int)(T - t < tl.tc ? T - t : tl.tc);
        for (int idx = tid; idx < steps * pairs * 4; idx += blockDim.x) {
          const int s_ = idx / (pairs * 4), rem = idx % (pairs * 4);
          const int pr = rem >> 2, gg = rem & 3;
          const int lb = pr / nu, jj = pr % nu;
          gxs[(s_ * pairs + pr) * 4 + gg] = a.gx[((t + s_) * B + b0 + lb) * 4 * H + gg * H + j0 + jj];
        }
      }
      // ---- 2. h_{t-1} of this batch slice, quantized per vector
      bool ok;
      if (t == 0) {
        ok = quant_tile<NVA, RBA, kSrcPlain>(nb, rowsA, R, 0u, (int)R, xc, tl.ldsX, tl.ldR, flag, rp,
                                    [&](int lb) -> const void * {
                                      return a.h0 ? a.h0 + (b0 + lb) * R : nullptr;
                                    });
      } else if (CNT) {
        const int64_t par = (t - 1) & 1;
        const int64_t hrow0 = (t - 1) * B + b0;
        if (tu < Qn) {
          if (!wait_count(counter(0, par, tb), (unsigned)(((t - 1) >> 1) + 1) * prod_h, flag))
            s_abort = 1;
          __syncthreads();
          if (s_abort) return;
          const float *prev = xhf + par * B * R;
          const int owords = (int)(a.ld_out / 8);
          for (int g = tu; g * 8 < nb; g += Qn) {
            const int lb = g * 8 + wave;
            if (lb >= nb) continue;
            quant_rows<NVA, 1, kSrcCoherent>(prev + (b0 + lb) * R, R, 1, 1, 0u, (int)R,
                                             xc + lb * tl.ldsX, tl.ldsX, tl.ldR, flag, rp + lb);
            // the wave's own LDS writes are complete in program order
            const int64_t row = hrow0 + lb;
            for (int wd = lane; wd < owords; wd += kWave) {
              uint64_t v = 0;
              if (wd * 8 < tl.ldR) v = *reinterpret_cast<const uint64_t *>(xc + lb * tl.ldsX + wd * 8);
              st_coherent64(reinterpret_cast<uint64_t *>(a.out_codes + row * a.ld_out) + wd, v);
            }
            if (lane == 0) {
              st_coherent_i(&a.out_zero[row], rp[lb].z);
              st_coherent(&a.out_inv_q[row], rp[lb].iqx);
              st_coherent_i(&a.out_sums[row], rp[lb].sum);
              if (a.tap_zero) a.tap_zero[row] = rp[lb].z;
              if (a.tap_inv_q) a.tap_inv_q[row] = rp[lb].iqx;
            }
            if (a.tap_codes)
              for (int k = lane; k < (int)R; k += kWave) a.tap_codes[row * R + k] = xc[lb * tl.ldsX + k];
          }
          // arrival once every wave's stores have completed
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          if (tid == 0)
            __hip_atomic_fetch_add(counter(2, par, tb), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (t == T) break;  // the codes of h_{T-1} are the output's last rows
        if (!wait_count(counter(2, par, tb), (unsigned)(((t - 1) >> 1) + 1) * Qn, flag)) s_abort = 1;
        __syncthreads();
        if (s_abort) return;
        // kLdW words per thread in flight together, then parked in LDS
        constexpr int kLdW = 8;
        const int rwords = tl.ldR / 8, nwords = rowsA * rwords;
        for (int base = 0; base < nwords; base += kLdW * (int)blockDim.x) {
          uint64_t v[kLdW];
#pragma unroll
          for (int i = 0; i < kLdW; ++i) {
            const int idx = base + i * (int)blockDim.x + tid, lb = idx / rwords, wd = idx % rwords;
            v[i] = 0;
            if (idx < nwords && lb < nb)
              v[i] = ld_coherent64(reinterpret_cast<const uint64_t *>(a.out_codes + (hrow0 + lb) * a.ld_out) + wd);
          }
#pragma unroll
          for (int i = 0; i < kLdW; ++i) {
            const int idx = base + i * (int)blockDim.x + tid, lb = idx / rwords, wd = idx % rwords;
            if (idx < nwords) *reinterpret_cast<uint64_t *>(xc + lb * tl.ldsX + wd * 8) = v[i];
          }
        }
        for (int lb = tid; lb < rowsA; lb += blockDim.x)
          rp[lb] = lb < nb ? row_param(ld_coherent_i(&a.out_zero[hrow0 + lb]),
                                       ld_coherent(&a.out_inv_q[hrow0 + lb]),
                                       ld_coherent_i(&a.out_sums[hrow0 + lb]), (int)R)
                           : row_param(0, 0.0f, 0, (int)R);
        ok = true;
      } else {
        const uint64_t *prev = xh_mine + ((t + 1) & 1) * B * R;
        ok = quant_tile<NVA, RBA, kSrcTagged>(nb, rowsA, R, (uint32_t)t, (int)R, xc, tl.ldsX, tl.ldR,
                                              flag, rp, [&](int lb) -> const void * {
                                                return prev + (b0 + lb) * R;
                                              });
      }
      if (!ok) s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      if (t == T) {
        if (!CNT && tu == 0) store_codes(a, tl, xc, rp, nb, (T - 1) * B + b0);
        break;
      }
      // ---- 3. Mult against the resident slice
      if (MFA)
        products_mfma(xc, tl.ldsX, tl.bB, wsl, tl.ldsW, nrows, nrows, tl.ldR, S, ldS);
      else
        products_valu(xc, tl.ldsX, nb, wsl, tl.ldsW, nrows, nrows, tl.ldR, S, ldS);
      __syncthreads();
      // ---- 4. recover, gates, cell update; publish h_t (or m_t)
      const int64_t mcur = (t & 1) * B * H;
      const float *gxt = tl.tc > 0 ? gxs + (t % tl.tc) * pairs * 4 : nullptr;
      // W_x x + b of gate gg of pair pr, from the LDS staging or global memory
      auto gx_of = [&](int pr, int gg) {
        const int lb = pr / nu, jj = pr % nu;
        return gxt ? gxt[pr * 4 + gg] : a.gx[(t * B + b0 + lb) * 4 * H + gg * H + j0 + jj];
      };
      // activation of gate gg of pair pr (sigmoid for i, f, o; tanh(x) =
      // 2 sigmoid(2x) - 1 for g), with the raw accumulator tap
      auto act_x = [&](int pr, int gg, float gxv) {
        const int lb = pr / nu, jj = pr % nu;
        const RowParam r = rp[lb];
        const int64_t b = b0 + lb, j = j0 + jj;
        const int n = gg * tl.u + jj;
        const ColParam c = cp[n];
        const int32_t sv = S[lb * ldS + n];
        const float yh = recover(sv, c.colterm, c.ztw, r.ztx, r.sigx, c.iqw, r.iqx);
        const float av = gxv + yh;
        if (a.acc_h) a.acc_h[(t * B + b) * 4 * H + gg * H + j] = acc_u8(sv, c.sigw, r.sigx, R);
        const float sg = sigmoid_cw(gg == 2 ? 2.0f * av : av);
        return gg == 2 ? 2.0f * sg - 1.0f : sg;
      };
      auto act = [&](int pr, int gg) { return act_x(pr, gg, gx_of(pr, gg)); };
      // cell update and publication of pair (lb, jj)
      auto finish_lj = [&](int lb, int jj, float ig, float fg, float gv, float og) {
        const int64_t b = b0 + lb, j = j0 + jj;
        const float cn = (fg * cst[lb * tl.u + jj]) + (ig * gv);
        cst[lb * tl.u + jj] = cn;
        const float m = og * tanh_cw(cn);
        if (a.tap_gates) {
          float *gp = a.tap_gates + (t * B + b) * 4 * H + j;
          gp[0] = ig, gp[H] = fg, gp[2 * H] = gv, gp[3 * H] = og;
        }
        if (a.tap_c) a.tap_c[(t * B + b) * H + j] = cn;
        if (a.tap_m) a.tap_m[(t * B + b) * H + j] = m;
        if (NVB == 0) {
          if (CNT)
            st_coherent(&xhf[hcur + b * R + j], m);
          else
            for (int c2 = 0; c2 < tl.reph; ++c2) publish(&xh[c2 * tl.strideh + hcur + b * R + j], (uint32_t)(t + 1), m);
          a.h[(t * B + b) * R + j] = m;
          if (t == T - 1 && a.hT) a.hT[b * R + j] = m;
        } else {
          if (CNT)
            st_coherent(&xmf[mcur + b * H + j], m);
          else
            for (int c2 = 0; c2 < tl.repm; ++c2) publish(&xm[c2 * tl.stridem + mcur + b * H + j], (uint32_t)(t + 1), m);
        }
        if (t == T - 1 && a.cT) a.cT[b * H + j] = cn;
      };
      auto finish = [&](int pr, float ig, float fg, float gv, float og) {
        finish_lj(pr / nu, pr % nu, ig, fg, gv, og);
      };
      // pairs one per lane in full rounds of the workgroup; the remainder
      // over four lanes per pair (lane g of a quad computes gate g) when that
      // fits, so no lane does much more than its share
      const int nt = nthr, full = fullr, remp = pairs % nt;
      const bool pre = CNT && tl.tc == 0;
      if (cfix && !a.acc_h) {
        // fixed cell per lane: column params from registers, one decision
        // per pair for the 24-bit recovery (the same values as recover())
        for (int k = 0; k < full; ++k) {
          const int pr = k * nt + tid, lb = lbL + k * dlb;
          const RowParam r = rp[lb];
          const bool fast = fcf && (uint32_t)(r.ztx + 127) <= 255u;
          float av4[4];
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) {
            const float gxv = pre && k < kGxPre
                                  ? (k == 0 ? gxr[0][gg] : k == 1 ? gxr[1][gg] : k == 2 ? gxr[2][gg] : gxr[3][gg])
                                  : gx_of(pr, gg);
            const int32_t sv = S[lb * ldS + gg * tl.u + jjL];
            float yh;
            if (fast) {
              const uint32_t tt = (uint32_t)sv + (uint32_t)mul_i24(r.ztx, fcol[gg]) +
                                  (uint32_t)mul_i24(fztw[gg], r.sigx);
              yh = ((float)(int32_t)tt * fiqw[gg]) * r.iqx;
            } else {
              const ColParam c = cp[gg * tl.u + jjL];
              yh = recover(sv, c.colterm, c.ztw, r.ztx, r.sigx, c.iqw, r.iqx);
            }
            const float av = gxv + yh;
            const float sg = sigmoid_cw(gg == 2 ? 2.0f * av : av);
            av4[gg] = gg == 2 ? 2.0f * sg - 1.0f : sg;
          }
          finish_lj(lb, jjL, av4[0], av4[1], av4[2], av4[3]);
        }
      } else
      for (int k = 0; k < full; ++k) {
        const int pr = k * nt + tid;
        if (pre && k < kGxPre) {
          // the round's prefetched values, picked by selects (no indexed
          // register array)
          float gv4[4];
#pragma unroll
          for (int gg = 0; gg < 4; ++gg)
            gv4[gg] = k == 0 ? gxr[0][gg] : k == 1 ? gxr[1][gg] : k == 2 ? gxr[2][gg] : gxr[3][gg];
          finish(pr, act_x(pr, 0, gv4[0]), act_x(pr, 1, gv4[1]), act_x(pr, 2, gv4[2]),
                 act_x(pr, 3, gv4[3]));
        } else {
          finish(pr, act(pr, 0), act(pr, 1), act(pr, 2), act(pr, 3));
        }
      }
      if (remp > 0) {
        const int p0 = full * nt;
        if (4 * remp <= nt) {
          if (tid < 4 * remp) {  // whole quads active
            const int pr = p0 + (tid >> 2);
            const float av = act(pr, tid & 3);
            const float ig = quad_bcast<0>(av), fg = quad_bcast<1>(av);
            const float gv = quad_bcast<2>(av), og = quad_bcast<3>(av);
            if ((tid & 3) == 0) finish(pr, ig, fg, gv, og);
          }
        } else if (tid < remp) {
          const int pr = p0 + tid;
          finish(pr, act(pr, 0), act(pr, 1), act(pr, 2), act(pr, 3));
        }
      }
      // the codes of h_{t-1} become the layer's quantized output (batched
      // tiles: the designated quantizers stored them already)
      if (!CNT && t > 0 && tu == 0) store_codes(a, tl, xc, rp, nb, (t - 1) * B + b0);
      if (CNT) arrive(counter(NVB == 0 ? 0 : 1, t & 1, tb));
    }
    if (t == T) break;

    // ---- 5. projection h_t = R(Mult(Q(m_t), W_r'))
    if (NVB > 0 && activeB) {
      const int ldx2 = tl.ldH + 16;
      const uint64_t *mrows = xm_mine + (t & 1) * B * H;
      const int rowsB = MFB ? tl.bB2 : nb2;
      __syncthreads();  // LDS codes / params of phase 4 are no longer read
      bool ok;
      if (CNT) {
        // the codes of m_t are made once per projection slice, its rows
        // spread over its projection tiles (rows tp, tp + npt, ...; the whole
        // workgroup per row), into a double buffer of the workspace; every
        // projection tile of the slice loads them
        const int QnB = nb2 < tl.npt ? nb2 : tl.npt;
        const int64_t par = t & 1;
        char *mbase = static_cast<char *>(a.ws) + tl.off_mc;
        int8_t *mcodes = reinterpret_cast<int8_t *>(mbase) + par * B * tl.ldH;
        const size_t zoff = tl.mc_zoff, poff = tl.mc_poff;
        int32_t *mz = reinterpret_cast<int32_t *>(mbase + zoff) + par * B;
        float *miq = reinterpret_cast<float *>(mbase + zoff + poff) + par * B;
        int32_t *msum = reinterpret_cast<int32_t *>(mbase + zoff + 2 * poff) + par * B;
        if (tp < nb2) {
          if (!wait_count(counter(1, par, tbB), (unsigned)((t >> 1) + 1) * prod_m, flag)) s_abort = 1;
          __syncthreads();
          if (s_abort) return;
          const float *mf = xmf + par * B * H;
          for (int lb = tp; lb < nb2; lb += tl.npt) {
            const int64_t row = c0 + lb;
            quant_row_wg(mf + row * H, (int)H, tl.ldH, mcodes + row * tl.ldH, &mz[row], &miq[row],
                         &msum[row], s_red);
          }
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          if (tid == 0)
            __hip_atomic_fetch_add(counter(3, par, tb2), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (!wait_count(counter(3, par, tb2), (unsigned)((t >> 1) + 1) * QnB, flag)) s_abort = 1;
        __syncthreads();
        if (s_abort) return;
        constexpr int kLdW = 8;
        const int mwords = tl.ldH / 8, nwords = rowsB * mwords;
        for (int base = 0; base < nwords; base += kLdW * (int)blockDim.x) {
          uint64_t v[kLdW];
#pragma unroll
          for (int i = 0; i < kLdW; ++i) {
            const int idx = base + i * (int)blockDim.x + tid, lb = idx / mwords, wd = idx % mwords;
            v[i] = 0;
            if (idx < nwords && lb < nb2)
              v[i] = ld_coherent64(reinterpret_cast<const uint64_t *>(mcodes + (c0 + lb) * tl.ldH) + wd);
          }
#pragma unroll
          for (int i = 0; i < kLdW; ++i) {
            const int idx = base + i * (int)blockDim.x + tid, lb = idx / mwords, wd = idx % mwords;
            if (idx < nwords) *reinterpret_cast<uint64_t *>(xc + lb * ldx2 + wd * 8) = v[i];
          }
        }
        for (int lb = tid; lb < rowsB; lb += blockDim.x)
          rp[lb] = lb < nb2 ? row_param(ld_coherent_i(&mz[c0 + lb]), ld_coherent(&miq[c0 + lb]),
                                        ld_coherent_i(&msum[c0 + lb]), (int)H)
                            : row_param(0, 0.0f, 0, (int)H);
        ok = true;
      } else {
        ok = quant_tile<NVB, RBB, kSrcTagged>(nb2, rowsB, H, (uint32_t)(t + 1), (int)H, xc, ldx2,
                                              tl.ldH, flag, rp, [&](int lb) -> const void * {
                                                return mrows + (c0 + lb) * H;
                                              });
      }
      if (!ok) s_abort = 1;
      __syncthreads();
      if (s_abort) return;
      // W_r' rows p0 .. p0 + np2 - 1, read from global memory (L2 resident)
      const int8_t *wr = a.Wr.codes + p0 * a.Wr.ld;
      if (MFB && tl.wres) {
        // this wave's share of K against the resident fragments; partial
        // sums of wave w in S[(w * 16 + row) * p2 + col], then summed into
        // slot 0 (integer sums: the order does not matter)
        const int lane = tid & 63, wv = tid >> 6;
        const int8_t *xr = xc + (lane & 15) * ldx2 + kwave + (lane >> 4) * 16;
        v4i acc[kWrTiles] = {v4i{}, v4i{}};
#pragma unroll
        for (int ks = 0; ks < kWrSteps; ++ks) {
          if (ks >= ksw) break;
          const v4i av = *reinterpret_cast<const v4i *>(xr + ks * 64);
#pragma unroll
          for (int tj = 0; tj < kWrTiles; ++tj)
            if (tj < ntw) acc[tj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, wfr[tj][ks], acc[tj], 0, 0, 0);
        }
#pragma unroll
        for (int tj = 0; tj < kWrTiles; ++tj)
          if (tj < ntw)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              S[(wv * 16 + (lane >> 4) * 4 + r) * tl.p2 + tj * 16 + (lane & 15)] = acc[tj][r];
        __syncthreads();
        const int nwv = (int)blockDim.x >> 6;
        for (int idx = tid; idx < 16 * tl.p2; idx += blockDim.x) {
          int sum = S[idx];
          for (int w = 1; w < nwv; ++w) sum += S[w * 16 * tl.p2 + idx];
          S[idx] = sum;
        }
      } else if (MFB)
        products_mfma(xc, ldx2, tl.bB2, wr, a.Wr.ld, tl.p2, np2, tl.ldH, S, tl.p2);
      else
        products_valu(xc, ldx2, nb2, wr, a.Wr.ld, tl.p2, np2, tl.ldH, S, tl.p2);
      __syncthreads();
      for (int idx = tid; idx < nb2 * np2; idx += blockDim.x) {
        const int lb = idx / np2, pp = idx % np2;
        const int64_t b = c0 + lb, p = p0 + pp;
        const RowParam r = rp[lb];
        const int blk = (int)p / (int)a.Wr.rows_per_block;  // W_r's row block of output p
        const int32_t ztw = a.Wr.zero[blk] + 128;
        const float iqw = a.Wr.inv_q[blk];
        const int32_t sigw = a.Wr.row_sums[p] - 128 * (int32_t)H;
        const int64_t colterm = (int64_t)sigw + H * (int64_t)ztw;
        const int32_t sv = S[lb * tl.p2 + pp];
        const float hv = recover(sv, colterm, ztw, r.ztx, r.sigx, iqw, r.iqx);
        if (CNT)
          st_coherent(&xhf[hcur + b * P + p], hv);
        else
          for (int c = 0; c < tl.reph; ++c) publish(&xh[c * tl.strideh + hcur + b * P + p], (uint32_t)(t + 1), hv);
        a.h[(t * B + b) * P + p] = hv;
        if (t == T - 1 && a.hT) a.hT[b * P + p] = hv;
        if (a.acc_r) a.acc_r[(t * B + b) * P + p] = acc_u8(sv, sigw, r.sigx, H);
      }
      if (CNT) arrive(counter(0, t & 1, tbB));
    }
    __syncthreads();  // LDS of this step is free before the next step's quantization
  }
}

// Clears the arrival counters and the exchange buffers (n64 64-bit words
// after the header); the timeout flag only when asked (once per API call).
__global__ void k_clear_exchange(unsigned *hdr, int64_t n64, int with_flag) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0 && with_flag) hdr[kHdrFlag] = 0u;
  uint64_t *x = reinterpret_cast<uint64_t *>(reinterpret_cast<char *>(hdr) + kHeaderBytes);
  for (int64_t k = i; k < n64; k += (int64_t)gridDim.x * blockDim.x) x[k] = 0;
}

hipError_t clear_exchange(void *ws, int64_t n64, hipStream_t s) {
  const unsigned zb = (unsigned)std::min<int64_t>(1024, (n64 + 255) / 256 + 1);
  hipLaunchKernelGGL(k_clear_exchange, dim3(zb), dim3(256), 0, s, static_cast<unsigned *>(ws), n64,
                     0);
  return hipGetLastError();
}

hipError_t reset_recurrent_flag(void *ws, hipStream_t s) {
  hipLaunchKernelGGL(k_clear_exchange, dim3(1), dim3(64), 0, s, static_cast<unsigned *>(ws),
                     (int64_t)0, 1);
  return hipGetLastError();
}

hipError_t set_wait_bound_recurrent(int polls) { return set_wait_bound_here(polls); }

// The bound of every wait of the persistent kernels, on every device (a test
// hook that forces the timeout path without a kernel that hangs); without a
// device there is nothing to bound.
hipError_t set_wait_bound(int polls) {
  int n = 0, cur = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    return hipSuccess;
  }
  hipError_t e = hipGetDevice(&cur);
  for (int d = 0; d < n && e == hipSuccess; ++d) {
    e = hipSetDevice(d);
    if (e == hipSuccess) e = set_wait_bound_recurrent(polls);
    if (e == hipSuccess) e = set_wait_bound_stack(polls);
    if (e == hipSuccess) e = set_wait_bound_pstack(polls);
    if (e == hipSuccess) e = set_wait_bound_f32(polls);
    if (e == hipSuccess) e = set_wait_bound_train(polls);
    if (e == hipSuccess) e = set_wait_bound_xrec(polls);
    if (e == hipSuccess) e = set_wait_bound_xstack(polls);
  }
  const hipError_t r = hipSetDevice(cur);
  return e != hipSuccess ? e : r;
}

// ------------------------------------------------------------------ host side
constexpr int kMaxReplicas = 4;
constexpr int kPublishBudget = 2048;  // values x replicas a workgroup publishes per step

// 64-bit words between replicas of a double buffer of `words` words: a
// multiple of 64 KB plus 4 KB, so replicas start on different channels.
static int64_t replica_stride(int64_t words) { return round_up(words, 8192) + 512; }

static int64_t exchange_words(int64_t B, int64_t H, int64_t P) {
  const int64_t R = P > 0 ? P : H;
  int64_t n = kMaxReplicas * replica_stride(2 * B * R);  // >= the float buffers of counter mode
  if (P > 0) n += kMaxReplicas * replica_stride(2 * B * H);
  return kRecCounterBytes / 8 + n;
}

// Codes of m_t made once per projection slice (batched tiles): [2][B][ldH]
// bytes, then zero points, recovery factors and code sums, [2][B] each.
static size_t mcode_bytes(int64_t B, int64_t H, int64_t P) {
  if (P <= 0) return 0;
  return align_up((size_t)2 * B * round_up(H, 64), 256) + 3 * align_up((size_t)2 * B * 4, 256);
}

size_t recurrent_ws(int64_t B, int64_t H, int64_t P) {
  const size_t spread = kHeaderBytes +
                        align_up((size_t)exchange_words(B, H, P) * sizeof(uint64_t), 256) +
                        mcode_bytes(B, H, P);
  return std::max(spread, xrec_ws(B, H, P));
}

static int replicas(int values_per_block, int consumers) {
  int r = kPublishBudget / (values_per_block > 0 ? values_per_block : 1);
  r = r < consumers ? r : consumers;
  r = r < kMaxReplicas ? r : kMaxReplicas;
  return r > 0 ? r : 1;
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
    // Fewer unit tiles per batch slice means fewer re-reads of each h row per
    // step; aim for at most 32 tiles, as long as the W_h' slice fits LDS.
    for (int bB = 16; bB <= 256 && !ok; bB *= 2) {
      const int nbt = (int)((B + bB - 1) / bB);
      if (nbt > G) continue;
      const int max_nut = G / nbt;
      for (int nut_target = 32; nut_target <= max_nut * 2 && !ok; nut_target *= 2) {
        const int nut_try = nut_target < max_nut ? nut_target : max_nut;
        int u = (int)((H + nut_try - 1) / nut_try);
        u = (u + 3) / 4 * 4;
        if ((size_t)4 * u * (tl.ldR + 16) > (size_t)lds_max / 2) continue;
        if ((int64_t)nbt * ((H + u - 1) / u) > G) continue;
        tl.bB = bB;
        tl.nbt = nbt;
        tl.u = u;
        tl.nut = (int)((H + u - 1) / u);
        tl.mfmaA = 1;
        ok = true;
      }
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
  // replicas of the published buffers (consumers of one batch row: the unit
  // tiles of its slice for h, the projection tiles for m)
  {
    const int hvals = P > 0 ? tl.bB2 * tl.p2 : tl.bB * tl.u;
    tl.reph = replicas(hvals, tl.nut);
    tl.repm = P > 0 ? replicas(tl.bB * tl.u, tl.npt) : 1;
    tl.strideh = replica_stride(2 * B * a.R);
    tl.stridem = P > 0 ? replica_stride(2 * B * H) : 0;
  }
  if (tl.nbt > kMaxSlices || (P > 0 && tl.nbt2 > kMaxSlices)) return false;
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
  // 16-row projection tiles whose W_r' slice fits kWrTiles x kWrSteps
  // fragments per lane when K is split over the eight waves: the slice stays
  // in registers and the waves' partial products are summed through LDS
  tl.wres = P > 0 && tl.mfmaB && tl.bB2 == 16 && tl.p2 % 16 == 0 && tl.p2 / 16 <= kWrTiles &&
            tl.ldH % 512 == 0 && tl.ldH / 512 <= kWrSteps;
  if (tl.wres) {
    const size_t sb3 = (size_t)(kRecThreads / 64) * 16 * tl.p2 * 4;
    sbytes = sbytes > sb3 ? sbytes : sb3;
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
  // W_x x + b staging: as many steps as fit (up to 64), at least one
  {
    const size_t per_step = (size_t)tl.bB * tl.u * 4 * sizeof(float);
    const size_t room = (size_t)lds_max - 64 > off ? (size_t)lds_max - 64 - off : 0;
    int64_t tc = (int64_t)(room / per_step);
    tc = tc > 64 ? 64 : tc;
    tc = tc > a.T ? a.T : tc;
    tl.tc = tc > 0 ? (int)tc : 0;  // 0: read W_x x + b straight from memory
    tl.off_gx = off;
    off = align_up(off + per_step * tl.tc, 16);
  }
  tl.lds_bytes = off;
  if (tl.lds_bytes + 64 > (size_t)lds_max) return false;  // + static shared (barrier flag)
  *out = tl;
  return true;
}

using RecKernel = void (*)(RecurrentArgs, RecTiling);

// The instantiation for a shape class: row widths up to 512 or 2048 values.
static RecKernel pick_kernel(const RecurrentArgs &a, const RecTiling &tl) {
  const bool wideR = a.R > 512, wideH = a.H > 512;
  if (a.P == 0) {
    if (tl.mfmaA) return wideR ? k_recurrent<32, true, 0, false> : k_recurrent<8, true, 0, false>;
    return wideR ? k_recurrent<32, false, 0, false> : k_recurrent<8, false, 0, false>;
  }
  if (wideR) return nullptr;  // projection widths above 512 are not instantiated
  if (tl.mfmaA) return wideH ? k_recurrent<8, true, 32, true> : k_recurrent<8, true, 8, true>;
  return wideH ? k_recurrent<8, false, 32, false> : k_recurrent<8, false, 8, false>;
}

hipError_t launch_recurrent(const RecurrentArgs &a, hipStream_t s, bool *unsupported) {
  *unsupported = false;
  if (a.T == 0 || a.B == 0) return hipSuccess;
  if (a.R > 2048 || a.H > 2048) {  // one h / m row is held in 32 registers per lane
    *unsupported = true;
    return hipSuccess;
  }
  int lds_max = 0;
  const int cus = device_cus(&lds_max);
  // batched layers with a projection on the whole chip: the XCD-local layout
  bool done = false;
  hipError_t ex = launch_xrec(a, cus, lds_max, s, &done);
  if (ex != hipSuccess || done) return ex;
  RecTiling tl;
  if (!plan(a, cus, lds_max, &tl)) {
    *unsupported = true;
    return hipSuccess;
  }
  RecKernel kern = pick_kernel(a, tl);
  if (!kern) {
    *unsupported = true;
    return hipSuccess;
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)tl.lds_bytes);
  if (e != hipSuccess) return e;
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kRecThreads, tl.lds_bytes);
  if (e != hipSuccess) return e;
  if (per_cu * cus < tl.grid) {
    *unsupported = true;
    return hipSuccess;
  }
  const int64_t n64 = kRecCounterBytes / 8 + tl.reph * tl.strideh + tl.repm * tl.stridem;
  const unsigned zb = (unsigned)std::min<int64_t>(1024, (n64 + 255) / 256 + 1);
  hipLaunchKernelGGL(k_clear_exchange, dim3(zb), dim3(256), 0, s, static_cast<unsigned *>(a.ws),
                     n64, 0);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  tl.off_mc = kHeaderBytes + align_up((size_t)exchange_words(a.B, a.H, a.P) * sizeof(uint64_t), 256);
  tl.mc_zoff = align_up((size_t)2 * a.B * tl.ldH, 256);
  tl.mc_poff = align_up((size_t)2 * a.B * 4, 256);
  RecurrentArgs args = a;
  void *kargs[] = {&args, &tl};
  return hipLaunchCooperativeKernel(reinterpret_cast<void *>(kern), dim3(tl.grid), dim3(kRecThreads),
                                    kargs, (unsigned)tl.lds_bytes, s);
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
