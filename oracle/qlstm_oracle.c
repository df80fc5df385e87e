/*
 * qlstm_oracle.c -- CPU oracle for quantized LSTM acoustic-model inference.
 *
 * TEST INFRASTRUCTURE ONLY (see qlstm_oracle.h).  Plain loops, one function
 * per step of the paper's method, in the paper's order and notation:
 *
 *   S    = 255 (8-bit scale), R = Vmax - Vmin, Q = S/R    (Section 3, "Quantizing")
 *   V'   = round(Q V) - round(Q Vmin)                      (Section 3.1, eq. 2)
 *   V''  = V' + round(Q Vmin)                              (Section 3.1, eq. 1)
 *   Vc   = Va'' Vb'' / (Qa Qb)                             (Section 3.1, eq. 1)
 *   V    = (V' + round(Q Vmin)) / Q                        (Section 3.1, eq. 3)
 *   y    = F(R(Mult(Q(X), W')) + B)                        (Section 3.1, Fig. 1)
 *
 * Readings where the paper is silent (each one is listed with its reason in
 * the project's design notes):
 *   - Q is formed and applied in fp64; round() is round-half-up done exactly.
 *   - A set whose range is 0, or so narrow that Q*max|V| exceeds 2^24, has its
 *     range widened to include 0; an all-zero set gets Q = 1, zero point 0.
 *   - Codes are clamped to [0, 255] (a guard; the clamp never fires when
 *     rounding is exact).
 *   - The eq. 1 numerator sum_k Va'' Vb'' is an exact int64 sum; its recovery
 *     is ((float)sum * Qa^-1) * Qb^-1 with Q^-1 = (float)(R / S).
 *   - Bias is added after recovery (Fig. 1), gate pre-activations are
 *     (Wx x + b) + Wh h.
 *   - LSTM gate order i, f, g, o; no peepholes; c = f c + i g; m = o tanh(c);
 *     the projection (when present) is linear with no bias.
 *   - sigmoid(x) = 1 / (1 + e^-x), tanh(x) = 2 sigmoid(2x) - 1, with e^x by
 *     Cody-Waite reduction and a Taylor polynomial (oracle_expf), all in fp32
 *     with IEEE division; the reduction and the polynomial use fused
 *     multiply-add (fmaf, one rounding), nothing else is contracted.
 *   - Activations are quantized per vector (one frame of one utterance).
 *   - Softmax posteriors are computed in fp64 from the fp32 logits.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp -fPIC -shared.
 */
#include "qlstm_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_S 255.0 /* the 8-bit scale S of Section 3 */

/* ------------------------------------------------------------------------ */
/* Elementary functions (not given by the paper).                            */
/* ------------------------------------------------------------------------ */

/* e^x after W. J. Cody and W. Waite, "Software Manual for the Elementary
 * Functions" (1980): x = n ln2 + r with n the nearest integer to x / ln2 and
 * ln2 split into a short high part (n * hi is exact) and a low part, so that
 * |r| <= ln2 / 2 (about); e^r is the degree-7 Taylor polynomial of exp
 * evaluated in Horner form; e^x = 2^n e^r by an exact power-of-two scaling.
 * Every multiply-add of the reduction and of Horner's scheme is one fused
 * multiply-add (fmaf), so each step rounds once.  The argument is clamped to
 * [-87, 87], so every result, and 1 / (1 + e^x), is a normal float. */
float oracle_expf(float x) {
  const float log2e = 1.44269504088896340736f;
  const float ln2_hi = 0.693145751953125f;        /* 15 significant bits */
  const float ln2_lo = 1.42860682030941723212e-6f; /* ln 2 - ln2_hi      */
  if (x != x) return x;
  if (x > 87.0f) x = 87.0f;
  if (x < -87.0f) x = -87.0f;
  float n = floorf(fmaf(x, log2e, 0.5f));
  float r = fmaf(-n, ln2_hi, x);
  r = fmaf(-n, ln2_lo, r);
  float p = 1.0f / 5040.0f;
  p = fmaf(p, r, 1.0f / 720.0f);
  p = fmaf(p, r, 1.0f / 120.0f);
  p = fmaf(p, r, 1.0f / 24.0f);
  p = fmaf(p, r, 1.0f / 6.0f);
  p = fmaf(p, r, 0.5f);
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  union {
    uint32_t u;
    float f;
  } two_n;
  two_n.u = (uint32_t)((int32_t)n + 127) << 23;
  return p * two_n.f;
}

float oracle_sigmoidf(float x) { return 1.0f / (1.0f + oracle_expf(-x)); }

float oracle_tanhf(float x) { return 2.0f * oracle_sigmoidf(2.0f * x) - 1.0f; }

/* Elementwise over an array: fn 0 = exp, 1 = sigmoid, 2 = tanh. */
void oracle_elementwise(int32_t fn, const float *x, float *y, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    y[i] = fn == 0 ? oracle_expf(x[i]) : fn == 1 ? oracle_sigmoidf(x[i]) : oracle_tanhf(x[i]);
}

/* ------------------------------------------------------------------------ */
/* Quantizer (Section 3 "Quantizing", Section 3.1 eq. 2)                     */
/* ------------------------------------------------------------------------ */

/* round(): half up, decided exactly.  floor() is exact; x - floor(x) is exact
 * for |x| >= 1, and for -1 < x < 0 its rounding is monotone and cannot cross
 * 0.5 (doubles just below -0.5 are 2^-53 apart), so the tie test is exact. */
int64_t oracle_round_half_up(double x) {
  double r = floor(x);
  if (x - r >= 0.5) r += 1.0;
  return (int64_t)r;
}

/* Range R, factor Q = S / R, zero point round(Q Vmin), recovery Q^-1 = R / S. */
void oracle_qparams(float vmin_f, float vmax_f, orc_qparams *p) {
  double vmin = (double)vmin_f, vmax = (double)vmax_f;
  double R = vmax - vmin;
  double amax = fabs(vmin) > fabs(vmax) ? fabs(vmin) : fabs(vmax);
  if (R == 0.0 || ORC_S * amax > 16777216.0 * R) {
    /* degenerate or ill-conditioned range: widen it to include 0 */
    if (vmin > 0.0) vmin = 0.0;
    if (vmax < 0.0) vmax = 0.0;
    R = vmax - vmin;
  }
  p->vmin = vmin;
  p->vmax = vmax;
  p->R = R;
  if (R == 0.0) { /* all zeros */
    p->Q = 1.0;
    p->z = 0;
    p->inv_q = 1.0f;
    return;
  }
  p->Q = ORC_S / R;
  p->z = (int32_t)oracle_round_half_up(p->Q * vmin);
  p->inv_q = (float)(R / ORC_S);
}

/* eq. 2: V' = round(Q V) - round(Q Vmin), kept within [0, S]. */
uint8_t oracle_code(float v, const orc_qparams *p) {
  int64_t c = oracle_round_half_up(p->Q * (double)v) - (int64_t)p->z;
  if (c < 0) c = 0;
  if (c > 255) c = 255;
  return (uint8_t)c;
}

void oracle_quantize_set(const float *v, int64_t n, uint8_t *codes,
                         orc_qparams *p, int32_t *code_sum) {
  float vmin = 0.0f, vmax = 0.0f;
  for (int64_t i = 0; i < n; ++i) {
    if (i == 0 || v[i] < vmin) vmin = v[i];
    if (i == 0 || v[i] > vmax) vmax = v[i];
  }
  oracle_qparams(vmin, vmax, p);
  int64_t s = 0;
  for (int64_t i = 0; i < n; ++i) {
    codes[i] = oracle_code(v[i], p);
    s += codes[i];
  }
  if (code_sum) *code_sum = (int32_t)s;
}

/* Section 3.1, granularity: each of `nblocks` row blocks (e.g. the four gate
 * matrices of an LSTM weight) is its own quantized set. */
int oracle_quantize(const float *src, int64_t rows, int64_t cols, int32_t nblocks,
                    uint8_t *codes, double *range, int32_t *zero, float *inv_q,
                    int32_t *row_sums) {
  if (rows < 0 || cols < 0 || nblocks <= 0 || rows % nblocks != 0) return -2;
  const int64_t rpb = rows / nblocks;
  for (int32_t blk = 0; blk < nblocks; ++blk) {
    orc_qparams p;
    oracle_quantize_set(src + blk * rpb * cols, rpb * cols,
                        codes + blk * rpb * cols, &p, NULL);
    if (range) range[blk] = p.R;
    if (zero) zero[blk] = p.z;
    if (inv_q) inv_q[blk] = p.inv_q;
  }
  if (row_sums)
    for (int64_t r = 0; r < rows; ++r) {
      int64_t s = 0;
      for (int64_t k = 0; k < cols; ++k) s += codes[r * cols + k];
      row_sums[r] = (int32_t)s;
    }
  return 0;
}

/* eq. 3: V = (V' + round(Q Vmin)) / Q, with 1/Q taken as the fp32 Q^-1. */
int oracle_dequantize(const uint8_t *codes, int64_t rows, int64_t cols,
                      int32_t nblocks, const int32_t *zero, const float *inv_q,
                      float *dst) {
  if (rows < 0 || cols < 0 || nblocks <= 0 || rows % nblocks != 0) return -2;
  const int64_t rpb = rows / nblocks;
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t blk = r / rpb;
    for (int64_t k = 0; k < cols; ++k)
      dst[r * cols + k] =
          (float)((int32_t)codes[r * cols + k] + zero[blk]) * inv_q[blk];
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Quantized product (Section 3.1, eq. 1) and recovery R(.)                  */
/* ------------------------------------------------------------------------ */

/* For one quantized activation vector x' (zero point zx, recovery invqx):
 *   acc[n] = sum_k W'[n][k] x'[k]                      (8-bit products, int32)
 *   tot    = sum_k (W'[n][k] + zW) (x'[k] + zx)        (eq. 1 numerator, V''V'')
 *   y[n]   = ((float)tot * QW^-1) * Qx^-1               (eq. 1 denominator)   */
static void qlinear_vec(const orc_qmat *W, const uint8_t *xc, int32_t zx,
                        float invqx, float *y, int32_t *acc) {
  const int64_t K = W->cols, rpb = W->rows / W->nblocks;
  /* rows are independent; this only runs in parallel when no enclosing
   * parallel region is active (batch of one) */
#pragma omp parallel for schedule(static) if (W->rows * K >= 65536)
  for (int64_t n = 0; n < W->rows; ++n) {
    const uint8_t *w = W->codes + n * K;
    const int64_t blk = n / rpb;
    const int64_t zw = W->zero[blk];
    int64_t a = 0, t = 0;
    for (int64_t k = 0; k < K; ++k) {
      a += (int64_t)w[k] * (int64_t)xc[k];
      t += ((int64_t)w[k] + zw) * ((int64_t)xc[k] + (int64_t)zx);
    }
    if (acc) acc[n] = (int32_t)a;
    y[n] = ((float)t * W->inv_q[blk]) * invqx;
  }
}

static int qmat_ok(const orc_qmat *W) {
  return W && W->codes && W->zero && W->inv_q && W->rows >= 0 && W->cols >= 0 &&
         W->nblocks > 0 && W->rows % W->nblocks == 0;
}

/* Fig. 1: y = R(Mult(Q(X), W')) + B, inputs quantized on the fly. */
int oracle_quantized_matmul(const orc_qmat *W, const float *X, int64_t m,
                            int32_t act_gran, const float *bias, float *Y,
                            int32_t *acc, uint8_t *x_codes, int32_t *x_zero,
                            float *x_inv_q) {
  if (!qmat_ok(W) || m < 0 || (act_gran != 0 && act_gran != 1)) return -2;
  const int64_t K = W->cols, N = W->rows;
  uint8_t *xc = (uint8_t *)malloc((size_t)(m * K > 0 ? m * K : 1));
  int32_t *zx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(m > 0 ? m : 1));
  float *iq = (float *)malloc(sizeof(float) * (size_t)(m > 0 ? m : 1));
  if (act_gran == 0) { /* per tensor: the whole X is one set */
    orc_qparams p;
    oracle_quantize_set(X, m * K, xc, &p, NULL);
    for (int64_t i = 0; i < m; ++i) {
      zx[i] = p.z;
      iq[i] = p.inv_q;
    }
  } else { /* per row: each activation vector is one set */
    for (int64_t i = 0; i < m; ++i) {
      orc_qparams p;
      oracle_quantize_set(X + i * K, K, xc + i * K, &p, NULL);
      zx[i] = p.z;
      iq[i] = p.inv_q;
    }
  }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < m; ++i) {
    qlinear_vec(W, xc + i * K, zx[i], iq[i], Y + i * N, acc ? acc + i * N : NULL);
    if (bias)
      for (int64_t n = 0; n < N; ++n) Y[i * N + n] = Y[i * N + n] + bias[n];
  }
  if (x_codes) memcpy(x_codes, xc, (size_t)(m * K));
  if (x_zero) memcpy(x_zero, zx, sizeof(int32_t) * (size_t)m);
  if (x_inv_q) memcpy(x_inv_q, iq, sizeof(float) * (size_t)m);
  free(xc);
  free(zx);
  free(iq);
  return 0;
}

int oracle_gemm_u8(const uint8_t *A, const uint8_t *B, int32_t *C, int64_t M,
                   int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 0) return -2;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < M; ++i)
    for (int64_t j = 0; j < N; ++j) {
      int64_t s = 0;
      for (int64_t k = 0; k < K; ++k) s += (int64_t)A[i * K + k] * (int64_t)B[j * K + k];
      C[i * N + j] = (int32_t)s;
    }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Quantized LSTM layer (Section 4 architecture; Fig. 1 per matrix product)  */
/* ------------------------------------------------------------------------ */

int oracle_lstm_layer_forward(const orc_layer *L, const float *x, int64_t T,
                              int64_t B, const float *h0, const float *c0,
                              float *h, float *hT, float *cT,
                              const orc_layer_taps *taps) {
  const int64_t H = L->hidden, P = L->proj, IN = L->in;
  const int64_t RD = P ? P : H; /* width of h */
  if (T < 0 || B < 0 || H <= 0 || IN <= 0 || P < 0) return -2;
  if (!qmat_ok(&L->Wx) || L->Wx.rows != 4 * H || L->Wx.cols != IN) return -2;
  if (!qmat_ok(&L->Wh) || L->Wh.rows != 4 * H || L->Wh.cols != RD) return -2;
  if (P && (!qmat_ok(&L->Wr) || L->Wr.rows != P || L->Wr.cols != H)) return -2;
  if (!L->bias) return -2;

#pragma omp parallel for schedule(dynamic, 1) if (B > 1)
  for (int64_t b = 0; b < B; ++b) {
    float *hprev = (float *)calloc((size_t)RD, sizeof(float));
    float *cprev = (float *)calloc((size_t)H, sizeof(float));
    float *yx = (float *)malloc(sizeof(float) * (size_t)(4 * H));
    float *yh = (float *)malloc(sizeof(float) * (size_t)(4 * H));
    float *m = (float *)malloc(sizeof(float) * (size_t)H);
    float *hn = (float *)malloc(sizeof(float) * (size_t)RD);
    uint8_t *xc = (uint8_t *)malloc((size_t)IN);
    uint8_t *hc = (uint8_t *)malloc((size_t)RD);
    uint8_t *mc = (uint8_t *)malloc((size_t)H);
    if (h0) memcpy(hprev, h0 + b * RD, sizeof(float) * (size_t)RD);
    if (c0) memcpy(cprev, c0 + b * H, sizeof(float) * (size_t)H);

    for (int64_t t = 0; t < T; ++t) {
      const int64_t row = t * B + b;
      orc_qparams px, ph;
      /* input product: Q(x_t) on the fly, Mult, R */
      oracle_quantize_set(x + row * IN, IN, xc, &px, NULL);
      qlinear_vec(&L->Wx, xc, px.z, px.inv_q, yx,
                  taps && taps->acc_x ? taps->acc_x + row * 4 * H : NULL);
      /* recurrent product: Q(h_{t-1}), Mult, R */
      oracle_quantize_set(hprev, RD, hc, &ph, NULL);
      qlinear_vec(&L->Wh, hc, ph.z, ph.inv_q, yh,
                  taps && taps->acc_h ? taps->acc_h + row * 4 * H : NULL);
      /* biases, then the activation functions F */
      for (int64_t j = 0; j < H; ++j) {
        const float ai = (yx[j] + L->bias[j]) + yh[j];
        const float af = (yx[H + j] + L->bias[H + j]) + yh[H + j];
        const float ag = (yx[2 * H + j] + L->bias[2 * H + j]) + yh[2 * H + j];
        const float ao = (yx[3 * H + j] + L->bias[3 * H + j]) + yh[3 * H + j];
        const float ig = oracle_sigmoidf(ai);
        const float fg = oracle_sigmoidf(af);
        const float gg = oracle_tanhf(ag);
        const float og = oracle_sigmoidf(ao);
        const float c = (fg * cprev[j]) + (ig * gg);
        cprev[j] = c;
        m[j] = og * oracle_tanhf(c);
        if (taps && taps->preact) {
          float *pa = taps->preact + row * 4 * H;
          pa[j] = ai, pa[H + j] = af, pa[2 * H + j] = ag, pa[3 * H + j] = ao;
        }
        if (taps && taps->gates) {
          float *ga = taps->gates + row * 4 * H;
          ga[j] = ig, ga[H + j] = fg, ga[2 * H + j] = gg, ga[3 * H + j] = og;
        }
      }
      if (taps && taps->m) memcpy(taps->m + row * H, m, sizeof(float) * (size_t)H);
      if (P) { /* linear projection: h = R(Mult(Q(m), Wr')) */
        orc_qparams pm;
        oracle_quantize_set(m, H, mc, &pm, NULL);
        qlinear_vec(&L->Wr, mc, pm.z, pm.inv_q, hn,
                    taps && taps->acc_r ? taps->acc_r + row * P : NULL);
      } else {
        memcpy(hn, m, sizeof(float) * (size_t)H);
      }
      memcpy(h + row * RD, hn, sizeof(float) * (size_t)RD);
      memcpy(hprev, hn, sizeof(float) * (size_t)RD);
      if (taps && taps->c) memcpy(taps->c + row * H, cprev, sizeof(float) * (size_t)H);
      if (taps && taps->h) memcpy(taps->h + row * RD, hn, sizeof(float) * (size_t)RD);
      if (taps && (taps->h_codes || taps->h_zero || taps->h_inv_q)) {
        orc_qparams pn;
        oracle_quantize_set(hn, RD, hc, &pn, NULL);
        if (taps->h_codes) memcpy(taps->h_codes + row * RD, hc, (size_t)RD);
        if (taps->h_zero) taps->h_zero[row] = pn.z;
        if (taps->h_inv_q) taps->h_inv_q[row] = pn.inv_q;
      }
    }
    if (hT) memcpy(hT + b * RD, hprev, sizeof(float) * (size_t)RD);
    if (cT) memcpy(cT + b * H, cprev, sizeof(float) * (size_t)H);
    free(hprev);
    free(cprev);
    free(yx);
    free(yh);
    free(m);
    free(hn);
    free(xc);
    free(hc);
    free(mc);
  }
  return 0;
}

/* softmax of one row of fp32 logits, in fp64 */
static void softmax_row(const float *l, int64_t S, float *p) {
  double mx = (double)l[0];
  for (int64_t s = 1; s < S; ++s)
    if ((double)l[s] > mx) mx = (double)l[s];
  double sum = 0.0;
  for (int64_t s = 0; s < S; ++s) sum += exp((double)l[s] - mx);
  for (int64_t s = 0; s < S; ++s) p[s] = (float)(exp((double)l[s] - mx) / sum);
}

/* Section 4: stacked LSTM layers, then the output layer, quantized as every
 * other layer ('quant-all', Section 5), then softmax. */
int oracle_acoustic_model_forward(const orc_model *M, const float *feats,
                                  int64_t T, int64_t B, float *post,
                                  const orc_layer_taps *layer_taps,
                                  int32_t *acc_y, float *logits) {
  if (!M || M->nlayers <= 0 || !M->layers || !qmat_ok(&M->Wy) || !M->by) return -2;
  const float *x = feats;
  float *prev = NULL;
  int64_t width = M->layers[0].in;
  for (int32_t l = 0; l < M->nlayers; ++l) {
    const orc_layer *L = &M->layers[l];
    if (L->in != width) return -2;
    const int64_t RD = L->proj ? L->proj : L->hidden;
    float *hl = (float *)malloc(sizeof(float) * (size_t)(T * B * RD > 0 ? T * B * RD : 1));
    int rc = oracle_lstm_layer_forward(L, x, T, B, NULL, NULL, hl, NULL, NULL,
                                       layer_taps ? &layer_taps[l] : NULL);
    free(prev);
    if (rc) {
      free(hl);
      return rc;
    }
    prev = hl;
    x = hl;
    width = RD;
  }
  if (M->Wy.cols != width) {
    free(prev);
    return -2;
  }
  const int64_t S = M->Wy.rows;
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < T * B; ++row) {
    uint8_t *xc = (uint8_t *)malloc((size_t)width);
    float *lg = (float *)malloc(sizeof(float) * (size_t)S);
    orc_qparams p;
    oracle_quantize_set(x + row * width, width, xc, &p, NULL);
    qlinear_vec(&M->Wy, xc, p.z, p.inv_q, lg, acc_y ? acc_y + row * S : NULL);
    for (int64_t s = 0; s < S; ++s) lg[s] = lg[s] + M->by[s];
    if (logits) memcpy(logits + row * S, lg, sizeof(float) * (size_t)S);
    softmax_row(lg, S, post + row * S);
    free(xc);
    free(lg);
  }
  free(prev);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Unquantized fp32 model (the 'match' condition of Section 5)               */
/* ------------------------------------------------------------------------ */

static void flinear_vec(const float *W, int64_t N, int64_t K, const float *x,
                        float *y) {
  for (int64_t n = 0; n < N; ++n) {
    double s = 0.0;
    for (int64_t k = 0; k < K; ++k) s += (double)W[n * K + k] * (double)x[k];
    y[n] = (float)s;
  }
}

int oracle_lstm_layer_forward_f32(const orc_layer_f32 *L, const float *x,
                                  int64_t T, int64_t B, const float *h0,
                                  const float *c0, float *h, float *hT, float *cT,
                                  const orc_layer_taps *taps) {
  const int64_t H = L->hidden, P = L->proj, IN = L->in;
  const int64_t RD = P ? P : H;
  if (T < 0 || B < 0 || H <= 0 || IN <= 0 || P < 0 || !L->Wx || !L->Wh || !L->bias ||
      (P && !L->Wr))
    return -2;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t b = 0; b < B; ++b) {
    float *hprev = (float *)calloc((size_t)RD, sizeof(float));
    float *cprev = (float *)calloc((size_t)H, sizeof(float));
    float *yx = (float *)malloc(sizeof(float) * (size_t)(4 * H));
    float *yh = (float *)malloc(sizeof(float) * (size_t)(4 * H));
    float *m = (float *)malloc(sizeof(float) * (size_t)H);
    float *hn = (float *)malloc(sizeof(float) * (size_t)RD);
    if (h0) memcpy(hprev, h0 + b * RD, sizeof(float) * (size_t)RD);
    if (c0) memcpy(cprev, c0 + b * H, sizeof(float) * (size_t)H);
    for (int64_t t = 0; t < T; ++t) {
      const int64_t row = t * B + b;
      flinear_vec(L->Wx, 4 * H, IN, x + row * IN, yx);
      flinear_vec(L->Wh, 4 * H, RD, hprev, yh);
      for (int64_t j = 0; j < H; ++j) {
        const float ig = oracle_sigmoidf((yx[j] + L->bias[j]) + yh[j]);
        const float fg = oracle_sigmoidf((yx[H + j] + L->bias[H + j]) + yh[H + j]);
        const float gg = oracle_tanhf((yx[2 * H + j] + L->bias[2 * H + j]) + yh[2 * H + j]);
        const float og = oracle_sigmoidf((yx[3 * H + j] + L->bias[3 * H + j]) + yh[3 * H + j]);
        const float c = (fg * cprev[j]) + (ig * gg);
        cprev[j] = c;
        m[j] = og * oracle_tanhf(c);
        if (taps && taps->gates) {
          float *ga = taps->gates + row * 4 * H;
          ga[j] = ig, ga[H + j] = fg, ga[2 * H + j] = gg, ga[3 * H + j] = og;
        }
      }
      if (P)
        flinear_vec(L->Wr, P, H, m, hn);
      else
        memcpy(hn, m, sizeof(float) * (size_t)H);
      memcpy(h + row * RD, hn, sizeof(float) * (size_t)RD);
      memcpy(hprev, hn, sizeof(float) * (size_t)RD);
      if (taps && taps->c) memcpy(taps->c + row * H, cprev, sizeof(float) * (size_t)H);
      if (taps && taps->m) memcpy(taps->m + row * H, m, sizeof(float) * (size_t)H);
      if (taps && taps->h) memcpy(taps->h + row * RD, hn, sizeof(float) * (size_t)RD);
    }
    if (hT) memcpy(hT + b * RD, hprev, sizeof(float) * (size_t)RD);
    if (cT) memcpy(cT + b * H, cprev, sizeof(float) * (size_t)H);
    free(hprev);
    free(cprev);
    free(yx);
    free(yh);
    free(m);
    free(hn);
  }
  return 0;
}

int oracle_acoustic_model_forward_f32(const orc_model_f32 *M, const float *feats,
                                      int64_t T, int64_t B, float *post) {
  if (!M || M->nlayers <= 0 || !M->layers || !M->Wy || !M->by) return -2;
  const float *x = feats;
  float *prev = NULL;
  int64_t width = M->layers[0].in;
  for (int32_t l = 0; l < M->nlayers; ++l) {
    const orc_layer_f32 *L = &M->layers[l];
    if (L->in != width) return -2;
    const int64_t RD = L->proj ? L->proj : L->hidden;
    float *hl = (float *)malloc(sizeof(float) * (size_t)(T * B * RD > 0 ? T * B * RD : 1));
    int rc = oracle_lstm_layer_forward_f32(L, x, T, B, NULL, NULL, hl, NULL, NULL, NULL);
    free(prev);
    if (rc) {
      free(hl);
      return rc;
    }
    prev = hl;
    x = hl;
    width = RD;
  }
  const int64_t S = M->S;
  if (S <= 0) {
    free(prev);
    return -2;
  }
#pragma omp parallel for schedule(static)
  for (int64_t row = 0; row < T * B; ++row) {
    float *lg = (float *)malloc(sizeof(float) * (size_t)S);
    flinear_vec(M->Wy, S, width, x + row * width, lg);
    for (int64_t s = 0; s < S; ++s) lg[s] = lg[s] + M->by[s];
    softmax_row(lg, S, post + row * S);
    free(lg);
  }
  free(prev);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Quantization aware training (Section 3.2, Algorithm 1)                    */
/*                                                                           */
/* The forward pass runs in quantized form (infer-and-recover: the inference */
/* path above, on freshly quantized copies of the float parameters); the     */
/* error, the gradients and the update are ordinary floating-point           */
/* backpropagation with the float parameters, evaluated at the activations   */
/* the quantized forward pass produced.  Quantization itself is not          */
/* differentiated.  Float arithmetic of the backward pass is done in fp64.   */
/* ------------------------------------------------------------------------ */

/* LSTM backward through time, one layer (gate order i, f, g, o; c = f c + i g;
 * m = o tanh(c); h = m, or h = Wr m with a projection; zero initial state). */
int oracle_lstm_layer_backward(const orc_layer_f32 *L, const float *x, int64_t T, int64_t B,
                               const float *gates, const float *c, const float *m,
                               const float *h, const float *dy, float *dWx, float *dWh,
                               float *dWr, float *db, float *dx) {
  const int64_t H = L->hidden, P = L->proj, IN = L->in;
  const int64_t RD = P ? P : H, G = 4 * H, N = T * B;
  if (T < 0 || B < 0 || H <= 0 || IN <= 0 || P < 0 || !L->Wx || !L->Wh || (P && !L->Wr))
    return -2;
  if (N > 0 && (!x || !gates || !c || !m || !h || !dy)) return -2;
  /* dC/da for every step: the serial part, one utterance at a time */
  double *da = (double *)calloc((size_t)(N * G > 0 ? N * G : 1), sizeof(double));
  double *dh_all = (double *)calloc((size_t)(N * RD > 0 ? N * RD : 1), sizeof(double));
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t b = 0; b < B; ++b) {
    double *dh_next = (double *)calloc((size_t)RD, sizeof(double)); /* via W_h from step t+1 */
    double *dc_next = (double *)calloc((size_t)H, sizeof(double));  /* via f from step t+1 */
    double *dm = (double *)malloc(sizeof(double) * (size_t)H);
    for (int64_t t = T - 1; t >= 0; --t) {
      const int64_t row = t * B + b;
      double *dh = dh_all + row * RD;
      for (int64_t k = 0; k < RD; ++k) dh[k] = (double)dy[row * RD + k] + dh_next[k];
      if (P) { /* h = Wr m: dC/dm = Wr^T dC/dh */
        for (int64_t j = 0; j < H; ++j) {
          double s = 0.0;
          for (int64_t p = 0; p < P; ++p) s += (double)L->Wr[p * H + j] * dh[p];
          dm[j] = s;
        }
      } else {
        for (int64_t j = 0; j < H; ++j) dm[j] = dh[j];
      }
      const float *gt = gates + row * G;
      double *dat = da + row * G;
      for (int64_t j = 0; j < H; ++j) {
        const double ig = gt[j], fg = gt[H + j], gg = gt[2 * H + j], og = gt[3 * H + j];
        const double ct = c[row * H + j];
        const double cp = t > 0 ? (double)c[(row - B) * H + j] : 0.0;
        const double tc = tanh(ct);
        const double d_o = dm[j] * tc;
        const double d_c = dm[j] * og * (1.0 - tc * tc) + dc_next[j];
        const double d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * cp;
        dc_next[j] = d_c * fg;
        dat[j] = d_i * ig * (1.0 - ig);         /* sigmoid' = s (1 - s) */
        dat[H + j] = d_f * fg * (1.0 - fg);
        dat[2 * H + j] = d_g * (1.0 - gg * gg); /* tanh' = 1 - tanh^2 */
        dat[3 * H + j] = d_o * og * (1.0 - og);
      }
      /* to h_{t-1} through W_h */
      for (int64_t k = 0; k < RD; ++k) {
        double s = 0.0;
        for (int64_t n = 0; n < G; ++n) s += (double)L->Wh[n * RD + k] * dat[n];
        dh_next[k] = s;
      }
    }
    free(dh_next);
    free(dc_next);
    free(dm);
  }
  /* gradients of the parameters: sums over all T*B frames */
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < G; ++n) {
    double sb = 0.0;
    for (int64_t r = 0; r < N; ++r) sb += da[r * G + n];
    if (db) db[n] = (float)sb;
    if (dWx)
      for (int64_t i = 0; i < IN; ++i) {
        double s = 0.0;
        for (int64_t r = 0; r < N; ++r) s += da[r * G + n] * (double)x[r * IN + i];
        dWx[n * IN + i] = (float)s;
      }
    if (dWh)
      for (int64_t k = 0; k < RD; ++k) {
        double s = 0.0; /* h_{t-1} = 0 at t = 0 */
        for (int64_t r = B; r < N; ++r) s += da[r * G + n] * (double)h[(r - B) * RD + k];
        dWh[n * RD + k] = (float)s;
      }
  }
  if (P && dWr) {
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < P; ++p)
      for (int64_t j = 0; j < H; ++j) {
        double s = 0.0;
        for (int64_t r = 0; r < N; ++r) s += dh_all[r * RD + p] * (double)m[r * H + j];
        dWr[p * H + j] = (float)s;
      }
  }
  if (dx) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < N; ++r)
      for (int64_t i = 0; i < IN; ++i) {
        double s = 0.0;
        for (int64_t n = 0; n < G; ++n) s += (double)L->Wx[n * IN + i] * da[r * G + n];
        dx[r * IN + i] = (float)s;
      }
  }
  free(da);
  free(dh_all);
  return 0;
}

/* C = -(1/N) sum_r log p_r[target_r]; dC/dz = (p - onehot) / N for the
 * softmax of z = Wy hL + by. */
int oracle_output_backward(const float *Wy, int64_t S, int64_t R, const float *hL,
                           const float *post, const int32_t *targets, int64_t N,
                           double *loss, float *dWy, float *dby, float *dhL) {
  if (S <= 0 || R <= 0 || N < 0 || !Wy) return -2;
  for (int64_t r = 0; r < N; ++r)
    if (targets[r] < 0 || targets[r] >= S) return -2;
  double *dz = (double *)malloc(sizeof(double) * (size_t)(N * S > 0 ? N * S : 1));
  double l = 0.0;
  for (int64_t r = 0; r < N; ++r) {
    l -= log((double)post[r * S + targets[r]]);
    for (int64_t s = 0; s < S; ++s)
      dz[r * S + s] = ((double)post[r * S + s] - (s == targets[r] ? 1.0 : 0.0)) / (double)N;
  }
  if (loss) *loss = N > 0 ? l / (double)N : 0.0;
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < S; ++s) {
    double sb = 0.0;
    for (int64_t r = 0; r < N; ++r) sb += dz[r * S + s];
    if (dby) dby[s] = (float)sb;
    if (dWy)
      for (int64_t k = 0; k < R; ++k) {
        double sw = 0.0;
        for (int64_t r = 0; r < N; ++r) sw += dz[r * S + s] * (double)hL[r * R + k];
        dWy[s * R + k] = (float)sw;
      }
  }
  if (dhL) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < N; ++r)
      for (int64_t k = 0; k < R; ++k) {
        double sh = 0.0;
        for (int64_t s = 0; s < S; ++s) sh += (double)Wy[s * R + k] * dz[r * S + s];
        dhL[r * R + k] = (float)sh;
      }
  }
  free(dz);
  return 0;
}

/* One quantized copy of a float matrix (w^q of Algorithm 1). */
typedef struct {
  uint8_t *codes;
  int32_t *zero;
  float *inv_q;
  orc_qmat q;
} orc_qcopy;
static void qcopy_make(orc_qcopy *c, const float *W, int64_t rows, int64_t cols, int32_t nb) {
  c->codes = (uint8_t *)malloc((size_t)(rows * cols > 0 ? rows * cols : 1));
  c->zero = (int32_t *)malloc(sizeof(int32_t) * (size_t)nb);
  c->inv_q = (float *)malloc(sizeof(float) * (size_t)nb);
  oracle_quantize(W, rows, cols, nb, c->codes, NULL, c->zero, c->inv_q, NULL);
  c->q.rows = rows;
  c->q.cols = cols;
  c->q.nblocks = nb;
  c->q.codes = c->codes;
  c->q.zero = c->zero;
  c->q.inv_q = c->inv_q;
}
static void qcopy_free(orc_qcopy *c) {
  free(c->codes);
  free(c->zero);
  free(c->inv_q);
}

int oracle_train_step(const orc_train_model *M, const float *feats, const int32_t *targets,
                      int64_t T, int64_t B, float lr, int32_t gate_blocks,
                      int32_t quantize_layers, int32_t quantize_output, double *loss,
                      const orc_train_model *grads) {
  if (!M || M->nlayers <= 0 || !M->layers || !M->Wy || !M->by || M->S <= 0) return -2;
  if (T < 0 || B < 0 || gate_blocks <= 0 || (quantize_output && !quantize_layers)) return -2;
  if (!grads || !grads->layers || !grads->Wy || !grads->by) return -2;
  const int32_t NL = M->nlayers;
  const int64_t N = T * B, S = M->S;
  int64_t width = M->layers[0].in;
  for (int32_t l = 0; l < NL; ++l) {
    const orc_train_layer *L = &M->layers[l];
    if (L->in != width || (4 * L->hidden) % gate_blocks != 0) return -2;
    width = L->proj ? L->proj : L->hidden;
  }
  const int64_t RL = width;

  /* 1. w^q <- quantize(w) */
  orc_qcopy *qx = (orc_qcopy *)calloc((size_t)NL, sizeof(orc_qcopy));
  orc_qcopy *qh = (orc_qcopy *)calloc((size_t)NL, sizeof(orc_qcopy));
  orc_qcopy *qr = (orc_qcopy *)calloc((size_t)NL, sizeof(orc_qcopy));
  orc_qcopy qy;
  memset(&qy, 0, sizeof(qy));
  if (quantize_layers)
    for (int32_t l = 0; l < NL; ++l) {
      const orc_train_layer *L = &M->layers[l];
      const int64_t RD = L->proj ? L->proj : L->hidden;
      qcopy_make(&qx[l], L->Wx, 4 * L->hidden, L->in, gate_blocks);
      qcopy_make(&qh[l], L->Wh, 4 * L->hidden, RD, gate_blocks);
      if (L->proj) qcopy_make(&qr[l], L->Wr, L->proj, L->hidden, 1);
    }
  if (quantize_output) qcopy_make(&qy, M->Wy, S, RL, 1);

  /* 2. a_k <- infer-and-recover(a_{k-1}, w^q, b), keeping what the backward
   *    pass needs: every layer's input, gates, c, m and h */
  float **xin = (float **)calloc((size_t)NL + 1, sizeof(float *));
  float **gat = (float **)calloc((size_t)NL, sizeof(float *));
  float **cst = (float **)calloc((size_t)NL, sizeof(float *));
  float **mo = (float **)calloc((size_t)NL, sizeof(float *));
  xin[0] = (float *)feats;
  int rc = 0;
  for (int32_t l = 0; l < NL && rc == 0; ++l) {
    const orc_train_layer *L = &M->layers[l];
    const int64_t H = L->hidden, RD = L->proj ? L->proj : H;
    xin[l + 1] = (float *)malloc(sizeof(float) * (size_t)(N * RD > 0 ? N * RD : 1));
    gat[l] = (float *)malloc(sizeof(float) * (size_t)(N * 4 * H > 0 ? N * 4 * H : 1));
    cst[l] = (float *)malloc(sizeof(float) * (size_t)(N * H > 0 ? N * H : 1));
    mo[l] = (float *)malloc(sizeof(float) * (size_t)(N * H > 0 ? N * H : 1));
    orc_layer_taps tp;
    memset(&tp, 0, sizeof(tp));
    tp.gates = gat[l];
    tp.c = cst[l];
    tp.m = mo[l];
    if (quantize_layers) {
      orc_layer ql;
      ql.in = L->in;
      ql.hidden = H;
      ql.proj = L->proj;
      ql.Wx = qx[l].q;
      ql.Wh = qh[l].q;
      if (L->proj) ql.Wr = qr[l].q;
      else memset(&ql.Wr, 0, sizeof(ql.Wr));
      ql.bias = L->bias;
      rc = oracle_lstm_layer_forward(&ql, xin[l], T, B, NULL, NULL, xin[l + 1], NULL, NULL, &tp);
    } else {
      orc_layer_f32 fl = {L->in, H, L->proj, L->Wx, L->Wh, L->Wr, L->bias};
      rc = oracle_lstm_layer_forward_f32(&fl, xin[l], T, B, NULL, NULL, xin[l + 1], NULL, NULL,
                                         &tp);
    }
  }
  float *post = (float *)malloc(sizeof(float) * (size_t)(N * S > 0 ? N * S : 1));
  float *dh = (float *)malloc(sizeof(float) * (size_t)(N * RL > 0 ? N * RL : 1));
  if (rc == 0) {
    const float *hL = xin[NL];
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < N; ++r) {
      float *lg = (float *)malloc(sizeof(float) * (size_t)S);
      if (quantize_output) { /* 'quant-all': the output layer quantized too */
        uint8_t *hc = (uint8_t *)malloc((size_t)RL);
        orc_qparams p;
        oracle_quantize_set(hL + r * RL, RL, hc, &p, NULL);
        qlinear_vec(&qy.q, hc, p.z, p.inv_q, lg, NULL);
        free(hc);
      } else { /* 'quant': a float output layer */
        flinear_vec(M->Wy, S, RL, hL + r * RL, lg);
      }
      for (int64_t s = 0; s < S; ++s) lg[s] = lg[s] + M->by[s];
      softmax_row(lg, S, post + r * S);
      free(lg);
    }
    /* 3. output error, then the layers from the top (float parameters) */
    double l = 0.0;
    rc = oracle_output_backward(M->Wy, S, RL, hL, post, targets, N, &l,
                                grads->Wy, grads->by, dh);
    if (loss) *loss = l;
  }
  for (int32_t l = NL - 1; l >= 0 && rc == 0; --l) {
    const orc_train_layer *L = &M->layers[l];
    const orc_layer_f32 fl = {L->in, L->hidden, L->proj, L->Wx, L->Wh, L->Wr, L->bias};
    float *dx = l > 0 ? (float *)malloc(sizeof(float) * (size_t)(N * L->in > 0 ? N * L->in : 1))
                      : NULL;
    const orc_train_layer *g = &grads->layers[l];
    rc = oracle_lstm_layer_backward(&fl, xin[l], T, B, gat[l], cst[l], mo[l], xin[l + 1], dh,
                                    g->Wx, g->Wh, g->Wr, g->bias, dx);
    free(dh);
    dh = dx;
  }
  free(dh);
  /* 4. w <- w - lr dC/dw (fp32): every weight and bias */
  if (rc == 0) {
    for (int32_t l = 0; l < NL; ++l) {
      const orc_train_layer *L = &M->layers[l], *g = &grads->layers[l];
      const int64_t H = L->hidden, RD = L->proj ? L->proj : H;
      for (int64_t i = 0; i < 4 * H * L->in; ++i) L->Wx[i] = L->Wx[i] - lr * g->Wx[i];
      for (int64_t i = 0; i < 4 * H * RD; ++i) L->Wh[i] = L->Wh[i] - lr * g->Wh[i];
      for (int64_t i = 0; i < 4 * H; ++i) L->bias[i] = L->bias[i] - lr * g->bias[i];
      if (L->proj)
        for (int64_t i = 0; i < L->proj * H; ++i) L->Wr[i] = L->Wr[i] - lr * g->Wr[i];
    }
    for (int64_t i = 0; i < S * RL; ++i) M->Wy[i] = M->Wy[i] - lr * grads->Wy[i];
    for (int64_t i = 0; i < S; ++i) M->by[i] = M->by[i] - lr * grads->by[i];
  }
  for (int32_t l = 0; l < NL; ++l) {
    if (quantize_layers) {
      qcopy_free(&qx[l]);
      qcopy_free(&qh[l]);
      if (M->layers[l].proj) qcopy_free(&qr[l]);
    }
    free(xin[l + 1]);
    free(gat[l]);
    free(cst[l]);
    free(mo[l]);
  }
  if (quantize_output) qcopy_free(&qy);
  free(qx);
  free(qh);
  free(qr);
  free(xin);
  free(gat);
  free(cst);
  free(mo);
  free(post);
  return rc;
}
