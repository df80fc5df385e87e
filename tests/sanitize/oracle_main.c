/* Runs every entry point of the CPU oracle on small, ragged and degenerate
 * shapes so that a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * sees each of its code paths: quantizer (per matrix, per gate block, per
 * row, constant and all-zero sets), the quantized product (per tensor and per
 * row, all outputs), the 8-bit GEMM, the quantized and fp32 LSTM layers with
 * and without projection (initial state, final state, every tap), both model
 * forwards, the layer and output backward passes and the training step in its
 * three modes.  Exit status 0 when every call returned 0 and the checked
 * invariants hold.  Test infrastructure: built and run by the test suite. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "qlstm_oracle.h"

static unsigned long long g_state = 0x9E3779B97F4A7C15ull;

/* uniform in [lo, hi) from a 64-bit LCG (inputs only; no method arithmetic) */
static float uni(float lo, float hi) {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return lo + (hi - lo) * (float)((g_state >> 40) * (1.0 / 16777216.0));
}

static float *fill(int64_t n, float lo, float hi) {
  float *p = malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
  for (int64_t i = 0; i < n; ++i) p[i] = uni(lo, hi);
  return p;
}

static int g_fail = 0;
#define CHECK(cond)                                                     \
  do {                                                                  \
    if (!(cond)) {                                                      \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      g_fail = 1;                                                       \
    }                                                                   \
  } while (0)

/* A quantized matrix with its storage. */
typedef struct {
  orc_qmat m;
  uint8_t *codes;
  int32_t *zero, *row_sums;
  float *inv_q;
  double *range;
} qm_t;

static qm_t make_qm(const float *src, int64_t rows, int64_t cols, int32_t nblocks) {
  qm_t q;
  q.codes = malloc((size_t)(rows * cols > 0 ? rows * cols : 1));
  q.zero = malloc(sizeof(int32_t) * (size_t)nblocks);
  q.inv_q = malloc(sizeof(float) * (size_t)nblocks);
  q.range = malloc(sizeof(double) * (size_t)nblocks);
  q.row_sums = malloc(sizeof(int32_t) * (size_t)(rows > 0 ? rows : 1));
  CHECK(oracle_quantize(src, rows, cols, nblocks, q.codes, q.range, q.zero, q.inv_q,
                        q.row_sums) == 0);
  q.m.rows = rows, q.m.cols = cols, q.m.nblocks = nblocks;
  q.m.codes = q.codes, q.m.zero = q.zero, q.m.inv_q = q.inv_q;
  return q;
}

static void free_qm(qm_t *q) {
  free(q->codes), free(q->zero), free(q->inv_q), free(q->range), free(q->row_sums);
}

static void scalars(void) {
  float x[9] = {-100.f, -87.5f, -3.f, -1e-7f, 0.f, 1e-7f, 2.5f, 87.5f, 100.f}, y[9];
  for (int fn = 0; fn < 3; ++fn) oracle_elementwise(fn, x, y, 9);
  CHECK(y[4] == 0.f && y[0] == -1.f && y[8] == 1.f);  /* tanh */
  orc_qparams p;
  oracle_qparams(0.f, 0.f, &p);
  CHECK(oracle_code(0.f, &p) == 0);
  oracle_qparams(-1.f, 3.f, &p);
  CHECK(oracle_code(-1.f, &p) == 0 && oracle_code(3.f, &p) == 255);
  oracle_qparams(1e-30f, 1e-30f, &p);
  oracle_qparams(5.f, 5.f + 1e-6f, &p);
  CHECK(oracle_round_half_up(2.5) == 3 && oracle_round_half_up(-2.5) == -2);
}

static void quantizer(void) {
  const int64_t rows = 12, cols = 7;
  float *w = fill(rows * cols, -1.f, 1.f);
  const int32_t blocks[4] = {1, 4, 12, 3};
  for (int i = 0; i < 4; ++i) {
    qm_t q = make_qm(w, rows, cols, blocks[i]);
    float *back = malloc(sizeof(float) * rows * cols);
    CHECK(oracle_dequantize(q.codes, rows, cols, blocks[i], q.zero, q.inv_q, back) == 0);
    for (int64_t k = 0; k < rows * cols; ++k) CHECK(fabsf(back[k] - w[k]) <= 2.f / 255.f);
    free(back);
    free_qm(&q);
  }
  float zeros[20] = {0}, consts[20];
  for (int k = 0; k < 20; ++k) consts[k] = 0.75f;
  qm_t z = make_qm(zeros, 4, 5, 4), c = make_qm(consts, 4, 5, 1);
  free_qm(&z), free_qm(&c);
  uint8_t codes[20];
  orc_qparams p;
  int32_t sum = 0;
  oracle_quantize_set(consts, 20, codes, &p, &sum);
  oracle_quantize_set(consts, 0, codes, &p, &sum);
  free(w);
}

static void products(void) {
  const int64_t rows = 9, K = 33, m = 5;
  float *w = fill(rows * K, -0.5f, 0.5f), *x = fill(m * K, -1.f, 1.f), *b = fill(rows, -1.f, 1.f);
  qm_t q = make_qm(w, rows, K, 1);
  float *y = malloc(sizeof(float) * m * rows);
  int32_t *acc = malloc(sizeof(int32_t) * m * rows), *xz = malloc(sizeof(int32_t) * m);
  uint8_t *xc = malloc((size_t)(m * K));
  float *xi = malloc(sizeof(float) * m);
  for (int gran = 0; gran < 2; ++gran) {
    CHECK(oracle_quantized_matmul(&q.m, x, m, gran, b, y, acc, xc, xz, xi) == 0);
    CHECK(oracle_quantized_matmul(&q.m, x, m, gran, NULL, y, NULL, NULL, NULL, NULL) == 0);
  }
  CHECK(oracle_quantized_matmul(&q.m, x, 0, 1, b, y, acc, xc, xz, xi) == 0);
  int32_t *c = malloc(sizeof(int32_t) * m * rows);
  CHECK(oracle_gemm_u8(xc, q.codes, c, m, rows, K) == 0);
  CHECK(oracle_gemm_u8(xc, q.codes, c, m, rows, 1) == 0);
  free(c), free(y), free(acc), free(xz), free(xc), free(xi), free(w), free(x), free(b);
  free_qm(&q);
}

/* One layer's float weights and their quantized copies. */
typedef struct {
  int64_t in, H, P;
  float *Wx, *Wh, *Wr, *b;
  qm_t qx, qh, qr;
  orc_layer q;
  orc_layer_f32 f;
  orc_train_layer t;
} layer_t;

static void make_layer(layer_t *L, int64_t in, int64_t H, int64_t P, int32_t gate_blocks) {
  const int64_t R = P ? P : H;
  L->in = in, L->H = H, L->P = P;
  L->Wx = fill(4 * H * in, -0.3f, 0.3f);
  L->Wh = fill(4 * H * R, -0.3f, 0.3f);
  L->Wr = P ? fill(P * H, -0.3f, 0.3f) : NULL;
  L->b = fill(4 * H, -0.2f, 0.2f);
  L->qx = make_qm(L->Wx, 4 * H, in, gate_blocks);
  L->qh = make_qm(L->Wh, 4 * H, R, gate_blocks);
  memset(&L->q, 0, sizeof L->q);
  L->q.in = in, L->q.hidden = H, L->q.proj = P;
  L->q.Wx = L->qx.m, L->q.Wh = L->qh.m, L->q.bias = L->b;
  if (P) {
    L->qr = make_qm(L->Wr, P, H, 1);
    L->q.Wr = L->qr.m;
  }
  L->f.in = in, L->f.hidden = H, L->f.proj = P;
  L->f.Wx = L->Wx, L->f.Wh = L->Wh, L->f.Wr = L->Wr, L->f.bias = L->b;
  L->t.in = in, L->t.hidden = H, L->t.proj = P;
  L->t.Wx = L->Wx, L->t.Wh = L->Wh, L->t.Wr = L->Wr, L->t.bias = L->b;
}

static void free_layer(layer_t *L) {
  free(L->Wx), free(L->Wh), free(L->Wr), free(L->b);
  free_qm(&L->qx), free_qm(&L->qh);
  if (L->P) free_qm(&L->qr);
}

typedef struct {
  orc_layer_taps t;
  void *mem[11];
} taps_t;

static void make_taps(taps_t *tp, int64_t T, int64_t B, int64_t H, int64_t P) {
  const int64_t R = P ? P : H, n = T * B > 0 ? T * B : 1;
  void **m = tp->mem;
  tp->t.acc_x = m[0] = malloc(sizeof(int32_t) * n * 4 * H);
  tp->t.acc_h = m[1] = malloc(sizeof(int32_t) * n * 4 * H);
  tp->t.acc_r = m[2] = malloc(sizeof(int32_t) * n * (P ? P : 1));
  tp->t.h_codes = m[3] = malloc((size_t)(n * R));
  tp->t.h_zero = m[4] = malloc(sizeof(int32_t) * n);
  tp->t.h_inv_q = m[5] = malloc(sizeof(float) * n);
  tp->t.c = m[6] = malloc(sizeof(float) * n * H);
  tp->t.h = m[7] = malloc(sizeof(float) * n * R);
  tp->t.preact = m[8] = malloc(sizeof(float) * n * 4 * H);
  tp->t.gates = m[9] = malloc(sizeof(float) * n * 4 * H);
  tp->t.m = m[10] = malloc(sizeof(float) * n * H);
  if (!P) tp->t.acc_r = NULL;
}

static void free_taps(taps_t *tp) {
  for (int i = 0; i < 11; ++i) free(tp->mem[i]);
}

static void layers(void) {
  const int64_t T = 6, B = 3, in = 11;
  const int64_t shapes[3][2] = {{9, 0}, {9, 5}, {1, 0}};  /* H, P */
  for (int s = 0; s < 3; ++s) {
    const int64_t H = shapes[s][0], P = shapes[s][1], R = P ? P : H;
    layer_t L;
    make_layer(&L, in, H, P, H % 4 == 0 || H == 9 ? 4 : 1);
    float *x = fill(T * B * in, -1.f, 1.f), *h0 = fill(B * R, -0.5f, 0.5f),
          *c0 = fill(B * H, -0.5f, 0.5f);
    float *h = malloc(sizeof(float) * T * B * R), *hT = malloc(sizeof(float) * B * R),
          *cT = malloc(sizeof(float) * B * H);
    taps_t tp;
    make_taps(&tp, T, B, H, P);
    CHECK(oracle_lstm_layer_forward(&L.q, x, T, B, h0, c0, h, hT, cT, &tp.t) == 0);
    CHECK(oracle_lstm_layer_forward(&L.q, x, T, B, NULL, NULL, h, NULL, NULL, NULL) == 0);
    CHECK(oracle_lstm_layer_forward(&L.q, x, 0, B, NULL, NULL, h, NULL, NULL, NULL) == 0);
    CHECK(oracle_lstm_layer_forward_f32(&L.f, x, T, B, h0, c0, h, hT, cT, &tp.t) == 0);
    CHECK(oracle_lstm_layer_forward_f32(&L.f, x, T, B, NULL, NULL, h, NULL, NULL, NULL) == 0);
    /* the float backward at the float forward's activations */
    float *dy = fill(T * B * R, -1.f, 1.f);
    float *dWx = malloc(sizeof(float) * 4 * H * in), *dWh = malloc(sizeof(float) * 4 * H * R),
          *dWr = malloc(sizeof(float) * (P ? P * H : 1)), *db = malloc(sizeof(float) * 4 * H),
          *dx = malloc(sizeof(float) * T * B * in);
    CHECK(oracle_lstm_layer_forward_f32(&L.f, x, T, B, NULL, NULL, h, NULL, NULL, &tp.t) == 0);
    CHECK(oracle_lstm_layer_backward(&L.f, x, T, B, tp.t.gates, tp.t.c, tp.t.m, tp.t.h, dy, dWx,
                                     dWh, P ? dWr : NULL, db, dx) == 0);
    CHECK(oracle_lstm_layer_backward(&L.f, x, T, B, tp.t.gates, tp.t.c, tp.t.m, tp.t.h, dy, NULL,
                                     NULL, NULL, NULL, NULL) == 0);
    free(dy), free(dWx), free(dWh), free(dWr), free(db), free(dx);
    free_taps(&tp);
    free(x), free(h0), free(c0), free(h), free(hT), free(cT);
    free_layer(&L);
  }
}

static void models_and_training(void) {
  const int64_t T = 5, B = 2, in = 8, S = 7;
  const int64_t dims[2][2] = {{12, 0}, {8, 4}};  /* H, P of layers 0 and 1 */
  for (int proj = 0; proj < 2; ++proj) {
    layer_t L[2];
    int64_t width = in;
    for (int l = 0; l < 2; ++l) {
      const int64_t H = dims[l][0], P = proj ? dims[l][1] : 0;
      make_layer(&L[l], width, H, P, 4);
      width = P ? P : H;
    }
    float *Wy = fill(S * width, -0.3f, 0.3f), *by = fill(S, -0.1f, 0.1f);
    qm_t qy = make_qm(Wy, S, width, 1);
    orc_layer ql[2] = {L[0].q, L[1].q};
    orc_model M = {2, ql, qy.m, by};
    orc_layer_f32 fl[2] = {L[0].f, L[1].f};
    orc_model_f32 F = {2, fl, S, Wy, by};
    float *x = fill(T * B * in, -1.f, 1.f), *post = malloc(sizeof(float) * T * B * S);
    float *logits = malloc(sizeof(float) * T * B * S);
    int32_t *acc_y = malloc(sizeof(int32_t) * T * B * S);
    taps_t tp[2];
    for (int l = 0; l < 2; ++l) make_taps(&tp[l], T, B, L[l].H, L[l].P);
    orc_layer_taps lt[2] = {tp[0].t, tp[1].t};
    CHECK(oracle_acoustic_model_forward(&M, x, T, B, post, lt, acc_y, logits) == 0);
    for (int64_t r = 0; r < T * B; ++r) {
      double sum = 0;
      for (int64_t k = 0; k < S; ++k) sum += post[r * S + k];
      CHECK(fabs(sum - 1.0) < 1e-5);
    }
    CHECK(oracle_acoustic_model_forward(&M, x, T, B, post, NULL, NULL, NULL) == 0);
    CHECK(oracle_acoustic_model_forward_f32(&F, x, T, B, post) == 0);
    /* the output layer's backward on the last layer's output */
    int32_t *y = malloc(sizeof(int32_t) * T * B);
    for (int64_t r = 0; r < T * B; ++r) y[r] = (int32_t)(r * 5 % S);
    double loss = 0;
    float *dWy = malloc(sizeof(float) * S * width), *dby = malloc(sizeof(float) * S),
          *dhL = malloc(sizeof(float) * T * B * width);
    CHECK(oracle_output_backward(Wy, S, width, tp[1].t.h, post, y, T * B, &loss, dWy, dby,
                                 dhL) == 0);
    CHECK(isfinite(loss) && loss > 0);
    /* the training step: float, 'quant', 'quant-all' */
    const int modes[3][2] = {{0, 0}, {1, 0}, {1, 1}};
    for (int mo = 0; mo < 3; ++mo) {
      layer_t G[2];
      for (int l = 0; l < 2; ++l) make_layer(&G[l], L[l].in, L[l].H, L[l].P, 4);
      float *gWy = fill(S * width, 0.f, 0.f), *gby = fill(S, 0.f, 0.f);
      orc_train_layer tl[2] = {L[0].t, L[1].t}, gl[2] = {G[0].t, G[1].t};
      orc_train_model TM = {2, tl, S, Wy, by}, GM = {2, gl, S, gWy, gby};
      CHECK(oracle_train_step(&TM, x, y, T, B, 0.05f, 4, modes[mo][0], modes[mo][1], &loss,
                              &GM) == 0);
      CHECK(isfinite(loss));
      CHECK(oracle_train_step(&TM, x, y, T, B, 0.05f, 2, modes[mo][0], modes[mo][1], NULL,
                              &GM) == 0);
      for (int l = 0; l < 2; ++l) free_layer(&G[l]);
      free(gWy), free(gby);
    }
    free(y), free(dWy), free(dby), free(dhL);
    for (int l = 0; l < 2; ++l) free_taps(&tp[l]);
    free(x), free(post), free(logits), free(acc_y), free(Wy), free(by);
    free_qm(&qy);
    for (int l = 0; l < 2; ++l) free_layer(&L[l]);
  }
}

int main(void) {
  scalars();
  quantizer();
  products();
  layers();
  models_and_training();
  if (g_fail) return 1;
  printf("oracle sanitizer run: ok\n");
  return 0;
}
