/*
 * qlstm_oracle.h -- CPU oracle for quantized LSTM acoustic-model inference.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously-correct
 * reference that the GPU library is checked against.  It shares no code,
 * header, table or helper with the GPU library, and only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.
 *
 * Paper: R. Alvarez, R. Prabhavalkar, A. Bakhtin, "On the efficient
 * representation and execution of deep acoustic models", Interspeech 2016
 * (arXiv:1607.04683).
 *
 *   Section 3, "Quantizing" / "Recovery"      -> oracle_qparams, oracle_code,
 *                                               oracle_quantize
 *   Section 3.1, eq. 1 (quantized product)     -> oracle_qlinear (via acc/tot)
 *   Section 3.1, eq. 2 (bias-free rounding)    -> oracle_code
 *   Section 3.1, eq. 3 (consistent recovery)   -> oracle_dequantize, recovery
 *   Section 3.1, Fig. 1 (y = F(R(Mult(Q(X),W'))+B)) -> oracle_quantized_matmul,
 *                                               the LSTM cell
 *   Section 3.1, granularity paragraph         -> nblocks (per gate matrix)
 *   Section 4 (4-5 LSTM layers, projection P,
 *   320-dim stacked input, softmax output)     -> oracle_lstm_layer_forward,
 *                                               oracle_acoustic_model_forward
 *
 * Conventions (host memory, caller-owned, row-major):
 *   codes are the paper's V' in 0..255 (uint8);
 *   a matrix of `rows` rows split into `nblocks` equal row blocks, each block
 *   quantized independently (nblocks = 4 for the four LSTM gates i, f, g, o);
 *   sequences are time-major [T][B][D].
 */
#ifndef QLSTM_ORACLE_H
#define QLSTM_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Parameters of one independently quantized set of values. */
typedef struct {
  double vmin, vmax; /* range endpoints after the degenerate-range rule */
  double R;          /* range R = vmax - vmin */
  double Q;          /* quantization factor Q = S / R, S = 255 */
  int32_t z;         /* round(Q * vmin) */
  float inv_q;       /* recovery factor Q^-1 = R / S, rounded to fp32 */
} orc_qparams;

/* One quantized matrix: codes [rows][cols], per-block zero points / recovery. */
typedef struct {
  int64_t rows, cols;
  int32_t nblocks;
  const uint8_t *codes;
  const int32_t *zero;   /* [nblocks] */
  const float *inv_q;    /* [nblocks] */
} orc_qmat;

typedef struct {
  int64_t in, hidden, proj;  /* proj = 0: no projection layer */
  orc_qmat Wx;               /* [4H][in]            */
  orc_qmat Wh;               /* [4H][proj ? proj:H] */
  orc_qmat Wr;               /* [proj][H] (proj > 0) */
  const float *bias;         /* [4H] */
} orc_layer;

typedef struct {
  int32_t nlayers;
  const orc_layer *layers;
  orc_qmat Wy;               /* [S][H_last] */
  const float *by;           /* [S] */
} orc_model;

/* Optional per-layer taps (every pointer nullable).  R = proj ? proj : H. */
typedef struct {
  int32_t *acc_x;   /* [T][B][4H] sum_k Wx'[n][k] x'_t[k]        (int32)   */
  int32_t *acc_h;   /* [T][B][4H] sum_k Wh'[n][k] h'_{t-1}[k]    (int32)   */
  int32_t *acc_r;   /* [T][B][P]  sum_k Wr'[n][k] m'_t[k]        (int32)   */
  uint8_t *h_codes; /* [T][B][R]  codes of h_t                               */
  int32_t *h_zero;  /* [T][B]     zero point round(Q vmin) of h_t            */
  float *h_inv_q;   /* [T][B]     recovery factor of h_t                     */
  float *c;         /* [T][B][H]  cell state after step t                    */
  float *h;         /* [T][B][R]  the layer's fp32 output h_t                */
  float *preact;    /* [T][B][4H] gate pre-activations (Wx x + b) + Wh h     */
  float *gates;     /* [T][B][4H] i, f, g, o after their activation functions */
  float *m;         /* [T][B][H]  cell output o tanh(c) (before a projection) */
} orc_layer_taps;

/* ---- scalar pieces ------------------------------------------------------ */
float oracle_expf(float x);
float oracle_sigmoidf(float x);
float oracle_tanhf(float x);
void oracle_elementwise(int32_t fn, const float *x, float *y, int64_t n);
int64_t oracle_round_half_up(double x);
void oracle_qparams(float vmin, float vmax, orc_qparams *p);
uint8_t oracle_code(float v, const orc_qparams *p);

/* ---- sets and matrices -------------------------------------------------- */
/* Quantize n values as one set; returns params and the sum of the codes. */
void oracle_quantize_set(const float *v, int64_t n, uint8_t *codes,
                         orc_qparams *p, int32_t *code_sum);
/* Quantize a [rows][cols] matrix in `nblocks` independent row blocks. */
int oracle_quantize(const float *src, int64_t rows, int64_t cols, int32_t nblocks,
                    uint8_t *codes, double *range, int32_t *zero, float *inv_q,
                    int32_t *row_sums);
/* Recover floats from codes (eq. 3). */
int oracle_dequantize(const uint8_t *codes, int64_t rows, int64_t cols,
                      int32_t nblocks, const int32_t *zero, const float *inv_q,
                      float *dst);

/* y = R(Mult(Q(X), W')) (+ bias); X [m][K] float; act_gran 0 = per tensor,
 * 1 = per row.  acc [m][rows] = raw sum of code products; x_codes [m][K],
 * x_zero [m], x_inv_q [m] receive the activation quantization (all nullable). */
int oracle_quantized_matmul(const orc_qmat *W, const float *X, int64_t m,
                            int32_t act_gran, const float *bias, float *Y,
                            int32_t *acc, uint8_t *x_codes, int32_t *x_zero,
                            float *x_inv_q);
/* C[M][N] = A[M][K] . B[N][K]^T on uint8 operands, int32 result. */
int oracle_gemm_u8(const uint8_t *A, const uint8_t *B, int32_t *C, int64_t M,
                   int64_t N, int64_t K);

/* ---- LSTM --------------------------------------------------------------- */
int oracle_lstm_layer_forward(const orc_layer *L, const float *x, int64_t T,
                              int64_t B, const float *h0, const float *c0,
                              float *h, float *hT, float *cT,
                              const orc_layer_taps *taps);
/* posteriors [T][B][S]; layer_taps nullable or [nlayers]; acc_y [T][B][S]
 * nullable; logits [T][B][S] nullable. */
int oracle_acoustic_model_forward(const orc_model *M, const float *feats,
                                  int64_t T, int64_t B, float *post,
                                  const orc_layer_taps *layer_taps,
                                  int32_t *acc_y, float *logits);

/* ---- unquantized fp32 comparison model ("match" condition, Section 5) ---- */
typedef struct {
  int64_t in, hidden, proj;
  const float *Wx, *Wh, *Wr, *bias; /* [4H][in], [4H][R], [P][H], [4H] */
} orc_layer_f32;
typedef struct {
  int32_t nlayers;
  const orc_layer_f32 *layers;
  int64_t S;            /* number of output states */
  const float *Wy, *by; /* [S][H_last], [S] */
} orc_model_f32;
int oracle_lstm_layer_forward_f32(const orc_layer_f32 *L, const float *x,
                                  int64_t T, int64_t B, const float *h0,
                                  const float *c0, float *h, float *hT, float *cT,
                                  const orc_layer_taps *taps);
int oracle_acoustic_model_forward_f32(const orc_model_f32 *M, const float *feats,
                                      int64_t T, int64_t B, float *post);

/* ---- quantization aware training (Section 3.2, Algorithm 1) ------------ */
/* Float master parameters of an acoustic model (fp32, host, updated in
 * place by the training step); the same layout holds gradients. */
typedef struct {
  int64_t in, hidden, proj;
  float *Wx, *Wh, *Wr, *bias; /* [4H][in], [4H][R], [P][H], [4H] */
} orc_train_layer;
typedef struct {
  int32_t nlayers;
  const orc_train_layer *layers;
  int64_t S;
  float *Wy, *by; /* [S][R_last], [S] */
} orc_train_model;

/* Backward pass through time of one LSTM layer in floating point, with the
 * float weights of L, given what its forward pass produced: the layer input
 * x [T][B][in], gates [T][B][4H] (after activation), c [T][B][H], m
 * [T][B][H] (o tanh c), h [T][B][R], zero initial state, and dC/dh dy
 * [T][B][R].  Writes dC/dWx, dC/dWh, dC/dWr (P > 0), dC/db and dC/dx
 * [T][B][in] (each nullable). */
int oracle_lstm_layer_backward(const orc_layer_f32 *L, const float *x, int64_t T, int64_t B,
                               const float *gates, const float *c, const float *m,
                               const float *h, const float *dy, float *dWx, float *dWh,
                               float *dWr, float *db, float *dx);
/* Frame-level cross-entropy of N frames of posteriors post [N][S] against
 * targets [N], averaged over the frames; its gradient through the output
 * layer z = Wy hL + by (Wy [S][R] float) to dC/dWy, dC/dby and dC/dhL
 * [N][R]. */
int oracle_output_backward(const float *Wy, int64_t S, int64_t R, const float *hL,
                           const float *post, const int32_t *targets, int64_t N,
                           double *loss, float *dWy, float *dby, float *dhL);
/* One training step (Algorithm 1) on a mini-batch feats [T][B][in] with
 * frame targets [T][B]: the parameters are quantized (W_x, W_h in gate_blocks
 * row blocks, W_r and W_y per matrix) and the forward pass runs in quantized
 * form (quantize_layers = 1; the inference path of this oracle) or in float
 * (0), with the output layer quantized (quantize_output = 1, 'quant-all') or
 * float (0, 'quant'); the loss and the backward pass are float, with the
 * float parameters, at the forward pass's activations; every weight and bias
 * is then moved by -lr times its gradient.  loss (nullable) receives the
 * mini-batch loss, grads (required; the shapes of M) the gradients.
 * quantize_output = 1 needs quantize_layers = 1. */
int oracle_train_step(const orc_train_model *M, const float *feats, const int32_t *targets,
                      int64_t T, int64_t B, float lr, int32_t gate_blocks,
                      int32_t quantize_layers, int32_t quantize_output, double *loss,
                      const orc_train_model *grads);

#ifdef __cplusplus
}
#endif
#endif
