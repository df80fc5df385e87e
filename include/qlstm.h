/*
 * qlstm.h -- C ABI of the MI355X (gfx950) quantized LSTM acoustic-model library.
 *
 * Implements the inference side of R. Alvarez, R. Prabhavalkar, A. Bakhtin,
 * "On the efficient representation and execution of deep acoustic models"
 * (Interspeech 2016, arXiv:1607.04683):
 *
 *   - the uniform linear 8-bit quantizer of Section 3 ("Quantizing":
 *     R = Vmax - Vmin, Q = S/R with S = 255) with the bias-free integer
 *     rounding of Section 3.1, eq. 2: V' = round(Q V) - round(Q Vmin);
 *   - the quantized product of Section 3.1, eq. 1, Vc = Va'' Vb'' / (Qa Qb)
 *     with V'' = V' + round(Q Vmin), computed as uint8 x uint8 products in
 *     32-bit accumulators plus exact zero-point terms, and recovered to float
 *     consistently with eq. 3;
 *   - layers that take and return float (Section 3.1, Fig. 1):
 *     y = F(R(Mult(Q(X), W')) + B), parameters quantized offline, inputs on
 *     the fly; weight matrices quantized independently per gate block by
 *     default, or per matrix, per sub-matrix of whole rows, or per row
 *     (Section 3.1, granularity paragraph);
 *   - the LSTM acoustic models of Section 4: stacked LSTM layers (optionally
 *     with a linear projection after each layer) and a quantized softmax
 *     output layer ('quant-all', Section 5).
 *
 * Numerical conventions shared by every entry point:
 *   - round() is round-half-up; Q = 255 / R is formed and applied in fp64;
 *   - a set whose range is 0, or narrower than max|V| * 255 / 2^24, has its
 *     range widened to include 0; an all-zero set has Q = 1, zero point 0;
 *   - the recovery factor is Q^-1 = (float)(R / 255); a product's recovered
 *     value is ((float)T * Qw^-1) * Qx^-1 where T = sum_k W'' x'' exactly;
 *   - gate pre-activations are (Wx x + b) + Wh h in fp32; gates are i, f, g, o;
 *     sigmoid(x) = 1 / (1 + e^-x) (IEEE division), tanh(x) = 2 sigmoid(2x) - 1
 *     with a fixed fp32 e^x (Cody-Waite reduction + degree-7 Taylor polynomial,
 *     each of their steps one fused multiply-add, no other contraction);
 *     c = f c + i g; m = o tanh(c); projection h = W_r m (no bias);
 *   - activations are quantized per vector (one frame of one utterance);
 *   - softmax is fp32 with the row maximum subtracted.
 *
 * Memory: every pointer argument is a device pointer unless stated otherwise;
 * the caller owns all memory.  Scratch memory comes from a caller-provided
 * workspace of at least the size returned by the matching *_workspace query
 * (256-byte aligned).  The library holds no device allocations.
 *
 * Device code layout: a matrix of codes is stored row-major with a leading
 * dimension `ld` (a multiple of 64, >= cols) as signed bytes equal to V' - 128
 * (the bits of V' XOR 0x80); bytes in columns [cols, ld) are 0.
 *
 * Execution: every call is asynchronous on `stream` (a hipStream_t; NULL is
 * the default stream).  Argument errors return before anything is enqueued.
 * QL_EHIP reports a failed launch (or an error left by earlier work).
 * Sequences are time-major: x[T][B][D].
 */
#ifndef QLSTM_H
#define QLSTM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QL_OK = 0,
  QL_EINVAL = -1,       /* null pointer or invalid enum/flag                       */
  QL_ESHAPE = -2,       /* inconsistent sizes, rows % nblocks != 0, ld too small    */
  QL_EOVERFLOW = -3,    /* K > 33025: 255*255*K could overflow a 32-bit accumulator */
  QL_EWORKSPACE = -4,   /* workspace null or smaller than the query returned        */
  QL_EHIP = -5,         /* HIP runtime error                                        */
  QL_EUNSUPPORTED = -6, /* shape outside what the kernels implement                 */
  QL_ETIMEOUT = -7,     /* a persistent kernel's bounded inter-block wait expired   */
  QL_ESCRATCH = -8      /* needs more than the static scratch of the no-alloc call  */
} ql_status;

typedef enum { QL_ACT_PER_TENSOR = 0, QL_ACT_PER_ROW = 1 } ql_act_gran;

/* One quantized matrix (Section 3.1): rows split into `nblocks` equal row
 * blocks, each quantized as an independent set (nblocks = 1: per matrix;
 * nblocks = 4: per LSTM gate i, f, g, o; more: the granularity paragraph's
 * individually quantized sub-matrices, each a band of whole rows, down to
 * nblocks = rows, one set per row).  Blocks are bands of rows so that every
 * output of a product has one weight recovery factor over its whole sum.
 * Every entry point accepts any nblocks dividing rows.  All arrays are device
 * memory. */
typedef struct {
  int8_t *codes;     /* [rows][ld], V' - 128 (see "Device code layout")    */
  int64_t rows, cols, ld;
  int32_t nblocks;
  double *range;     /* [nblocks] R after the degenerate-range rule          */
  int32_t *zero;     /* [nblocks] round(Q Vmin)                              */
  float *inv_q;      /* [nblocks] Q^-1 = (float)(R / 255)                    */
  int32_t *row_sums; /* [rows] sum over the row of V' (0..255 domain)        */
} ql_qmatrix;

/* One LSTM layer (Section 4).  W_x [4H][in], W_h [4H][R], W_r [P][H] where
 * R = proj ? proj : hidden; gate blocks of W_x / W_h in the order i, f, g, o. */
typedef struct {
  int64_t in, hidden, proj; /* proj = 0: no projection                         */
  ql_qmatrix Wx, Wh, Wr;    /* Wr ignored when proj = 0                         */
  const float *bias;        /* [4H] fp32, device                                */
} ql_lstm_layer;

/* LSTM acoustic model: nlayers stacked layers and a quantized softmax layer. */
typedef struct {
  int32_t nlayers;
  const ql_lstm_layer *layers; /* host array of nlayers descriptors             */
  ql_qmatrix Wy;               /* [S][R_last]                                   */
  const float *by;             /* [S] fp32, device                              */
} ql_model;

/* Optional diagnostic outputs of one LSTM layer (every pointer nullable,
 * device memory).  acc_* are the raw 8-bit-domain accumulators
 * sum_k W'[n][k] x'[k] of eq. 1 before zero-point terms and recovery (gate
 * row n = g H + j, gates i, f, g, o).  Every kernel that runs the layer fills
 * every tap it is given, the layer wavefronts included. */
typedef struct {
  int32_t *acc_x;   /* [T][B][4H] input products                              */
  int32_t *acc_h;   /* [T][B][4H] recurrent products (h_{t-1})                */
  int32_t *acc_r;   /* [T][B][P]  projection products                         */
  int8_t *h_codes;  /* [T][B][R]  codes of h_t (device code layout, ld = R)   */
  int32_t *h_zero;  /* [T][B]     zero point of h_t                           */
  float *h_inv_q;   /* [T][B]     recovery factor of h_t                      */
  float *h;         /* [T][B][R]  fp32 h_t; honoured by the model and stack
                       forwards (the one-layer entry points return h anyway)  */
  float *gates;     /* [T][B][4H] i, f, g, o after their activation functions */
  float *c;         /* [T][B][H]  cell state c_t                              */
  float *m;         /* [T][B][H]  cell output o tanh(c_t) (before a projection) */
} ql_lstm_taps;

/* Recurrent state of one layer at a chunk boundary of a stream (Section 4:
 * the network runs on a live utterance, one frame per 30 ms): h [B][R] and
 * c [B][H] fp32, device memory.  Both pointers nullable (zeros in, not
 * written out). */
typedef struct {
  float *h;
  float *c;
} ql_lstm_state;

typedef struct {
  const ql_lstm_taps *layers; /* host array [nlayers] or NULL                 */
  int32_t *acc_y;             /* [T][B][S] softmax-layer accumulators, or NULL */
  float *logits;              /* [T][B][S] recovered logits + bias, or NULL    */
} ql_model_taps;

/* ---- quantization (Section 3; eq. 2) ---------------------------------------
 * Quantizes src [rows][cols] (fp32, device) in nblocks row blocks into dst,
 * whose arrays the caller allocated (codes rows*ld bytes, ld = dst->ld).
 * dst->rows/cols/nblocks must match; nblocks <= 65535 (QL_EUNSUPPORTED
 * beyond).  Offline step for weights. */
size_t ql_quantize_workspace(int64_t rows, int64_t cols, int32_t nblocks);
ql_status ql_quantize(const float *src, int64_t rows, int64_t cols, int32_t nblocks,
                      ql_qmatrix *dst, void *ws, size_t ws_bytes, void *stream);

/* Recovery (eq. 3): dst [rows][cols] fp32 = (V' + round(Q Vmin)) * Q^-1. */
ql_status ql_dequantize(const ql_qmatrix *q, float *dst, void *stream);

/* ---- quantized layer product (Fig. 1: R(Mult(Q(X), W')) + B) ---------------
 * X [m][cols] fp32 is quantized on the fly (per tensor or per row), multiplied
 * by W'^T and recovered: Y [m][rows] fp32 (+ bias[rows] when non-null).
 * acc [m][rows] (nullable) receives sum_k W'[n][k] x'[i][k]. */
size_t ql_quantized_matmul_workspace(int64_t m, int64_t rows, int64_t cols);
ql_status ql_quantized_matmul(const ql_qmatrix *W, const float *X, int64_t m,
                              ql_act_gran gran, const float *bias, float *Y,
                              int32_t *acc, void *ws, size_t ws_bytes, void *stream);

/* ---- raw 8-bit GEMM (eq. 1 integer core) ------------------------------------
 * C[M][N] = sum_k A'[i][k] B'[j][k] (int32) for code matrices in the device
 * code layout: A [M][lda], B [N][ldb] with lda, ldb multiples of 64 and
 * padding bytes 0.  a_sums [M] / b_sums [N] (nullable) are the row sums of
 * the 0..255 codes; when null they are computed into the workspace. */
size_t ql_gemm_u8_workspace(int64_t M, int64_t N, int64_t K);
ql_status ql_gemm_u8(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                     int32_t *C, int64_t M, int64_t N, int64_t K,
                     const int32_t *a_sums, const int32_t *b_sums,
                     void *ws, size_t ws_bytes, void *stream);

/* ---- LSTM layer (Section 4) ---------------------------------------------------
 * x [T][B][in] fp32 -> h [T][B][R] fp32.  h0 [B][R], c0 [B][H] (nullable =
 * zeros); hT [B][R], cT [B][H] (nullable) receive the final state, so a
 * stream split into chunks and chained through (hT, cT) -> (h0, c0) gives
 * the same bits as one call.  taps nullable. */
size_t ql_lstm_layer_workspace(const ql_lstm_layer *L, int64_t T, int64_t B);
ql_status ql_lstm_layer_forward(const ql_lstm_layer *L, const float *x, int64_t T,
                                int64_t B, const float *h0, const float *c0,
                                float *h, float *hT, float *cT,
                                const ql_lstm_taps *taps, void *ws, size_t ws_bytes,
                                void *stream);

/* Per-vector quantized activation rows (the codes one layer hands the next):
 * codes [rows][ld] in the device code layout, and per row its zero point,
 * recovery factor and the sum of its 0..255 codes.  Device memory. */
typedef struct {
  int8_t *codes;
  int64_t rows, cols, ld;
  int32_t *zero;
  float *inv_q;
  int32_t *sums;
} ql_qact;

/* ---- activation quantization on the fly (Section 3.1; eq. 2) ----------------------
 * Quantizes every row of X [m][cols] fp32 as its own vector: dst->codes
 * [m][dst->ld] (device code layout, padding 0), dst->zero / inv_q / sums per
 * row.  dst->rows must be m, dst->cols must be cols; the caller allocates. */
ql_status ql_quantize_activations(const float *X, int64_t m, int64_t cols, const ql_qact *dst,
                                  void *stream);

/* ---- several stacked layers in one launch (Section 4) ---------------------------
 * n layers (layer k > 0 takes layer k-1's output), run as one persistent launch
 * in which layer k works on frame t while layer k-1 is already on a later frame:
 * either layers without projection and of one width H <= 512, or (batch 1 only)
 * layers that all have a projection, with H, P and in <= 512.  Input: the
 * per-vector codes of x_t (x->rows = T*B, x->cols = layers[0].in).  Output: the
 * codes of every h_t of every layer, h_codes[k] (rows = T*B, cols = R = P or H,
 * ld a multiple of 64), and h_last [T][B][R] fp32 of the last layer (nullable).
 * state_in / state_out (host arrays of n descriptors, or NULL): each layer's
 * initial state (NULL or null pointers: zeros) and final state; in and out
 * must not overlap (QL_EINVAL).  taps: host array of n, or NULL.  QL_EUNSUPPORTED when the
 * n layers do not fit one launch (or projection layers at B > 1).  Same
 * results, bit for bit, as n calls of the one-layer path. */
size_t ql_lstm_stack_workspace(const ql_lstm_layer *layers, int32_t n, int64_t T, int64_t B);
/* How many of the first n layers one launch holds on the current device (the
 * grouping ql_acoustic_model_forward uses); 1 when they cannot share one.
 * Layers that all have a projection (H, P, in <= 512) share launches at batch 1:
 * ql_acoustic_model_forward and ql_lstm_stack_forward run them as a wavefront
 * too. */
int32_t ql_lstm_stack_layers_per_launch(const ql_lstm_layer *layers, int32_t n, int64_t T,
                                        int64_t B);
ql_status ql_lstm_stack_forward(const ql_lstm_layer *layers, int32_t n, const ql_qact *x,
                                int64_t T, int64_t B, const ql_qact *h_codes, float *h_last,
                                const ql_lstm_state *state_in, const ql_lstm_state *state_out,
                                const ql_lstm_taps *taps, void *ws, size_t ws_bytes,
                                void *stream);

/* ---- the recurrence of one layer alone (Section 4) ------------------------------
 * Given the input pre-activations gx [T][B][4H] fp32 = R(Mult(Q(x_t), W_x')) + b
 * for every frame (what ql_quantized_matmul with per-row quantization and the
 * bias computes), runs the serial part: per step, Q(h_{t-1}) per vector, the
 * W_h' product, recovery, gates, c and h (and the projection when present).
 * Writes h [T][B][R] fp32 and hT / cT (nullable).  h_codes (nullable; rows =
 * T*B, cols = R, ld a multiple of 64 >= R) receives the per-vector codes of
 * every h_t, i.e. the next layer's quantized input.  taps: acc_h, acc_r and the
 * h_* fields are honoured (acc_x is not produced here). */
size_t ql_lstm_recurrence_workspace(const ql_lstm_layer *L, int64_t T, int64_t B);
ql_status ql_lstm_recurrence(const ql_lstm_layer *L, const float *gx, int64_t T, int64_t B,
                             const float *h0, const float *c0, float *h, float *hT,
                             float *cT, const ql_qact *h_codes, const ql_lstm_taps *taps,
                             void *ws, size_t ws_bytes, void *stream);

/* ---- acoustic model (Section 4; quantized softmax, Section 5 'quant-all') ----
 * feats [T][B][in] fp32 -> posteriors post [T][B][S] fp32.  taps nullable. */
size_t ql_acoustic_model_workspace(const ql_model *M, int64_t T, int64_t B);
ql_status ql_acoustic_model_forward(const ql_model *M, const float *feats, int64_t T,
                                    int64_t B, float *post, const ql_model_taps *taps,
                                    void *ws, size_t ws_bytes, void *stream);
/* The same for one chunk of a stream (Section 4: a live utterance evaluated
 * as its frames arrive): state_in / state_out are host arrays of nlayers
 * per-layer states (either NULL: zeros in / nothing out); they must not
 * overlap (QL_EINVAL).  Calls chained through state_out -> state_in give, bit for bit,
 * the posteriors of one call over the whole utterance.  Workspace as
 * ql_acoustic_model_workspace. */
ql_status ql_acoustic_model_forward_stream(const ql_model *M, const float *feats, int64_t T,
                                           int64_t B, const ql_lstm_state *state_in,
                                           const ql_lstm_state *state_out, float *post,
                                           const ql_model_taps *taps, void *ws, size_t ws_bytes,
                                           void *stream);

/* ---- the stream step for callers that cannot allocate -------------------------
 * For callers that must not allocate device memory or hand over a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The same computation as ql_acoustic_model_forward_stream
 * (without taps), on a scratch buffer the library holds in a static device
 * array of QL_NOALLOC_SCRATCH_BYTES per GPU (resolved once per device on the
 * first call there and kept until the process ends).  Calls whose
 * ql_acoustic_model_workspace(M, T, B) exceeds it return QL_ESCRATCH before
 * anything is enqueued (the 5 x 500 model with an 8192-way softmax fits chunks
 * of up to about 1700 frames at batch 1).  Every call on one GPU uses that
 * GPU's one scratch array: calls that overlap in time on one GPU (other
 * streams, other threads) race and give undefined results; calls ordered on
 * one stream are safe (each clears what it needs).  timed_out (device int32,
 * nullable) receives 1 if a persistent kernel's bounded wait expired (the
 * outputs are then undefined), else 0, in stream order.  Allocates nothing:
 * no hipMalloc, no hipFree, no allocating library call. */
#define QL_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
ql_status ql_acoustic_model_forward_stream_noalloc(const ql_model *M, const float *feats,
                                                   int64_t T, int64_t B,
                                                   const ql_lstm_state *state_in,
                                                   const ql_lstm_state *state_out, float *post,
                                                   int32_t *timed_out, void *stream);

/* ---- frontend fused into the input quantizer (Section 4) ------------------------
 * The network's input at presented step t of utterance b is the concatenation of
 * `stack` consecutive base frames skip*t, ..., skip*t + stack - 1 of that utterance
 * (the paper stacks 8 frames of 40 log-mel energies, 7 of right context, and
 * presents every third stacked frame: one network step per 30 ms).  frames
 * [nframes][B][dim] fp32 (device, time-major).  The number of presented steps is
 * T = ql_stacked_input_count(nframes, stack, skip) = (nframes - stack) / skip + 1
 * when nframes >= stack, else 0 (trailing frames that do not complete a stack are
 * not presented).  The stacked vectors are never written: each is gathered from
 * the base frames while it is quantized, per vector, exactly as
 * ql_quantize_activations quantizes the same vector. */
int64_t ql_stacked_input_count(int64_t nframes, int32_t stack, int32_t skip);
/* dst->rows must be T * B, dst->cols = stack * dim (QL_ESHAPE otherwise);
 * codes and per-row zero point, recovery factor and code sum as in
 * ql_quantize_activations.  stack, skip, dim > 0. */
ql_status ql_quantize_stacked_frames(const float *frames, int64_t nframes, int64_t B, int64_t dim,
                                     int32_t stack, int32_t skip, const ql_qact *dst,
                                     void *stream);
/* ql_acoustic_model_forward on the stacked inputs of frames [nframes][B][dim]:
 * layers[0].in must equal stack * dim; post [T][B][S] with T as above.  Same bits
 * as stacking on the host and calling ql_acoustic_model_forward. */
size_t ql_acoustic_model_frames_workspace(const ql_model *M, int64_t nframes, int64_t B,
                                          int32_t stack, int32_t skip);
ql_status ql_acoustic_model_forward_frames(const ql_model *M, const float *frames,
                                           int64_t nframes, int64_t B, int64_t dim,
                                           int32_t stack, int32_t skip, float *post,
                                           const ql_model_taps *taps, void *ws, size_t ws_bytes,
                                           void *stream);

/* ---- unquantized fp32 model (the float baseline of Section 5) -----------------
 * The same layers and model with fp32 weights and no quantization: products
 * accumulate in fp32, gate math is the same as above, the output layer is a
 * plain fp32 softmax.  Weights are device fp32 arrays, row-major and dense:
 * Wx [4H][in], Wh [4H][R], Wr [P][H] (P > 0), bias [4H]; the model's layers
 * array is a host array, Wy [states][R_last], by [states].  Float results
 * follow the summation order of the GPU kernels, so they agree with a
 * reference evaluation to rounding, not bit for bit. */
typedef struct {
  int64_t in, hidden, proj;
  const float *Wx, *Wh, *Wr, *bias;
} ql_f32_layer;
typedef struct {
  int32_t nlayers;
  const ql_f32_layer *layers;
  int64_t states;
  const float *Wy, *by;
} ql_f32_model;

/* Y [m][rows] = X [m][cols] W^T + bias (bias nullable); W [rows][cols]. */
ql_status ql_f32_matmul(const float *W, int64_t rows, int64_t cols, const float *X, int64_t m,
                        const float *bias, float *Y, void *stream);
/* As ql_lstm_layer_forward, without taps. */
size_t ql_f32_lstm_layer_workspace(const ql_f32_layer *L, int64_t T, int64_t B);
ql_status ql_f32_lstm_layer_forward(const ql_f32_layer *L, const float *x, int64_t T,
                                    int64_t B, const float *h0, const float *c0, float *h,
                                    float *hT, float *cT, void *ws, size_t ws_bytes,
                                    void *stream);
/* As ql_acoustic_model_forward: feats [T][B][in] -> post [T][B][states]. */
size_t ql_f32_acoustic_model_workspace(const ql_f32_model *M, int64_t T, int64_t B);
ql_status ql_f32_acoustic_model_forward(const ql_f32_model *M, const float *feats, int64_t T,
                                        int64_t B, float *post, void *ws, size_t ws_bytes,
                                        void *stream);

/* ---- quantization-aware training step (Section 3.2, Algorithm 1) ---------------
 * Float master parameters of an acoustic model (device fp32, row-major, the
 * layouts of ql_f32_layer / ql_f32_model), updated in place by the step. */
typedef struct {
  int64_t in, hidden, proj;  /* proj must be 0 (QL_EUNSUPPORTED otherwise)     */
  float *Wx, *Wh, *Wr, *bias; /* [4H][in], [4H][H], unused, [4H]               */
} ql_train_layer;
typedef struct {
  int32_t nlayers;
  const ql_train_layer *layers; /* host array of nlayers descriptors            */
  int64_t states;
  float *Wy, *by;               /* [states][H_last], [states]                    */
} ql_train_model;
/* One training step on a mini-batch feats [T][B][in] (fp32, device) with frame
 * targets [T][B] (int32 state indices, device), as Algorithm 1 lays it out:
 *   1. the parameters are quantized (W_x and W_h in gate_blocks row blocks,
 *      4 = per gate; the output layer's W_y per matrix);
 *   2. the forward pass runs in quantized form, the inference path of this
 *      library (ql_acoustic_model_forward, bit for bit), its activations kept;
 *      quantize_output = 1 quantizes the output layer too ('quant-all'),
 *      0 keeps it float ('quant', Section 5);
 *   3. the loss is frame-level cross-entropy of the posteriors, averaged over
 *      the T*B frames (*loss, device float, nullable);
 *   4. the backward pass is floating point, with the float parameters,
 *      evaluated at the quantized forward pass's activations (quantization is
 *      not differentiated); grads (required; device arrays of the shapes of M)
 *      receives every gradient;
 *   5. every weight and bias moves by -lr times its gradient (fp32).
 * Layers without projection, hidden <= 512 (QL_EUNSUPPORTED otherwise).  Zero
 * initial state per utterance.  Workspace from ql_train_step_workspace (0 for
 * an invalid model).  QL_EINVAL: a null pointer (feats / targets may be null
 * when T*B = 0), quantize_output not 0 or 1, lr not finite, grads not of the
 * model's layer count and states; QL_ESHAPE: widths that do not chain, 4H not
 * a multiple of gate_blocks, grads of other shapes, T or B < 0. */
size_t ql_train_step_workspace(const ql_train_model *M, int64_t T, int64_t B,
                               int32_t gate_blocks);
ql_status ql_train_step(const ql_train_model *M, const float *feats, const int32_t *targets,
                        int64_t T, int64_t B, float lr, int32_t gate_blocks,
                        int32_t quantize_output, float *loss, const ql_train_model *grads,
                        void *ws, size_t ws_bytes, void *stream);

/* ---- misc -------------------------------------------------------------------- */
/* Synchronizes `stream`, then reports QL_ETIMEOUT if a persistent kernel of the
 * last layer / model forward call (8-bit or fp32) that used this
 * workspace gave up waiting for the rest of its grid (its outputs are then
 * undefined), else QL_OK. */
ql_status ql_workspace_status(const void *ws, void *stream);
const char *ql_status_str(ql_status s);
/* Test hook for the timeout path: calls made after it bound every inter-
 * workgroup wait of their persistent kernels to `polls` re-reads (0 restores
 * the default bound), so a wait that is not met within them expires, every
 * workgroup leaves at its next wait, and ql_workspace_status reports
 * QL_ETIMEOUT (the outputs are then undefined).  Applies to every device of
 * the process (none: nothing to do) and must not overlap a call of this
 * library in flight; QL_EINVAL for a negative count, QL_EHIP if a device
 * could not be set. */
ql_status ql_debug_set_wait_bound(int32_t polls);
/* Test hook: which layout the recurrence of layer L runs in at batch B on the
 * current device -- 1: one persistent launch over the whole chip with each
 * XCD holding an eighth of the batch (layers with a projection, batch 16 to
 * 256, 256 CUs), 0: any other path; -1 for an invalid layer or B < 0. */
int32_t ql_debug_recurrence_layout(const ql_lstm_layer *L, int64_t B);
/* Test hook: which layout the first wavefront launch over the n stacked
 * layers (no projection) runs in for T frames at batch B on the current
 * device -- 1: one persistent launch over the whole chip with one XCD per
 * layer (batch 16 to 64, 2 to 8 layers, widths up to 512, 256 CUs), 0: any
 * other path (including none); -1 for an invalid layer, n < 1, T < 0 or
 * B < 0.  The layers are read, never written. */
int32_t ql_debug_stack_layout(const ql_lstm_layer *layers, int32_t n, int64_t T, int64_t B);
/* Elementwise gate functions on device arrays (fn 0 = e^x, 1 = sigmoid,
 * 2 = tanh, 3 = the reciprocal 1 / d that sigmoid applies to d = 1 + e^-x,
 * defined for d in [1, 2^126) and equal there to IEEE division) -- the exact
 * functions the LSTM kernels use. */
ql_status ql_gate_fn(int32_t fn, const float *x, float *y, int64_t n, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* QLSTM_H */
