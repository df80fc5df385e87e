// ql_launch.h -- host-side launchers of the gfx950 kernels (internal).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ql {

constexpr int kSetParts = 128;  // partial min/max blocks per quantized set

inline size_t align_up(size_t n, size_t a) { return (n + a - 1) / a * a; }
inline int64_t round_up(int64_t n, int64_t a) { return (n + a - 1) / a * a; }

// ---- quantizer (ql_quantize.hip)
hipError_t launch_quantize_rows(const float *X, int64_t ldx, int64_t m, int64_t K, int8_t *codes,
                                int64_t ld, int32_t *zero, float *inv_q, int32_t *sums,
                                hipStream_t s);
size_t set_quantize_ws(int nsets);
hipError_t launch_quantize_stacked(const float *frames, int64_t B, int dim, int stack, int skip,
                                   int64_t T, int8_t *codes, int64_t ld, int32_t *zero,
                                   float *inv_q, int32_t *sums, hipStream_t s);
hipError_t launch_set_quantize(const float *X, int64_t ldx, int64_t rows, int64_t cols,
                               int nsets, int8_t *codes, int64_t ld, double *range,
                               int32_t *zero, float *inv_q, int32_t *row_sums,
                               int32_t *row_zero, float *row_inv_q, void *ws, hipStream_t s);
hipError_t launch_dequantize(const int8_t *codes, int64_t ld, int64_t rows, int64_t cols,
                             int nblocks, const int32_t *zero, const float *inv_q, float *dst,
                             hipStream_t s);
hipError_t launch_code_row_sums(const int8_t *codes, int64_t ld, int64_t rows, int64_t K,
                                int32_t *sums, hipStream_t s);
hipError_t launch_gate_fn(int fn, const float *x, float *y, int64_t n, hipStream_t s);

// ---- 8-bit GEMM (ql_gemm.hip)
// Per-row description of a quantized activation matrix X' [M][ld].
struct ActRows {
  const int8_t *codes;
  int64_t ld;
  const int32_t *zero;   // [M] round(Q Vmin) per row
  const float *inv_q;    // [M]
  const int32_t *sums;   // [M] sum of V' (0..255)
};
// Quantized weight matrix W' [N][ld] with per-block params.
struct WeightMat {
  const int8_t *codes;
  int64_t ld;
  int64_t rows_per_block;
  const int32_t *zero;     // [nblocks]
  const float *inv_q;      // [nblocks]
  const int32_t *row_sums; // [N]
};

// Y[m][n] = recover(X'[m] . W'[n]) (+ bias[n]); acc (nullable) = raw sums.
hipError_t launch_gemm_recover(const ActRows &X, const WeightMat &W, int64_t M, int64_t N,
                               int64_t K, const float *bias, float *Y, int32_t *acc,
                               hipStream_t s);
// C[m][n] = sum_k A'[m][k] B'[n][k] in the 0..255 domain.
hipError_t launch_gemm_raw(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb,
                           int32_t *C, int64_t M, int64_t N, int64_t K, const int32_t *a_sums,
                           const int32_t *b_sums, hipStream_t s);
// Softmax output layer: post[m][n] = softmax_n(recover(X'[m] . W'[n]) + bias[n]).
size_t softmax_ws(int64_t M, int64_t N);
hipError_t launch_softmax_layer(const ActRows &X, const WeightMat &W, int64_t M, int64_t N,
                                int64_t K, const float *bias, float *post, int32_t *acc,
                                float *logits, void *ws, hipStream_t s);

// ---- recurrence (ql_recurrent.hip)
struct RecurrentArgs {
  int64_t T, B, H, P, R;     // R = P ? P : H
  const float *gx;           // [T][B][4H] (W_x x_t + b), fp32
  WeightMat Wh;              // [4H][ldR]
  WeightMat Wr;              // [P][ldH] (P > 0)
  const float *h0, *c0;      // nullable
  float *h;                  // [T][B][R] output
  float *hT, *cT;            // nullable
  // codes of every h_t for the next layer / output layer
  int8_t *out_codes;         // [T*B][ld_out]
  int64_t ld_out;
  int32_t *out_zero;         // [T*B]
  float *out_inv_q;          // [T*B]
  int32_t *out_sums;         // [T*B]
  // optional taps
  int32_t *acc_h;            // [T][B][4H]
  int32_t *acc_r;            // [T][B][P]
  int8_t *tap_codes;         // [T][B][R] (ld = R)
  int32_t *tap_zero;         // [T][B]
  float *tap_inv_q;          // [T][B]
  float *tap_gates;          // [T][B][4H] activated gates i, f, g, o
  float *tap_c;              // [T][B][H] cell state
  float *tap_m;              // [T][B][H] cell output o tanh(c)
  // scratch
  void *ws;
};
size_t recurrent_ws(int64_t B, int64_t H, int64_t P);
// Batched layers with a projection on the whole chip (ql_xrec.hip): each XCD
// runs the layer for an eighth of the batch.  *done false when the shapes or
// the device do not fit that layout (nothing launched).
size_t xrec_ws(int64_t B, int64_t H, int64_t P);
hipError_t launch_xrec(const RecurrentArgs &a, int cus, int lds_max, hipStream_t s, bool *done);
// 1 when launch_recurrent would run `a` in the XCD-local layout on the current
// device, else 0.
int recurrent_layout(const RecurrentArgs &a);
// returns hipSuccess, or an error; *unsupported set if shapes do not fit.
hipError_t launch_recurrent(const RecurrentArgs &a, hipStream_t s, bool *unsupported);
// Clears the timeout flag (once per API call, before the first layer).
hipError_t reset_recurrent_flag(void *ws, hipStream_t s);
// Bounds every wait of the persistent kernels to `polls` re-reads (0: the
// default), on every device; one setter per source file with such kernels.
hipError_t set_wait_bound(int polls);
hipError_t set_wait_bound_recurrent(int polls);
hipError_t set_wait_bound_stack(int polls);
hipError_t set_wait_bound_pstack(int polls);
hipError_t set_wait_bound_f32(int polls);
hipError_t set_wait_bound_train(int polls);
hipError_t set_wait_bound_xrec(int polls);
hipError_t set_wait_bound_xstack(int polls);
// Reads the timeout flag a persistent launch left in its workspace (syncs s).
hipError_t recurrent_timed_out(const void *ws, hipStream_t s, bool *timed_out);
// Zeroes the n64 64-bit words after the workspace header (counters first).
hipError_t clear_exchange(void *ws, int64_t n64, hipStream_t s);

// ---- several stacked layers in one launch (ql_stack.hip)
constexpr int kMaxStack = 8;
// Codes + row params a layer writes for every frame (its output).
struct OutRows {
  int8_t *codes;
  int64_t ld;
  int32_t *zero;
  float *inv_q;
  int32_t *sums;
};
struct StackLayer {
  WeightMat Wx, Wh;        // [4H][ld] each
  const float *bias;       // [4H]
  int64_t in;              // input width
  ActRows xin;             // input codes: the launch's first layer reads finished data,
                           // a later layer reads the previous layer's `out`
  OutRows out;             // [T*B] rows of codes of h_t + params
  float *h;                // [T][B][H] fp32 (nullable)
  int8_t *tap_codes;       // optional taps: [T][B][H] codes (ld = H), zero, inv_q
  int32_t *tap_zero;
  float *tap_inv_q;
  int32_t *acc_x, *acc_h;  // optional taps: [T][B][4H] raw input / recurrent sums
  float *tap_gates;        // optional taps: [T][B][4H] activated gates, [T][B][H] c and
  float *tap_c, *tap_m;    // m (= h without a projection)
  const float *h0, *c0;    // [B][H] initial state (nullable = zeros)
  float *hT, *cT;          // [B][H] final state (nullable)
};
struct StackArgs {
  int nl;                  // layers in this launch (2 .. kMaxStack)
  int64_t T, B, H;         // all layers: hidden width H, no projection
  StackLayer L[kMaxStack];
  void *ws;                // stack_ws bytes; timeout flag cleared by the caller
};
size_t stack_ws(int nl, int64_t T, int64_t B, int64_t H);
// ---- stacked layers with a projection, one batch row (ql_pstack.hip)
struct PStackLayer {
  WeightMat Wx, Wh, Wr;    // [4H][in], [4H][P], [P][H]
  const float *bias;       // [4H]
  int64_t in, H, P;        // input width (layer k > 0: P of layer k-1), cells, projection
  ActRows xin;             // the launch's first layer only: codes of every x_t
  OutRows out;             // [T] rows of codes of h_t + params
  float *h;                // [T][P] fp32 (nullable)
  int8_t *tap_codes;       // optional taps: [T][P] codes (ld = P), zero, inv_q
  int32_t *tap_zero;
  float *tap_inv_q;
  int32_t *acc_x, *acc_h;  // optional taps: [T][4H] raw input / recurrent sums
  int32_t *acc_r;          // optional tap: [T][P] raw projection sums
  float *tap_gates;        // optional taps: [T][4H] activated gates, [T][H] c and m
  float *tap_c, *tap_m;
  const float *h0, *c0;    // [P], [H] initial state (nullable = zeros)
  float *hT, *cT;          // [P], [H] final state (nullable)
};
struct PStackArgs {
  int nl;                  // layers in this launch (1 .. kMaxStack)
  int64_t T;               // frames (batch 1)
  PStackLayer L[kMaxStack];
  void *ws;                // pstack_ws bytes; timeout flag cleared by the caller
};
size_t pstack_ws(const int64_t *H, const int64_t *P, int nl, int64_t T);
hipError_t launch_pstack(const PStackArgs &a, hipStream_t s, bool *unsupported);
// How many of a.nl layers fit one launch (1: none; use the one-layer path).
int pstack_layers_per_launch(const PStackArgs &a);

hipError_t launch_stack(const StackArgs &a, hipStream_t s, bool *unsupported);
// Batch 16 to 64 on the whole chip (ql_xstack.hip): one XCD per layer.  *done
// false when the shapes or the device do not fit that layout (nothing
// launched).
size_t xstack_ws(int nl);
bool xstack_applies(const StackArgs &a, int cus, int lds_max);
hipError_t launch_xstack(const StackArgs &a, int cus, int lds_max, bool taps, hipStream_t s,
                         bool *done);
// 1 when launch_stack would run a in that layout on the current device, else 0.
int stack_layout(const StackArgs &a);
// How many layers of such a stack fit one launch (1: none, use the one-layer path).
int stack_layers_per_launch(int n, int64_t T, int64_t B, int64_t H, int64_t in0, int64_t in1);

// ---- unquantized fp32 model (ql_f32.hip)
// C[m][n] = sum_k A[m][k] B[n][k] (+ bias[n]); bias nullable.
hipError_t launch_sgemm(const float *A, int64_t lda, const float *B, int64_t ldb, int64_t M,
                        int64_t N, int64_t K, const float *bias, float *C, int64_t ldc,
                        hipStream_t s);
// The same with either operand transposed: A(m, k) = A[k*lda + m] when ta,
// B(n, k) = B[k*ldb + n] when tb.  splits > 1 (with part: splits*M*N floats)
// splits K over more workgroups and sums the partial products in order.
hipError_t launch_sgemm_ex(bool ta, bool tb, const float *A, int64_t lda, const float *B,
                           int64_t ldb, int64_t M, int64_t N, int64_t K, const float *bias,
                           float *C, int64_t ldc, int splits, float *part, hipStream_t s);
// In-place softmax of each of `rows` rows of S floats.
hipError_t launch_softmax_rows(float *x, int64_t rows, int64_t S, hipStream_t s);
struct F32RecArgs {
  int64_t T, B, H, P, R;     // R = P ? P : H
  const float *gx;           // [T][B][4H] (W_x x_t + b)
  const float *Wh;           // [4H][R]
  const float *Wr;           // [P][H] (P > 0)
  const float *h0, *c0;      // nullable
  float *h;                  // [T][B][R]
  float *hT, *cT;            // nullable
  void *ws;                  // recurrent_f32_ws bytes, timeout flag cleared by the caller
};
size_t recurrent_f32_ws(int64_t B, int64_t H, int64_t P);
hipError_t launch_recurrent_f32(const F32RecArgs &a, hipStream_t s, bool *unsupported);

// ---- quantization-aware training step (ql_train.hip)
// Cross-entropy of the posteriors post [N][S] against targets [N]: dC/dz =
// (p - onehot) / N written over post, -log p[target] per row into row_loss,
// their mean into *loss (nullable).
hipError_t launch_xent_grad(float *post, const int32_t *targets, int64_t N, int64_t S,
                            float *row_loss, float *loss, hipStream_t s);
// out[n] = sum_m X[m][n] (fixed order); part: colsum_ws(N) bytes.
size_t colsum_ws(int64_t N);
hipError_t launch_colsum(const float *X, int64_t M, int64_t N, float *out, float *part,
                         hipStream_t s);
// w <- w - lr g
hipError_t launch_sgd(float *w, const float *g, int64_t n, float lr, hipStream_t s);
// Backpropagation through time of one layer without projection: da [T][B][4H]
// = dC/d(gate pre-activations) from dy [T][B][H] = dC/dh (from above) and the
// forward pass's gates [T][B][4H] and c [T][B][H], with W_h [4H][H] fp32.
struct BpttArgs {
  int64_t T, B, H;
  const float *Wh, *dy, *gates, *c;
  float *da;
  void *ws;  // bptt_ws bytes; timeout flag cleared by the caller
};
size_t bptt_ws(int64_t T, int64_t B);
hipError_t launch_bptt(const BpttArgs &a, hipStream_t s, bool *unsupported);

}  // namespace ql
