// ql_api.cpp -- the C ABI of include/qlstm.h: argument checks, workspace
// carving and stream-ordered launches of the gfx950 kernels.
#include "../../include/qlstm.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>

#include "ql_launch.h"

using namespace ql;

namespace {

constexpr int64_t kMaxK = 33025;  // 255 * 255 * K must fit a 32-bit accumulator
constexpr size_t kHeader = 256;   // persistent-kernel barrier counter and flag

hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

ql_status from_hip(hipError_t e) { return e == hipSuccess ? QL_OK : QL_EHIP; }

// Bump allocator over a caller workspace (256-byte aligned pieces).
struct Carve {
  char *base;
  size_t off = 0;
  explicit Carve(void *p) : base(static_cast<char *>(p)) {}
  template <class T>
  T *take(size_t count) {
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += align_up(count * sizeof(T), 256);
    return p;
  }
};

ql_status check_qmatrix(const ql_qmatrix *q, bool need_sums) {
  if (!q || !q->codes || !q->zero || !q->inv_q || (need_sums && !q->row_sums)) return QL_EINVAL;
  if (q->rows < 0 || q->cols < 0 || q->nblocks <= 0) return QL_ESHAPE;
  if (q->rows % q->nblocks != 0) return QL_ESHAPE;
  if (q->ld < q->cols || q->ld % 64 != 0) return QL_ESHAPE;
  if (q->cols > kMaxK) return QL_EOVERFLOW;
  return QL_OK;
}

WeightMat weight(const ql_qmatrix &q) {
  WeightMat w;
  w.codes = q.codes;
  w.ld = q.ld;
  w.rows_per_block = q.rows / q.nblocks;
  w.zero = q.zero;
  w.inv_q = q.inv_q;
  w.row_sums = q.row_sums;
  return w;
}

// Activation rows quantized on the fly: [m][ld] codes + per-row params.
struct ActBuf {
  int8_t *codes;
  int64_t ld;
  int32_t *zero, *sums;
  float *inv_q;
  ActRows rows() const { return ActRows{codes, ld, zero, inv_q, sums}; }
};
ActBuf take_act(Carve &c, int64_t m, int64_t cols) {
  ActBuf a;
  a.ld = round_up(cols, 64);
  a.codes = c.take<int8_t>((size_t)(m * a.ld));
  a.zero = c.take<int32_t>((size_t)m);
  a.inv_q = c.take<float>((size_t)m);
  a.sums = c.take<int32_t>((size_t)m);
  return a;
}

int64_t layer_width(const ql_lstm_layer &L) { return L.proj ? L.proj : L.hidden; }

// The int a C caller passed for an enum argument.  C lets an enum carry any
// int; in C++ only its enumerators' range is a valid value, so the argument
// is read through its bytes, never as the enum.
template <class E>
int enum_arg(const E &e) {
  static_assert(sizeof(E) == sizeof(int), "C enums are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

// True when a buffer of the initial states (per layer h [B][R], c [B][H])
// shares a byte with a buffer of the final states: the kernels read the one
// and write the other within a launch.
bool states_overlap(const ql_lstm_layer *layers, int n, int64_t B, const ql_lstm_state *in,
                    const ql_lstm_state *out) {
  if (!in || !out || B <= 0) return false;
  auto span = [&](const ql_lstm_state &st, int l, bool cell, uintptr_t *lo, uintptr_t *hi) {
    const float *p = cell ? st.c : st.h;
    if (!p) return false;
    const int64_t w = cell ? layers[l].hidden : layer_width(layers[l]);
    *lo = reinterpret_cast<uintptr_t>(p);
    *hi = *lo + static_cast<uintptr_t>(B * w) * sizeof(float);
    return true;
  };
  for (int a = 0; a < n; ++a)
    for (int ca = 0; ca < 2; ++ca) {
      uintptr_t alo, ahi;
      if (!span(in[a], a, ca == 1, &alo, &ahi)) continue;
      for (int b = 0; b < n; ++b)
        for (int cb = 0; cb < 2; ++cb) {
          uintptr_t blo, bhi;
          if (span(out[b], b, cb == 1, &blo, &bhi) && alo < bhi && blo < ahi) return true;
        }
    }
  return false;
}

ql_status check_layer(const ql_lstm_layer *L) {
  if (!L || !L->bias) return QL_EINVAL;
  if (L->in <= 0 || L->hidden <= 0 || L->proj < 0) return QL_ESHAPE;
  const int64_t H = L->hidden, R = layer_width(*L);
  ql_status st = check_qmatrix(&L->Wx, true);
  if (st == QL_OK) st = check_qmatrix(&L->Wh, true);
  if (st == QL_OK && L->proj) st = check_qmatrix(&L->Wr, true);
  if (st != QL_OK) return st;
  if (L->Wx.rows != 4 * H || L->Wx.cols != L->in) return QL_ESHAPE;
  if (L->Wh.rows != 4 * H || L->Wh.cols != R) return QL_ESHAPE;
  if (L->proj && (L->Wr.rows != L->proj || L->Wr.cols != H)) return QL_ESHAPE;
  if (H > kMaxK) return QL_EOVERFLOW;
  return QL_OK;
}

// Workspace of one layer's forward pass, carved in a fixed order.
struct LayerWs {
  void *rec;       // recurrent header + scratch (first: holds the timeout flag)
  ActBuf xin;      // codes of the layer input
  float *gx;       // [T*B][4H]
  ActBuf hout;     // codes of every h_t
};
LayerWs carve_layer(Carve &c, const ql_lstm_layer &L, int64_t T, int64_t B, bool quantize_input) {
  LayerWs w;
  w.rec = c.take<char>(recurrent_ws(B, L.hidden, L.proj));
  if (quantize_input) w.xin = take_act(c, T * B, L.in);
  w.gx = c.take<float>((size_t)(T * B * 4 * L.hidden));
  w.hout = take_act(c, T * B, layer_width(L));
  return w;
}

RecurrentArgs rec_args(const ql_lstm_layer &L, int64_t T, int64_t B, const float *gx,
                       const float *h0, const float *c0, float *h, float *hT, float *cT,
                       const ActBuf &hout, const ql_lstm_taps *taps, void *rec) {
  RecurrentArgs a{};
  a.T = T;
  a.B = B;
  a.H = L.hidden;
  a.P = L.proj;
  a.R = layer_width(L);
  a.gx = gx;
  a.Wh = weight(L.Wh);
  if (L.proj) a.Wr = weight(L.Wr);
  a.h0 = h0;
  a.c0 = c0;
  a.h = h;
  a.hT = hT;
  a.cT = cT;
  a.out_codes = hout.codes;
  a.ld_out = hout.ld;
  a.out_zero = hout.zero;
  a.out_inv_q = hout.inv_q;
  a.out_sums = hout.sums;
  if (taps) {
    a.acc_h = taps->acc_h;
    a.acc_r = taps->acc_r;
    a.tap_codes = taps->h_codes;
    a.tap_zero = taps->h_zero;
    a.tap_inv_q = taps->h_inv_q;
    a.tap_gates = taps->gates;
    a.tap_c = taps->c;
    a.tap_m = taps->m;
  }
  a.ws = rec;
  return a;
}

// One layer given its input codes; writes h (float) and hout (codes).
ql_status run_layer(const ql_lstm_layer &L, const ActRows &xin, int64_t T, int64_t B,
                    const float *h0, const float *c0, float *h, float *hT, float *cT,
                    const LayerWs &w, const ql_lstm_taps *taps, hipStream_t s) {
  const int64_t M = T * B, H = L.hidden;
  hipError_t e = launch_gemm_recover(xin, weight(L.Wx), M, 4 * H, L.in, L.bias, w.gx,
                                     taps ? taps->acc_x : nullptr, s);
  if (e != hipSuccess) return QL_EHIP;
  bool unsupported = false;
  RecurrentArgs a = rec_args(L, T, B, w.gx, h0, c0, h, hT, cT, w.hout, taps, w.rec);
  e = launch_recurrent(a, s, &unsupported);
  if (e != hipSuccess) return QL_EHIP;
  return unsupported ? QL_EUNSUPPORTED : QL_OK;
}

}  // namespace

extern "C" {

const char *ql_status_str(ql_status s) {
  switch (enum_arg(s)) {
    case QL_OK: return "ok";
    case QL_EINVAL: return "invalid argument";
    case QL_ESHAPE: return "inconsistent shapes";
    case QL_EOVERFLOW: return "K too large for 32-bit accumulators";
    case QL_EWORKSPACE: return "workspace too small";
    case QL_EHIP: return "HIP runtime error";
    case QL_EUNSUPPORTED: return "shape not supported by the kernels";
    case QL_ETIMEOUT: return "persistent kernel wait timed out";
    case QL_ESCRATCH: return "call needs more than the no-alloc entry point's static scratch";
  }
  return "unknown status";
}

size_t ql_quantize_workspace(int64_t rows, int64_t cols, int32_t nblocks) {
  (void)rows;
  (void)cols;
  return set_quantize_ws(nblocks > 0 ? nblocks : 1);
}

ql_status ql_quantize(const float *src, int64_t rows, int64_t cols, int32_t nblocks,
                      ql_qmatrix *dst, void *ws, size_t ws_bytes, void *stream) {
  if (!dst || !dst->zero || !dst->inv_q) return QL_EINVAL;
  if (rows * cols > 0 && (!src || !dst->codes)) return QL_EINVAL;
  if (rows < 0 || cols < 0 || nblocks <= 0 || rows % nblocks != 0) return QL_ESHAPE;
  if (nblocks > 65535) return QL_EUNSUPPORTED;  // one grid row of partial min/max per set
  if (dst->rows != rows || dst->cols != cols || dst->nblocks != nblocks) return QL_ESHAPE;
  if (dst->ld < cols || dst->ld % 64 != 0) return QL_ESHAPE;
  if (!ws || ws_bytes < ql_quantize_workspace(rows, cols, nblocks)) return QL_EWORKSPACE;
  return from_hip(launch_set_quantize(src, cols, rows, cols, nblocks, dst->codes, dst->ld,
                                      dst->range, dst->zero, dst->inv_q, dst->row_sums, nullptr,
                                      nullptr, ws, as_stream(stream)));
}

ql_status ql_dequantize(const ql_qmatrix *q, float *dst, void *stream) {
  if (!q || !q->codes || !q->zero || !q->inv_q) return QL_EINVAL;
  if (q->rows * q->cols > 0 && !dst) return QL_EINVAL;
  if (q->rows < 0 || q->cols < 0 || q->nblocks <= 0 || q->rows % q->nblocks != 0 ||
      q->ld < q->cols)
    return QL_ESHAPE;
  return from_hip(launch_dequantize(q->codes, q->ld, q->rows, q->cols, q->nblocks, q->zero,
                                    q->inv_q, dst, as_stream(stream)));
}

size_t ql_quantized_matmul_workspace(int64_t m, int64_t rows, int64_t cols) {
  (void)rows;
  Carve c(nullptr);
  take_act(c, m, cols);
  c.take<char>(set_quantize_ws(1));
  return c.off;
}

ql_status ql_quantized_matmul(const ql_qmatrix *W, const float *X, int64_t m, ql_act_gran gran,
                              const float *bias, float *Y, int32_t *acc, void *ws,
                              size_t ws_bytes, void *stream) {
  ql_status st = check_qmatrix(W, true);
  if (st != QL_OK) return st;
  if (m > 0 && (!X || !Y)) return QL_EINVAL;
  const int g = enum_arg(gran);
  if (g != QL_ACT_PER_TENSOR && g != QL_ACT_PER_ROW) return QL_EINVAL;
  if (m < 0) return QL_ESHAPE;
  if (!ws || ws_bytes < ql_quantized_matmul_workspace(m, W->rows, W->cols)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  Carve c(ws);
  ActBuf x = take_act(c, m, W->cols);
  void *qws = c.take<char>(set_quantize_ws(1));
  hipError_t e;
  if (g == QL_ACT_PER_ROW)
    e = launch_quantize_rows(X, W->cols, m, W->cols, x.codes, x.ld, x.zero, x.inv_q, x.sums, s);
  else
    e = launch_set_quantize(X, W->cols, m, W->cols, 1, x.codes, x.ld, nullptr, nullptr, nullptr,
                            x.sums, x.zero, x.inv_q, qws, s);
  if (e != hipSuccess) return QL_EHIP;
  return from_hip(launch_gemm_recover(x.rows(), weight(*W), m, W->rows, W->cols, bias, Y, acc, s));
}

size_t ql_gemm_u8_workspace(int64_t M, int64_t N, int64_t K) {
  (void)K;
  return align_up((size_t)M * 4, 256) + align_up((size_t)N * 4, 256);
}

ql_status ql_gemm_u8(const int8_t *A, int64_t lda, const int8_t *B, int64_t ldb, int32_t *C,
                     int64_t M, int64_t N, int64_t K, const int32_t *a_sums,
                     const int32_t *b_sums, void *ws, size_t ws_bytes, void *stream) {
  if (M < 0 || N < 0 || K < 0) return QL_ESHAPE;
  if ((M > 0 && !A) || (N > 0 && !B) || (M > 0 && N > 0 && !C)) return QL_EINVAL;
  if (M < 0 || N < 0 || K < 0 || lda < K || ldb < K || lda % 64 || ldb % 64) return QL_ESHAPE;
  if (K > kMaxK) return QL_EOVERFLOW;
  hipStream_t s = as_stream(stream);
  if (!a_sums || !b_sums) {
    if (!ws || ws_bytes < ql_gemm_u8_workspace(M, N, K)) return QL_EWORKSPACE;
    Carve c(ws);
    int32_t *sa = c.take<int32_t>((size_t)M), *sb = c.take<int32_t>((size_t)N);
    if (!a_sums) {
      if (launch_code_row_sums(A, lda, M, K, sa, s) != hipSuccess) return QL_EHIP;
      a_sums = sa;
    }
    if (!b_sums) {
      if (launch_code_row_sums(B, ldb, N, K, sb, s) != hipSuccess) return QL_EHIP;
      b_sums = sb;
    }
  }
  return from_hip(launch_gemm_raw(A, lda, B, ldb, C, M, N, K, a_sums, b_sums, s));
}

size_t ql_lstm_layer_workspace(const ql_lstm_layer *L, int64_t T, int64_t B) {
  if (!L || T < 0 || B < 0) return 0;
  Carve c(nullptr);
  carve_layer(c, *L, T, B, true);
  return c.off;
}

ql_status ql_lstm_layer_forward(const ql_lstm_layer *L, const float *x, int64_t T, int64_t B,
                                const float *h0, const float *c0, float *h, float *hT,
                                float *cT, const ql_lstm_taps *taps, void *ws, size_t ws_bytes,
                                void *stream) {
  ql_status st = check_layer(L);
  if (st != QL_OK) return st;
  if (T < 0 || B < 0) return QL_ESHAPE;
  if (T * B > 0 && (!x || !h)) return QL_EINVAL;
  if (!ws || ws_bytes < ql_lstm_layer_workspace(L, T, B)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  Carve c(ws);
  LayerWs w = carve_layer(c, *L, T, B, true);
  if (reset_recurrent_flag(w.rec, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;
  if (launch_quantize_rows(x, L->in, T * B, L->in, w.xin.codes, w.xin.ld, w.xin.zero,
                           w.xin.inv_q, w.xin.sums, s) != hipSuccess)
    return QL_EHIP;
  return run_layer(*L, w.xin.rows(), T, B, h0, c0, h, hT, cT, w, taps, s);
}

}  // extern "C"

namespace {
// A model whose layers share one width H <= 512 and have no projection can
// run several layers per persistent launch (a wavefront); per-layer
// accumulator taps need the one-layer path.
bool stackable(const ql_model &M) {
  if (M.nlayers < 2) return false;
  for (int l = 0; l < M.nlayers; ++l) {
    const ql_lstm_layer &L = M.layers[l];
    if (L.proj != 0 || L.hidden != M.layers[0].hidden || L.hidden > 512) return false;
  }
  return true;
}
// Initial / final state of layer l of a call (host arrays of per-layer
// descriptors, each nullable).
const float *st_h(const ql_lstm_state *s, int l) { return s ? s[l].h : nullptr; }
const float *st_c(const ql_lstm_state *s, int l) { return s ? s[l].c : nullptr; }
float *st_hout(const ql_lstm_state *s, int l) { return s ? s[l].h : nullptr; }
float *st_cout(const ql_lstm_state *s, int l) { return s ? s[l].c : nullptr; }

// Layers that all have a projection, at one batch row, run as the projection
// wavefront (ql_pstack.hip) when at least two of them share a launch.
bool pstack_shapes(const ql_lstm_layer *layers, int n, int64_t B) {
  if (B != 1 || n < 2) return false;
  for (int l = 0; l < n; ++l) {
    const ql_lstm_layer &L = layers[l];
    if (L.proj <= 0 || L.hidden > 512 || L.proj > 512 || L.in > 512) return false;
  }
  return true;
}
PStackArgs pstack_shape_args(const ql_lstm_layer *layers, int n, int64_t T) {
  PStackArgs a{};
  a.nl = n < kMaxStack ? n : kMaxStack;
  a.T = T;
  for (int k = 0; k < a.nl; ++k) {
    a.L[k].in = layers[k].in;
    a.L[k].H = layers[k].hidden;
    a.L[k].P = layers[k].proj;
  }
  return a;
}
int pstack_per_launch(const ql_lstm_layer *layers, int n, int64_t T, int64_t B) {
  if (!pstack_shapes(layers, n, B)) return 1;
  return pstack_layers_per_launch(pstack_shape_args(layers, n, T));
}
PStackLayer pstack_layer(const ql_lstm_layer &L, const ActRows &xin, const ActBuf &out,
                         const ql_lstm_taps *t, const ql_lstm_state *s0, const ql_lstm_state *s1,
                         int l) {
  PStackLayer s{};
  s.Wx = weight(L.Wx);
  s.Wh = weight(L.Wh);
  s.Wr = weight(L.Wr);
  s.bias = L.bias;
  s.in = L.in;
  s.H = L.hidden;
  s.P = L.proj;
  s.xin = xin;
  s.out = OutRows{out.codes, out.ld, out.zero, out.inv_q, out.sums};
  s.h = nullptr;
  if (t) {
    s.tap_codes = t->h_codes;
    s.tap_zero = t->h_zero;
    s.tap_inv_q = t->h_inv_q;
    s.acc_x = t->acc_x;
    s.acc_h = t->acc_h;
    s.acc_r = t->acc_r;
    s.h = t->h;
    s.tap_gates = t->gates;
    s.tap_c = t->c;
    s.tap_m = t->m;
  }
  s.h0 = st_h(s0, l);
  s.c0 = st_c(s0, l);
  s.hT = st_hout(s1, l);
  s.cT = st_cout(s1, l);
  return s;
}

// Workspace of a model forward: exchange scratch first (it holds the timeout
// flag), then the input codes, W_x x + b, one code buffer per layer, h.
struct ModelWs {
  void *rec;
  ActBuf xin;
  float *gx;
  ActBuf out[kMaxStack > 16 ? kMaxStack : 16];
  float *hf;
  void *sws;
};
ModelWs carve_model(Carve &c, const ql_model &M, int64_t T, int64_t B) {
  int64_t maxH = 0, maxR = 0, maxP = 0;
  for (int l = 0; l < M.nlayers; ++l) {
    const ql_lstm_layer &L = M.layers[l];
    maxH = L.hidden > maxH ? L.hidden : maxH;
    maxR = layer_width(L) > maxR ? layer_width(L) : maxR;
    maxP = L.proj > maxP ? L.proj : maxP;
  }
  const int64_t MB = T * B;
  size_t rec = recurrent_ws(B, maxH, maxP);
  if (stackable(M)) {
    const size_t st = stack_ws(M.nlayers < kMaxStack ? M.nlayers : kMaxStack, T, B, maxH);
    rec = rec > st ? rec : st;
  }
  const bool pst = pstack_shapes(M.layers, M.nlayers, B);
  if (pst) {
    int64_t hs[kMaxStack], ps[kMaxStack];
    const int nl = M.nlayers < kMaxStack ? M.nlayers : kMaxStack;
    for (int k = 0; k < nl; ++k) hs[k] = maxH, ps[k] = maxP;
    const size_t st = pstack_ws(hs, ps, nl, T);
    rec = rec > st ? rec : st;
  }
  ModelWs w{};
  w.rec = c.take<char>(rec);
  w.xin = take_act(c, MB, M.layers[0].in);
  w.gx = c.take<float>((size_t)(MB * 4 * maxH));
  // one output code buffer per layer (two alternate when layers run one by one)
  const int nbuf = stackable(M) || pst ? (M.nlayers < 16 ? M.nlayers : 16) : 2;
  for (int i = 0; i < nbuf; ++i) w.out[i] = take_act(c, MB, maxR);
  w.hf = c.take<float>((size_t)(MB * maxR));
  w.sws = c.take<char>(softmax_ws(MB, M.Wy.rows));
  return w;
}

StackLayer stack_layer(const ql_lstm_layer &L, const ActRows &xin, const ActBuf &out,
                       const ql_lstm_taps *t, const ql_lstm_state *s0, const ql_lstm_state *s1,
                       int l) {
  StackLayer s{};
  s.Wx = weight(L.Wx);
  s.Wh = weight(L.Wh);
  s.bias = L.bias;
  s.in = L.in;
  s.xin = xin;
  s.out = OutRows{out.codes, out.ld, out.zero, out.inv_q, out.sums};
  s.h = nullptr;
  if (t) {
    s.tap_codes = t->h_codes;
    s.tap_zero = t->h_zero;
    s.tap_inv_q = t->h_inv_q;
    s.acc_x = t->acc_x;
    s.acc_h = t->acc_h;
    s.h = t->h;
    s.tap_gates = t->gates;
    s.tap_c = t->c;
    s.tap_m = t->m;
  }
  s.h0 = st_h(s0, l);
  s.c0 = st_c(s0, l);
  s.hT = st_hout(s1, l);
  s.cT = st_cout(s1, l);
  return s;
}

size_t model_ws_bytes(const ql_model *M, int64_t T, int64_t B) {
  Carve c(nullptr);
  carve_model(c, *M, T, B);
  return c.off;
}
}  // namespace

extern "C" {
size_t ql_acoustic_model_workspace(const ql_model *M, int64_t T, int64_t B) {
  if (!M || M->nlayers <= 0 || !M->layers || T < 0 || B < 0) return 0;
  return model_ws_bytes(M, T, B);
}

}  // extern "C"

namespace {
// Where the first layer's input comes from: a dense [T][B][in] array of
// presented inputs, or the frontend's base frames [nframes][B][dim] stacked
// `stack` at a time with every `skip`-th stack presented (Section 4).
struct Frontend {
  const float *x;
  bool stacked;
  int32_t dim, stack, skip;
};

hipError_t quantize_input(const Frontend &f, int64_t T, int64_t B, int64_t in, const ActBuf &dst,
                          hipStream_t s) {
  if (f.stacked)
    return launch_quantize_stacked(f.x, B, f.dim, f.stack, f.skip, T, dst.codes, dst.ld,
                                   dst.zero, dst.inv_q, dst.sums, s);
  return launch_quantize_rows(f.x, in, T * B, in, dst.codes, dst.ld, dst.zero, dst.inv_q,
                              dst.sums, s);
}

ql_status model_forward(const ql_model *M, const Frontend &fe, int64_t T, int64_t B, float *post,
                        const ql_lstm_state *s0, const ql_lstm_state *s1,
                        const ql_model_taps *taps, void *ws, size_t ws_bytes, void *stream,
                        bool output_layer = true) {
  if (!M || !M->layers || !M->by) return QL_EINVAL;
  if (M->nlayers <= 0 || T < 0 || B < 0) return QL_ESHAPE;
  if (T * B > 0 && (!fe.x || !post)) return QL_EINVAL;
  for (int l = 0; l < M->nlayers; ++l) {
    ql_status st = check_layer(&M->layers[l]);
    if (st != QL_OK) return st;
    const int64_t want_in = l == 0 ? M->layers[0].in : layer_width(M->layers[l - 1]);
    if (M->layers[l].in != want_in) return QL_ESHAPE;
  }
  if (states_overlap(M->layers, M->nlayers, B, s0, s1)) return QL_EINVAL;
  ql_status st = QL_OK;
  if (output_layer) {
    st = check_qmatrix(&M->Wy, true);
    if (st != QL_OK) return st;
    if (M->Wy.cols != layer_width(M->layers[M->nlayers - 1])) return QL_ESHAPE;
  }
  if (!ws || ws_bytes < ql_acoustic_model_workspace(M, T, B)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  // the timeout flag sits at the start of the workspace in every forward call
  if (reset_recurrent_flag(ws, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;

  int64_t maxH = 0, maxR = 0, maxP = 0;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_lstm_layer &L = M->layers[l];
    maxH = L.hidden > maxH ? L.hidden : maxH;
    maxR = layer_width(L) > maxR ? layer_width(L) : maxR;
    maxP = L.proj > maxP ? L.proj : maxP;
  }
  const int64_t MB = T * B;
  (void)maxP;
  Carve c(ws);
  ModelWs mw = carve_model(c, *M, T, B);

  if (quantize_input(fe, T, B, M->layers[0].in, mw.xin, s) != hipSuccess) return QL_EHIP;
  ActRows cur = mw.xin.rows();
  const bool stack = stackable(*M);
  const bool pst = !stack && pstack_shapes(M->layers, M->nlayers, B);
  int per_launch = 1;
  if (stack) {
    const int64_t in1 = M->nlayers > 1 ? M->layers[1].in : M->layers[0].in;
    per_launch = stack_layers_per_launch(M->nlayers, T, B, maxH, M->layers[0].in, in1);
  } else if (pst) {
    per_launch = pstack_per_launch(M->layers, M->nlayers, T, B);
  }
  for (int l = 0; l < M->nlayers;) {
    const int left = M->nlayers - l;
    // split the layers into launches of nearly equal size
    const int launches = (left + per_launch - 1) / per_launch;
    const int n = (left + launches - 1) / launches;
    if (stack && n >= 2) {
      StackArgs sa{};
      sa.nl = n;
      sa.T = T;
      sa.B = B;
      sa.H = maxH;
      sa.ws = mw.rec;
      for (int k = 0; k < n; ++k) {
        const ql_lstm_taps *lt = taps && taps->layers ? &taps->layers[l + k] : nullptr;
        const ActRows xin = k == 0 ? cur : mw.out[l + k - 1].rows();
        sa.L[k] = stack_layer(M->layers[l + k], xin, mw.out[l + k], lt, s0, s1, l + k);
      }
      bool unsupported = false;
      if (launch_stack(sa, s, &unsupported) != hipSuccess) return QL_EHIP;
      if (unsupported) return QL_EUNSUPPORTED;
      cur = mw.out[l + n - 1].rows();
      l += n;
      continue;
    }
    if (pst && n >= 2) {
      PStackArgs pa{};
      pa.nl = n;
      pa.T = T;
      pa.ws = mw.rec;
      for (int k = 0; k < n; ++k) {
        const ql_lstm_taps *lt = taps && taps->layers ? &taps->layers[l + k] : nullptr;
        pa.L[k] = pstack_layer(M->layers[l + k], k == 0 ? cur : ActRows{}, mw.out[l + k], lt, s0,
                               s1, l + k);
      }
      bool unsupported = false;
      if (launch_pstack(pa, s, &unsupported) != hipSuccess) return QL_EHIP;
      if (unsupported) return QL_EUNSUPPORTED;
      cur = mw.out[l + n - 1].rows();
      l += n;
      continue;
    }
    const ql_lstm_layer &L = M->layers[l];
    LayerWs w;
    w.rec = mw.rec;
    w.gx = mw.gx;
    w.hout = mw.out[stack || pst ? l : (l & 1)];
    w.hout.ld = round_up(layer_width(L), 64);
    const ql_lstm_taps *lt = taps && taps->layers ? &taps->layers[l] : nullptr;
    st = run_layer(L, cur, T, B, st_h(s0, l), st_c(s0, l), lt && lt->h ? lt->h : mw.hf,
                   st_hout(s1, l), st_cout(s1, l), w, lt, s);
    if (st != QL_OK) return st;
    cur = w.hout.rows();
    ++l;
  }
  if (!output_layer) return QL_OK;
  const int64_t K = layer_width(M->layers[M->nlayers - 1]);
  return from_hip(launch_softmax_layer(cur, weight(M->Wy), MB, M->Wy.rows, K, M->by, post,
                                       taps ? taps->acc_y : nullptr,
                                       taps ? taps->logits : nullptr, mw.sws, s));
}
}  // namespace

extern "C" {
ql_status ql_acoustic_model_forward(const ql_model *M, const float *feats, int64_t T, int64_t B,
                                    float *post, const ql_model_taps *taps, void *ws,
                                    size_t ws_bytes, void *stream) {
  return model_forward(M, Frontend{feats, false, 0, 0, 0}, T, B, post, nullptr, nullptr, taps, ws,
                       ws_bytes, stream);
}

ql_status ql_acoustic_model_forward_stream(const ql_model *M, const float *feats, int64_t T,
                                           int64_t B, const ql_lstm_state *state_in,
                                           const ql_lstm_state *state_out, float *post,
                                           const ql_model_taps *taps, void *ws, size_t ws_bytes,
                                           void *stream) {
  return model_forward(M, Frontend{feats, false, 0, 0, 0}, T, B, post, state_in, state_out, taps,
                       ws, ws_bytes, stream);
}

int64_t ql_stacked_input_count(int64_t nframes, int32_t stack, int32_t skip) {
  if (nframes < 0 || stack <= 0 || skip <= 0 || nframes < stack) return 0;
  return (nframes - stack) / skip + 1;
}

namespace {
ql_status check_frontend(int64_t nframes, int64_t B, int64_t dim, int32_t stack, int32_t skip,
                         int64_t in) {
  if (nframes < 0 || B < 0 || dim <= 0 || stack <= 0 || skip <= 0) return QL_ESHAPE;
  if (dim * stack != in || in > INT32_MAX) return QL_ESHAPE;
  return QL_OK;
}
}  // namespace

ql_status ql_quantize_stacked_frames(const float *frames, int64_t nframes, int64_t B, int64_t dim,
                                     int32_t stack, int32_t skip, const ql_qact *dst,
                                     void *stream) {
  if (!dst) return QL_EINVAL;
  ql_status st = check_frontend(nframes, B, dim, stack, skip, dst->cols);
  if (st != QL_OK) return st;
  const int64_t T = ql_stacked_input_count(nframes, stack, skip);
  if (dst->rows != T * B || dst->ld < round_up(dst->cols, 64) || dst->ld % 64) return QL_ESHAPE;
  if (T * B == 0) return QL_OK;
  if (!frames || !dst->codes || !dst->zero || !dst->inv_q || !dst->sums) return QL_EINVAL;
  return from_hip(launch_quantize_stacked(frames, B, (int)dim, stack, skip, T, dst->codes,
                                          dst->ld, dst->zero, dst->inv_q, dst->sums,
                                          as_stream(stream)));
}

size_t ql_acoustic_model_frames_workspace(const ql_model *M, int64_t nframes, int64_t B,
                                          int32_t stack, int32_t skip) {
  return ql_acoustic_model_workspace(M, ql_stacked_input_count(nframes, stack, skip), B);
}

ql_status ql_acoustic_model_forward_frames(const ql_model *M, const float *frames,
                                           int64_t nframes, int64_t B, int64_t dim,
                                           int32_t stack, int32_t skip, float *post,
                                           const ql_model_taps *taps, void *ws, size_t ws_bytes,
                                           void *stream) {
  if (!M || !M->layers) return QL_EINVAL;
  if (M->nlayers <= 0) return QL_ESHAPE;
  ql_status st = check_frontend(nframes, B, dim, stack, skip, M->layers[0].in);
  if (st != QL_OK) return st;
  const int64_t T = ql_stacked_input_count(nframes, stack, skip);
  return model_forward(M, Frontend{frames, true, (int32_t)dim, stack, skip}, T, B, post, nullptr,
                       nullptr, taps, ws, ws_bytes, stream);
}

size_t ql_lstm_recurrence_workspace(const ql_lstm_layer *L, int64_t T, int64_t B) {
  if (!L || T < 0 || B < 0) return 0;
  Carve c(nullptr);
  c.take<char>(recurrent_ws(B, L->hidden, L->proj));
  take_act(c, T * B, layer_width(*L));
  return c.off;
}

ql_status ql_lstm_recurrence(const ql_lstm_layer *L, const float *gx, int64_t T, int64_t B,
                             const float *h0, const float *c0, float *h, float *hT, float *cT,
                             const ql_qact *h_codes, const ql_lstm_taps *taps, void *ws,
                             size_t ws_bytes, void *stream) {
  ql_status st = check_layer(L);
  if (st != QL_OK) return st;
  if (T < 0 || B < 0) return QL_ESHAPE;
  if (T * B > 0 && (!gx || !h)) return QL_EINVAL;
  const int64_t R = layer_width(*L);
  if (h_codes) {
    if (!h_codes->codes || !h_codes->zero || !h_codes->inv_q || !h_codes->sums) return QL_EINVAL;
    if (h_codes->rows != T * B || h_codes->cols != R || h_codes->ld < round_up(R, 64) ||
        h_codes->ld % 64)
      return QL_ESHAPE;
  }
  if (!ws || ws_bytes < ql_lstm_recurrence_workspace(L, T, B)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  Carve c(ws);
  void *rec = c.take<char>(recurrent_ws(B, L->hidden, L->proj));
  if (reset_recurrent_flag(rec, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;
  ActBuf out = take_act(c, T * B, R);
  if (h_codes) {
    out.codes = h_codes->codes;
    out.ld = h_codes->ld;
    out.zero = h_codes->zero;
    out.inv_q = h_codes->inv_q;
    out.sums = h_codes->sums;
  }
  bool unsupported = false;
  RecurrentArgs a = rec_args(*L, T, B, gx, h0, c0, h, hT, cT, out, taps, rec);
  if (launch_recurrent(a, s, &unsupported) != hipSuccess) return QL_EHIP;
  return unsupported ? QL_EUNSUPPORTED : QL_OK;
}

// ---------------------------------------------------------------- fp32 model
namespace {
int64_t f32_width(const ql_f32_layer &L) { return L.proj ? L.proj : L.hidden; }

ql_status check_f32_layer(const ql_f32_layer *L) {
  if (!L || !L->Wx || !L->Wh || !L->bias || (L->proj && !L->Wr)) return QL_EINVAL;
  if (L->in <= 0 || L->hidden <= 0 || L->proj < 0) return QL_ESHAPE;
  return QL_OK;
}

// gx = x Wx^T + b over all frames, then the recurrence.
ql_status run_f32_layer(const ql_f32_layer &L, const float *x, int64_t T, int64_t B,
                        const float *h0, const float *c0, float *h, float *hT, float *cT,
                        float *gx, void *rec, hipStream_t s) {
  const int64_t H = L.hidden;
  if (launch_sgemm(x, L.in, L.Wx, L.in, T * B, 4 * H, L.in, L.bias, gx, 4 * H, s) != hipSuccess)
    return QL_EHIP;
  F32RecArgs a{};
  a.T = T;
  a.B = B;
  a.H = H;
  a.P = L.proj;
  a.R = f32_width(L);
  a.gx = gx;
  a.Wh = L.Wh;
  a.Wr = L.Wr;
  a.h0 = h0;
  a.c0 = c0;
  a.h = h;
  a.hT = hT;
  a.cT = cT;
  a.ws = rec;
  bool unsupported = false;
  if (launch_recurrent_f32(a, s, &unsupported) != hipSuccess) return QL_EHIP;
  return unsupported ? QL_EUNSUPPORTED : QL_OK;
}
}  // namespace

ql_status ql_f32_matmul(const float *W, int64_t rows, int64_t cols, const float *X, int64_t m,
                        const float *bias, float *Y, void *stream) {
  if (rows < 0 || cols < 0 || m < 0) return QL_ESHAPE;
  if (rows * m > 0 && (!W || !X || !Y)) return QL_EINVAL;
  return from_hip(launch_sgemm(X, cols, W, cols, m, rows, cols, bias, Y, rows, as_stream(stream)));
}

size_t ql_f32_lstm_layer_workspace(const ql_f32_layer *L, int64_t T, int64_t B) {
  if (!L || T < 0 || B < 0) return 0;
  Carve c(nullptr);
  c.take<char>(recurrent_f32_ws(B, L->hidden, L->proj));
  c.take<float>((size_t)(T * B * 4 * L->hidden));
  return c.off;
}

ql_status ql_f32_lstm_layer_forward(const ql_f32_layer *L, const float *x, int64_t T,
                                    int64_t B, const float *h0, const float *c0, float *h,
                                    float *hT, float *cT, void *ws, size_t ws_bytes,
                                    void *stream) {
  ql_status st = check_f32_layer(L);
  if (st != QL_OK) return st;
  if (T < 0 || B < 0) return QL_ESHAPE;
  if (T * B > 0 && (!x || !h)) return QL_EINVAL;
  if (!ws || ws_bytes < ql_f32_lstm_layer_workspace(L, T, B)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  Carve c(ws);
  void *rec = c.take<char>(recurrent_f32_ws(B, L->hidden, L->proj));
  float *gx = c.take<float>((size_t)(T * B * 4 * L->hidden));
  if (reset_recurrent_flag(rec, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;
  return run_f32_layer(*L, x, T, B, h0, c0, h, hT, cT, gx, rec, s);
}

size_t ql_f32_acoustic_model_workspace(const ql_f32_model *M, int64_t T, int64_t B) {
  if (!M || M->nlayers <= 0 || !M->layers || T < 0 || B < 0) return 0;
  int64_t maxH = 0, maxR = 0, maxP = 0;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_f32_layer &L = M->layers[l];
    maxH = L.hidden > maxH ? L.hidden : maxH;
    maxR = f32_width(L) > maxR ? f32_width(L) : maxR;
    maxP = L.proj > maxP ? L.proj : maxP;
  }
  Carve c(nullptr);
  c.take<char>(recurrent_f32_ws(B, maxH, maxP));
  c.take<float>((size_t)(T * B * 4 * maxH));
  c.take<float>((size_t)(T * B * maxR));
  c.take<float>((size_t)(T * B * maxR));
  return c.off;
}

ql_status ql_f32_acoustic_model_forward(const ql_f32_model *M, const float *feats, int64_t T,
                                        int64_t B, float *post, void *ws, size_t ws_bytes,
                                        void *stream) {
  if (!M || !M->layers || !M->Wy || !M->by) return QL_EINVAL;
  if (M->nlayers <= 0 || M->states <= 0 || T < 0 || B < 0) return QL_ESHAPE;
  if (T * B > 0 && (!feats || !post)) return QL_EINVAL;
  for (int l = 0; l < M->nlayers; ++l) {
    ql_status st = check_f32_layer(&M->layers[l]);
    if (st != QL_OK) return st;
    const int64_t want_in = l == 0 ? M->layers[0].in : f32_width(M->layers[l - 1]);
    if (M->layers[l].in != want_in) return QL_ESHAPE;
  }
  if (!ws || ws_bytes < ql_f32_acoustic_model_workspace(M, T, B)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  if (reset_recurrent_flag(ws, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;
  int64_t maxH = 0, maxR = 0, maxP = 0;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_f32_layer &L = M->layers[l];
    maxH = L.hidden > maxH ? L.hidden : maxH;
    maxR = f32_width(L) > maxR ? f32_width(L) : maxR;
    maxP = L.proj > maxP ? L.proj : maxP;
  }
  const int64_t MB = T * B;
  Carve c(ws);
  void *rec = c.take<char>(recurrent_f32_ws(B, maxH, maxP));
  float *gx = c.take<float>((size_t)(MB * 4 * maxH));
  float *hbuf[2] = {c.take<float>((size_t)(MB * maxR)), c.take<float>((size_t)(MB * maxR))};
  const float *cur = feats;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_f32_layer &L = M->layers[l];
    ql_status st = run_f32_layer(L, cur, T, B, nullptr, nullptr, hbuf[l & 1], nullptr, nullptr,
                                 gx, rec, s);
    if (st != QL_OK) return st;
    cur = hbuf[l & 1];
  }
  const int64_t K = f32_width(M->layers[M->nlayers - 1]);
  if (launch_sgemm(cur, K, M->Wy, K, MB, M->states, K, M->by, post, M->states, s) != hipSuccess)
    return QL_EHIP;
  return from_hip(launch_softmax_rows(post, MB, M->states, s));
}

ql_status ql_quantize_activations(const float *X, int64_t m, int64_t cols, const ql_qact *dst,
                                  void *stream) {
  if (!dst) return QL_EINVAL;
  if (m < 0 || cols < 0) return QL_ESHAPE;
  if (dst->rows != m || dst->cols != cols || dst->ld < round_up(cols, 64) || dst->ld % 64)
    return QL_ESHAPE;
  if (m == 0) return QL_OK;
  if (!X || !dst->codes || !dst->zero || !dst->inv_q || !dst->sums) return QL_EINVAL;
  return from_hip(launch_quantize_rows(X, cols, m, cols, dst->codes, dst->ld, dst->zero,
                                       dst->inv_q, dst->sums, as_stream(stream)));
}

namespace {
// The last layer's h went to its tap when one was given: h_last gets a copy.
ql_status copy_last_h(float *h_last, const float *written, int64_t count, hipStream_t s) {
  if (!h_last || written == h_last || count == 0) return QL_OK;
  return from_hip(hipMemcpyAsync(h_last, written, (size_t)count * sizeof(float),
                                 hipMemcpyDeviceToDevice, s));
}
}  // namespace

size_t ql_lstm_stack_workspace(const ql_lstm_layer *layers, int32_t n, int64_t T, int64_t B) {
  if (!layers || n < 1 || n > kMaxStack || T < 0 || B < 0) return 0;
  if (layers[0].proj > 0) {  // the projection wavefront (batch 1)
    int64_t hs[kMaxStack], ps[kMaxStack];
    for (int k = 0; k < n; ++k) hs[k] = layers[k].hidden, ps[k] = layers[k].proj;
    return align_up(pstack_ws(hs, ps, n, T), 256);
  }
  return align_up(stack_ws(n, T, B, layers[0].hidden), 256);
}

int32_t ql_lstm_stack_layers_per_launch(const ql_lstm_layer *layers, int32_t n, int64_t T,
                                        int64_t B) {
  if (!layers || n < 2 || T < 0 || B < 0) return 1;
  if (pstack_shapes(layers, n, B)) return pstack_per_launch(layers, n, T, B);
  const int64_t H = layers[0].hidden;
  for (int k = 0; k < n; ++k)
    if (layers[k].proj != 0 || layers[k].hidden != H || (k > 0 && layers[k].in != H)) return 1;
  return stack_layers_per_launch(n, T, B, H, layers[0].in, n > 1 ? layers[1].in : layers[0].in);
}

ql_status ql_lstm_stack_forward(const ql_lstm_layer *layers, int32_t n, const ql_qact *x,
                                int64_t T, int64_t B, const ql_qact *h_codes, float *h_last,
                                const ql_lstm_state *state_in, const ql_lstm_state *state_out,
                                const ql_lstm_taps *taps, void *ws, size_t ws_bytes,
                                void *stream) {
  if (!layers || !x || !h_codes) return QL_EINVAL;
  if (n < 1 || n > kMaxStack || T < 0 || B < 0) return QL_ESHAPE;
  const int64_t H = layers[0].hidden;
  const bool proj = layers[0].proj > 0;
  for (int k = 0; k < n; ++k) {
    const ql_status st = check_layer(&layers[k]);
    if (st != QL_OK) return st;
    if (proj) {  // every layer projected, each taking the previous one's P outputs
      if (layers[k].proj <= 0 || (k > 0 && layers[k].in != layers[k - 1].proj)) return QL_ESHAPE;
    } else {
      if (layers[k].proj != 0 || layers[k].hidden != H) return QL_ESHAPE;
      if (k > 0 && layers[k].in != H) return QL_ESHAPE;
    }
    const int64_t R = layer_width(layers[k]);
    const ql_qact &o = h_codes[k];
    if (o.rows != T * B || o.cols != R || o.ld < round_up(R, 64) || o.ld % 64) return QL_ESHAPE;
    if (T * B > 0 && (!o.codes || !o.zero || !o.inv_q || !o.sums)) return QL_EINVAL;
  }
  if (x->rows != T * B || x->cols != layers[0].in || x->ld < round_up(x->cols, 64) || x->ld % 64)
    return QL_ESHAPE;
  if (T * B > 0 && (!x->codes || !x->zero || !x->inv_q || !x->sums)) return QL_EINVAL;
  if (states_overlap(layers, n, B, state_in, state_out)) return QL_EINVAL;
  if (!ws || ws_bytes < ql_lstm_stack_workspace(layers, n, T, B)) return QL_EWORKSPACE;
  if (n == 1) return QL_EUNSUPPORTED;  // one layer: ql_lstm_layer_forward
  hipStream_t s = as_stream(stream);
  if (reset_recurrent_flag(ws, s) != hipSuccess) return QL_EHIP;
  if (T == 0 || B == 0) return QL_OK;
  if (proj) {
    if (B != 1) return QL_EUNSUPPORTED;  // batched projection layers: one layer per call
    PStackArgs pa{};
    pa.nl = n;
    pa.T = T;
    pa.ws = ws;
    for (int k = 0; k < n; ++k) {
      const ActRows xin = k == 0 ? ActRows{x->codes, x->ld, x->zero, x->inv_q, x->sums} : ActRows{};
      ActBuf out{h_codes[k].codes, h_codes[k].ld, h_codes[k].zero, h_codes[k].sums, h_codes[k].inv_q};
      pa.L[k] = pstack_layer(layers[k], xin, out, taps ? &taps[k] : nullptr, state_in,
                             state_out, k);
      if (k == n - 1 && h_last && !pa.L[k].h) pa.L[k].h = h_last;
    }
    bool unsupported = false;
    if (launch_pstack(pa, s, &unsupported) != hipSuccess) return QL_EHIP;
    if (unsupported) return QL_EUNSUPPORTED;
    return copy_last_h(h_last, pa.L[n - 1].h, T * B * layers[n - 1].proj, s);
  }
  StackArgs sa{};
  sa.nl = n;
  sa.T = T;
  sa.B = B;
  sa.H = H;
  sa.ws = ws;
  for (int k = 0; k < n; ++k) {
    const ActRows xin = k == 0 ? ActRows{x->codes, x->ld, x->zero, x->inv_q, x->sums}
                               : ActRows{h_codes[k - 1].codes, h_codes[k - 1].ld, h_codes[k - 1].zero,
                                         h_codes[k - 1].inv_q, h_codes[k - 1].sums};
    ActBuf out{h_codes[k].codes, h_codes[k].ld, h_codes[k].zero, h_codes[k].sums, h_codes[k].inv_q};
    sa.L[k] = stack_layer(layers[k], xin, out, taps ? &taps[k] : nullptr, state_in, state_out,
                          k);
    if (k == n - 1 && h_last && !sa.L[k].h) sa.L[k].h = h_last;
  }
  bool unsupported = false;
  if (launch_stack(sa, s, &unsupported) != hipSuccess) return QL_EHIP;
  if (unsupported) return QL_EUNSUPPORTED;
  return copy_last_h(h_last, sa.L[n - 1].h, T * B * H, s);
}

ql_status ql_workspace_status(const void *ws, void *stream) {
  if (!ws) return QL_EINVAL;
  bool to = false;
  if (recurrent_timed_out(ws, as_stream(stream), &to) != hipSuccess) return QL_EHIP;
  return to ? QL_ETIMEOUT : QL_OK;
}

ql_status ql_debug_set_wait_bound(int32_t polls) {
  if (polls < 0) return QL_EINVAL;
  return set_wait_bound(polls) == hipSuccess ? QL_OK : QL_EHIP;
}

int32_t ql_debug_recurrence_layout(const ql_lstm_layer *L, int64_t B) {
  if (check_layer(L) != QL_OK || B < 0) return -1;
  ActBuf out{};
  out.ld = round_up(layer_width(*L), 64);
  RecurrentArgs a = rec_args(*L, 1, B, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                             out, nullptr, nullptr);
  return recurrent_layout(a);
}

int32_t ql_debug_stack_layout(const ql_lstm_layer *layers, int32_t n, int64_t T, int64_t B) {
  if (!layers || n < 1 || T < 0 || B < 0) return -1;
  for (int k = 0; k < n; ++k)
    if (check_layer(&layers[k]) != QL_OK) return -1;
  const int per = ql_lstm_stack_layers_per_launch(layers, n, T, B);
  if (per < 2 || layers[0].proj != 0) return 0;
  // the first launch of the model forward's split into nearly equal launches
  const int launches = (n + per - 1) / per;
  const int nl = (n + launches - 1) / launches;
  if (nl < 2) return 0;
  StackArgs sa{};
  sa.nl = nl;
  sa.T = T;
  sa.B = B;
  sa.H = layers[0].hidden;
  for (int k = 0; k < nl; ++k) {
    ActBuf out{};
    out.ld = round_up(layer_width(layers[k]), 64);
    sa.L[k] = stack_layer(layers[k], ActRows{}, out, nullptr, nullptr, nullptr, k);
  }
  return stack_layout(sa);
}

ql_status ql_gate_fn(int32_t fn, const float *x, float *y, int64_t n, void *stream) {
  if (n > 0 && (!x || !y)) return QL_EINVAL;
  if (fn < 0 || fn > 3) return QL_EINVAL;
  if (n < 0) return QL_ESHAPE;
  return from_hip(launch_gate_fn(fn, x, y, n, as_stream(stream)));
}

}  // extern "C"

// ------------------------------------------------ quantization-aware training
namespace {

// Workspace of a training step, carved in a fixed order.  The exchange
// region at the head serves the forward pass, then the backward pass (its
// first bytes hold the timeout flag of both).
struct TrainWs {
  void *xch;
  size_t xch_bytes;
  struct QCopy {
    int8_t *codes;
    double *range;
    int32_t *zero;
    float *inv_q;
    int32_t *row_sums;
  } qx[kMaxStack > 16 ? kMaxStack : 16], qh[16], qy;
  void *qws;                          // set-quantizer scratch
  float *gates[16], *c[16], *h[16];   // forward activations per layer
  float *post;                        // posteriors, then dC/dz
  float *row_loss;
  float *dy, *dx, *da;                // dC/dh of the current layer, of its input, dC/da
  float *part;                        // split-K partial products
  float *cpart;                       // column-sum partials
};

constexpr int kMaxTrainLayers = 16;

int64_t train_width_max(const ql_train_model &M, int64_t *maxH, int64_t *maxIn) {
  int64_t mh = 0, mi = 0;
  for (int l = 0; l < M.nlayers; ++l) {
    mh = std::max<int64_t>(mh, M.layers[l].hidden);
    mi = std::max<int64_t>(mi, M.layers[l].in);
  }
  *maxH = mh;
  *maxIn = mi;
  return mh;
}

// K split of a gradient product with an M x N result: enough workgroups for
// the chip when the result is small and K is long.
int grad_splits(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  const int64_t by_k = std::max<int64_t>(1, K / 1024);
  return (int)std::max<int64_t>(1, std::min<int64_t>({512 / std::max<int64_t>(tiles, 1), by_k, 64}));
}

size_t grad_part_floats(const ql_train_model &M, int64_t T, int64_t B) {
  const int64_t N = T * B;
  size_t mx = 0;
  auto need = [&](int64_t m, int64_t n, int64_t k) {
    const int sp = grad_splits(m, n, k);
    if (sp > 1) mx = std::max(mx, (size_t)sp * (size_t)(m * n));
  };
  for (int l = 0; l < M.nlayers; ++l) {
    const int64_t H = M.layers[l].hidden;
    need(4 * H, M.layers[l].in, N);
    need(4 * H, H, N > B ? N - B : 0);
  }
  need(M.states, M.layers[M.nlayers - 1].hidden, N);
  return mx;
}

// A model of the quantized copies in w (descriptor arrays owned by the caller).
void train_qmodel(const ql_train_model &M, const TrainWs &w, int32_t gb, bool qout,
                  ql_lstm_layer *layers, ql_model *qm) {
  for (int l = 0; l < M.nlayers; ++l) {
    const ql_train_layer &L = M.layers[l];
    const int64_t H = L.hidden;
    ql_lstm_layer q{};
    q.in = L.in;
    q.hidden = H;
    q.proj = 0;
    q.Wx = ql_qmatrix{w.qx[l].codes, 4 * H, L.in, round_up(L.in, 64), gb, w.qx[l].range,
                      w.qx[l].zero, w.qx[l].inv_q, w.qx[l].row_sums};
    q.Wh = ql_qmatrix{w.qh[l].codes, 4 * H, H, round_up(H, 64), gb, w.qh[l].range,
                      w.qh[l].zero, w.qh[l].inv_q, w.qh[l].row_sums};
    q.bias = L.bias;
    layers[l] = q;
  }
  qm->nlayers = M.nlayers;
  qm->layers = layers;
  const int64_t HL = M.layers[M.nlayers - 1].hidden;
  qm->Wy = qout ? ql_qmatrix{w.qy.codes, M.states, HL, round_up(HL, 64), 1, w.qy.range,
                             w.qy.zero, w.qy.inv_q, w.qy.row_sums}
                : ql_qmatrix{nullptr, 0, HL, round_up(HL, 64), 1, nullptr, nullptr, nullptr, nullptr};
  qm->by = M.by;
}

TrainWs carve_train(Carve &c, const ql_train_model &M, int64_t T, int64_t B, int32_t gb,
                    bool qout) {
  TrainWs w{};
  const int64_t N = T * B;
  int64_t maxH = 0, maxIn = 0;
  train_width_max(M, &maxH, &maxIn);
  // exchange region: the forward pass's whole workspace, or the backward's
  // counters, whichever is larger
  ql_lstm_layer layers[kMaxTrainLayers];
  ql_model qm{};
  train_qmodel(M, w, gb, qout, layers, &qm);
  if (!qout) qm.Wy.rows = 0;
  w.xch_bytes = std::max(model_ws_bytes(&qm, T, B), bptt_ws(T, B));
  w.xch = c.take<char>(w.xch_bytes);
  auto qcopy = [&](TrainWs::QCopy &q, int64_t rows, int64_t cols, int nb) {
    q.codes = c.take<int8_t>((size_t)(rows * round_up(cols, 64)));
    q.range = c.take<double>((size_t)nb);
    q.zero = c.take<int32_t>((size_t)nb);
    q.inv_q = c.take<float>((size_t)nb);
    q.row_sums = c.take<int32_t>((size_t)rows);
  };
  for (int l = 0; l < M.nlayers; ++l) {
    const int64_t H = M.layers[l].hidden;
    qcopy(w.qx[l], 4 * H, M.layers[l].in, gb);
    qcopy(w.qh[l], 4 * H, H, gb);
  }
  const int64_t HL = M.layers[M.nlayers - 1].hidden;
  if (qout) qcopy(w.qy, M.states, HL, 1);
  w.qws = c.take<char>(set_quantize_ws(gb));
  for (int l = 0; l < M.nlayers; ++l) {
    const int64_t H = M.layers[l].hidden;
    w.gates[l] = c.take<float>((size_t)(N * 4 * H));
    w.c[l] = c.take<float>((size_t)(N * H));
    w.h[l] = c.take<float>((size_t)(N * H));
  }
  w.post = c.take<float>((size_t)(N * M.states));
  w.row_loss = c.take<float>((size_t)std::max<int64_t>(N, 1) + 1);
  w.dy = c.take<float>((size_t)(N * std::max(maxH, maxIn)));
  w.dx = c.take<float>((size_t)(N * std::max(maxH, maxIn)));
  w.da = c.take<float>((size_t)(N * 4 * maxH));
  w.part = c.take<float>(grad_part_floats(M, T, B));
  w.cpart = c.take<float>(colsum_ws(std::max<int64_t>(4 * maxH, M.states)) / sizeof(float));
  return w;
}

ql_status check_train_model(const ql_train_model *M, int32_t gb, bool need_ptrs) {
  if (!M || !M->layers || M->nlayers <= 0) return QL_EINVAL;
  if (M->nlayers > kMaxTrainLayers || M->states <= 0 || gb <= 0) return QL_ESHAPE;
  if (need_ptrs && (!M->Wy || !M->by)) return QL_EINVAL;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_train_layer &L = M->layers[l];
    if (L.proj != 0) return QL_EUNSUPPORTED;
    if (L.in <= 0 || L.hidden <= 0) return QL_ESHAPE;
    if (L.hidden > 512) return QL_EUNSUPPORTED;
    if (l > 0 && L.in != M->layers[l - 1].hidden) return QL_ESHAPE;
    if ((4 * L.hidden) % gb != 0) return QL_ESHAPE;
    if (L.in > kMaxK || gb > 65535) return QL_EOVERFLOW;
    if (need_ptrs && (!L.Wx || !L.Wh || !L.bias)) return QL_EINVAL;
  }
  return QL_OK;
}

}  // namespace

extern "C" {

size_t ql_train_step_workspace(const ql_train_model *M, int64_t T, int64_t B,
                               int32_t gate_blocks) {
  if (check_train_model(M, gate_blocks, false) != QL_OK || T < 0 || B < 0) return 0;
  Carve c(nullptr);
  carve_train(c, *M, T, B, gate_blocks, true);
  return c.off;
}

ql_status ql_train_step(const ql_train_model *M, const float *feats, const int32_t *targets,
                        int64_t T, int64_t B, float lr, int32_t gate_blocks,
                        int32_t quantize_output, float *loss, const ql_train_model *grads,
                        void *ws, size_t ws_bytes, void *stream) {
  ql_status st = check_train_model(M, gate_blocks, true);
  if (st != QL_OK) return st;
  if (T < 0 || B < 0) return QL_ESHAPE;
  if (quantize_output != 0 && quantize_output != 1) return QL_EINVAL;
  if (!std::isfinite(lr)) return QL_EINVAL;
  if (!grads || !grads->layers || grads->nlayers != M->nlayers || grads->states != M->states ||
      !grads->Wy || !grads->by)
    return QL_EINVAL;
  for (int l = 0; l < M->nlayers; ++l) {
    const ql_train_layer &g = grads->layers[l], &L = M->layers[l];
    if (!g.Wx || !g.Wh || !g.bias) return QL_EINVAL;
    if (g.in != L.in || g.hidden != L.hidden || g.proj != 0) return QL_ESHAPE;
  }
  if (T * B > 0 && (!feats || !targets)) return QL_EINVAL;
  if (!ws || ws_bytes < ql_train_step_workspace(M, T, B, gate_blocks)) return QL_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  const bool qout = quantize_output == 1;
  Carve c(ws);
  TrainWs w = carve_train(c, *M, T, B, gate_blocks, qout);
  if (reset_recurrent_flag(w.xch, s) != hipSuccess) return QL_EHIP;
  const int64_t N = T * B, S = M->states, NL = M->nlayers;
  const int64_t HL = M->layers[NL - 1].hidden;

  // 1. w^q <- quantize(w)
  for (int l = 0; l < NL; ++l) {
    const ql_train_layer &L = M->layers[l];
    const int64_t H = L.hidden;
    if (launch_set_quantize(L.Wx, L.in, 4 * H, L.in, gate_blocks, w.qx[l].codes,
                            round_up(L.in, 64), w.qx[l].range, w.qx[l].zero, w.qx[l].inv_q,
                            w.qx[l].row_sums, nullptr, nullptr, w.qws, s) != hipSuccess ||
        launch_set_quantize(L.Wh, H, 4 * H, H, gate_blocks, w.qh[l].codes, round_up(H, 64),
                            w.qh[l].range, w.qh[l].zero, w.qh[l].inv_q, w.qh[l].row_sums,
                            nullptr, nullptr, w.qws, s) != hipSuccess)
      return QL_EHIP;
  }
  if (qout && launch_set_quantize(M->Wy, HL, S, HL, 1, w.qy.codes, round_up(HL, 64), w.qy.range,
                                  w.qy.zero, w.qy.inv_q, w.qy.row_sums, nullptr, nullptr, w.qws,
                                  s) != hipSuccess)
    return QL_EHIP;

  // 2. the quantized forward pass (the inference path), its activations kept
  ql_lstm_layer layers[kMaxTrainLayers];
  ql_model qm{};
  train_qmodel(*M, w, gate_blocks, qout, layers, &qm);
  ql_lstm_taps lt[kMaxTrainLayers];
  for (int l = 0; l < NL; ++l) {
    lt[l] = ql_lstm_taps{};
    lt[l].gates = w.gates[l];
    lt[l].c = w.c[l];
    lt[l].h = w.h[l];
  }
  const ql_model_taps mt{lt, nullptr, nullptr};
  if (N > 0) {
    st = model_forward(&qm, Frontend{feats, false, 0, 0, 0}, T, B, w.post, nullptr, nullptr, &mt,
                       w.xch, w.xch_bytes, stream, qout);
    if (st != QL_OK) return st;
    if (!qout) {  // 'quant': float output layer on the quantized layers' h
      if (launch_sgemm(w.h[NL - 1], HL, M->Wy, HL, N, S, HL, M->by, w.post, S, s) != hipSuccess ||
          launch_softmax_rows(w.post, N, S, s) != hipSuccess)
        return QL_EHIP;
    }
  }

  // 3. loss and output error; gradients of the output layer; dC/dh of the top layer
  if (launch_xent_grad(w.post, targets, N, S, w.row_loss, loss, s) != hipSuccess) return QL_EHIP;
  auto gemm_grad = [&](const float *A, int64_t lda, const float *Bm, int64_t ldb, int64_t m,
                       int64_t n, int64_t k, float *C) {
    return launch_sgemm_ex(true, true, A, lda, Bm, ldb, m, n, k, nullptr, C, n,
                           grad_splits(m, n, k), w.part, s);
  };
  if (gemm_grad(w.post, S, w.h[NL - 1], HL, S, HL, N, grads->Wy) != hipSuccess ||
      launch_colsum(w.post, N, S, grads->by, w.cpart, s) != hipSuccess ||
      launch_sgemm_ex(false, true, w.post, S, M->Wy, HL, N, HL, S, nullptr, w.dy, HL, 1, nullptr,
                      s) != hipSuccess)
    return QL_EHIP;

  // 4. the layers from the top: BPTT, then the gradient products
  float *dy = w.dy, *dx = w.dx;
  for (int l = (int)NL - 1; l >= 0; --l) {
    const ql_train_layer &L = M->layers[l];
    const ql_train_layer &g = grads->layers[l];
    const int64_t H = L.hidden, IN = L.in;
    const float *xin = l == 0 ? feats : w.h[l - 1];
    BpttArgs ba{T, B, H, L.Wh, dy, w.gates[l], w.c[l], w.da, w.xch};
    bool unsupported = false;
    if (launch_bptt(ba, s, &unsupported) != hipSuccess) return QL_EHIP;
    if (unsupported) return QL_EUNSUPPORTED;
    if (gemm_grad(w.da, 4 * H, xin, IN, 4 * H, IN, N, g.Wx) != hipSuccess ||
        gemm_grad(w.da + B * 4 * H, 4 * H, w.h[l], H, 4 * H, H, N > B ? N - B : 0, g.Wh) !=
            hipSuccess ||
        launch_colsum(w.da, N, 4 * H, g.bias, w.cpart, s) != hipSuccess)
      return QL_EHIP;
    if (l > 0) {
      if (launch_sgemm_ex(false, true, w.da, 4 * H, L.Wx, IN, N, IN, 4 * H, nullptr, dx, IN, 1,
                          nullptr, s) != hipSuccess)
        return QL_EHIP;
      std::swap(dy, dx);
    }
  }

  // 5. w <- w - lr dC/dw
  for (int l = 0; l < NL; ++l) {
    const ql_train_layer &L = M->layers[l], &g = grads->layers[l];
    const int64_t H = L.hidden;
    if (launch_sgd(L.Wx, g.Wx, 4 * H * L.in, lr, s) != hipSuccess ||
        launch_sgd(L.Wh, g.Wh, 4 * H * H, lr, s) != hipSuccess ||
        launch_sgd(L.bias, g.bias, 4 * H, lr, s) != hipSuccess)
      return QL_EHIP;
  }
  if (launch_sgd(M->Wy, grads->Wy, S * HL, lr, s) != hipSuccess ||
      launch_sgd(M->by, grads->by, S, lr, s) != hipSuccess)
    return QL_EHIP;
  return QL_OK;
}

}  // extern "C"
