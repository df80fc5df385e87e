// Drives the host side of the C ABI (include/qlstm.h) -- argument checks,
// workspace queries and workspace carving -- through every entry point, with
// invalid arguments and with descriptors of the evaluated models, so that a
// build of the library's host code with AddressSanitizer and
// UndefinedBehaviorSanitizer sees each of those paths.  Needs no GPU: no call
// here gets past its checks to a launch (device pointers are placeholders the
// checks must never dereference).  Exit status 0 when every call returned
// what its declaration promises.  Test infrastructure: built and run by the
// test suite.
#include <cmath>
#include <cstdio>
#include <vector>

#include "qlstm.h"

namespace {

int g_fail = 0;
#define EXPECT(call, want)                                                               \
  do {                                                                                   \
    const long long got_ = (long long)(call);                                            \
    if (got_ != (long long)(want)) {                                                     \
      std::fprintf(stderr, "%s:%d: %s = %lld, want %lld\n", __FILE__, __LINE__, #call,   \
                   got_, (long long)(want));                                             \
      g_fail = 1;                                                                        \
    }                                                                                    \
  } while (0)
#define EXPECT_POS(call)                                                                 \
  do {                                                                                   \
    if (!((call) > 0)) {                                                                 \
      std::fprintf(stderr, "%s:%d: %s not > 0\n", __FILE__, __LINE__, #call);            \
      g_fail = 1;                                                                        \
    }                                                                                    \
  } while (0)

// placeholder device addresses: never dereferenced on the host
template <class T>
T *fake() {
  return reinterpret_cast<T *>(static_cast<uintptr_t>(0x7f0000001000ull));
}

ql_qmatrix qm(int64_t rows, int64_t cols, int32_t nblocks, bool null_codes = false) {
  ql_qmatrix q{};
  q.codes = null_codes ? nullptr : fake<int8_t>();
  q.rows = rows, q.cols = cols, q.ld = (cols + 63) / 64 * 64, q.nblocks = nblocks;
  q.range = fake<double>(), q.zero = fake<int32_t>(), q.inv_q = fake<float>();
  q.row_sums = fake<int32_t>();
  return q;
}

ql_lstm_layer layer(int64_t in, int64_t H, int64_t P = 0) {
  ql_lstm_layer L{};
  const int64_t R = P ? P : H;
  L.in = in, L.hidden = H, L.proj = P;
  L.Wx = qm(4 * H, in, 4), L.Wh = qm(4 * H, R, 4);
  if (P) L.Wr = qm(P, H, 1);
  L.bias = fake<float>();
  return L;
}

ql_qact qact(int64_t rows, int64_t cols) {
  ql_qact a{};
  a.codes = fake<int8_t>(), a.rows = rows, a.cols = cols, a.ld = (cols + 63) / 64 * 64;
  a.zero = fake<int32_t>(), a.inv_q = fake<float>(), a.sums = fake<int32_t>();
  return a;
}

void wait_bound_hook() {
  EXPECT(ql_debug_set_wait_bound(-1), QL_EINVAL);
  EXPECT(ql_debug_set_wait_bound(5), QL_OK);
  EXPECT(ql_debug_set_wait_bound(0), QL_OK);
}

void status_strings() {
  for (int s = -8; s <= 0; ++s) EXPECT(ql_status_str(static_cast<ql_status>(s)) != nullptr, 1);
  EXPECT(ql_status_str(static_cast<ql_status>(-100)) != nullptr, 1);
}

void quantize_and_products() {
  ql_qmatrix dst = qm(32, 16, 4);
  EXPECT_POS(ql_quantize_workspace(32, 16, 4));
  EXPECT(ql_quantize(nullptr, 32, 16, 4, &dst, fake<void>(), 1 << 20, nullptr), QL_EINVAL);
  EXPECT(ql_dequantize(nullptr, fake<float>(), nullptr), QL_EINVAL);
  const size_t ws = ql_quantized_matmul_workspace(4, 8, 16);
  EXPECT_POS(ws);
  ql_qmatrix W = qm(8, 16, 4);
  auto mm = [&](const ql_qmatrix &q, const float *X, int64_t m, int gran, size_t wsb) {
    return ql_quantized_matmul(&q, X, m, static_cast<ql_act_gran>(gran), nullptr, fake<float>(),
                               nullptr, fake<void>(), wsb, nullptr);
  };
  EXPECT(mm(qm(8, 16, 4, true), fake<float>(), 4, 1, ws), QL_EINVAL);
  EXPECT(mm(W, nullptr, 4, 1, ws), QL_EINVAL);
  EXPECT(mm(W, fake<float>(), 4, 7, ws), QL_EINVAL);
  EXPECT(mm(qm(9, 16, 4), fake<float>(), 4, 1, ws), QL_ESHAPE);
  ql_qmatrix narrow = W;
  narrow.ld = 8;
  EXPECT(mm(narrow, fake<float>(), 4, 1, ws), QL_ESHAPE);
  EXPECT(mm(qm(8, 33026, 4), fake<float>(), 4, 1, ws), QL_EOVERFLOW);
  EXPECT(mm(W, fake<float>(), 4, 1, ws - 1), QL_EWORKSPACE);
  EXPECT(mm(W, fake<float>(), -1, 1, ws), QL_ESHAPE);
  EXPECT_POS(ql_gemm_u8_workspace(64, 64, 64));
  auto g = [&](int64_t lda, int64_t K) {
    return ql_gemm_u8(fake<int8_t>(), lda, fake<int8_t>(), lda, fake<int32_t>(), 4, 4, K,
                      nullptr, nullptr, nullptr, 0, nullptr);
  };
  EXPECT(g(32, 64), QL_ESHAPE);
  EXPECT(g(96, 64), QL_ESHAPE);
  EXPECT(g(33088, 33026), QL_EOVERFLOW);
  EXPECT(g(64, 64), QL_EWORKSPACE);
  EXPECT(ql_gate_fn(9, fake<float>(), fake<float>(), 4, nullptr), QL_EINVAL);
  EXPECT(ql_gate_fn(0, nullptr, fake<float>(), 4, nullptr), QL_EINVAL);
  EXPECT(ql_gate_fn(0, fake<float>(), fake<float>(), -1, nullptr), QL_ESHAPE);
  ql_qact a = qact(4, 16);
  EXPECT(ql_quantize_activations(fake<float>(), 5, 16, &a, nullptr), QL_ESHAPE);
  EXPECT(ql_quantize_activations(nullptr, 4, 16, &a, nullptr), QL_EINVAL);
}

void layers_and_models() {
  // the evaluated shapes: 5 x 500 on 320 inputs, 4 x LSTMP 2048/512 on 640, Table 1 P = 200
  const ql_lstm_layer l500 = layer(320, 500), l500b = layer(500, 500);
  const ql_lstm_layer lp0 = layer(640, 2048, 512), lp1 = layer(512, 2048, 512);
  const ql_lstm_layer t0 = layer(320, 500, 200), t1 = layer(200, 500, 200);
  EXPECT_POS(ql_lstm_layer_workspace(&l500, 300, 1));
  EXPECT_POS(ql_lstm_layer_workspace(&lp0, 800, 256));
  EXPECT_POS(ql_lstm_recurrence_workspace(&lp1, 800, 256));
  EXPECT(ql_lstm_layer_forward(&l500, nullptr, 5, 2, nullptr, nullptr, fake<float>(), nullptr,
                               nullptr, nullptr, fake<void>(), 1 << 30, nullptr),
         QL_EINVAL);
  ql_lstm_layer bad = l500;
  bad.Wx = qm(2000, 321, 4);
  EXPECT(ql_lstm_layer_forward(&bad, fake<float>(), 5, 2, nullptr, nullptr, fake<float>(),
                               nullptr, nullptr, nullptr, fake<void>(), 1 << 30, nullptr),
         QL_ESHAPE);
  bad = layer(16, 8, 3);
  bad.bias = nullptr;
  EXPECT(ql_lstm_layer_forward(&bad, fake<float>(), 5, 2, nullptr, nullptr, fake<float>(),
                               nullptr, nullptr, nullptr, fake<void>(), 1 << 30, nullptr),
         QL_EINVAL);

  std::vector<ql_lstm_layer> five{l500, l500b, l500b, l500b, l500b};
  std::vector<ql_lstm_layer> four{lp0, lp1, lp1, lp1};
  std::vector<ql_lstm_layer> proj{t0, t1, t1, t1, t1};
  ql_model m5{5, five.data(), qm(8192, 500, 1), fake<float>()};
  ql_model mp{4, four.data(), qm(16384, 512, 1), fake<float>()};
  ql_model mt{5, proj.data(), qm(8192, 200, 1), fake<float>()};
  for (const ql_model *m : {&m5, &mp, &mt})
    for (int64_t B : {1, 16, 64, 256}) EXPECT_POS(ql_acoustic_model_workspace(m, 100, B));
  EXPECT_POS(ql_acoustic_model_frames_workspace(&m5, 308, 64, 8, 3));
  EXPECT_POS(ql_lstm_stack_workspace(five.data(), 5, 1000, 64));
  EXPECT_POS(ql_lstm_stack_workspace(proj.data(), 5, 500, 1));
  std::vector<ql_lstm_layer> broken{l500, layer(501, 500)};
  ql_model mb{2, broken.data(), qm(8192, 500, 1), fake<float>()};
  EXPECT(ql_acoustic_model_forward(&mb, fake<float>(), 3, 2, fake<float>(), nullptr, fake<void>(),
                                   size_t(1) << 40, nullptr),
         QL_ESHAPE);
  ql_model my{5, five.data(), qm(8192, 501, 1), fake<float>()};
  EXPECT(ql_acoustic_model_forward(&my, fake<float>(), 3, 2, fake<float>(), nullptr, fake<void>(),
                                   size_t(1) << 40, nullptr),
         QL_ESHAPE);
  const size_t need = ql_acoustic_model_workspace(&m5, 3, 2);
  EXPECT(ql_acoustic_model_forward(&m5, fake<float>(), 3, 2, fake<float>(), nullptr, fake<void>(),
                                   need - 1, nullptr),
         QL_EWORKSPACE);
  std::vector<ql_lstm_state> st(5, ql_lstm_state{fake<float>(), fake<float>()});
  EXPECT(ql_acoustic_model_forward_stream(&m5, fake<float>(), 3, 2, st.data(), st.data(),
                                          fake<float>(), nullptr, fake<void>(), need, nullptr),
         QL_EINVAL);  // state in and out overlap
  EXPECT(ql_acoustic_model_forward_stream_noalloc(nullptr, fake<float>(), 3, 2, nullptr, nullptr,
                                                  fake<float>(), nullptr, nullptr),
         QL_EINVAL);
  EXPECT(ql_acoustic_model_forward_stream_noalloc(&m5, fake<float>(), -3, 2, nullptr, nullptr,
                                                  fake<float>(), nullptr, nullptr),
         QL_ESHAPE);
  EXPECT(ql_acoustic_model_forward_stream_noalloc(&m5, fake<float>(), 100000, 64, nullptr,
                                                  nullptr, fake<float>(), nullptr, nullptr),
         QL_ESCRATCH);

  const int64_t T = 5, B = 2;
  std::vector<ql_lstm_layer> two{layer(16, 8), layer(8, 8)};
  ql_qact x = qact(T * B, 16);
  std::vector<ql_qact> outs{qact(T * B, 8), qact(T * B, 8)};
  const size_t sneed = ql_lstm_stack_workspace(two.data(), 2, T, B);
  EXPECT_POS(sneed);
  EXPECT(ql_lstm_stack_forward(two.data(), 2, &x, T, B, outs.data(), nullptr, nullptr, nullptr,
                               nullptr, fake<void>(), sneed - 1, nullptr),
         QL_EWORKSPACE);
  ql_qact x_bad = qact(T * B + 1, 16);
  EXPECT(ql_lstm_stack_forward(two.data(), 2, &x_bad, T, B, outs.data(), nullptr, nullptr,
                               nullptr, nullptr, fake<void>(), sneed, nullptr),
         QL_ESHAPE);
  EXPECT(ql_lstm_stack_forward(two.data(), 2, nullptr, T, B, outs.data(), nullptr, nullptr,
                               nullptr, nullptr, fake<void>(), sneed, nullptr),
         QL_EINVAL);

  EXPECT(ql_stacked_input_count(308, 8, 3), 101);
  EXPECT(ql_stacked_input_count(7, 8, 3), 0);
  ql_qact q = qact(5 * 2, 320);
  EXPECT(ql_quantize_stacked_frames(fake<float>(), 20, 2, 41, 8, 3, &q, nullptr), QL_ESHAPE);
  EXPECT(ql_quantize_stacked_frames(fake<float>(), 23, 2, 40, 8, 3, &q, nullptr), QL_ESHAPE);
}

void fp32_model() {
  ql_f32_layer good{16, 8, 0, fake<float>(), fake<float>(), nullptr, fake<float>()};
  const size_t n = ql_f32_lstm_layer_workspace(&good, 5, 2);
  EXPECT_POS(n);
  EXPECT(ql_f32_lstm_layer_forward(&good, nullptr, 5, 2, nullptr, nullptr, fake<float>(), nullptr,
                                   nullptr, fake<void>(), n, nullptr),
         QL_EINVAL);
  EXPECT(ql_f32_lstm_layer_forward(&good, fake<float>(), -1, 2, nullptr, nullptr, fake<float>(),
                                   nullptr, nullptr, fake<void>(), n, nullptr),
         QL_ESHAPE);
  std::vector<ql_f32_layer> two{good, ql_f32_layer{9, 8, 0, fake<float>(), fake<float>(), nullptr,
                                                   fake<float>()}};
  ql_f32_model m{2, two.data(), 10, fake<float>(), fake<float>()};
  EXPECT(ql_f32_acoustic_model_forward(&m, fake<float>(), 3, 2, fake<float>(), fake<void>(),
                                       size_t(1) << 40, nullptr),
         QL_ESHAPE);
  ql_f32_model m1{1, two.data(), 10, fake<float>(), fake<float>()};
  EXPECT_POS(ql_f32_acoustic_model_workspace(&m1, 1000, 64));
  EXPECT(ql_f32_matmul(nullptr, 4, 4, fake<float>(), 2, nullptr, fake<float>(), nullptr),
         QL_EINVAL);
}

ql_train_layer tlayer(int64_t in, int64_t H, int64_t P = 0) {
  return ql_train_layer{in, H, P, fake<float>(), fake<float>(), nullptr, fake<float>()};
}

void training() {
  std::vector<ql_train_layer> five{tlayer(320, 500), tlayer(500, 500), tlayer(500, 500),
                                   tlayer(500, 500), tlayer(500, 500)};
  ql_train_model M{5, five.data(), 8192, fake<float>(), fake<float>()};
  std::vector<ql_train_layer> gl = five;
  ql_train_model G{5, gl.data(), 8192, fake<float>(), fake<float>()};
  const size_t need = ql_train_step_workspace(&M, 1000, 64, 4);
  EXPECT_POS(need);
  EXPECT_POS(ql_train_step_workspace(&M, 12, 1, 2000));  // per-row weight blocks
  EXPECT(ql_train_step_workspace(&M, 12, 1, 3), 0);      // 4H not a multiple of 3
  auto step = [&](const ql_train_model *m, const ql_train_model *g, int64_t T, float lr,
                  int32_t qout, size_t wsb) {
    return ql_train_step(m, fake<float>(), fake<int32_t>(), T, 64, lr, 4, qout, fake<float>(), g,
                         fake<void>(), wsb, nullptr);
  };
  EXPECT(step(nullptr, &G, 1000, 0.1f, 1, need), QL_EINVAL);
  EXPECT(step(&M, nullptr, 1000, 0.1f, 1, need), QL_EINVAL);
  EXPECT(step(&M, &G, 1000, 0.1f, 2, need), QL_EINVAL);
  EXPECT(step(&M, &G, 1000, NAN, 1, need), QL_EINVAL);
  EXPECT(step(&M, &G, 1000, INFINITY, 1, need), QL_EINVAL);
  EXPECT(step(&M, &G, -1, 0.1f, 1, need), QL_ESHAPE);
  EXPECT(step(&M, &G, 1000, 0.1f, 1, need - 1), QL_EWORKSPACE);
  EXPECT(ql_train_step(&M, nullptr, fake<int32_t>(), 1000, 64, 0.1f, 4, 1, nullptr, &G,
                       fake<void>(), need, nullptr),
         QL_EINVAL);
  std::vector<ql_train_layer> g_small = five;
  g_small[2] = tlayer(500, 400);
  ql_train_model G2{5, g_small.data(), 8192, fake<float>(), fake<float>()};
  EXPECT(step(&M, &G2, 1000, 0.1f, 1, need), QL_ESHAPE);
  ql_train_model G3{5, gl.data(), 8191, fake<float>(), fake<float>()};
  EXPECT(step(&M, &G3, 1000, 0.1f, 1, need), QL_EINVAL);
  std::vector<ql_train_layer> proj{tlayer(320, 500, 200)};
  ql_train_model MP{1, proj.data(), 8192, fake<float>(), fake<float>()};
  EXPECT(ql_train_step_workspace(&MP, 10, 2, 4), 0);
  EXPECT(step(&MP, &G, 10, 0.1f, 1, need), QL_EUNSUPPORTED);
  std::vector<ql_train_layer> wide{tlayer(320, 513)};
  ql_train_model MW{1, wide.data(), 8192, fake<float>(), fake<float>()};
  EXPECT(step(&MW, &G, 10, 0.1f, 1, need), QL_EUNSUPPORTED);
  std::vector<ql_train_layer> chain{tlayer(320, 500), tlayer(499, 500)};
  ql_train_model MC{2, chain.data(), 8192, fake<float>(), fake<float>()};
  EXPECT(step(&MC, &G, 10, 0.1f, 1, need), QL_ESHAPE);
}

}  // namespace

int main() {
  status_strings();
  wait_bound_hook();
  quantize_and_products();
  layers_and_models();
  fp32_model();
  training();
  if (g_fail) return 1;
  std::printf("ABI sanitizer run: ok\n");
  return 0;
}
