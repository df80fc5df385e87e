"""C ABI checks that need no GPU: the library loads, exports every function
include/qlstm.h declares, and rejects bad arguments before enqueuing work.

Every call below fails validation before the library touches memory or the
HIP runtime (the pointers passed are never dereferenced)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlstm.h")


@pytest.fixture(scope="module")
def ql():
    from paper_1607_04683_amd import qlstm
    if not os.path.exists(qlstm.LIB_PATH):
        from paper_1607_04683_amd import build
        build.build(force=False)
    return qlstm


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ql_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_four_paper_calls():
    names = declared_functions()
    for f in ("ql_quantize", "ql_quantized_matmul", "ql_lstm_layer_forward",
              "ql_acoustic_model_forward"):
        assert f in names


def test_library_exports_every_declared_symbol(ql):
    lib = C.CDLL(ql.LIB_PATH)
    missing = [f for f in declared_functions() if not hasattr(lib, f)]
    assert not missing, missing
    assert sorted(ql.EXPORTS) == declared_functions()


def test_status_strings(ql):
    for s in range(0, -8, -1):
        assert ql.status_str(s) and ql.status_str(s) != "unknown status"


FAKE = 0x1000  # never dereferenced: each call below fails validation first


def qm(rows=8, cols=16, ld=64, nblocks=1, null=False):
    return ql_mod().CQMatrix(None if null else FAKE, rows, cols, ld, nblocks, FAKE, FAKE, FAKE, FAKE)


def ql_mod():
    from paper_1607_04683_amd import qlstm
    return qlstm


def test_quantized_matmul_argument_errors(ql):
    lib = ql.load()
    ws = lib.ql_quantized_matmul_workspace(4, 8, 16)
    call = lambda q, X=FAKE, m=4, gran=1, Y=FAKE, wsb=ws: lib.ql_quantized_matmul(
        C.byref(q), X, m, gran, None, Y, None, FAKE, wsb, None)
    assert call(qm(null=True)) == ql.QL_EINVAL
    assert call(qm(), X=None) == ql.QL_EINVAL
    assert call(qm(), gran=7) == ql.QL_EINVAL
    assert call(qm(rows=9, nblocks=4)) == ql.QL_ESHAPE          # rows % nblocks
    assert call(qm(ld=8)) == ql.QL_ESHAPE                        # ld < cols
    assert call(qm(cols=33026, ld=33088)) == ql.QL_EOVERFLOW     # int32 accumulator guard
    assert call(qm(), wsb=ws - 1) == ql.QL_EWORKSPACE
    assert call(qm(), m=-1) == ql.QL_ESHAPE


def test_gemm_argument_errors(ql):
    lib = ql.load()
    g = lambda lda=64, ldb=64, K=64, M=4, N=4, ws=None, wsb=0: lib.ql_gemm_u8(
        FAKE, lda, FAKE, ldb, FAKE, M, N, K, None, None, ws, wsb, None)
    assert g(lda=32) == ql.QL_ESHAPE
    assert g(lda=96) == ql.QL_ESHAPE       # not a multiple of 64
    assert g(K=33026, lda=33088, ldb=33088) == ql.QL_EOVERFLOW
    assert g() == ql.QL_EWORKSPACE         # sums not given and no workspace
    assert lib.ql_gemm_u8(None, 64, FAKE, 64, FAKE, 4, 4, 64, None, None, None, 0, None) == ql.QL_EINVAL


def test_layer_argument_errors(ql):
    lib = ql.load()
    H, IN = 8, 16
    good = ql.CLayer(IN, H, 0, qm(4 * H, IN, 64, 4), qm(4 * H, H, 64, 4),
                     ql.CQMatrix(None, 0, 0, 0, 1, None, None, None, None), FAKE)
    nbytes = lib.ql_lstm_layer_workspace(C.byref(good), 5, 2)
    assert nbytes > 0
    f = lambda L, wsb=nbytes, x=FAKE: lib.ql_lstm_layer_forward(
        C.byref(L), x, 5, 2, None, None, FAKE, None, None, None, FAKE, wsb, None)
    assert f(good, x=None) == ql.QL_EINVAL
    assert f(good, wsb=nbytes - 1) == ql.QL_EWORKSPACE
    bad = ql.CLayer(IN, H, 0, qm(4 * H, IN + 1, 64, 4), qm(4 * H, H, 64, 4), good.Wr, FAKE)
    assert f(bad) == ql.QL_ESHAPE
    bad = ql.CLayer(IN, H, 0, qm(4 * H, IN, 64, 4), qm(4 * H, H + 1, 64, 4), good.Wr, FAKE)
    assert f(bad) == ql.QL_ESHAPE
    bad = ql.CLayer(IN, H, 3, qm(4 * H, IN, 64, 4), qm(4 * H, 3, 64, 4), qm(3, H, 64, 1), None)
    assert f(bad) == ql.QL_EINVAL          # null bias
    bad = ql.CLayer(IN, H, 3, qm(4 * H, IN, 64, 4), qm(4 * H, 3, 64, 4), qm(3, H, 64, 2), FAKE)
    assert f(bad) == ql.QL_ESHAPE          # W_r rows % nblocks


def test_model_argument_errors(ql):
    lib = ql.load()
    H, IN, S = 8, 16, 10
    empty = ql.CQMatrix(None, 0, 0, 0, 1, None, None, None, None)
    l0 = ql.CLayer(IN, H, 0, qm(4 * H, IN, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    l1 = ql.CLayer(H + 1, H, 0, qm(4 * H, H + 1, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    arr = (ql.CLayer * 2)(l0, l1)
    m = ql.CModel(2, arr, qm(S, H, 64, 1), FAKE)
    assert lib.ql_acoustic_model_forward(C.byref(m), FAKE, 3, 2, FAKE, None, FAKE, 1 << 40,
                                         None) == ql.QL_ESHAPE   # layer widths do not chain
    arr2 = (ql.CLayer * 1)(l0)
    m2 = ql.CModel(1, arr2, qm(S, H + 2, 64, 1), FAKE)
    assert lib.ql_acoustic_model_forward(C.byref(m2), FAKE, 3, 2, FAKE, None, FAKE, 1 << 40,
                                         None) == ql.QL_ESHAPE   # W_y width
    m3 = ql.CModel(1, arr2, qm(S, H, 64, 1), FAKE)
    need = lib.ql_acoustic_model_workspace(C.byref(m3), 3, 2)
    assert need > 0
    assert lib.ql_acoustic_model_forward(C.byref(m3), FAKE, 3, 2, FAKE, None, FAKE, need - 1,
                                         None) == ql.QL_EWORKSPACE


def test_f32_argument_errors(ql):
    lib = ql.load()
    H, IN, S = 8, 16, 10
    good = ql.CF32Layer(IN, H, 0, FAKE, FAKE, None, FAKE)
    nbytes = lib.ql_f32_lstm_layer_workspace(C.byref(good), 5, 2)
    assert nbytes > 0
    f = lambda L, wsb=nbytes, x=FAKE, T=5: lib.ql_f32_lstm_layer_forward(
        C.byref(L), x, T, 2, None, None, FAKE, None, None, FAKE, wsb, None)
    assert f(good, x=None) == ql.QL_EINVAL
    assert f(good, wsb=nbytes - 1) == ql.QL_EWORKSPACE
    assert f(good, T=-1) == ql.QL_ESHAPE
    assert f(ql.CF32Layer(IN, H, 0, None, FAKE, None, FAKE)) == ql.QL_EINVAL   # no W_x
    assert f(ql.CF32Layer(IN, H, 3, FAKE, FAKE, None, FAKE)) == ql.QL_EINVAL   # no W_r
    assert f(ql.CF32Layer(IN, 0, 0, FAKE, FAKE, None, FAKE)) == ql.QL_ESHAPE
    l1 = ql.CF32Layer(H + 1, H, 0, FAKE, FAKE, None, FAKE)
    arr = (ql.CF32Layer * 2)(good, l1)
    m = ql.CF32Model(2, arr, S, FAKE, FAKE)
    assert lib.ql_f32_acoustic_model_forward(C.byref(m), FAKE, 3, 2, FAKE, FAKE, 1 << 40,
                                             None) == ql.QL_ESHAPE   # widths do not chain
    arr1 = (ql.CF32Layer * 1)(good)
    m1 = ql.CF32Model(1, arr1, S, FAKE, FAKE)
    need = lib.ql_f32_acoustic_model_workspace(C.byref(m1), 3, 2)
    assert need > 0
    assert lib.ql_f32_acoustic_model_forward(C.byref(m1), FAKE, 3, 2, FAKE, FAKE, need - 1,
                                             None) == ql.QL_EWORKSPACE
    assert lib.ql_f32_matmul(None, 4, 4, FAKE, 2, None, FAKE, None) == ql.QL_EINVAL
    assert lib.ql_f32_matmul(FAKE, -4, 4, FAKE, 2, None, FAKE, None) == ql.QL_ESHAPE


def test_activation_and_stack_argument_errors(ql):
    lib = ql.load()
    q = ql.CQAct(FAKE, 4, 16, 64, FAKE, FAKE, FAKE)
    assert lib.ql_quantize_activations(FAKE, 5, 16, C.byref(q), None) == ql.QL_ESHAPE   # rows
    q_bad_ld = ql.CQAct(FAKE, 4, 16, 32, FAKE, FAKE, FAKE)
    assert lib.ql_quantize_activations(FAKE, 4, 16, C.byref(q_bad_ld), None) == ql.QL_ESHAPE
    assert lib.ql_quantize_activations(None, 4, 16, C.byref(q), None) == ql.QL_EINVAL
    H, IN, T, B = 8, 16, 5, 2
    empty = ql.CQMatrix(None, 0, 0, 0, 1, None, None, None, None)
    L0 = ql.CLayer(IN, H, 0, qm(4 * H, IN, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    L1 = ql.CLayer(H, H, 0, qm(4 * H, H, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    arr = (ql.CLayer * 2)(L0, L1)
    x = ql.CQAct(FAKE, T * B, IN, 64, FAKE, FAKE, FAKE)
    outs = (ql.CQAct * 2)(ql.CQAct(FAKE, T * B, H, 64, FAKE, FAKE, FAKE),
                          ql.CQAct(FAKE, T * B, H, 64, FAKE, FAKE, FAKE))
    need = lib.ql_lstm_stack_workspace(arr, 2, T, B)
    assert need > 0
    f = lambda layers=arr, xx=x, wsb=need: lib.ql_lstm_stack_forward(
        layers, 2, C.byref(xx), T, B, outs, None, None, None, None, FAKE, wsb, None)
    assert f(wsb=need - 1) == ql.QL_EWORKSPACE
    assert f(xx=ql.CQAct(FAKE, T * B + 1, IN, 64, FAKE, FAKE, FAKE)) == ql.QL_ESHAPE
    bad = (ql.CLayer * 2)(L0, ql.CLayer(H, H + 1, 0, qm(4 * H + 4, H, 64, 4),
                                        qm(4 * H + 4, H + 1, 64, 4), empty, FAKE))
    assert f(layers=bad) == ql.QL_ESHAPE   # widths differ
    assert lib.ql_lstm_stack_forward(arr, 2, None, T, B, outs, None, None, None, None, FAKE, need,
                                     None) == ql.QL_EINVAL


def test_frontend_argument_errors(ql):
    """Stacked-frame entry points: presented-step count and argument checks."""
    lib = ql.load()
    cnt = lib.ql_stacked_input_count
    assert [cnt(n, 8, 3) for n in (0, 7, 8, 10, 11, 14, 308)] == [0, 0, 1, 1, 2, 3, 101]
    assert cnt(5, 0, 3) == 0 and cnt(5, 1, 0) == 0 and cnt(-1, 8, 3) == 0
    T = cnt(20, 8, 3)  # 5 presented steps
    q = ql.CQAct(FAKE, T * 2, 320, 320, FAKE, FAKE, FAKE)
    f = lambda frames=FAKE, n=20, B=2, dim=40, st=8, sk=3, qq=q: lib.ql_quantize_stacked_frames(
        frames, n, B, dim, st, sk, C.byref(qq), None)
    assert f(dim=41) == ql.QL_ESHAPE                                   # stack*dim != cols
    assert f(n=23) == ql.QL_ESHAPE                                     # 6 steps, 5 rows given
    assert f(sk=0) == ql.QL_ESHAPE and f(st=0) == ql.QL_ESHAPE
    assert f(qq=ql.CQAct(FAKE, T * 2, 320, 300, FAKE, FAKE, FAKE)) == ql.QL_ESHAPE  # ld
    assert f(frames=None) == ql.QL_EINVAL
    assert lib.ql_quantize_stacked_frames(FAKE, 20, 2, 40, 8, 3, None, None) == ql.QL_EINVAL
    assert f(n=7, qq=ql.CQAct(FAKE, 0, 320, 320, FAKE, FAKE, FAKE)) == ql.QL_OK  # nothing to do
    H, IN = 8, 320
    empty = ql.CQMatrix(None, 0, 0, 0, 1, None, None, None, None)
    L0 = ql.CLayer(IN, H, 0, qm(4 * H, IN, 320, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    arr = (ql.CLayer * 1)(L0)
    m = ql.CModel(1, arr, qm(16, H, 64, 1), FAKE)
    need = lib.ql_acoustic_model_frames_workspace(C.byref(m), 20, 2, 8, 3)
    assert need == lib.ql_acoustic_model_workspace(C.byref(m), T, 2) > 0
    g = lambda dim=40, wsb=need: lib.ql_acoustic_model_forward_frames(
        C.byref(m), FAKE, 20, 2, dim, 8, 3, FAKE, None, FAKE, wsb, None)
    assert g(dim=20) == ql.QL_ESHAPE                                   # 8*20 != layers[0].in
    assert g(wsb=need - 1) == ql.QL_EWORKSPACE


def test_train_step_argument_errors(ql):
    """ql_train_step (Section 3.2, Algorithm 1): every documented error."""
    lib = ql.load()
    TL, TM = ql.CTrainLayer, ql.CTrainModel

    def model(*layers, states=10):
        arr = (TL * len(layers))(*layers)
        return TM(len(layers), arr, states, FAKE, FAKE), arr

    M, _keep = model(TL(16, 8, 0, FAKE, FAKE, None, FAKE), TL(8, 8, 0, FAKE, FAKE, None, FAKE))
    G, _keepg = model(TL(16, 8, 0, FAKE, FAKE, None, FAKE), TL(8, 8, 0, FAKE, FAKE, None, FAKE))
    need = lib.ql_train_step_workspace(C.byref(M), 5, 2, 4)
    assert need > 0
    assert lib.ql_train_step_workspace(C.byref(M), 5, 2, 3) == 0        # 4H % 3

    def step(m=M, g=G, T=5, lr=0.1, qout=1, wsb=need, feats=FAKE, gb=4):
        return lib.ql_train_step(C.byref(m) if m is not None else None, feats, FAKE, T, 2, lr, gb,
                                 qout, None, C.byref(g) if g is not None else None, FAKE, wsb,
                                 None)

    assert step(m=None) == ql.QL_EINVAL
    assert step(g=None) == ql.QL_EINVAL
    assert step(qout=2) == ql.QL_EINVAL
    assert step(lr=float("nan")) == ql.QL_EINVAL
    assert step(lr=float("inf")) == ql.QL_EINVAL
    assert step(feats=None) == ql.QL_EINVAL
    assert step(T=-1) == ql.QL_ESHAPE
    assert step(gb=3) == ql.QL_ESHAPE
    assert step(wsb=need - 1) == ql.QL_EWORKSPACE
    G2, _k2 = model(TL(16, 8, 0, FAKE, FAKE, None, FAKE), TL(8, 7, 0, FAKE, FAKE, None, FAKE))
    assert step(g=G2) == ql.QL_ESHAPE                                   # gradient shapes
    G3, _k3 = model(TL(16, 8, 0, FAKE, FAKE, None, FAKE), TL(8, 8, 0, FAKE, FAKE, None, FAKE),
                    states=11)
    assert step(g=G3) == ql.QL_EINVAL                                   # states differ
    MP, _kp = model(TL(16, 8, 4, FAKE, FAKE, FAKE, FAKE))
    assert lib.ql_train_step_workspace(C.byref(MP), 5, 2, 4) == 0
    assert step(m=MP) == ql.QL_EUNSUPPORTED                             # projection
    MW, _kw = model(TL(16, 513, 0, FAKE, FAKE, None, FAKE))
    assert step(m=MW) == ql.QL_EUNSUPPORTED                             # H > 512
    MC, _kc = model(TL(16, 8, 0, FAKE, FAKE, None, FAKE), TL(9, 8, 0, FAKE, FAKE, None, FAKE))
    assert step(m=MC) == ql.QL_ESHAPE                                   # widths do not chain


def test_stream_state_in_and_out_must_not_overlap(ql):
    """The stream entry points reject initial and final states that share
    memory (the kernels read the one while writing the other)."""
    lib = ql.load()
    H, IN, S, T, B = 8, 16, 10, 3, 2
    empty = ql.CQMatrix(None, 0, 0, 0, 1, None, None, None, None)
    L0 = ql.CLayer(IN, H, 0, qm(4 * H, IN, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    L1 = ql.CLayer(H, H, 0, qm(4 * H, H, 64, 4), qm(4 * H, H, 64, 4), empty, FAKE)
    arr = (ql.CLayer * 2)(L0, L1)
    m = ql.CModel(2, arr, qm(S, H, 64, 1), FAKE)
    need = lib.ql_acoustic_model_workspace(C.byref(m), T, B)
    base = 0x100000
    s_in = (ql.CState * 2)(ql.CState(base, base + 0x1000), ql.CState(base + 0x2000, base + 0x3000))

    def call(s_out):
        return lib.ql_acoustic_model_forward_stream(C.byref(m), FAKE, T, B, s_in, s_out, FAKE,
                                                    None, FAKE, need, None)

    # layer 1's c out starts inside layer 0's h in (B * H floats = 64 bytes from base)
    overl = (ql.CState * 2)(ql.CState(base + 0x5000, base + 0x6000),
                            ql.CState(base + 0x7000, base + 60))
    assert call(overl) == ql.QL_EINVAL
    same = (ql.CState * 2)(ql.CState(base + 0x5000, base + 0x6000),
                           ql.CState(base + 0x2000, None))
    assert call(same) == ql.QL_EINVAL
    outs = (ql.CQAct * 2)(ql.CQAct(FAKE, T * B, H, 64, FAKE, FAKE, FAKE),
                          ql.CQAct(FAKE, T * B, H, 64, FAKE, FAKE, FAKE))
    x = ql.CQAct(FAKE, T * B, IN, 64, FAKE, FAKE, FAKE)
    sneed = lib.ql_lstm_stack_workspace(arr, 2, T, B)
    assert lib.ql_lstm_stack_forward(arr, 2, C.byref(x), T, B, outs, None, s_in, same, None, FAKE,
                                     sneed, None) == ql.QL_EINVAL


def test_wait_bound_hook_arguments(ql):
    lib = ql.load()
    assert lib.ql_debug_set_wait_bound(-1) == ql.QL_EINVAL
    assert lib.ql_debug_set_wait_bound(0) == ql.QL_OK
