"""ctypes front end of the CPU oracle (qlstm_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library.  The arithmetic lives
in qlstm_oracle.c; this file builds it, marshals numpy arrays, packs the
results and stacks the frontend's base frames (a plain gather, Section 4).  Codes here are the paper's V' in 0..255 (uint8).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "qlstm_oracle.c")
LIB = os.path.join(HERE, "libqlstm_oracle.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C, no GPU)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < max(
            os.path.getmtime(SRC), os.path.getmtime(os.path.join(HERE, "qlstm_oracle.h"))):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        _declare(_lib)
    return _lib


class QParams(C.Structure):
    _fields_ = [("vmin", C.c_double), ("vmax", C.c_double), ("R", C.c_double),
                ("Q", C.c_double), ("z", C.c_int32), ("inv_q", C.c_float)]


class QMat(C.Structure):
    _fields_ = [("rows", C.c_int64), ("cols", C.c_int64), ("nblocks", C.c_int32),
                ("codes", C.c_void_p), ("zero", C.c_void_p), ("inv_q", C.c_void_p)]


class Layer(C.Structure):
    _fields_ = [("in_", C.c_int64), ("hidden", C.c_int64), ("proj", C.c_int64),
                ("Wx", QMat), ("Wh", QMat), ("Wr", QMat), ("bias", C.c_void_p)]


class Model(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(Layer)), ("Wy", QMat),
                ("by", C.c_void_p)]


class Taps(C.Structure):
    _fields_ = [("acc_x", C.c_void_p), ("acc_h", C.c_void_p), ("acc_r", C.c_void_p),
                ("h_codes", C.c_void_p), ("h_zero", C.c_void_p), ("h_inv_q", C.c_void_p),
                ("c", C.c_void_p), ("h", C.c_void_p), ("preact", C.c_void_p),
                ("gates", C.c_void_p), ("m", C.c_void_p)]


class LayerF32(C.Structure):
    _fields_ = [("in_", C.c_int64), ("hidden", C.c_int64), ("proj", C.c_int64),
                ("Wx", C.c_void_p), ("Wh", C.c_void_p), ("Wr", C.c_void_p),
                ("bias", C.c_void_p)]


class ModelF32(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(LayerF32)), ("S", C.c_int64),
                ("Wy", C.c_void_p), ("by", C.c_void_p)]


class TrainModel(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(LayerF32)), ("S", C.c_int64),
                ("Wy", C.c_void_p), ("by", C.c_void_p)]


def _declare(L):
    vp, i64, i32 = C.c_void_p, C.c_int64, C.c_int32
    L.oracle_expf.argtypes = [C.c_float]
    L.oracle_expf.restype = C.c_float
    L.oracle_elementwise.argtypes = [i32, vp, vp, i64]
    L.oracle_round_half_up.argtypes = [C.c_double]
    L.oracle_round_half_up.restype = i64
    L.oracle_qparams.argtypes = [C.c_float, C.c_float, C.POINTER(QParams)]
    L.oracle_code.argtypes = [C.c_float, C.POINTER(QParams)]
    L.oracle_code.restype = C.c_uint8
    L.oracle_quantize_set.argtypes = [vp, i64, vp, C.POINTER(QParams), vp]
    L.oracle_quantize.argtypes = [vp, i64, i64, i32, vp, vp, vp, vp, vp]
    L.oracle_dequantize.argtypes = [vp, i64, i64, i32, vp, vp, vp]
    L.oracle_quantized_matmul.argtypes = [C.POINTER(QMat), vp, i64, i32, vp, vp, vp, vp,
                                          vp, vp]
    L.oracle_gemm_u8.argtypes = [vp, vp, vp, i64, i64, i64]
    L.oracle_lstm_layer_forward.argtypes = [C.POINTER(Layer), vp, i64, i64, vp, vp, vp,
                                            vp, vp, C.POINTER(Taps)]
    L.oracle_acoustic_model_forward.argtypes = [C.POINTER(Model), vp, i64, i64, vp,
                                                C.POINTER(Taps), vp, vp]
    L.oracle_lstm_layer_forward_f32.argtypes = [C.POINTER(LayerF32), vp, i64, i64, vp, vp,
                                                vp, vp, vp, C.POINTER(Taps)]
    L.oracle_lstm_layer_backward.argtypes = [C.POINTER(LayerF32), vp, i64, i64, vp, vp, vp, vp,
                                             vp, vp, vp, vp, vp, vp]
    L.oracle_output_backward.argtypes = [vp, i64, i64, vp, vp, vp, i64, C.POINTER(C.c_double),
                                         vp, vp, vp]
    L.oracle_train_step.argtypes = [C.POINTER(TrainModel), vp, vp, i64, i64, C.c_float, i32,
                                    i32, i32, C.POINTER(C.c_double), C.POINTER(TrainModel)]
    L.oracle_acoustic_model_forward_f32.argtypes = [C.POINTER(ModelF32), vp, i64, i64, vp]
    for f in ("oracle_quantize", "oracle_dequantize", "oracle_quantized_matmul",
              "oracle_gemm_u8", "oracle_lstm_layer_forward",
              "oracle_acoustic_model_forward", "oracle_lstm_layer_forward_f32",
              "oracle_acoustic_model_forward_f32", "oracle_lstm_layer_backward",
              "oracle_output_backward", "oracle_train_step"):
        getattr(L, f).restype = i32


def set_threads(n: int) -> None:
    """OpenMP threads the oracle runs on (omp_set_num_threads of its runtime)."""
    lib().omp_set_num_threads(int(n))


def threads() -> int:
    lib().omp_get_max_threads.restype = C.c_int
    return int(lib().omp_get_max_threads())


def _p(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


# ---------------------------------------------------------------- scalars
def expf(x):
    return _elementwise(0, x)


def sigmoidf(x):
    return _elementwise(1, x)


def tanhf(x):
    return _elementwise(2, x)


def _elementwise(fn, x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty_like(x)
    lib().oracle_elementwise(fn, _p(x), _p(y), x.size)
    return y


def round_half_up(x: float) -> int:
    return int(lib().oracle_round_half_up(float(x)))


def qparams(vmin: float, vmax: float) -> dict:
    p = QParams()
    lib().oracle_qparams(float(vmin), float(vmax), C.byref(p))
    return dict(vmin=p.vmin, vmax=p.vmax, R=p.R, Q=p.Q, z=p.z, inv_q=np.float32(p.inv_q))


def quantize_set(v):
    """Quantize all of v as one set -> (codes uint8 same shape, params, code_sum)."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    codes = np.empty(v.shape, dtype=np.uint8)
    p = QParams()
    s = C.c_int32()
    lib().oracle_quantize_set(_p(v), v.size, _p(codes), C.byref(p), C.byref(s))
    return codes, dict(vmin=p.vmin, vmax=p.vmax, R=p.R, Q=p.Q, z=p.z,
                       inv_q=np.float32(p.inv_q)), int(s.value)


# ---------------------------------------------------------------- matrices
@dataclass
class QMatrix:
    codes: np.ndarray      # [rows][cols] uint8
    range: np.ndarray      # [nblocks] float64
    zero: np.ndarray       # [nblocks] int32
    inv_q: np.ndarray      # [nblocks] float32
    row_sums: np.ndarray   # [rows] int32
    nblocks: int

    @property
    def shape(self):
        return self.codes.shape

    def cstruct(self) -> QMat:
        r, c = self.codes.shape
        return QMat(r, c, self.nblocks, _p(self.codes), _p(self.zero), _p(self.inv_q))


def quantize(W, nblocks: int = 1) -> QMatrix:
    W = np.ascontiguousarray(W, dtype=np.float32)
    rows, cols = W.shape
    q = QMatrix(np.empty((rows, cols), np.uint8), np.empty(nblocks, np.float64),
                np.empty(nblocks, np.int32), np.empty(nblocks, np.float32),
                np.empty(rows, np.int32), nblocks)
    _check(lib().oracle_quantize(_p(W), rows, cols, nblocks, _p(q.codes), _p(q.range),
                                 _p(q.zero), _p(q.inv_q), _p(q.row_sums)), "quantize")
    return q


def dequantize(q: QMatrix) -> np.ndarray:
    rows, cols = q.codes.shape
    out = np.empty((rows, cols), np.float32)
    _check(lib().oracle_dequantize(_p(q.codes), rows, cols, q.nblocks, _p(q.zero),
                                   _p(q.inv_q), _p(out)), "dequantize")
    return out


def quantized_matmul(q: QMatrix, X, act_gran: int = 1, bias=None):
    """-> dict(Y [m][rows] fp32, acc [m][rows] int32, x_codes, x_zero, x_inv_q)."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    m, K = X.shape
    N = q.codes.shape[0]
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    Y = np.empty((m, N), np.float32)
    acc = np.empty((m, N), np.int32)
    xc = np.empty((m, K), np.uint8)
    xz = np.empty(m, np.int32)
    xi = np.empty(m, np.float32)
    qs = q.cstruct()
    _check(lib().oracle_quantized_matmul(C.byref(qs), _p(X), m, act_gran, _p(bias), _p(Y),
                                         _p(acc), _p(xc), _p(xz), _p(xi)), "quantized_matmul")
    return dict(Y=Y, acc=acc, x_codes=xc, x_zero=xz, x_inv_q=xi)


def gemm_u8(A, B):
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, K = A.shape
    N = B.shape[0]
    Cm = np.empty((M, N), np.int32)
    _check(lib().oracle_gemm_u8(_p(A), _p(B), _p(Cm), M, N, K), "gemm_u8")
    return Cm


# ---------------------------------------------------------------- LSTM models
@dataclass
class QLayer:
    n_in: int
    hidden: int
    proj: int
    Wx: QMatrix
    Wh: QMatrix
    Wr: QMatrix | None
    bias: np.ndarray

    def cstruct(self) -> Layer:
        empty = QMat(0, 0, 1, None, None, None)
        return Layer(self.n_in, self.hidden, self.proj, self.Wx.cstruct(), self.Wh.cstruct(),
                     self.Wr.cstruct() if self.Wr is not None else empty, _p(self.bias))


def quantize_layer(L: dict, gate_blocks: int = 4, proj_blocks: int = 1) -> QLayer:
    """Float layer {'Wx','Wh','b','Wr'} -> quantized: W_x, W_h in gate_blocks
    row blocks (4: per gate), W_r in proj_blocks (Section 3.1, granularity)."""
    Wx, Wh = L["Wx"], L["Wh"]
    H = Wx.shape[0] // 4
    Wr = L.get("Wr")
    return QLayer(Wx.shape[1], H, 0 if Wr is None else Wr.shape[0],
                  quantize(Wx, gate_blocks), quantize(Wh, gate_blocks),
                  None if Wr is None else quantize(Wr, proj_blocks),
                  np.ascontiguousarray(L["b"], dtype=np.float32))


@dataclass
class QModel:
    layers: list
    Wy: QMatrix
    by: np.ndarray


def quantize_model(weights: dict, gate_blocks: int = 4, proj_blocks: int = 1,
                   out_blocks: int = 1) -> QModel:
    return QModel([quantize_layer(L, gate_blocks, proj_blocks) for L in weights["layers"]],
                  quantize(weights["Wy"], out_blocks),
                  np.ascontiguousarray(weights["by"], np.float32))


def _taps_arrays(T, B, H, P):
    RD = P if P else H
    t = dict(acc_x=np.empty((T, B, 4 * H), np.int32), acc_h=np.empty((T, B, 4 * H), np.int32),
             acc_r=np.empty((T, B, P), np.int32) if P else None,
             h_codes=np.empty((T, B, RD), np.uint8), h_zero=np.empty((T, B), np.int32),
             h_inv_q=np.empty((T, B), np.float32), c=np.empty((T, B, H), np.float32),
             h=np.empty((T, B, RD), np.float32), preact=np.empty((T, B, 4 * H), np.float32),
             gates=np.empty((T, B, 4 * H), np.float32), m=np.empty((T, B, H), np.float32))
    ts = Taps(*[_p(t[k]) for k in ("acc_x", "acc_h", "acc_r", "h_codes", "h_zero",
                                   "h_inv_q", "c", "h", "preact", "gates", "m")])
    return t, ts


def lstm_layer_forward(L: QLayer, x, h0=None, c0=None, taps: bool = False):
    """x [T][B][in] fp32 -> dict(h [T][B][R], hT, cT, and taps if asked)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    T, B, _ = x.shape
    H, P = L.hidden, L.proj
    RD = P if P else H
    h = np.empty((T, B, RD), np.float32)
    hT = np.empty((B, RD), np.float32)
    cT = np.empty((B, H), np.float32)
    h0 = None if h0 is None else np.ascontiguousarray(h0, np.float32)
    c0 = None if c0 is None else np.ascontiguousarray(c0, np.float32)
    ls = L.cstruct()
    out = dict(h=h, hT=hT, cT=cT)
    tp = None
    if taps:
        t, ts = _taps_arrays(T, B, H, P)
        out.update(t)
        tp = C.byref(ts)
    _check(lib().oracle_lstm_layer_forward(C.byref(ls), _p(x), T, B, _p(h0), _p(c0), _p(h),
                                           _p(hT), _p(cT), tp), "lstm_layer_forward")
    return out


def acoustic_model_forward(Mq: QModel, feats, taps: bool = False):
    """feats [T][B][in] -> dict(post [T][B][S], logits, acc_y, layer taps)."""
    feats = np.ascontiguousarray(feats, dtype=np.float32)
    T, B, _ = feats.shape
    S = Mq.Wy.codes.shape[0]
    layers = (Layer * len(Mq.layers))(*[L.cstruct() for L in Mq.layers])
    model = Model(len(Mq.layers), layers, Mq.Wy.cstruct(), _p(Mq.by))
    post = np.empty((T, B, S), np.float32)
    out = dict(post=post)
    tp = None
    acc_y = logits = None
    if taps:
        lt = []
        arr = (Taps * len(Mq.layers))()
        for i, L in enumerate(Mq.layers):
            t, ts = _taps_arrays(T, B, L.hidden, L.proj)
            lt.append(t)
            arr[i] = ts
        out["layers"] = lt
        tp = arr
        acc_y = np.empty((T, B, S), np.int32)
        logits = np.empty((T, B, S), np.float32)
        out.update(acc_y=acc_y, logits=logits)
    _check(lib().oracle_acoustic_model_forward(C.byref(model), _p(feats), T, B, _p(post), tp,
                                               _p(acc_y), _p(logits)),
           "acoustic_model_forward")
    return out


def stacked_input_count(nframes: int, stack: int = 8, skip: int = 3) -> int:
    """Section 4 frontend: a stacked frame needs `stack` base frames (the first
    plus stack-1 of right context); only every skip-th stacked frame, starting
    with the first, is presented to the network."""
    if nframes < stack:
        return 0
    return (nframes - stack) // skip + 1


def stack_frames(frames, stack: int = 8, skip: int = 3) -> np.ndarray:
    """Section 4 frontend: base frames [nframes][B][d] -> presented inputs
    [T][B][stack*d], input t = base frames skip*t .. skip*t+stack-1 laid end to
    end (plain loops: one copy per (t, b, j))."""
    frames = np.asarray(frames, dtype=np.float32)
    nframes, B, d = frames.shape
    T = stacked_input_count(nframes, stack, skip)
    out = np.empty((T, B, stack * d), np.float32)
    for t in range(T):
        for b in range(B):
            for j in range(stack):
                out[t, b, j * d:(j + 1) * d] = frames[skip * t + j, b, :]
    return out


def acoustic_model_forward_frames(Mq: QModel, frames, stack: int = 8, skip: int = 3,
                                  taps: bool = False):
    """The model on the presented inputs of base frames [nframes][B][d]."""
    return acoustic_model_forward(Mq, stack_frames(frames, stack, skip), taps)


# ---------------------------------------------------------------- fp32 model
def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def lstm_layer_forward_f32(L: dict, x, h0=None, c0=None, taps: bool = False):
    """The unquantized layer -> dict(h, hT, cT[, c, m, gates, h taps])."""
    x = _f32(x)
    T, B, n_in = x.shape
    Wx, Wh, b, Wr = _f32(L["Wx"]), _f32(L["Wh"]), _f32(L["b"]), _f32(L.get("Wr"))
    H = Wx.shape[0] // 4
    P = 0 if Wr is None else Wr.shape[0]
    RD = P if P else H
    ls = LayerF32(n_in, H, P, _p(Wx), _p(Wh), _p(Wr), _p(b))
    h = np.empty((T, B, RD), np.float32)
    hT = np.empty((B, RD), np.float32)
    cT = np.empty((B, H), np.float32)
    h0, c0 = _f32(h0), _f32(c0)
    out = dict(h=h, hT=hT, cT=cT)
    tp = None
    if taps:
        t, ts = _taps_arrays(T, B, H, P)
        out.update({k: t[k] for k in ("c", "m", "gates")})
        ts.h = None
        tp = C.byref(ts)
        out["_keep"] = t
    _check(lib().oracle_lstm_layer_forward_f32(C.byref(ls), _p(x), T, B, _p(h0), _p(c0),
                                               _p(h), _p(hT), _p(cT), tp), "lstm_f32")
    return out


def acoustic_model_forward_f32(weights: dict, feats):
    feats = _f32(feats)
    T, B, _ = feats.shape
    keep = []
    ls = []
    for L in weights["layers"]:
        Wx, Wh, b, Wr = _f32(L["Wx"]), _f32(L["Wh"]), _f32(L["b"]), _f32(L.get("Wr"))
        keep += [Wx, Wh, b, Wr]
        H = Wx.shape[0] // 4
        ls.append(LayerF32(Wx.shape[1], H, 0 if Wr is None else Wr.shape[0], _p(Wx), _p(Wh),
                           _p(Wr), _p(b)))
    arr = (LayerF32 * len(ls))(*ls)
    Wy, by = _f32(weights["Wy"]), _f32(weights["by"])
    m = ModelF32(len(ls), arr, Wy.shape[0], _p(Wy), _p(by))
    post = np.empty((T, B, Wy.shape[0]), np.float32)
    _check(lib().oracle_acoustic_model_forward_f32(C.byref(m), _p(feats), T, B, _p(post)),
           "model_f32")
    return dict(post=post)


# ------------------------------------------------- quantization aware training
def _train_struct(weights: dict):
    """Host fp32 copies of a model's parameters and the C struct over them."""
    keep, ls = [], []
    for L in weights["layers"]:
        Wx, Wh, b = (np.array(L[k], dtype=np.float32, copy=True) for k in ("Wx", "Wh", "b"))
        Wr = None if L.get("Wr") is None else np.array(L["Wr"], dtype=np.float32, copy=True)
        keep.append(dict(Wx=Wx, Wh=Wh, b=b, Wr=Wr))
        H = Wx.shape[0] // 4
        ls.append(LayerF32(Wx.shape[1], H, 0 if Wr is None else Wr.shape[0], _p(Wx), _p(Wh),
                           _p(Wr), _p(b)))
    Wy = np.array(weights["Wy"], dtype=np.float32, copy=True)
    by = np.array(weights["by"], dtype=np.float32, copy=True)
    arr = (LayerF32 * len(ls))(*ls)
    st = TrainModel(len(ls), arr, Wy.shape[0], _p(Wy), _p(by))
    return dict(layers=keep, Wy=Wy, by=by), st, arr


def train_step(weights: dict, feats, targets, lr: float, gate_blocks: int = 4,
               quantize_layers: bool = True, quantize_output: bool = True):
    """Algorithm 1 on one mini-batch -> (updated weights, gradients, loss).
    weights is not modified."""
    feats = _f32(feats)
    T, B, _ = feats.shape
    targets = np.ascontiguousarray(targets, dtype=np.int32)
    assert targets.shape == (T, B)
    new, st, keep1 = _train_struct(weights)
    zeros = {"layers": [dict(Wx=np.zeros_like(L["Wx"]), Wh=np.zeros_like(L["Wh"]),
                             b=np.zeros_like(L["b"]),
                             Wr=None if L["Wr"] is None else np.zeros_like(L["Wr"]))
                        for L in new["layers"]],
             "Wy": np.zeros_like(new["Wy"]), "by": np.zeros_like(new["by"])}
    grads, gst, keep2 = _train_struct(zeros)
    loss = C.c_double()
    _check(lib().oracle_train_step(C.byref(st), _p(feats), _p(targets), T, B, float(lr),
                                   gate_blocks, int(quantize_layers), int(quantize_output),
                                   C.byref(loss), C.byref(gst)), "train_step")
    return new, grads, float(loss.value)


def lstm_layer_backward(L: dict, x, gates, c, m, h, dy):
    """Float BPTT of one layer at the given forward activations -> dict of
    gradients (Wx, Wh, Wr, b) and dx."""
    x, gates, c, m, h, dy = (_f32(a) for a in (x, gates, c, m, h, dy))
    T, B, n_in = x.shape
    Wx, Wh, b, Wr = _f32(L["Wx"]), _f32(L["Wh"]), _f32(L["b"]), _f32(L.get("Wr"))
    H = Wx.shape[0] // 4
    P = 0 if Wr is None else Wr.shape[0]
    ls = LayerF32(n_in, H, P, _p(Wx), _p(Wh), _p(Wr), _p(b))
    out = dict(Wx=np.empty_like(Wx), Wh=np.empty_like(Wh), b=np.empty_like(b),
               Wr=None if Wr is None else np.empty_like(Wr), dx=np.empty_like(x))
    _check(lib().oracle_lstm_layer_backward(C.byref(ls), _p(x), T, B, _p(gates), _p(c), _p(m),
                                            _p(h), _p(dy), _p(out["Wx"]), _p(out["Wh"]),
                                            _p(out["Wr"]), _p(out["b"]), _p(out["dx"])),
           "lstm_layer_backward")
    return out
