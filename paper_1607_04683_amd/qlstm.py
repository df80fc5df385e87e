"""Thin Python binding of libqlstm.so (include/qlstm.h).

Argument marshalling only: every step of quantized inference runs in the
library's gfx950 kernels.  PyTorch supplies device memory (tensors) and the
current HIP stream.  If the shared library is missing this module raises; it
never falls back to another implementation.

Codes on the device use the library's layout: row-major with a leading
dimension `ld` (multiple of 64) and bytes equal to V' - 128 (int8).
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqlstm.so")

QL_OK, QL_EINVAL, QL_ESHAPE, QL_EOVERFLOW, QL_EWORKSPACE, QL_EHIP, QL_EUNSUPPORTED, \
    QL_ETIMEOUT, QL_ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7, -8
NOALLOC_SCRATCH_BYTES = 32 << 20  # QL_NOALLOC_SCRATCH_BYTES
QL_ACT_PER_TENSOR, QL_ACT_PER_ROW = 0, 1

EXPORTS = [
    "ql_quantize_workspace", "ql_quantize", "ql_dequantize", "ql_quantized_matmul_workspace",
    "ql_quantized_matmul", "ql_gemm_u8_workspace", "ql_gemm_u8", "ql_lstm_layer_workspace",
    "ql_lstm_layer_forward", "ql_acoustic_model_workspace", "ql_acoustic_model_forward",
    "ql_status_str", "ql_workspace_status", "ql_gate_fn", "ql_lstm_recurrence_workspace",
    "ql_lstm_recurrence", "ql_f32_matmul", "ql_f32_lstm_layer_workspace",
    "ql_f32_lstm_layer_forward", "ql_f32_acoustic_model_workspace",
    "ql_f32_acoustic_model_forward", "ql_quantize_activations", "ql_lstm_stack_workspace",
    "ql_lstm_stack_forward", "ql_lstm_stack_layers_per_launch", "ql_stacked_input_count",
    "ql_quantize_stacked_frames", "ql_acoustic_model_frames_workspace",
    "ql_acoustic_model_forward_frames", "ql_acoustic_model_forward_stream",
    "ql_acoustic_model_forward_stream_noalloc", "ql_train_step_workspace", "ql_train_step",
    "ql_debug_set_wait_bound", "ql_debug_recurrence_layout", "ql_debug_stack_layout",
]


class QLError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} ({status})")
        self.status = status


class CQMatrix(C.Structure):
    _fields_ = [("codes", C.c_void_p), ("rows", C.c_int64), ("cols", C.c_int64),
                ("ld", C.c_int64), ("nblocks", C.c_int32), ("range", C.c_void_p),
                ("zero", C.c_void_p), ("inv_q", C.c_void_p), ("row_sums", C.c_void_p)]


class CLayer(C.Structure):
    _fields_ = [("in_", C.c_int64), ("hidden", C.c_int64), ("proj", C.c_int64),
                ("Wx", CQMatrix), ("Wh", CQMatrix), ("Wr", CQMatrix), ("bias", C.c_void_p)]


class CModel(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(CLayer)), ("Wy", CQMatrix),
                ("by", C.c_void_p)]


class CTaps(C.Structure):
    _fields_ = [("acc_x", C.c_void_p), ("acc_h", C.c_void_p), ("acc_r", C.c_void_p),
                ("h_codes", C.c_void_p), ("h_zero", C.c_void_p), ("h_inv_q", C.c_void_p),
                ("h", C.c_void_p), ("gates", C.c_void_p), ("c", C.c_void_p), ("m", C.c_void_p)]


class CState(C.Structure):
    _fields_ = [("h", C.c_void_p), ("c", C.c_void_p)]


class CQAct(C.Structure):
    _fields_ = [("codes", C.c_void_p), ("rows", C.c_int64), ("cols", C.c_int64),
                ("ld", C.c_int64), ("zero", C.c_void_p), ("inv_q", C.c_void_p),
                ("sums", C.c_void_p)]


class CF32Layer(C.Structure):
    _fields_ = [("in_", C.c_int64), ("hidden", C.c_int64), ("proj", C.c_int64),
                ("Wx", C.c_void_p), ("Wh", C.c_void_p), ("Wr", C.c_void_p), ("bias", C.c_void_p)]


class CF32Model(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(CF32Layer)), ("states", C.c_int64),
                ("Wy", C.c_void_p), ("by", C.c_void_p)]


class CTrainLayer(C.Structure):
    _fields_ = [("in_", C.c_int64), ("hidden", C.c_int64), ("proj", C.c_int64),
                ("Wx", C.c_void_p), ("Wh", C.c_void_p), ("Wr", C.c_void_p), ("bias", C.c_void_p)]


class CTrainModel(C.Structure):
    _fields_ = [("nlayers", C.c_int32), ("layers", C.POINTER(CTrainLayer)), ("states", C.c_int64),
                ("Wy", C.c_void_p), ("by", C.c_void_p)]


class CModelTaps(C.Structure):
    _fields_ = [("layers", C.POINTER(CTaps)), ("acc_y", C.c_void_p), ("logits", C.c_void_p)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libqlstm.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build it with `python -m paper_1607_04683_amd.build`")
    L = C.CDLL(path)
    vp, i64, i32, sz = C.c_void_p, C.c_int64, C.c_int32, C.c_size_t
    L.ql_status_str.argtypes = [i32]
    L.ql_status_str.restype = C.c_char_p
    L.ql_quantize_workspace.argtypes = [i64, i64, i32]
    L.ql_quantize_workspace.restype = sz
    L.ql_quantize.argtypes = [vp, i64, i64, i32, C.POINTER(CQMatrix), vp, sz, vp]
    L.ql_dequantize.argtypes = [C.POINTER(CQMatrix), vp, vp]
    L.ql_quantized_matmul_workspace.argtypes = [i64, i64, i64]
    L.ql_quantized_matmul_workspace.restype = sz
    L.ql_quantized_matmul.argtypes = [C.POINTER(CQMatrix), vp, i64, i32, vp, vp, vp, vp, sz, vp]
    L.ql_gemm_u8_workspace.argtypes = [i64, i64, i64]
    L.ql_gemm_u8_workspace.restype = sz
    L.ql_gemm_u8.argtypes = [vp, i64, vp, i64, vp, i64, i64, i64, vp, vp, vp, sz, vp]
    L.ql_lstm_layer_workspace.argtypes = [C.POINTER(CLayer), i64, i64]
    L.ql_lstm_layer_workspace.restype = sz
    L.ql_lstm_layer_forward.argtypes = [C.POINTER(CLayer), vp, i64, i64, vp, vp, vp, vp, vp,
                                        C.POINTER(CTaps), vp, sz, vp]
    L.ql_acoustic_model_workspace.argtypes = [C.POINTER(CModel), i64, i64]
    L.ql_acoustic_model_workspace.restype = sz
    L.ql_acoustic_model_forward.argtypes = [C.POINTER(CModel), vp, i64, i64, vp,
                                            C.POINTER(CModelTaps), vp, sz, vp]
    L.ql_lstm_recurrence_workspace.argtypes = [C.POINTER(CLayer), i64, i64]
    L.ql_lstm_recurrence_workspace.restype = sz
    L.ql_lstm_recurrence.argtypes = [C.POINTER(CLayer), vp, i64, i64, vp, vp, vp, vp, vp,
                                     C.POINTER(CQAct), C.POINTER(CTaps), vp, sz, vp]
    L.ql_workspace_status.argtypes = [vp, vp]
    L.ql_gate_fn.argtypes = [i32, vp, vp, i64, vp]
    L.ql_debug_set_wait_bound.argtypes = [i32]
    L.ql_debug_recurrence_layout.argtypes = [C.POINTER(CLayer), i64]
    L.ql_debug_recurrence_layout.restype = i32
    L.ql_debug_stack_layout.argtypes = [C.POINTER(CLayer), i32, i64, i64]
    L.ql_debug_stack_layout.restype = i32
    L.ql_f32_matmul.argtypes = [vp, i64, i64, vp, i64, vp, vp, vp]
    L.ql_quantize_activations.argtypes = [vp, i64, i64, C.POINTER(CQAct), vp]
    L.ql_lstm_stack_workspace.argtypes = [C.POINTER(CLayer), i32, i64, i64]
    L.ql_lstm_stack_workspace.restype = sz
    L.ql_lstm_stack_forward.argtypes = [C.POINTER(CLayer), i32, C.POINTER(CQAct), i64, i64,
                                        C.POINTER(CQAct), vp, C.POINTER(CState),
                                        C.POINTER(CState), C.POINTER(CTaps), vp, sz, vp]
    L.ql_acoustic_model_forward_stream.argtypes = [C.POINTER(CModel), vp, i64, i64,
                                                   C.POINTER(CState), C.POINTER(CState), vp,
                                                   C.POINTER(CModelTaps), vp, sz, vp]
    L.ql_train_step_workspace.argtypes = [C.POINTER(CTrainModel), i64, i64, i32]
    L.ql_train_step_workspace.restype = sz
    L.ql_train_step.argtypes = [C.POINTER(CTrainModel), vp, vp, i64, i64, C.c_float, i32, i32,
                                vp, C.POINTER(CTrainModel), vp, sz, vp]
    L.ql_acoustic_model_forward_stream_noalloc.argtypes = [C.POINTER(CModel), vp, i64, i64,
                                                           C.POINTER(CState), C.POINTER(CState),
                                                           vp, vp, vp]
    L.ql_lstm_stack_layers_per_launch.argtypes = [C.POINTER(CLayer), i32, i64, i64]
    L.ql_lstm_stack_layers_per_launch.restype = i32
    L.ql_stacked_input_count.argtypes = [i64, i32, i32]
    L.ql_stacked_input_count.restype = i64
    L.ql_quantize_stacked_frames.argtypes = [vp, i64, i64, i64, i32, i32, C.POINTER(CQAct), vp]
    L.ql_acoustic_model_frames_workspace.argtypes = [C.POINTER(CModel), i64, i64, i32, i32]
    L.ql_acoustic_model_frames_workspace.restype = sz
    L.ql_acoustic_model_forward_frames.argtypes = [C.POINTER(CModel), vp, i64, i64, i64, i32,
                                                   i32, vp, C.POINTER(CModelTaps), vp, sz, vp]
    L.ql_f32_lstm_layer_workspace.argtypes = [C.POINTER(CF32Layer), i64, i64]
    L.ql_f32_lstm_layer_workspace.restype = sz
    L.ql_f32_lstm_layer_forward.argtypes = [C.POINTER(CF32Layer), vp, i64, i64, vp, vp, vp, vp,
                                            vp, vp, sz, vp]
    L.ql_f32_acoustic_model_workspace.argtypes = [C.POINTER(CF32Model), i64, i64]
    L.ql_f32_acoustic_model_workspace.restype = sz
    L.ql_f32_acoustic_model_forward.argtypes = [C.POINTER(CF32Model), vp, i64, i64, vp, vp, sz,
                                                vp]
    for f in ("ql_quantize", "ql_dequantize", "ql_quantized_matmul", "ql_gemm_u8",
              "ql_lstm_layer_forward", "ql_acoustic_model_forward", "ql_workspace_status",
              "ql_gate_fn", "ql_lstm_recurrence", "ql_f32_matmul", "ql_f32_lstm_layer_forward",
              "ql_f32_acoustic_model_forward", "ql_quantize_activations",
              "ql_lstm_stack_forward", "ql_quantize_stacked_frames",
              "ql_acoustic_model_forward_frames", "ql_acoustic_model_forward_stream",
              "ql_acoustic_model_forward_stream_noalloc", "ql_train_step",
              "ql_debug_set_wait_bound"):
        getattr(L, f).restype = i32
    _lib = L
    return L


def status_str(s: int) -> str:
    return load().ql_status_str(s).decode()


def _check(st: int, what: str):
    if st != QL_OK:
        raise QLError(st, what)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ws(nbytes: int, device):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def ld_for(cols: int) -> int:
    return (cols + 63) // 64 * 64


# ------------------------------------------------------------------- matrices
@dataclass
class QMatrix:
    """A quantized matrix on the device (see ql_qmatrix)."""
    codes: torch.Tensor     # int8 [rows][ld]
    rows: int
    cols: int
    nblocks: int
    range: torch.Tensor     # float64 [nblocks]
    zero: torch.Tensor      # int32 [nblocks]
    inv_q: torch.Tensor     # float32 [nblocks]
    row_sums: torch.Tensor  # int32 [rows]

    @property
    def ld(self) -> int:
        return self.codes.shape[1]

    def cstruct(self) -> CQMatrix:
        return CQMatrix(self.codes.data_ptr(), self.rows, self.cols, self.ld, self.nblocks,
                        self.range.data_ptr(), self.zero.data_ptr(), self.inv_q.data_ptr(),
                        self.row_sums.data_ptr())

    def codes_u8(self) -> torch.Tensor:
        """The paper's V' (0..255) as uint8 [rows][cols] (device)."""
        return (self.codes[:, :self.cols].view(torch.uint8) ^ 0x80)

    @staticmethod
    def empty(rows: int, cols: int, nblocks: int, device) -> "QMatrix":
        return QMatrix(torch.zeros(rows, ld_for(cols), dtype=torch.int8, device=device), rows,
                       cols, nblocks, torch.empty(nblocks, dtype=torch.float64, device=device),
                       torch.empty(nblocks, dtype=torch.int32, device=device),
                       torch.empty(nblocks, dtype=torch.float32, device=device),
                       torch.empty(rows, dtype=torch.int32, device=device))


def quantize(W: torch.Tensor, nblocks: int = 1) -> QMatrix:
    """Section 3 quantizer: W [rows][cols] fp32 (device) -> QMatrix."""
    W = W.contiguous()
    assert W.dtype == torch.float32 and W.dim() == 2
    rows, cols = W.shape
    q = QMatrix.empty(rows, cols, nblocks, W.device)
    lib = load()
    nbytes = lib.ql_quantize_workspace(rows, cols, nblocks)
    ws = _ws(nbytes, W.device)
    cs = q.cstruct()
    _check(lib.ql_quantize(_ptr(W), rows, cols, nblocks, C.byref(cs), _ptr(ws), ws.numel(),
                           _stream()), "ql_quantize")
    return q


def dequantize(q: QMatrix) -> torch.Tensor:
    out = torch.empty(q.rows, q.cols, dtype=torch.float32, device=q.codes.device)
    cs = q.cstruct()
    _check(load().ql_dequantize(C.byref(cs), _ptr(out), _stream()), "ql_dequantize")
    return out


def quantized_matmul(q: QMatrix, X: torch.Tensor, gran: int = QL_ACT_PER_ROW, bias=None,
                     want_acc: bool = False):
    """Fig. 1: R(Mult(Q(X), W')) + B -> (Y [m][rows], acc or None)."""
    X = X.contiguous()
    m = X.shape[0]
    lib = load()
    Y = torch.empty(m, q.rows, dtype=torch.float32, device=X.device)
    acc = torch.empty(m, q.rows, dtype=torch.int32, device=X.device) if want_acc else None
    ws = _ws(lib.ql_quantized_matmul_workspace(m, q.rows, q.cols), X.device)
    cs = q.cstruct()
    _check(lib.ql_quantized_matmul(C.byref(cs), _ptr(X), m, gran, _ptr(bias), _ptr(Y), _ptr(acc),
                                   _ptr(ws), ws.numel(), _stream()), "ql_quantized_matmul")
    return Y, acc


def device_codes(u8, ld: int | None = None, device="cuda") -> torch.Tensor:
    """uint8 codes [rows][cols] (numpy or tensor) -> device layout int8 [rows][ld]."""
    t = torch.as_tensor(u8).to(device)
    rows, cols = t.shape
    ld = ld or ld_for(cols)
    out = torch.zeros(rows, ld, dtype=torch.int8, device=device)
    out[:, :cols] = (t.to(torch.uint8) ^ 0x80).view(torch.int8)
    return out


def gemm_u8(A: torch.Tensor, B: torch.Tensor, K: int, a_sums=None, b_sums=None, out=None,
            ws=None):
    """C = A' B'^T (int32) for device-layout codes A [M][lda], B [N][ldb]."""
    M, lda = A.shape
    N, ldb = B.shape
    lib = load()
    Cm = out if out is not None else torch.empty(M, N, dtype=torch.int32, device=A.device)
    if ws is None and (a_sums is None or b_sums is None):
        ws = _ws(lib.ql_gemm_u8_workspace(M, N, K), A.device)
    _check(lib.ql_gemm_u8(_ptr(A), lda, _ptr(B), ldb, _ptr(Cm), M, N, K, _ptr(a_sums),
                          _ptr(b_sums), _ptr(ws), 0 if ws is None else ws.numel(), _stream()),
           "ql_gemm_u8")
    return Cm


def gate_fn(fn: int, x: torch.Tensor) -> torch.Tensor:
    x = x.contiguous()
    y = torch.empty_like(x)
    _check(load().ql_gate_fn(fn, _ptr(x), _ptr(y), x.numel(), _stream()), "ql_gate_fn")
    return y


# ------------------------------------------------------------------- LSTM
@dataclass
class Layer:
    n_in: int
    hidden: int
    proj: int
    Wx: QMatrix
    Wh: QMatrix
    Wr: QMatrix | None
    bias: torch.Tensor

    @property
    def width(self) -> int:
        return self.proj if self.proj else self.hidden

    def cstruct(self) -> CLayer:
        empty = CQMatrix(None, 0, 0, 0, 1, None, None, None, None)
        return CLayer(self.n_in, self.hidden, self.proj, self.Wx.cstruct(), self.Wh.cstruct(),
                      self.Wr.cstruct() if self.Wr is not None else empty, self.bias.data_ptr())


def quantize_layer(L: dict, device="cuda", gate_blocks: int = 4, proj_blocks: int = 1) -> Layer:
    """Float layer {'Wx','Wh','b','Wr'} (numpy/tensors) -> quantized layer on the device:
    W_x, W_h in gate_blocks row blocks (4: one per gate i, f, g, o; 4H: per row),
    W_r in proj_blocks row blocks (1: per matrix)."""
    t = lambda a: torch.as_tensor(a, dtype=torch.float32).to(device).contiguous()
    Wx, Wh = t(L["Wx"]), t(L["Wh"])
    Wr = None if L.get("Wr") is None else t(L["Wr"])
    H = Wx.shape[0] // 4
    return Layer(Wx.shape[1], H, 0 if Wr is None else Wr.shape[0], quantize(Wx, gate_blocks),
                 quantize(Wh, gate_blocks),
                 None if Wr is None else quantize(Wr, proj_blocks), t(L["b"]))


@dataclass
class Model:
    layers: list
    Wy: QMatrix
    by: torch.Tensor

    def cstruct(self):
        arr = (CLayer * len(self.layers))(*[L.cstruct() for L in self.layers])
        return CModel(len(self.layers), arr, self.Wy.cstruct(), self.by.data_ptr()), arr


def quantize_model(weights: dict, device="cuda", gate_blocks: int = 4, proj_blocks: int = 1,
                   out_blocks: int = 1) -> Model:
    """Row blocks per matrix: gate_blocks for W_x / W_h, proj_blocks for W_r,
    out_blocks for the softmax layer's W_y (Section 3.1, granularity)."""
    return Model([quantize_layer(L, device, gate_blocks, proj_blocks) for L in weights["layers"]],
                 quantize(torch.as_tensor(weights["Wy"], dtype=torch.float32).to(device),
                          out_blocks),
                 torch.as_tensor(weights["by"], dtype=torch.float32).to(device).contiguous())


TAP_NAMES = ("acc_x", "acc_h", "acc_r", "h_codes", "h_zero", "h_inv_q", "h", "gates", "c", "m")


def _taps(T, B, L: Layer, device, which=True, layer_h=True):
    """Allocate the requested taps (True = all, or a collection of names);
    layer_h=False leaves out the fp32 h tap (the one-layer calls return h)."""
    H, P, R = L.hidden, L.proj, L.width
    want = set(TAP_NAMES) if which is True else set(which)
    if not layer_h:
        want.discard("h")
    z = lambda name, *s, dt: torch.empty(*s, dtype=dt, device=device) if name in want else None
    t = dict(acc_x=z("acc_x", T, B, 4 * H, dt=torch.int32),
             acc_h=z("acc_h", T, B, 4 * H, dt=torch.int32),
             acc_r=z("acc_r", T, B, P, dt=torch.int32) if P else None,
             h_codes=z("h_codes", T, B, R, dt=torch.int8), h_zero=z("h_zero", T, B, dt=torch.int32),
             h_inv_q=z("h_inv_q", T, B, dt=torch.float32), h=z("h", T, B, R, dt=torch.float32),
             gates=z("gates", T, B, 4 * H, dt=torch.float32), c=z("c", T, B, H, dt=torch.float32),
             m=z("m", T, B, H, dt=torch.float32))
    c = CTaps(*[None if t[k] is None else t[k].data_ptr() for k in TAP_NAMES])
    if not layer_h:
        del t["h"]  # the caller's own h output keeps its name
    return t, c


class Workspace:
    """Reusable device workspace (grows on demand)."""

    def __init__(self):
        self.buf = None

    def get(self, nbytes: int, device):
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != torch.device(device):
            self.buf = _ws(nbytes, device)
        return self.buf


def lstm_layer_forward(L: Layer, x: torch.Tensor, h0=None, c0=None, taps: bool = False,
                       workspace: Workspace | None = None, check: bool = True):
    """x [T][B][in] fp32 (device) -> dict(h, hT, cT[, taps])."""
    x = x.contiguous()
    T, B, _ = x.shape
    dev = x.device
    lib = load()
    cl = L.cstruct()
    h = torch.empty(T, B, L.width, dtype=torch.float32, device=dev)
    hT = torch.empty(B, L.width, dtype=torch.float32, device=dev)
    cT = torch.empty(B, L.hidden, dtype=torch.float32, device=dev)
    nbytes = lib.ql_lstm_layer_workspace(C.byref(cl), T, B)
    ws = (workspace or Workspace()).get(nbytes, dev)
    out = dict(h=h, hT=hT, cT=cT)
    tp = None
    if taps:
        t, ct = _taps(T, B, L, dev, taps, layer_h=False)
        out.update(t)
        tp = C.byref(ct)
    _check(lib.ql_lstm_layer_forward(C.byref(cl), _ptr(x), T, B, _ptr(h0), _ptr(c0), _ptr(h),
                                     _ptr(hT), _ptr(cT), tp, _ptr(ws), ws.numel(), _stream()),
           "ql_lstm_layer_forward")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_lstm_layer_forward")
    return out


def lstm_recurrence(L: Layer, gx: torch.Tensor, h0=None, c0=None, taps=False,
                    workspace: Workspace | None = None, out=None, check: bool = True):
    """gx [T][B][4H] fp32 pre-activations (device) -> dict(h, hT, cT, codes...)."""
    gx = gx.contiguous()
    T, B, _ = gx.shape
    dev = gx.device
    lib = load()
    cl = L.cstruct()
    o = out or {}
    h = o.get("h")
    if h is None:
        h = torch.empty(T, B, L.width, dtype=torch.float32, device=dev)
    ws = (workspace or Workspace()).get(lib.ql_lstm_recurrence_workspace(C.byref(cl), T, B), dev)
    res = dict(h=h)
    tp = None
    if taps:
        t, ct = _taps(T, B, L, dev, taps, layer_h=False)
        res.update(t)
        tp = C.byref(ct)
    _check(lib.ql_lstm_recurrence(C.byref(cl), _ptr(gx), T, B, _ptr(h0), _ptr(c0), _ptr(h),
                                  None, None, None, tp, _ptr(ws), ws.numel(), _stream()),
           "ql_lstm_recurrence")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_lstm_recurrence")
    return res


def _model_taps(M: Model, T: int, B: int, dev, taps, out: dict):
    """Tap buffers of a model forward (None when taps is falsy)."""
    if not taps:
        return None
    S = M.Wy.rows
    lt = []
    arr = (CTaps * len(M.layers))()
    for i, L in enumerate(M.layers):
        t, ct = _taps(T, B, L, dev, taps)
        lt.append(t)
        arr[i] = ct
    full = taps is True or "acc_y" in taps
    acc_y = torch.empty(T, B, S, dtype=torch.int32, device=dev) if full else None
    logits = torch.empty(T, B, S, dtype=torch.float32, device=dev) if full else None
    out.update(layers=lt, acc_y=acc_y, logits=logits, _keep=arr)
    return CModelTaps(arr, None if acc_y is None else acc_y.data_ptr(),
                      None if logits is None else logits.data_ptr())


def _state_array(states):
    """Host array of per-layer ql_lstm_state from [(h, c), ...] (tensors or None)."""
    if states is None:
        return None
    return (CState * len(states))(*[CState(_ptr(h), _ptr(c)) for h, c in states])


def empty_state(M: Model, B: int, device="cuda"):
    """Per-layer (h [B][R], c [B][H]) fp32 buffers for a stream's state."""
    return [(torch.empty(B, L.width, dtype=torch.float32, device=device),
             torch.empty(B, L.hidden, dtype=torch.float32, device=device)) for L in M.layers]


def acoustic_model_forward(M: Model, feats: torch.Tensor, taps: bool = False,
                           workspace: Workspace | None = None, post: torch.Tensor | None = None,
                           check: bool = True, state_in=None, state_out=None):
    """feats [T][B][in] fp32 (device) -> dict(post [T][B][S][, taps]).
    state_in / state_out: per-layer [(h, c)] of a stream (ql_acoustic_model_forward_stream);
    they must not share memory."""
    feats = feats.contiguous()
    T, B, _ = feats.shape
    dev = feats.device
    lib = load()
    cm, keep = M.cstruct()
    if post is None:
        post = torch.empty(T, B, M.Wy.rows, dtype=torch.float32, device=dev)
    nbytes = lib.ql_acoustic_model_workspace(C.byref(cm), T, B)
    ws = (workspace or Workspace()).get(nbytes, dev)
    out = dict(post=post)
    mt = _model_taps(M, T, B, dev, taps, out)
    mtp = C.byref(mt) if mt is not None else None
    if state_in is None and state_out is None:
        _check(lib.ql_acoustic_model_forward(C.byref(cm), _ptr(feats), T, B, _ptr(post), mtp,
                                             _ptr(ws), ws.numel(), _stream()),
               "ql_acoustic_model_forward")
    else:
        si, so = _state_array(state_in), _state_array(state_out)
        _check(lib.ql_acoustic_model_forward_stream(C.byref(cm), _ptr(feats), T, B, si, so,
                                                    _ptr(post), mtp, _ptr(ws), ws.numel(),
                                                    _stream()),
               "ql_acoustic_model_forward_stream")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_acoustic_model_forward")
    return out


def acoustic_model_forward_stream_noalloc(M: Model, feats: torch.Tensor, post: torch.Tensor,
                                          state_in=None, state_out=None, timed_out=None):
    """One chunk of a stream on the library's static scratch
    (ql_acoustic_model_forward_stream_noalloc): post [T][B][S] and the optional
    timed_out (int32 device tensor of one element) are the caller's; nothing
    is allocated here or in the library."""
    feats = feats.contiguous()
    T, B, _ = feats.shape
    cm, keep = M.cstruct()
    _check(load().ql_acoustic_model_forward_stream_noalloc(
        C.byref(cm), _ptr(feats), T, B, _state_array(state_in), _state_array(state_out),
        _ptr(post), _ptr(timed_out), _stream()), "ql_acoustic_model_forward_stream_noalloc")
    return post


def stacked_input_count(nframes: int, stack: int = 8, skip: int = 3) -> int:
    """Presented steps of nframes base frames (stack frames per input, every
    skip-th stack presented)."""
    return int(load().ql_stacked_input_count(nframes, stack, skip))


def quantize_stacked_frames(frames: torch.Tensor, stack: int = 8, skip: int = 3,
                            out: QAct | None = None) -> QAct:
    """Base frames [nframes][B][dim] fp32 (device) -> per-vector codes of the
    presented stacked inputs (T*B rows of stack*dim values)."""
    frames = frames.contiguous()
    nframes, B, dim = frames.shape
    T = stacked_input_count(nframes, stack, skip)
    q = out or QAct.empty(T * B, stack * dim, frames.device)
    cq = q.cstruct()
    _check(load().ql_quantize_stacked_frames(_ptr(frames), nframes, B, dim, stack, skip,
                                             C.byref(cq), _stream()),
           "ql_quantize_stacked_frames")
    return q


def acoustic_model_forward_frames(M: Model, frames: torch.Tensor, stack: int = 8, skip: int = 3,
                                  taps: bool = False, workspace: Workspace | None = None,
                                  post: torch.Tensor | None = None, check: bool = True):
    """Base frames [nframes][B][dim] fp32 (device) -> dict(post [T][B][S][, taps]),
    the frontend's stacking fused into the input quantizer."""
    frames = frames.contiguous()
    nframes, B, dim = frames.shape
    dev = frames.device
    lib = load()
    T = stacked_input_count(nframes, stack, skip)
    cm, keep = M.cstruct()
    if post is None:
        post = torch.empty(T, B, M.Wy.rows, dtype=torch.float32, device=dev)
    nbytes = lib.ql_acoustic_model_frames_workspace(C.byref(cm), nframes, B, stack, skip)
    ws = (workspace or Workspace()).get(nbytes, dev)
    out = dict(post=post)
    mt = _model_taps(M, T, B, dev, taps, out)
    _check(lib.ql_acoustic_model_forward_frames(C.byref(cm), _ptr(frames), nframes, B, dim,
                                                stack, skip, _ptr(post),
                                                C.byref(mt) if mt is not None else None,
                                                _ptr(ws), ws.numel(), _stream()),
           "ql_acoustic_model_forward_frames")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_acoustic_model_forward_frames")
    return out


# ------------------------------------------------------------- fp32 model
def f32_matmul(W: torch.Tensor, X: torch.Tensor, bias=None) -> torch.Tensor:
    """Y [m][rows] = X [m][cols] W^T (+ bias), fp32 accumulation."""
    W, X = W.contiguous(), X.contiguous()
    rows, cols = W.shape
    m = X.shape[0]
    Y = torch.empty(m, rows, dtype=torch.float32, device=X.device)
    _check(load().ql_f32_matmul(_ptr(W), rows, cols, _ptr(X), m, _ptr(bias), _ptr(Y), _stream()),
           "ql_f32_matmul")
    return Y


@dataclass
class F32Layer:
    n_in: int
    hidden: int
    proj: int
    Wx: torch.Tensor
    Wh: torch.Tensor
    Wr: torch.Tensor | None
    bias: torch.Tensor

    @property
    def width(self) -> int:
        return self.proj if self.proj else self.hidden

    def cstruct(self) -> CF32Layer:
        return CF32Layer(self.n_in, self.hidden, self.proj, _ptr(self.Wx), _ptr(self.Wh),
                         _ptr(self.Wr), _ptr(self.bias))


def f32_layer(L: dict, device="cuda") -> F32Layer:
    """Device copy of one layer's float weights (Wx, Wh, b[, Wr])."""
    t = lambda a: torch.as_tensor(a, dtype=torch.float32).contiguous().to(device)
    Wr = None if L.get("Wr") is None else t(L["Wr"])
    Wx = t(L["Wx"])
    return F32Layer(Wx.shape[1], Wx.shape[0] // 4, 0 if Wr is None else Wr.shape[0], Wx,
                    t(L["Wh"]), Wr, t(L["b"]))


@dataclass
class F32Model:
    layers: list
    Wy: torch.Tensor
    by: torch.Tensor

    def cstruct(self):
        arr = (CF32Layer * len(self.layers))(*[L.cstruct() for L in self.layers])
        return CF32Model(len(self.layers), arr, self.Wy.shape[0], _ptr(self.Wy), _ptr(self.by)), arr


def f32_model(weights: dict, device="cuda") -> F32Model:
    t = lambda a: torch.as_tensor(a, dtype=torch.float32).contiguous().to(device)
    return F32Model([f32_layer(L, device) for L in weights["layers"]], t(weights["Wy"]),
                    t(weights["by"]))


def f32_lstm_layer_forward(L: F32Layer, x: torch.Tensor, h0=None, c0=None,
                           workspace: Workspace | None = None, check: bool = True):
    """x [T][B][in] fp32 (device) -> dict(h [T][B][R], hT, cT)."""
    x = x.contiguous()
    T, B, _ = x.shape
    dev = x.device
    lib = load()
    cl = L.cstruct()
    h = torch.empty(T, B, L.width, dtype=torch.float32, device=dev)
    hT = torch.empty(B, L.width, dtype=torch.float32, device=dev)
    cT = torch.empty(B, L.hidden, dtype=torch.float32, device=dev)
    ws = (workspace or Workspace()).get(lib.ql_f32_lstm_layer_workspace(C.byref(cl), T, B), dev)
    _check(lib.ql_f32_lstm_layer_forward(C.byref(cl), _ptr(x), T, B, _ptr(h0), _ptr(c0), _ptr(h),
                                         _ptr(hT), _ptr(cT), _ptr(ws), ws.numel(), _stream()),
           "ql_f32_lstm_layer_forward")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_f32_lstm_layer_forward")
    return dict(h=h, hT=hT, cT=cT)


def f32_acoustic_model_forward(M: F32Model, feats: torch.Tensor,
                               workspace: Workspace | None = None,
                               post: torch.Tensor | None = None, check: bool = True):
    """feats [T][B][in] fp32 (device) -> dict(post [T][B][states])."""
    feats = feats.contiguous()
    T, B, _ = feats.shape
    dev = feats.device
    lib = load()
    cm, keep = M.cstruct()
    S = M.Wy.shape[0]
    if post is None:
        post = torch.empty(T, B, S, dtype=torch.float32, device=dev)
    ws = (workspace or Workspace()).get(lib.ql_f32_acoustic_model_workspace(C.byref(cm), T, B), dev)
    _check(lib.ql_f32_acoustic_model_forward(C.byref(cm), _ptr(feats), T, B, _ptr(post), _ptr(ws),
                                             ws.numel(), _stream()),
           "ql_f32_acoustic_model_forward")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_f32_acoustic_model_forward")
    return dict(post=post)


# ------------------------------------------------- activation codes and stacks
@dataclass
class QAct:
    """Per-vector quantized rows: codes [rows][ld] (device layout), zero,
    inv_q, sums per row."""
    codes: torch.Tensor
    cols: int
    zero: torch.Tensor
    inv_q: torch.Tensor
    sums: torch.Tensor

    @staticmethod
    def empty(rows: int, cols: int, device) -> "QAct":
        return QAct(torch.zeros(rows, ld_for(cols), dtype=torch.int8, device=device), cols,
                    torch.empty(rows, dtype=torch.int32, device=device),
                    torch.empty(rows, dtype=torch.float32, device=device),
                    torch.empty(rows, dtype=torch.int32, device=device))

    def cstruct(self) -> CQAct:
        return CQAct(_ptr(self.codes), self.codes.shape[0], self.cols, self.codes.shape[1],
                     _ptr(self.zero), _ptr(self.inv_q), _ptr(self.sums))


def quantize_activations(X: torch.Tensor, out: QAct | None = None) -> QAct:
    """Each row of X [m][cols] quantized as its own vector (eq. 2)."""
    X = X.contiguous()
    m, cols = X.shape
    q = out or QAct.empty(m, cols, X.device)
    cq = q.cstruct()
    _check(load().ql_quantize_activations(_ptr(X), m, cols, C.byref(cq), _stream()),
           "ql_quantize_activations")
    return q


def lstm_stack_forward(layers: list, x: QAct, T: int, B: int, want_h: bool = False,
                       outs: list | None = None, workspace: Workspace | None = None,
                       check: bool = True, taps=False, state_in=None, state_out=None):
    """n stacked layers (no projection and one width, or all projected at
    B = 1) in one launch from input codes x (T*B rows) -> dict(codes=[QAct per
    layer], h=[T][B][R] of the last[, layers=per-layer taps]).  state_in /
    state_out: per-layer [(h, c)] (must not share memory)."""
    lib = load()
    n = len(layers)
    dev = x.codes.device
    arr = (CLayer * n)(*[L.cstruct() for L in layers])
    outs = outs or [QAct.empty(T * B, L.width, dev) for L in layers]
    oarr = (CQAct * n)(*[o.cstruct() for o in outs])
    h = torch.empty(T, B, layers[-1].width, dtype=torch.float32, device=dev) if want_h else None
    nbytes = lib.ql_lstm_stack_workspace(arr, n, T, B)
    ws = (workspace or Workspace()).get(nbytes, dev)
    cx = x.cstruct()
    res = dict(codes=outs, h=h)
    tarr = None
    if taps:
        lt = []
        tarr = (CTaps * n)()
        for i, L in enumerate(layers):
            t, ct = _taps(T, B, L, dev, taps)
            lt.append(t)
            tarr[i] = ct
        res["layers"] = lt
    _check(lib.ql_lstm_stack_forward(arr, n, C.byref(cx), T, B, oarr, _ptr(h),
                                     _state_array(state_in), _state_array(state_out), tarr,
                                     _ptr(ws), ws.numel(), _stream()), "ql_lstm_stack_forward")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_lstm_stack_forward")
    return res


def stack_layers_per_launch(M: Model, T: int, B: int) -> int:
    """How many of M's layers one wavefront launch holds (1: none; the model
    forward then runs one layer per launch)."""
    arr = (CLayer * len(M.layers))(*[L.cstruct() for L in M.layers])
    return int(load().ql_lstm_stack_layers_per_launch(arr, len(M.layers), T, B))


def recurrence_layout(L: Layer, B: int) -> int:
    """1 when L's recurrence at batch B runs with each XCD holding an eighth of
    the batch (layers with a projection on the whole chip), else 0."""
    c = L.cstruct()
    return int(load().ql_debug_recurrence_layout(C.byref(c), B))


def stack_layout(M: Model, T: int, B: int) -> int:
    """1 when the first wavefront launch over M's layers runs with one XCD per
    layer (batch 16 to 64 on the whole chip), else 0."""
    arr = (CLayer * len(M.layers))(*[L.cstruct() for L in M.layers])
    return int(load().ql_debug_stack_layout(arr, len(M.layers), T, B))


# ------------------------------------------- quantization-aware training step
def train_params(weights: dict, device="cuda") -> dict:
    """Device fp32 copies of a model's float parameters (layers without
    projection): {'layers': [{'Wx','Wh','b'}], 'Wy', 'by'}."""
    t = lambda a: torch.as_tensor(a, dtype=torch.float32).to(device).contiguous().clone()
    return {"layers": [{k: t(L[k]) for k in ("Wx", "Wh", "b")} for L in weights["layers"]],
            "Wy": t(weights["Wy"]), "by": t(weights["by"])}


def _train_struct(P: dict):
    arr = (CTrainLayer * len(P["layers"]))(*[
        CTrainLayer(L["Wx"].shape[1], L["Wx"].shape[0] // 4, 0, _ptr(L["Wx"]), _ptr(L["Wh"]),
                    None, _ptr(L["b"])) for L in P["layers"]])
    return CTrainModel(len(P["layers"]), arr, P["Wy"].shape[0], _ptr(P["Wy"]), _ptr(P["by"])), arr


def train_step(P: dict, feats: torch.Tensor, targets: torch.Tensor, lr: float,
               gate_blocks: int = 4, quantize_output: bool = True, grads: dict | None = None,
               workspace: Workspace | None = None, check: bool = True):
    """One quantization-aware SGD step (ql_train_step) on device parameters P
    (updated in place) -> (loss tensor [1], grads dict of P's shapes)."""
    feats = feats.contiguous()
    targets = targets.to(torch.int32).contiguous()
    T, B, _ = feats.shape
    dev = feats.device
    lib = load()
    if grads is None:
        grads = {"layers": [{k: torch.empty_like(v) for k, v in L.items()} for L in P["layers"]],
                 "Wy": torch.empty_like(P["Wy"]), "by": torch.empty_like(P["by"])}
    cm, keep1 = _train_struct(P)
    cg, keep2 = _train_struct(grads)
    ws = (workspace or Workspace()).get(lib.ql_train_step_workspace(C.byref(cm), T, B,
                                                                    gate_blocks), dev)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    _check(lib.ql_train_step(C.byref(cm), _ptr(feats), _ptr(targets), T, B, float(lr), gate_blocks,
                             int(bool(quantize_output)), _ptr(loss), C.byref(cg), _ptr(ws),
                             ws.numel(), _stream()), "ql_train_step")
    if check:
        _check(lib.ql_workspace_status(_ptr(ws), _stream()), "ql_train_step")
    return loss, grads
