"""Seeded synthetic workloads shaped like the paper's embedded LSTM acoustic models.

This module only draws random numbers and fixes shapes; it contains none of
the quantization or LSTM arithmetic.  Both the GPU library's tests/benchmark
and the CPU oracle take their inputs from here.

Shapes follow Section 4 of the paper (Alvarez, Prabhavalkar, Bakhtin,
Interspeech 2016): 40-dim log-mel frames every 10 ms, 8 consecutive frames
stacked (7 frames of right context) into a 320-dim vector, and only every
third stacked frame presented to the network; 4-5 LSTM layers of N cells,
optionally with a linear projection of P units after each layer, and a
softmax output layer.  The paper's speech data is not available, so inputs
are standard-normal "features" with the same stacking/overlap structure and
weights are uniform or normal with the stated spread.

Draw order (one numpy PCG64 generator per workload, float64 draws cast to
fp32): for each layer W_x, W_h, b, [W_r]; then W_y, b_y; then the features,
utterance by utterance.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class LSTMModelShape:
    """Architecture of a stacked (projected) LSTM acoustic model."""

    n_in: int                 # stacked feature width (8 x frame dim)
    hidden: int               # LSTM cells per layer (N)
    layers: int
    proj: int = 0             # projection units P (0 = no projection)
    states: int = 0           # softmax output states (0 = no output layer)
    frame_dim: int = 40       # base log-mel frame width
    stack: int = 8            # frames stacked per input vector
    skip: int = 3             # present every `skip`-th stacked frame

    def layer_dims(self):
        """[(in, hidden, proj)] per layer; W_x is 4N x in, W_h is 4N x (P or N)."""
        dims = []
        width = self.n_in
        for _ in range(self.layers):
            dims.append((width, self.hidden, self.proj))
            width = self.proj if self.proj else self.hidden
        return dims

    @property
    def out_width(self) -> int:
        return self.proj if self.proj else self.hidden

    def param_count(self, include_output: bool = False) -> int:
        """Weights + biases (no peepholes), optionally with the output layer."""
        n = 0
        for (i, h, p) in self.layer_dims():
            r = p if p else h
            n += 4 * h * i + 4 * h * r + 4 * h + (p * h if p else 0)
        if include_output and self.states:
            n += self.states * self.out_width + self.states
        return n


@dataclass(frozen=True)
class Workload:
    name: str
    model: LSTMModelShape | None
    T: int = 0
    B: int = 0
    dist: str = "uniform"     # weight distribution: "uniform" (+-scale) or "normal" (std=scale)
    scale: float = 0.08
    seed: int = 0
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def frames(self) -> int:
        return self.T * self.B


# The five evaluation workloads.  Index 0 is the small standalone quantized
# matmul, 1-4 are LSTM models of increasing size.
QMATMUL_16x128x256 = Workload(
    name="qmatmul W256x128 X16x128 per-tensor", model=None, seed=0,
    extra=dict(rows=256, cols=128, m=16, w_std=0.1, x_lo=-1.0, x_hi=1.0),
)
LSTM1x500_T300_B1 = Workload(
    name="1xLSTM500 in320 T300 B1",
    model=LSTMModelShape(n_in=320, hidden=500, layers=1),
    T=300, B=1, dist="uniform", scale=0.08, seed=0)
LSTM5x500_S8192_T500_B1 = Workload(
    name="5xLSTM500 + softmax8192, T500 B1",
    model=LSTMModelShape(n_in=320, hidden=500, layers=5, states=8192),
    T=500, B=1, dist="uniform", scale=0.08, seed=0)
LSTM5x500_S8192_T1000_B64 = Workload(
    name="5xLSTM500 + softmax8192, T1000 B64",
    model=LSTMModelShape(n_in=320, hidden=500, layers=5, states=8192),
    T=1000, B=64, dist="uniform", scale=0.08, seed=0)
LSTMP4x2048P512_S16384_T800_B256 = Workload(
    name="4xLSTMP2048/P512 in640 + softmax16384, T800 B256",
    model=LSTMModelShape(n_in=640, hidden=2048, layers=4, proj=512, states=16384,
                         frame_dim=80),
    T=800, B=256, dist="normal", scale=0.02, seed=0)
GEMM_SWEEP = (4096, 8192)

WORKLOADS = [QMATMUL_16x128x256, LSTM1x500_T300_B1, LSTM5x500_S8192_T500_B1,
             LSTM5x500_S8192_T1000_B64, LSTMP4x2048P512_S16384_T800_B256]


def _draw(rng: np.random.Generator, shape, dist: str, scale: float) -> np.ndarray:
    if dist == "uniform":
        a = rng.uniform(-scale, scale, size=shape)
    elif dist == "normal":
        a = rng.normal(0.0, scale, size=shape)
    else:
        raise ValueError(dist)
    return a.astype(np.float32)


def model_weights(w: Workload):
    """Float weights {'layers': [{'Wx','Wh','b','Wr'}], 'Wy', 'by'} and the rng
    positioned after the weight draws (features are drawn from it next)."""
    m = w.model
    rng = np.random.Generator(np.random.PCG64(w.seed))
    layers = []
    for (i, h, p) in m.layer_dims():
        r = p if p else h
        L = {"Wx": _draw(rng, (4 * h, i), w.dist, w.scale),
             "Wh": _draw(rng, (4 * h, r), w.dist, w.scale),
             "b": _draw(rng, (4 * h,), w.dist, w.scale)}
        L["Wr"] = _draw(rng, (p, h), w.dist, w.scale) if p else None
        layers.append(L)
    out = {"layers": layers, "Wy": None, "by": None}
    if m.states:
        out["Wy"] = _draw(rng, (m.states, m.out_width), w.dist, w.scale)
        out["by"] = _draw(rng, (m.states,), w.dist, w.scale)
    return out, rng


def stacked_features(rng: np.random.Generator, T: int, B: int, frame_dim: int = 40,
                     stack: int = 8, skip: int = 3, utterances=None) -> np.ndarray:
    """[T][B][stack*frame_dim] fp32.  Per utterance, base frames f_j ~ N(0,1)
    (j = 0 .. skip*(T-1)+stack-1); input t is concat(f_{skip t}, ..., f_{skip t+stack-1}),
    so consecutive inputs share stack-skip base frames, as with the paper's
    frontend.  `utterances` (optional) keeps only those batch entries (the draws
    for all B utterances are still made, in order, so a subset is identical to
    the same slice of the full tensor)."""
    nbase = skip * (T - 1) + stack if T > 0 else 0
    keep = list(range(B)) if utterances is None else list(utterances)
    out = np.empty((T, len(keep), stack * frame_dim), dtype=np.float32)
    slot = {b: k for k, b in enumerate(keep)}
    for b in range(B):
        base = rng.standard_normal((nbase, frame_dim))
        if b not in slot:
            continue
        idx = skip * np.arange(T)[:, None] + np.arange(stack)[None, :]
        out[:, slot[b], :] = base[idx].reshape(T, stack * frame_dim).astype(np.float32)
    return out


def base_frames(rng: np.random.Generator, T: int, B: int, frame_dim: int = 40, stack: int = 8,
                skip: int = 3, utterances=None) -> np.ndarray:
    """The base frames behind stacked_features, time-major [nbase][B][frame_dim]
    fp32 with nbase = skip*(T-1)+stack: the same draws, in the same order, before
    any stacking (the input of the fused frontend)."""
    nbase = skip * (T - 1) + stack if T > 0 else 0
    keep = list(range(B)) if utterances is None else list(utterances)
    out = np.empty((nbase, len(keep), frame_dim), dtype=np.float32)
    slot = {b: k for k, b in enumerate(keep)}
    for b in range(B):
        base = rng.standard_normal((nbase, frame_dim))
        if b in slot:
            out[:, slot[b], :] = base.astype(np.float32)
    return out


def frames(w: Workload, utterances=None) -> np.ndarray:
    _, rng = model_weights(w)
    m = w.model
    return base_frames(rng, w.T, w.B, m.frame_dim, m.stack, m.skip, utterances)


def features(w: Workload, utterances=None) -> np.ndarray:
    _, rng = model_weights(w)
    m = w.model
    return stacked_features(rng, w.T, w.B, m.frame_dim, m.stack, m.skip, utterances)


def frame_targets(w: Workload, seed: int = 1) -> np.ndarray:
    """Synthetic frame-level state targets [T][B] (int32, uniform over the
    output states) for a training mini-batch of workload w: the paper's
    alignments need its transcribed data, and a training step's work does not
    depend on the label values."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, w.model.states, size=(w.T, w.B)).astype(np.int32)


def qmatmul_operands(w: Workload = QMATMUL_16x128x256):
    """(W [rows][cols], X [m][cols]) fp32: W ~ N(0, 0.1), X ~ U[-1, 1]."""
    e = w.extra
    rng = np.random.Generator(np.random.PCG64(w.seed))
    W = rng.normal(0.0, e["w_std"], size=(e["rows"], e["cols"])).astype(np.float32)
    X = rng.uniform(e["x_lo"], e["x_hi"], size=(e["m"], e["cols"])).astype(np.float32)
    return W, X


def gemm_operands(M: int, N: int, K: int, seed: int = 0):
    """(A [M][K], B [N][K]) uint8 ~ U{0..255}."""
    rng = np.random.Generator(np.random.PCG64(seed))
    A = rng.integers(0, 256, size=(M, K), dtype=np.uint8)
    B = rng.integers(0, 256, size=(N, K), dtype=np.uint8)
    return A, B


def random_model(n_in: int, hidden: int, layers: int, proj: int = 0, states: int = 0,
                 seed: int = 0, dist: str = "uniform", scale: float = 0.08):
    """Weights for an arbitrary small model (tests)."""
    w = Workload(name="custom", model=LSTMModelShape(n_in=n_in, hidden=hidden,
                 layers=layers, proj=proj, states=states), dist=dist, scale=scale,
                 seed=seed)
    return model_weights(w)[0]
