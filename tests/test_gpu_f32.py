"""The unquantized fp32 model path against the oracle's float model.

The GPU accumulates products in fp32 (MFMA), the oracle in fp64, so results
agree to rounding rather than bit for bit: the bar is 1e-4 absolute on h, the
final state and the posteriors.  The GEMM alone is held to the standard
worst-case bound of fp32 summation, K * 2^-24 * sum_k |x_k w_k|."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


def dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("m,rows,cols", [(1, 1, 1), (5, 33, 7), (130, 257, 129), (300, 2000, 320),
                                         (64, 8192, 500), (129, 130, 1023)])
def test_f32_matmul(ql, m, rows, cols):
    rng = np.random.default_rng(m + rows + cols)
    W = rng.normal(0, 0.05, (rows, cols)).astype(np.float32)
    X = rng.standard_normal((m, cols)).astype(np.float32)
    b = rng.normal(0, 0.1, rows).astype(np.float32)
    Y = ql.f32_matmul(dev(W), dev(X), dev(b)).cpu().numpy().astype(np.float64)
    ref = X.astype(np.float64) @ W.astype(np.float64).T + b
    mag = np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T + np.abs(b)
    bound = (cols + 2) * 2.0 ** -24 * mag
    assert np.all(np.abs(Y - ref) <= bound)


def _layer(ql, orc, n_in, H, P, T, B, seed, h0c0=False):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(n_in, H, 1, proj=P, seed=seed)["layers"][0]
    rng = np.random.default_rng(seed + 7)
    x = rng.standard_normal((T, B, n_in)).astype(np.float32)
    R = P if P else H
    h0 = c0 = None
    if h0c0:
        h0 = (np.tanh(rng.standard_normal((B, R))) * 0.5).astype(np.float32)
        c0 = rng.standard_normal((B, H)).astype(np.float32)
    g = ql.f32_lstm_layer_forward(ql.f32_layer(w), dev(x), dev(h0), dev(c0))
    o = orc.lstm_layer_forward_f32(w, x, h0, c0)
    for k in ("h", "hT", "cT"):
        assert np.max(np.abs(g[k].cpu().numpy() - o[k])) <= TOL, k


@pytest.mark.parametrize("n_in,H,P,T,B,h0c0", [
    (40, 37, 0, 7, 3, False),        # one batch row per tile, ragged units
    (320, 500, 0, 40, 64, True),     # 16-row MFMA tiles, W_h slice in LDS
    (64, 96, 32, 12, 20, True),      # projection, MFMA, ragged batch slice
    (48, 64, 16, 9, 2, False),       # projection, one batch row per tile
    (640, 2048, 512, 3, 16, False),  # the LSTMP layer's shapes
    (64, 2048, 512, 2, 256, False),  # batch 256: W_h slice read from L2
])
def test_f32_layer_shapes(ql, orc, n_in, H, P, T, B, h0c0):
    _layer(ql, orc, n_in, H, P, T, B, seed=n_in + H + P + B, h0c0=h0c0)


def test_f32_layer_500_T300_B1(ql, orc):
    """One 500-cell layer, 320-dim stacked features, T = 300, batch 1."""
    from paper_1607_04683_amd import workloads as wl
    w, _ = wl.model_weights(wl.LSTM1x500_T300_B1)
    x = wl.features(wl.LSTM1x500_T300_B1)
    L = w["layers"][0]
    g = ql.f32_lstm_layer_forward(ql.f32_layer(L), dev(x))
    o = orc.lstm_layer_forward_f32(L, x)
    for k in ("h", "hT", "cT"):
        assert np.max(np.abs(g[k].cpu().numpy() - o[k])) <= TOL, k


def test_f32_model_small(ql, orc):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 48, 2, states=100, seed=3)
    x = np.random.default_rng(4).standard_normal((11, 5, 40)).astype(np.float32)
    g = ql.f32_acoustic_model_forward(ql.f32_model(w), dev(x))["post"].cpu().numpy()
    o = orc.acoustic_model_forward_f32(w, x)["post"]
    assert np.max(np.abs(g - o)) <= TOL
    assert np.allclose(g.sum(-1), 1.0, atol=1e-5)


def test_f32_model_5x500_B1(ql, orc):
    """The 5-layer 500-cell model with the 8192-way softmax, T = 500, batch 1."""
    from paper_1607_04683_amd import workloads as wl
    W = wl.LSTM5x500_S8192_T500_B1
    w, _ = wl.model_weights(W)
    x = wl.features(W)
    g = ql.f32_acoustic_model_forward(ql.f32_model(w), dev(x))["post"].cpu().numpy()
    o = orc.acoustic_model_forward_f32(w, x)["post"]
    assert np.max(np.abs(g - o)) <= TOL


def test_f32_model_B64_sampled_utterance(ql, orc):
    """Batch 64 x T = 1000 on the GPU; utterance 45 against the oracle
    (utterances are independent)."""
    from paper_1607_04683_amd import workloads as wl
    W = wl.LSTM5x500_S8192_T1000_B64
    w, _ = wl.model_weights(W)
    x = wl.features(W)
    g = ql.f32_acoustic_model_forward(ql.f32_model(w), dev(x))["post"][:, 45].cpu().numpy()
    o = orc.acoustic_model_forward_f32(w, x[:, 45:46])["post"][:, 0]
    assert np.max(np.abs(g - o)) <= TOL
