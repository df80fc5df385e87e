"""The quantization-aware training step on the GPU (ql_train_step; Section
3.2, Algorithm 1) against the oracle's (oracle_train_step): the loss, every
gradient and every updated parameter.

Tolerance: the forward pass is the inference path and bit-exact with the
oracle's; the backward pass sums in fp32 on the GPU (MFMA products, split
sums) and in fp64 in the oracle, over up to T*B frames and 4H gate rows, so
each gradient is held to 1e-4 of its largest element (observed errors are
around 1e-6 of it; a missing or wrong term moves a gradient by far more), the
loss to 1e-5 relative, and the update of the GPU's own parameters is checked
bit for bit as w - lr g of its own gradient."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

GRAD_RTOL = 1e-4


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


def _compare(ql, orc, w, x, y, lr, gate_blocks=4, quantize_output=True):
    P = ql.train_params(w)
    before = {"layers": [{k: v.clone() for k, v in L.items()} for L in P["layers"]],
              "Wy": P["Wy"].clone(), "by": P["by"].clone()}
    loss, g = ql.train_step(P, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), lr,
                            gate_blocks=gate_blocks, quantize_output=quantize_output)
    new_o, g_o, loss_o = orc.train_step(w, x, y, lr, gate_blocks=gate_blocks,
                                        quantize_output=quantize_output)
    assert abs(loss.item() - loss_o) <= 1e-5 * abs(loss_o), (loss.item(), loss_o)
    pairs = [("Wy", g["Wy"], g_o["Wy"], P["Wy"], before["Wy"]),
             ("by", g["by"], g_o["by"], P["by"], before["by"])]
    for l in range(len(w["layers"])):
        for k in ("Wx", "Wh", "b"):
            pairs.append((f"layer {l} {k}", g["layers"][l][k], g_o["layers"][l][k],
                          P["layers"][l][k], before["layers"][l][k]))
    lr32 = np.float32(lr)
    worst = 0.0
    for name, gg, go, pn, pb in pairs:
        gn = gg.cpu().numpy()
        scale = float(np.max(np.abs(go)))
        assert scale > 0, name
        err = float(np.max(np.abs(gn.astype(np.float64) - go))) / scale
        worst = max(worst, err)
        assert err <= GRAD_RTOL, (name, err)
        # the GPU's update of its own parameters: w - lr g, bit for bit
        assert np.array_equal(pn.cpu().numpy(), pb.cpu().numpy() - lr32 * gn), name
    return worst


def _case(in_, H, layers, S, T, B, seed):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(in_, H, layers, states=S, seed=seed)
    rng = np.random.default_rng(seed + 1)
    x = rng.standard_normal((T, B, in_)).astype(np.float32)
    y = rng.integers(0, S, (T, B)).astype(np.int32)
    return w, x, y


@pytest.mark.parametrize("layers,B", [(3, 1), (3, 5), (3, 20), (1, 3), (2, 37)])
@pytest.mark.parametrize("quantize_output", [True, False])
def test_train_step_equals_oracle(ql, orc, layers, B, quantize_output):
    """One row per tile (B = 1, 5), 16-row tiles (B = 20, 37: a ragged last
    slice), one layer per launch (1 layer); 'quant-all' and 'quant'."""
    w, x, y = _case(40, 48, layers, 96, 13, B, seed=layers * 100 + B)
    _compare(ql, orc, w, x, y, lr=0.5, quantize_output=quantize_output)


def test_train_step_per_row_weight_blocks(ql, orc):
    w, x, y = _case(24, 32, 2, 50, 9, 4, seed=5)
    _compare(ql, orc, w, x, y, lr=0.3, gate_blocks=128)


def test_train_step_5x500_softmax8192_B64(ql, orc):
    """The 5 x 500 model with the 8192-way softmax at batch 64 on a short
    mini-batch (T = 12): every gradient against the oracle."""
    from paper_1607_04683_amd.workloads import LSTM5x500_S8192_T1000_B64 as W_, features, model_weights
    w = model_weights(W_)[0]
    x = np.ascontiguousarray(features(W_)[:12])
    y = np.random.default_rng(0).integers(0, 8192, (12, 64)).astype(np.int32)
    _compare(ql, orc, w, x, y, lr=1.0)


@pytest.mark.parametrize("H,B", [(500, 64), (128, 64), (48, 20)])
def test_train_step_repeats_bit_for_bit(ql, H, B):
    """The same step on the same inputs gives the same gradients, bit for bit,
    every time: the backward recurrence and the products sum in fixed orders,
    so a difference means some value was read before it was final.  At 500
    cells and batch 64 every CU of the chip holds a backward tile."""
    w, x, y = _case(40, H, 1, 96, 12, B, seed=H + B)
    x, y = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    _, ref = ql.train_step(ql.train_params(w), x, y, 1.0)
    for _ in range(4):
        _, g = ql.train_step(ql.train_params(w), x, y, 1.0)
        for k in ("Wx", "Wh", "b"):
            assert torch.equal(g["layers"][0][k], ref["layers"][0][k]), k
        assert torch.equal(g["Wy"], ref["Wy"]) and torch.equal(g["by"], ref["by"])


def test_train_steps_lower_the_loss(ql, orc):
    """Repeated quantization-aware steps on one mini-batch (targets a function
    of the current frame) lower its loss at every step, as the oracle's
    steps do."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 64, 2, states=4, seed=9)
    x = np.random.default_rng(10).standard_normal((30, 16, 40)).astype(np.float32)
    y = ((x[..., 0] > 0).astype(np.int32) + 2 * (x[..., 1] > 0)).astype(np.int32)
    P = ql.train_params(w)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    losses = [ql.train_step(P, xd, yd, 5.0)[0].item() for _ in range(10)]
    assert all(b < a for a, b in zip(losses, losses[1:])), losses
    assert losses[-1] < losses[0] - 0.005, losses
    wo, ref = w, []
    for _ in range(10):
        wo, _, l = orc.train_step(wo, x, y, 5.0)
        ref.append(l)
    assert np.max(np.abs(np.array(losses) - ref)) < 1e-4, (losses, ref)


def test_train_step_rejects_projection_layers(ql):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(8, 16, 1, proj=4, states=5, seed=1)
    cm = ql.CTrainModel(1, (ql.CTrainLayer * 1)(ql.CTrainLayer(8, 16, 4, 1, 1, 1, 1)), 5, 1, 1)
    assert ql.load().ql_train_step_workspace(cm, 3, 2, 4) == 0
