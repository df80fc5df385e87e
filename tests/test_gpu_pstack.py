"""Stacked projection layers at one batch row in one wavefront launch (the
5 x 500 / P models of Section 4 streamed frame by frame): every layer's input,
recurrent and projection int32 sums, codes, row params and fp32 h bit-exact
and posteriors within 1e-4 of the oracle."""
import numpy as np
import pytest
import torch
from model_parity import assert_model_taps

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


def u8(t):
    return t.cpu().numpy().view(np.uint8) ^ 0x80


def _weights(n_in, dims, states, seed):
    """Layers of different widths: dims = [(H, P), ...], layer k's input = P of k-1."""
    from paper_1607_04683_amd.workloads import random_model
    layers = []
    width = n_in
    for k, (H, P) in enumerate(dims):
        layers.append(random_model(width, H, 1, proj=P, seed=seed + k)["layers"][0])
        width = P
    rng = np.random.default_rng(seed + 99)
    return {"layers": layers,
            "Wy": rng.uniform(-0.08, 0.08, (states, width)).astype(np.float32),
            "by": rng.uniform(-0.08, 0.08, states).astype(np.float32)}


def _case(ql, orc, w, T, seed, gate_blocks=4, proj_blocks=1):
    x = np.random.default_rng(seed).standard_normal((T, 1, w["layers"][0]["Wx"].shape[1]))
    x = x.astype(np.float32)
    Mg = ql.quantize_model(w, gate_blocks=gate_blocks, proj_blocks=proj_blocks)
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=True)
    o = orc.acoustic_model_forward(orc.quantize_model(w, gate_blocks, proj_blocks), x, taps=True)
    assert_model_taps(g, o)
    return Mg, x, g


@pytest.mark.parametrize("dims,T", [
    ([(500, 100)] * 5, 60),                     # Table 1 shapes
    ([(500, 400)] * 5, 30),
    ([(64, 24), (40, 30), (64, 5)], 25),        # mixed widths; 5 outputs over 4 tiles
    ([(48, 16)] * 9, 12),                       # two launches (at most 8 layers in one)
    ([(500, 200)] * 2, 1),                      # one frame
])
def test_projection_wavefront(ql, orc, dims, T):
    w = _weights(320, dims, 300, seed=len(dims) * 10 + T)
    Mg, x, g = _case(ql, orc, w, T, seed=T)
    assert ql.stack_layers_per_launch(Mg, T, 1) >= 2


def test_projection_wavefront_row_blocks(ql, orc):
    w = _weights(320, [(100, 40)] * 3, 200, seed=3)
    _case(ql, orc, w, 20, seed=4, gate_blocks=400, proj_blocks=40)


def test_projection_wavefront_equals_one_layer_path(ql):
    """The wavefront and one launch per layer (ql_lstm_layer_forward chained on
    each layer's fp32 h) give the same sums, codes and h, bit for bit; taps
    cost the wavefront nothing but the stores."""
    w = _weights(320, [(500, 200)] * 5, 8192, seed=7)
    x = torch.from_numpy(np.random.default_rng(9).standard_normal((50, 1, 320)).astype(np.float32))
    Mg = ql.quantize_model(w)
    a = ql.acoustic_model_forward(Mg, x.cuda(), taps=("h_codes",))
    b = ql.acoustic_model_forward(Mg, x.cuda(), taps=True)
    assert torch.equal(a["post"], b["post"])
    cur = x.cuda()
    for l in range(5):
        assert torch.equal(a["layers"][l]["h_codes"], b["layers"][l]["h_codes"])
        one = ql.lstm_layer_forward(Mg.layers[l], cur, taps=True)
        for k in ("acc_x", "acc_h", "acc_r", "h_codes", "h_zero", "h_inv_q"):
            assert torch.equal(one[k], b["layers"][l][k]), (l, k)
        assert torch.equal(one["h"], b["layers"][l]["h"]), l
        cur = one["h"]


def test_projection_wavefront_empty(ql):
    w = _weights(16, [(24, 8)] * 2, 10, seed=1)
    Mg = ql.quantize_model(w)
    g = ql.acoustic_model_forward(Mg, torch.zeros(0, 1, 16, device="cuda"))
    assert g["post"].shape == (0, 1, 10)


def test_lstm_stack_forward_entry_projection(ql, orc):
    """ql_lstm_stack_forward with projection layers at batch 1: every layer's
    codes and row params and the last layer's fp32 h equal the oracle's
    layer-by-layer evaluation."""
    T = 13
    w = _weights(40, [(48, 20), (36, 28), (48, 12)], 10, seed=5)
    x = np.random.default_rng(2).standard_normal((T, 1, 40)).astype(np.float32)
    layers = [ql.quantize_layer(L) for L in w["layers"]]
    xq = ql.quantize_activations(torch.from_numpy(x.reshape(T, 40)).cuda())
    rng = np.random.default_rng(6)
    dims = [(48, 20), (36, 28), (48, 12)]
    h0 = [(np.tanh(rng.standard_normal((1, P))) * 0.6).astype(np.float32) for _, P in dims]
    c0 = [rng.standard_normal((1, H)).astype(np.float32) for H, _ in dims]
    s_in = [(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()) for a, b in zip(h0, c0)]
    s_out = [(torch.empty(1, P, device="cuda"), torch.empty(1, H, device="cuda")) for H, P in dims]
    g = ql.lstm_stack_forward(layers, xq, T, 1, want_h=True, taps=True, state_in=s_in,
                              state_out=s_out)
    cur = x
    for k, (L, P) in enumerate(zip(w["layers"], (20, 28, 12))):
        o = orc.lstm_layer_forward(orc.quantize_layer(L), cur, h0[k], c0[k], taps=True)
        got = u8(g["codes"][k].codes)[:, :P].reshape(T, 1, P)
        assert np.array_equal(got, o["h_codes"]), f"layer {k}"
        assert np.array_equal(g["codes"][k].zero.cpu().numpy().reshape(T, 1), o["h_zero"])
        assert np.array_equal(g["codes"][k].inv_q.cpu().numpy().reshape(T, 1), o["h_inv_q"])
        for name in ("acc_x", "acc_h", "acc_r", "h"):
            assert np.array_equal(g["layers"][k][name].cpu().numpy(), o[name]), f"layer {k} {name}"
        assert np.array_equal(s_out[k][0].cpu().numpy(), o["hT"]), f"layer {k} hT"
        assert np.array_equal(s_out[k][1].cpu().numpy(), o["cT"]), f"layer {k} cT"
        cur = o["h"]
    assert np.array_equal(g["h"].cpu().numpy(), cur)
    # batched projection layers are not taken by this entry point
    xb = ql.quantize_activations(torch.zeros(T * 2, 40, device="cuda"))
    with pytest.raises(ql.QLError):
        ql.lstm_stack_forward(layers, xb, T, 2)


@pytest.mark.parametrize("P", [100, 400])
def test_projection_wavefront_table1_full_size(ql, orc, P):
    """The bench's Table 1 configuration: 5 x 500 cells with P projections and
    an 8192-way softmax, one utterance of T = 500 presented frames (seed 0)."""
    from paper_1607_04683_amd.workloads import random_model, stacked_features
    T = 500
    w = random_model(320, 500, 5, proj=P, states=8192, seed=0)
    x = stacked_features(np.random.Generator(np.random.PCG64(0)), T, 1)
    Mg = ql.quantize_model(w)
    assert ql.stack_layers_per_launch(Mg, T, 1) == 5
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=True)
    o = orc.acoustic_model_forward(orc.quantize_model(w), x, taps=True)
    assert_model_taps(g, o)
