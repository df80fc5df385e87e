"""Quantization granularity (Section 3.1): weight matrices quantized per matrix,
per gate block, in sub-matrices of whole rows, or per row, through every GPU
path (quantizer, hoisted and large-tile products, the one-layer recurrence with
and without projection in both exchange modes, the layer wavefront, the
softmax layer), bit-exact against the oracle quantized the same way."""
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


def np_(t):
    return t.cpu().numpy()


def u8(t):
    return np_(t).view(np.uint8) ^ 0x80


@pytest.mark.parametrize("rows,cols,nblocks", [(2000, 320, 2000), (2000, 500, 40), (512, 2048, 512),
                                               (8192, 500, 8192), (7, 3, 7)])
def test_quantize_row_blocks(ql, orc, rows, cols, nblocks):
    """Every block its own set: per-block params and codes bit-exact, and each
    block's extremes land on codes 0 and 255."""
    rng = np.random.default_rng(rows + cols + nblocks)
    W = rng.uniform(-0.08, 0.08, (rows, cols)).astype(np.float32)
    W *= rng.uniform(0.1, 3.0, (rows, 1)).astype(np.float32)    # rows of different ranges
    q = ql.quantize(torch.from_numpy(W).cuda(), nblocks)
    o = orc.quantize(W, nblocks)
    got = u8(q.codes)[:, :cols]
    assert np.array_equal(got, o.codes)
    assert np.array_equal(np_(q.zero), o.zero)
    assert np.array_equal(np_(q.inv_q).view(np.uint32), o.inv_q.view(np.uint32))
    assert np.array_equal(np_(q.row_sums), o.codes.astype(np.int64).sum(1))
    blk = got.reshape(nblocks, -1)
    assert (blk.min(1) == 0).all() and (blk.max(1) == 255).all()


@pytest.mark.parametrize("nblocks", [4100, 20])
def test_qmatmul_large_tiles_row_blocks(ql, orc, nblocks):
    """256x256 tiles whose columns carry different zero points and factors."""
    m, rows, cols = 4096, 4100, 320
    rng = np.random.default_rng(nblocks)
    W = (rng.normal(0, 0.05, (rows, cols)) * rng.uniform(0.2, 2.0, (rows, 1))).astype(np.float32)
    X = rng.standard_normal((m, cols)).astype(np.float32)
    bias = rng.normal(0, 0.1, rows).astype(np.float32)
    q = ql.quantize(torch.from_numpy(W).cuda(), nblocks)
    Y, acc = ql.quantized_matmul(q, torch.from_numpy(X).cuda(), 1, torch.from_numpy(bias).cuda(),
                                 want_acc=True)
    sel = np.unique(np.concatenate([[0, 255, 256, m - 1], rng.choice(m, 16, replace=False)]))
    o = orc.quantized_matmul(orc.quantize(W, nblocks), X[sel], act_gran=1, bias=bias)
    idx = torch.from_numpy(sel).cuda()
    assert np.array_equal(acc[idx].cpu().numpy(), o["acc"])
    assert np.array_equal(Y[idx].cpu().numpy().view(np.uint32), o["Y"].view(np.uint32))


@pytest.mark.parametrize("P,gate_blocks,proj_blocks", [(0, 160, 1), (0, 20, 1), (24, 160, 24),
                                                       (24, 1, 4), (24, 4, 1)])
@pytest.mark.parametrize("B", [1, 20])
def test_layer_granularity(ql, orc, P, gate_blocks, proj_blocks, B):
    """One 40-cell layer (gate rows 160), T = 9, free-running: accumulators,
    codes of h and the fp32 h, c bit-exact."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(33, 40, 1, proj=P, seed=gate_blocks + proj_blocks)["layers"][0]
    w["Wh"] = w["Wh"] * np.linspace(0.3, 2.0, w["Wh"].shape[0], dtype=np.float32)[:, None]
    x = np.random.default_rng(B).standard_normal((9, B, 33)).astype(np.float32)
    L = ql.quantize_layer(w, gate_blocks=gate_blocks, proj_blocks=proj_blocks)
    g = ql.lstm_layer_forward(L, torch.from_numpy(x).cuda(), taps=True)
    o = orc.lstm_layer_forward(orc.quantize_layer(w, gate_blocks, proj_blocks), x, taps=True)
    for k in ("acc_x", "acc_h") + (("acc_r",) if P else ()):
        assert np.array_equal(np_(g[k]), o[k]), k
    assert np.array_equal(u8(g["h_codes"]), o["h_codes"])
    for k in ("h", "hT", "cT"):
        assert np.array_equal(np_(g[k]), o[k]), k


@pytest.mark.parametrize("B", [1, 20])
def test_model_wavefront_per_row(ql, orc, B):
    """Three 40-cell layers in one wavefront launch and a 300-way softmax, every
    matrix quantized per row."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(32, 40, 3, states=300, seed=9)
    x = np.random.default_rng(4).standard_normal((11, B, 32)).astype(np.float32)
    Mg = ql.quantize_model(w, gate_blocks=160, out_blocks=300)
    assert ql.stack_layers_per_launch(Mg, 11, B) >= 2
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=("h_codes",))
    o = orc.acoustic_model_forward(orc.quantize_model(w, 160, 1, 300), x, taps=True)
    for l in range(3):
        assert np.array_equal(u8(g["layers"][l]["h_codes"]), o["layers"][l]["h_codes"]), l
    assert np.max(np.abs(np_(g["post"]) - o["post"])) <= TOL


def test_model_lstmp_sub_matrices(ql, orc):
    """Two LSTMP layers (64 cells, P = 24) with W_x, W_h in 16 sub-matrices,
    W_r per row and W_y in 4 sub-matrices; batch 16 (counter exchange)."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(32, 64, 2, proj=24, states=100, seed=13)
    x = np.random.default_rng(6).standard_normal((7, 16, 32)).astype(np.float32)
    Mg = ql.quantize_model(w, gate_blocks=16, proj_blocks=24, out_blocks=4)
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=True)
    o = orc.acoustic_model_forward(orc.quantize_model(w, 16, 24, 4), x, taps=True)
    for l in range(2):
        for k in ("acc_x", "acc_h", "acc_r", "h_codes"):
            got = u8(g["layers"][l][k]) if k == "h_codes" else np_(g["layers"][l][k])
            assert np.array_equal(got, o["layers"][l][k]), (l, k)
    assert np.array_equal(np_(g["acc_y"]), o["acc_y"])
    assert np.array_equal(np_(g["logits"]), o["logits"])
    assert np.max(np.abs(np_(g["post"]) - o["post"])) <= TOL


def test_model_softmax_large_tiles_per_row(ql, orc):
    """Softmax layer on the 256x256 tiles with W_y quantized per row (8200
    states, ragged last tile), sampled utterances."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(32, 40, 1, states=8200, seed=43)
    x = np.random.default_rng(8).standard_normal((30, 80, 32)).astype(np.float32)
    utts = [0, 41, 79]
    Mg = ql.quantize_model(w, out_blocks=8200)
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=True)
    o = orc.acoustic_model_forward(orc.quantize_model(w, 4, 1, 8200),
                                   np.ascontiguousarray(x[:, utts]), taps=True)
    assert np.array_equal(np_(g["acc_y"])[:, utts], o["acc_y"])
    assert np.array_equal(np_(g["logits"])[:, utts], o["logits"])
    assert np.max(np.abs(np_(g["post"])[:, utts] - o["post"])) <= TOL
