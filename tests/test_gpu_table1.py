"""The ten acoustic-model architectures of Table 1 (Section 4: 4 or 5 layers
of 300, 400 or 500 cells; 5 x 500 with a projection of 100 to 400 units after
every layer), 320-dim stacked input, with synthetic U[-0.08, 0.08] weights and
an 8192-way quantized softmax, at batch 1 (one-row exchange) and batch 16
(batched tiles): codes of every layer bit-exact, posteriors within 1e-4."""
import json
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

TOL = 1e-4
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_params.json")
ARCHS = [(m["layers"], m["hidden"], m["proj"]) for m in json.load(open(GOLDEN))["models"]]


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


@pytest.mark.parametrize("layers,hidden,proj", ARCHS)
@pytest.mark.parametrize("T,B", [(40, 1), (16, 16)])
def test_table1_architecture(ql, orc, layers, hidden, proj, T, B):
    from paper_1607_04683_amd.workloads import random_model, stacked_features
    w = random_model(320, hidden, layers, proj=proj, states=8192, seed=layers * 1000 + hidden + proj)
    x = stacked_features(np.random.Generator(np.random.PCG64(T + B)), T, B)
    Mg = ql.quantize_model(w)
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(x).cuda(), taps=("h_codes",))
    o = orc.acoustic_model_forward(orc.quantize_model(w), x, taps=True)
    for l in range(layers):
        got = g["layers"][l]["h_codes"].cpu().numpy().view(np.uint8) ^ 0x80
        assert np.array_equal(got, o["layers"][l]["h_codes"]), f"layer {l} codes"
    err = np.max(np.abs(g["post"].cpu().numpy() - o["post"]))
    assert err <= TOL, err
