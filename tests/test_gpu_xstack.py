"""Stacked layers without a projection (Section 4) at batch 16 to 64 on the
whole chip run in the XCD-local layer wavefront: XCD l runs layer l for the
whole sequence, its 32 workgroups (2 row groups x 16 cell tiles) hand the
codes of h_t and the rows' min / max to each other through the XCD's own L2,
and each layer's quantized output crosses to the next XCD.  Every tap of
every layer (input and recurrent sums, codes, row params, fp32 h, gates, c)
is compared with the oracle bit for bit on ragged shapes: the smallest and
largest batch, odd batches (the second row group one row short), cell counts
that leave tiles without cells, the widest input and cell count, the most
layers one launch holds, and sequences of one and two frames."""
import numpy as np
import pytest
import torch
from model_parity import assert_model_taps

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


# layers, n_in, H, T, B
CASES = [
    (2, 40, 48, 9, 16),      # the smallest batch: 8 rows per group (one 16-row MFMA tile)
    (3, 24, 100, 6, 33),     # 17 + 16 rows; 100 cells: tiles 4..15 of a group hold none
    (8, 40, 64, 5, 21),      # the most layers of one launch; 11 + 10 rows
    (2, 512, 512, 4, 64),    # the widest input and cell count at full batch
    (3, 320, 500, 4, 64),    # the 5 x 500 model's widths
    (4, 70, 36, 7, 47),      # 36 cells: one full tile and one with 4 cells
    (3, 40, 48, 1, 20),      # one frame: x_1 never loaded, the last output at once
    (2, 24, 64, 2, 64),      # two frames: x_2 never loaded
]


@pytest.mark.parametrize("layers,n_in,H,T,B", CASES)
def test_xcd_stack_equals_oracle(ql, orc, layers, n_in, H, T, B):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(n_in, H, layers, states=40, seed=layers * 1000 + H + B)
    x = np.random.default_rng(B + H).standard_normal((T, B, n_in)).astype(np.float32)
    M = ql.quantize_model(w)
    assert ql.stack_layers_per_launch(M, T, B) == layers
    assert ql.stack_layout(M, T, B) == 1
    g = ql.acoustic_model_forward(M, torch.from_numpy(x).cuda(), taps=True)
    o = orc.acoustic_model_forward(orc.quantize_model(w), x, taps=True)
    assert_model_taps(g, o, None, names=ql.TAP_NAMES)


def test_layout_choice(ql):
    """Batches 16 to 64 of 2 or more stacked layers take the XCD layout; one
    row, batch 15 or 65, a single layer or a layer with a projection do not."""
    from paper_1607_04683_amd.workloads import random_model
    M = lambda n, H=48, P=0: ql.quantize_model(random_model(40, H, n, proj=P, states=20, seed=3))
    assert ql.stack_layout(M(3), 10, 16) == 1
    assert ql.stack_layout(M(3), 10, 64) == 1
    assert ql.stack_layout(M(3), 10, 15) == 0
    assert ql.stack_layout(M(3), 10, 65) == 0
    assert ql.stack_layout(M(3), 10, 1) == 0
    assert ql.stack_layout(M(1), 10, 32) == 0
    assert ql.stack_layout(M(3, 64, 24), 10, 32) == 0


def test_xcd_stack_repeats_bit_for_bit(ql):
    """The 5 x 500 model's stack at batch 64, 60 frames: the build without taps
    twice and the build with taps once give the same codes."""
    from paper_1607_04683_amd.workloads import random_model
    M = ql.quantize_model(random_model(320, 500, 5, states=64, seed=4))
    x = torch.randn(60, 64, 320, device="cuda")
    assert ql.stack_layout(M, 60, 64) == 1
    ref = ql.acoustic_model_forward(M, x, taps=True)
    for _ in range(2):
        got = ql.acoustic_model_forward(M, x, taps=("h_codes",))
        for l in range(5):
            assert torch.equal(got["layers"][l]["h_codes"], ref["layers"][l]["h_codes"]), l
        assert torch.equal(got["post"], ref["post"])
