"""Layers with a projection (Section 4, LSTMP) at batch 16 to 256 on the whole
chip run in the XCD-local layout: each XCD holds an eighth of the batch for
the whole sequence, and its 32 workgroups hand m_t and h_t to each other
through its own L2.  Every input, recurrent and projection sum, code, row
param, gate, c, m, h and final state is compared with the oracle bit for
bit, on ragged shapes: batches that leave some XCDs short or without rows,
cell counts that leave tiles without cells, projection widths that leave
output groups without outputs, and a given h0 / c0."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_1607_04683_amd import qlstm
    qlstm.load()
    return qlstm


def np_(t):
    return t.cpu().numpy()


def _case(ql, orc, n_in, H, P, T, B, seed, h0c0=False):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(n_in, H, 1, proj=P, seed=seed)["layers"][0]
    rng = np.random.default_rng(seed + 100)
    x = rng.standard_normal((T, B, n_in)).astype(np.float32)
    h0 = c0 = None
    if h0c0:
        h0 = (np.tanh(rng.standard_normal((B, P))) * 0.5).astype(np.float32)
        c0 = rng.standard_normal((B, H)).astype(np.float32)
    L = ql.quantize_layer(w)
    g = ql.lstm_layer_forward(L, torch.from_numpy(x).cuda(),
                              None if h0 is None else torch.from_numpy(h0).cuda(),
                              None if c0 is None else torch.from_numpy(c0).cuda(), taps=True)
    o = orc.lstm_layer_forward(orc.quantize_layer(w), x, h0, c0, taps=True)
    return L, g, o


def _assert_equal(g, o):
    for k in ("acc_x", "acc_h", "acc_r", "h_zero", "h_inv_q", "h", "hT", "cT"):
        assert np.array_equal(np_(g[k]), o[k]), k
    assert np.array_equal(np_(g["h_codes"]).view(np.uint8) ^ 0x80, o["h_codes"])


# n_in, H, P, T, B
CASES = [
    (40, 96, 32, 7, 100),     # 32-cell tiles, 13 rows per XCD (one 16-row MFMA tile)
    (33, 64, 24, 9, 17),      # 3 rows per XCD: the last two XCDs hold none
    (64, 1100, 300, 4, 130),  # 64-cell tiles, tiles past H, P = 300; 17 rows, the last XCD 11
    (40, 500, 100, 6, 200),   # 25 rows per XCD (two MFMA tiles)
    (48, 2048, 512, 3, 256),  # the LSTMP layer's widths at full batch
    (24, 256, 200, 5, 250),   # the last XCD 26 rows
    (20, 64, 16, 5, 16),      # the smallest batch: 2 rows per XCD
]


@pytest.mark.parametrize("n_in,H,P,T,B", CASES)
def test_xcd_layout_equals_oracle(ql, orc, n_in, H, P, T, B):
    L, g, o = _case(ql, orc, n_in, H, P, T, B, seed=n_in + H + P + T + B)
    assert ql.recurrence_layout(L, B) == 1
    _assert_equal(g, o)


def test_xcd_layout_h0_c0(ql, orc):
    L, g, o = _case(ql, orc, 24, 64, 16, 6, 40, seed=7, h0c0=True)
    assert ql.recurrence_layout(L, 40) == 1
    _assert_equal(g, o)


def test_layout_choice(ql):
    """The XCD-local layout takes batched projection layers only; others keep
    the spread layout (which a cell count that is not a multiple of 4 still
    takes at batch 40, compared with the oracle below)."""
    from paper_1607_04683_amd.workloads import random_model
    lay = lambda H, P: ql.quantize_layer(random_model(16, H, 1, proj=P, seed=1)["layers"][0])
    assert ql.recurrence_layout(lay(64, 24), 16) == 1
    assert ql.recurrence_layout(lay(64, 24), 256) == 1
    assert ql.recurrence_layout(lay(64, 24), 15) == 0
    assert ql.recurrence_layout(lay(64, 24), 257) == 0
    assert ql.recurrence_layout(lay(64, 0), 64) == 0
    assert ql.recurrence_layout(lay(42, 24), 64) == 0


def test_spread_layout_with_projection_equals_oracle(ql, orc):
    L, g, o = _case(ql, orc, 30, 42, 24, 8, 40, seed=9)
    assert ql.recurrence_layout(L, 40) == 0
    _assert_equal(g, o)


def test_xcd_layout_repeats_bit_for_bit(ql):
    """The LSTMP layer's widths, batch 256, 40 frames: the build without taps
    twice and the build with taps once give the same bits."""
    from paper_1607_04683_amd.workloads import random_model
    L = ql.quantize_layer(random_model(64, 2048, 1, proj=512, seed=2)["layers"][0])
    x = torch.randn(40, 256, 64, device="cuda")
    ref = ql.lstm_layer_forward(L, x, taps=("h_codes",))
    for _ in range(2):
        got = ql.lstm_layer_forward(L, x)
        for k in ("h", "hT", "cT"):
            assert torch.equal(got[k], ref[k]), k
