"""The frontend (Section 4: 8 frames stacked, every third stack presented)
fused into the input quantizer, against the oracle's own stacking followed by
its per-vector quantizer.  Codes, zero points, recovery factors and code sums
bit-exact; posteriors of a model fed base frames within 1e-4 of the oracle,
and bit-identical to the same model fed the stacked inputs."""
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


def u8(t, cols):
    return np_(t)[:, :cols].view(np.uint8) ^ 0x80


@pytest.mark.parametrize("nframes,B,dim,stack,skip", [
    (20, 3, 40, 8, 3),       # 5 presented steps
    (8, 1, 40, 8, 3),        # exactly one stack
    (7, 2, 40, 8, 3),        # too short: nothing presented
    (31, 5, 13, 8, 3),       # odd frame width: scalar loads; 2 leftover frames
    (26, 2, 80, 8, 3),       # 640-wide inputs
    (3 * 99 + 8, 64, 40, 8, 3),
    (17, 4, 12, 4, 1),       # other stack / skip
])
def test_quantize_stacked_frames(ql, orc, nframes, B, dim, stack, skip):
    rng = np.random.default_rng(nframes * 7 + B)
    f = rng.standard_normal((nframes, B, dim)).astype(np.float32)
    if nframes >= 14:
        f[:, 0, :] = 0.0      # utterance 0 silent: every presented vector all zero
        f[3:11, 1, :] = 0.5   # utterance 1: one stack of constant frames
    T = orc.stacked_input_count(nframes, stack, skip)
    assert ql.stacked_input_count(nframes, stack, skip) == T
    q = ql.quantize_stacked_frames(torch.from_numpy(f).cuda(), stack, skip)
    torch.cuda.synchronize()
    K = stack * dim
    assert q.codes.shape[0] == T * B
    if T == 0:
        return
    X = orc.stack_frames(f, stack, skip).reshape(T * B, K)
    o = orc.quantize(X, T * B)            # one block per row = per-vector quantization
    assert np.array_equal(u8(q.codes, K), o.codes)
    assert np.array_equal(np_(q.zero), o.zero)
    assert np.array_equal(np_(q.inv_q).view(np.uint32), o.inv_q.view(np.uint32))
    assert np.array_equal(np_(q.sums), o.codes.astype(np.int64).sum(1))
    assert (q.codes[:, K:] == 0).all()
    # same bits as quantizing the stacked copy with the dense quantizer
    qd = ql.quantize_activations(torch.from_numpy(X).cuda())
    assert torch.equal(qd.codes, q.codes) and torch.equal(qd.zero, q.zero)


def test_model_forward_frames_small(ql, orc):
    """Two 48-cell layers + 300-way softmax on base frames of 5-dim features."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 48, 2, states=300, seed=5)
    f = np.random.default_rng(3).standard_normal((3 * 10 + 6, 3, 5)).astype(np.float32)
    Mg = ql.quantize_model(w)
    g = ql.acoustic_model_forward_frames(Mg, torch.from_numpy(f).cuda(), taps=("h_codes",))
    o = orc.acoustic_model_forward_frames(orc.quantize_model(w), f, taps=True)
    assert g["post"].shape == (10, 3, 300)
    for l in range(2):
        assert np.array_equal(u8(g["layers"][l]["h_codes"].reshape(30, -1), 48),
                              o["layers"][l]["h_codes"].reshape(30, 48)), l
    assert np.max(np.abs(np_(g["post"]) - o["post"])) <= TOL


def test_model_forward_frames_empty(ql):
    from paper_1607_04683_amd.workloads import random_model
    Mg = ql.quantize_model(random_model(16, 8, 1, states=10, seed=2))
    g = ql.acoustic_model_forward_frames(Mg, torch.zeros(6, 2, 2, device="cuda"))
    assert g["post"].shape == (0, 2, 10)


def test_model_forward_frames_5x500_T1000_B64(ql, orc):
    """The batch-64 workload fed its base frames: posteriors bit-identical to
    the forward on the stacked inputs; the oracle recomputes one utterance."""
    from paper_1607_04683_amd.workloads import (LSTM5x500_S8192_T1000_B64 as W_, model_weights,
                                                features, frames)
    w = model_weights(W_)[0]
    f = frames(W_)
    Mg = ql.quantize_model(w)
    gf = ql.acoustic_model_forward_frames(Mg, torch.from_numpy(f).cuda())["post"]
    gx = ql.acoustic_model_forward(Mg, torch.from_numpy(features(W_)).cuda())["post"]
    assert gf.shape == (W_.T, W_.B, 8192)
    assert torch.equal(gf, gx)
    o = orc.acoustic_model_forward_frames(orc.quantize_model(w), np.ascontiguousarray(f[:, [17]]))
    assert np.max(np.abs(np_(gf[:, 17]) - o["post"][:, 0])) <= TOL
