"""The allocation-free stream step (ql_acoustic_model_forward_stream_noalloc)
against the workspace entry point it shares its kernels with
(ql_acoustic_model_forward_stream): the same posteriors and final state, bit
for bit, over calls in a row on the one static scratch array, each smaller
than the one before (what a call leaves behind must not leak into the next),
and the size limit rejected before anything runs."""
import ctypes as C

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


def _pair(ql, M, x, s_in, out_a, out_b):
    """The same chunk through both entry points; returns both posteriors."""
    T, B, _ = x.shape
    S = M.Wy.rows
    ref = ql.acoustic_model_forward(M, x, state_in=s_in, state_out=out_a)["post"]
    post = torch.full((T, B, S), float("nan"), device="cuda")
    flag = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    ql.acoustic_model_forward_stream_noalloc(M, x, post, state_in=s_in, state_out=out_b,
                                             timed_out=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    return ref, post


@pytest.mark.parametrize("P", [0, 16])
def test_noalloc_stream_equals_workspace_entry(ql, P):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 48, 3, proj=P, states=96, seed=71 + P)
    M = ql.quantize_model(w)
    rng = np.random.default_rng(5 + P)
    # batch 20 (batched wavefront / one layer per launch), then a smaller
    # continuation of the same stream, then a smaller stream at batch 1
    # (projection wavefront for P > 0)
    x20 = torch.from_numpy(rng.standard_normal((60, 20, 40)).astype(np.float32)).cuda()
    x1 = torch.from_numpy(rng.standard_normal((9, 1, 40)).astype(np.float32)).cuda()
    sa, sb = ql.empty_state(M, 20), ql.empty_state(M, 20)
    ref, got = _pair(ql, M, x20[:45], None, sa, sb)
    assert torch.equal(ref, got)
    for (ha, ca), (hb, cb) in zip(sa, sb):
        assert torch.equal(ha, hb) and torch.equal(ca, cb)
    sa2, sb2 = ql.empty_state(M, 20), ql.empty_state(M, 20)
    ref, got = _pair(ql, M, x20[45:], sa, sa2, sb2)
    assert torch.equal(ref, got)
    for (ha, ca), (hb, cb) in zip(sa2, sb2):
        assert torch.equal(ha, hb) and torch.equal(ca, cb)
    s1a, s1b = ql.empty_state(M, 1), ql.empty_state(M, 1)
    ref, got = _pair(ql, M, x1, None, s1a, s1b)
    assert torch.equal(ref, got)
    for (ha, ca), (hb, cb) in zip(s1a, s1b):
        assert torch.equal(ha, hb) and torch.equal(ca, cb)


def test_noalloc_5x500_stream_B1(ql):
    """The 5 x 500 + 8192 softmax model at batch 1: a 300-frame chunk, then a
    200-frame continuation, equal to the workspace entry point's."""
    from paper_1607_04683_amd.workloads import LSTM5x500_S8192_T500_B1 as W_, model_weights, features
    M = ql.quantize_model(model_weights(W_)[0])
    x = torch.from_numpy(features(W_)).cuda()
    sa, sb = ql.empty_state(M, 1), ql.empty_state(M, 1)
    ref, got = _pair(ql, M, x[:300], None, sa, sb)
    assert torch.equal(ref, got)
    sa2, sb2 = ql.empty_state(M, 1), ql.empty_state(M, 1)
    ref, got = _pair(ql, M, x[300:], sa, sa2, sb2)
    assert torch.equal(ref, got)


def test_noalloc_rejects_calls_beyond_the_scratch(ql):
    from paper_1607_04683_amd.workloads import random_model
    M = ql.quantize_model(random_model(320, 500, 5, states=8192, seed=1))
    cm, keep = M.cstruct()
    lib = ql.load()
    T_ok = 1600
    assert lib.ql_acoustic_model_workspace(C.byref(cm), T_ok, 1) <= ql.NOALLOC_SCRATCH_BYTES
    T_big = 2000
    assert lib.ql_acoustic_model_workspace(C.byref(cm), T_big, 1) > ql.NOALLOC_SCRATCH_BYTES
    x = torch.zeros(T_big, 1, 320, device="cuda")
    post = torch.full((T_big, 1, 8192), -1.0, device="cuda")
    with pytest.raises(ql.QLError) as e:
        ql.acoustic_model_forward_stream_noalloc(M, x, post)
    assert e.value.status == ql.QL_ESCRATCH
    torch.cuda.synchronize()
    assert bool((post == -1.0).all())  # nothing ran
