"""The timeout path of the persistent kernels' bounded waits, forced from the
host.  With every wait bounded to one re-read (ql_debug_set_wait_bound), a
call whose workgroups must wait for each other gives up: the first wait that
is not met at once raises the workspace flag, every workgroup leaves at its
next wait (so the launch drains and the kernel ends normally), and the call
reports QL_ETIMEOUT.  The next call with the default bound gives the same
results, bit for bit, as a call made before.  Covers each persistent kernel:
the batched and the one-row layer wavefronts, the one-layer recurrence with a
projection (XCD-local and spread layouts), the fp32 recurrence, the training step's backward recurrence and
the allocation-free entry point."""
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


@pytest.fixture(autouse=True)
def default_bound(ql):
    yield
    ql.load().ql_debug_set_wait_bound(0)


def _times_out(ql, call):
    lib = ql.load()
    assert lib.ql_debug_set_wait_bound(1) == ql.QL_OK
    try:
        with pytest.raises(ql.QLError) as err:
            call()
            torch.cuda.synchronize()
        assert err.value.status == ql.QL_ETIMEOUT, err.value
    finally:
        assert lib.ql_debug_set_wait_bound(0) == ql.QL_OK


def _model(ql, B, layers=3, H=48, proj=0, seed=1):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(24, H, layers, proj=proj, states=20, seed=seed)
    x = torch.from_numpy(np.random.default_rng(seed).standard_normal((12, B, 24))
                         .astype(np.float32)).cuda()
    return w, x


@pytest.mark.parametrize("B", [32, 1])
def test_layer_wavefront_times_out_and_recovers(ql, B):
    """B = 32: batched tiles (counters, quantizing workgroups); B = 1: one-row
    tiles (tagged words)."""
    w, x = _model(ql, B)
    M = ql.quantize_model(w)
    assert ql.stack_layers_per_launch(M, x.shape[0], B) >= 2
    ref = ql.acoustic_model_forward(M, x)["post"]
    _times_out(ql, lambda: ql.acoustic_model_forward(M, x))
    assert torch.equal(ql.acoustic_model_forward(M, x)["post"], ref)


@pytest.mark.parametrize("H,B,layout", [(64, 20, 1), (42, 20, 0), (64, 5, 0)])
def test_projection_recurrence_times_out_and_recovers(ql, H, B, layout):
    """The XCD-local layout (batch 20) and the spread one (42 cells; batch 5)."""
    from paper_1607_04683_amd.workloads import random_model
    L = ql.quantize_layer(random_model(24, H, 1, proj=24, seed=3)["layers"][0])
    assert ql.recurrence_layout(L, B) == layout
    x = torch.randn(9, B, 24, device="cuda")
    ref = ql.lstm_layer_forward(L, x)["h"]
    _times_out(ql, lambda: ql.lstm_layer_forward(L, x))
    assert torch.equal(ql.lstm_layer_forward(L, x)["h"], ref)


def test_fp32_recurrence_times_out_and_recovers(ql):
    w, x = _model(ql, 20, layers=2, seed=4)
    M = ql.f32_model(w)
    ref = ql.f32_acoustic_model_forward(M, x)["post"]
    _times_out(ql, lambda: ql.f32_acoustic_model_forward(M, x))
    assert torch.equal(ql.f32_acoustic_model_forward(M, x)["post"], ref)


def test_training_step_times_out_and_recovers(ql):
    """Fresh parameters for every call (a step that timed out has updated its
    copy with undefined gradients)."""
    w, x = _model(ql, 5, layers=2, H=32, seed=5)
    y = torch.randint(0, 20, (x.shape[0], x.shape[1]), dtype=torch.int32, device="cuda")
    _, ref = ql.train_step(ql.train_params(w), x, y, 0.1)
    _times_out(ql, lambda: ql.train_step(ql.train_params(w), x, y, 0.1))
    _, g = ql.train_step(ql.train_params(w), x, y, 0.1)
    for k in ("Wy", "by"):
        assert torch.equal(g[k], ref[k]), k
    for Lg, Lr in zip(g["layers"], ref["layers"]):
        for k in Lr:
            assert torch.equal(Lg[k], Lr[k]), k


def test_no_alloc_entry_point_reports_the_timeout(ql):
    w, x = _model(ql, 20, seed=6)
    M = ql.quantize_model(w)
    T, B, _ = x.shape
    post = torch.empty(T, B, 20, device="cuda")
    flag = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    lib = ql.load()
    assert lib.ql_debug_set_wait_bound(1) == ql.QL_OK
    try:
        ql.acoustic_model_forward_stream_noalloc(M, x, post, timed_out=flag)
        torch.cuda.synchronize()
        assert int(flag.item()) == 1
    finally:
        assert lib.ql_debug_set_wait_bound(0) == ql.QL_OK
    ql.acoustic_model_forward_stream_noalloc(M, x, post, timed_out=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    assert torch.equal(post, ql.acoustic_model_forward(M, x)["post"])
