"""LSTM layer / acoustic model parity of the GPU path with the CPU oracle.

Free-running: the GPU's h_t feeds its own next quantization, so codes and
int32 accumulators can only stay bit-exact if every fp32 operation of the
chain matches; float outputs are additionally held to the 1e-4 bar and
posteriors (a different summation order in the softmax) to 1e-4 absolute."""
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


def np_(t):
    return t.cpu().numpy()


def u8(t):
    return np_(t).view(np.uint8) ^ 0x80


def _layer_case(ql, orc, n_in, H, P, T, B, seed, h0c0=False, taps=True):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(n_in, H, 1, proj=P, seed=seed)["layers"][0]
    rng = np.random.default_rng(seed + 100)
    x = rng.standard_normal((T, B, n_in)).astype(np.float32)
    R = P if P else H
    h0 = c0 = None
    if h0c0:
        h0 = (np.tanh(rng.standard_normal((B, R))) * 0.5).astype(np.float32)
        c0 = rng.standard_normal((B, H)).astype(np.float32)
    L = ql.quantize_layer(w)
    g = ql.lstm_layer_forward(L, torch.from_numpy(x).cuda(),
                              None if h0 is None else torch.from_numpy(h0).cuda(),
                              None if c0 is None else torch.from_numpy(c0).cuda(), taps=taps)
    o = orc.lstm_layer_forward(orc.quantize_layer(w), x, h0, c0, taps=taps)
    return g, o


def _assert_layer(g, o, P):
    assert np.array_equal(np_(g["acc_x"]), o["acc_x"])
    assert np.array_equal(np_(g["acc_h"]), o["acc_h"])
    if P:
        assert np.array_equal(np_(g["acc_r"]), o["acc_r"])
    assert np.array_equal(u8(g["h_codes"]), o["h_codes"])
    assert np.array_equal(np_(g["h_zero"]), o["h_zero"])
    assert np.array_equal(np_(g["h_inv_q"]), o["h_inv_q"])
    for k in ("h", "hT", "cT"):
        assert np.max(np.abs(np_(g[k]) - o[k])) <= TOL, k
        assert np.array_equal(np_(g[k]), o[k]), k   # the fp32 chain is bit-exact


def test_lstm_layer_500_cells_T300_B1(ql, orc):
    """One LSTM layer of 500 cells on 320-dim stacked features, T=300, B=1,
    W_x 2000x320 and W_h 2000x500 ~ U[-0.08, 0.08] (per-gate quantized)."""
    from paper_1607_04683_amd.workloads import LSTM1x500_T300_B1 as W_, model_weights, features
    w = model_weights(W_)[0]["layers"][0]
    x = features(W_)
    L = ql.quantize_layer(w)
    g = ql.lstm_layer_forward(L, torch.from_numpy(x).cuda(), taps=True)
    o = orc.lstm_layer_forward(orc.quantize_layer(w), x, taps=True)
    _assert_layer(g, o, 0)


@pytest.mark.parametrize("n_in,H,P,T,B", [(50, 37, 0, 13, 1), (50, 37, 0, 13, 3),
                                          (64, 40, 0, 9, 20), (33, 64, 24, 9, 2),
                                          (33, 64, 24, 9, 17), (33, 64, 24, 9, 45),
                                          (40, 96, 32, 7, 100), (64, 512, 32, 6, 40),
                                          (48, 1024, 48, 5, 24), (130, 129, 0, 5, 64)])
def test_lstm_layer_shapes(ql, orc, n_in, H, P, T, B):
    g, o = _layer_case(ql, orc, n_in, H, P, T, B, seed=n_in + H + P + T + B)
    _assert_layer(g, o, P)


@pytest.mark.parametrize("P", [0, 16])
def test_lstm_layer_h0_c0(ql, orc, P):
    g, o = _layer_case(ql, orc, 24, 32, P, 6, 18, seed=5, h0c0=True)
    _assert_layer(g, o, P)


def test_lstm_layer_chunked_streaming(ql):
    """(hT, cT) -> (h0, c0) across two calls equals one call, bit for bit."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 48, 1, proj=0, seed=11)["layers"][0]
    L = ql.quantize_layer(w)
    x = torch.randn(20, 4, 40, device="cuda")
    full = ql.lstm_layer_forward(L, x)
    a = ql.lstm_layer_forward(L, x[:8])
    b = ql.lstm_layer_forward(L, x[8:], a["hT"], a["cT"])
    assert torch.equal(torch.cat([a["h"], b["h"]]), full["h"])
    assert torch.equal(b["cT"], full["cT"])


def test_lstm_layer_empty(ql):
    from paper_1607_04683_amd.workloads import random_model
    L = ql.quantize_layer(random_model(8, 8, 1, seed=1)["layers"][0])
    out = ql.lstm_layer_forward(L, torch.empty(0, 3, 8, device="cuda"))
    assert out["h"].shape == (0, 3, 8)


def _model_case(ql, orc, weights, feats, utts=None, taps=("h_codes",)):
    """GPU forward of the whole batch; the oracle on the sampled utterances
    (per-vector quantization makes them independent of their batch-mates);
    every requested tap compared element by element."""
    Mg = ql.quantize_model(weights)
    g = ql.acoustic_model_forward(Mg, torch.from_numpy(feats).cuda(), taps=taps)
    fo = feats if utts is None else np.ascontiguousarray(feats[:, list(utts)])
    o = orc.acoustic_model_forward(orc.quantize_model(weights), fo, taps=True)
    assert_model_taps(g, o, utts, names=ql.TAP_NAMES if taps is True else taps)
    return g, o


def test_model_small_all_taps(ql, orc):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(32, 40, 2, states=300, seed=21)
    x = np.random.default_rng(1).standard_normal((7, 3, 32)).astype(np.float32)
    g, o = _model_case(ql, orc, w, x, taps=True)
    assert np.array_equal(np_(g["acc_y"]), o["acc_y"])
    assert np.array_equal(np_(g["logits"]), o["logits"])
    for l in range(2):
        assert np.array_equal(np_(g["layers"][l]["acc_h"]), o["layers"][l]["acc_h"])
    p = np_(g["post"]).astype(np.float64)
    assert np.max(np.abs(p.sum(-1) - 1.0)) < 1e-5


def test_model_softmax_large_tiles_ragged_states(ql, orc):
    """2400 frames x 8200 states: enough for the 256x256 product tiles, with
    a ragged last column tile.  Logits and accumulators bit-exact and
    posteriors to 1e-4 on sampled utterances."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(32, 40, 1, states=8200, seed=41)
    x = np.random.default_rng(2).standard_normal((30, 80, 32)).astype(np.float32)
    utts = [0, 37, 79]
    g, o = _model_case(ql, orc, w, x, utts=utts, taps=True)
    assert np.array_equal(np_(g["acc_y"])[:, utts], o["acc_y"])
    assert np.array_equal(np_(g["logits"])[:, utts], o["logits"])
    p = np_(g["post"]).astype(np.float64)
    assert np.max(np.abs(p.sum(-1) - 1.0)) < 1e-5


@pytest.mark.parametrize("H,S", [(40, 300), (130, 8200)])
def test_model_softmax_long_runs_ragged(ql, orc, H, S):
    """33020 frames (260 x 127, a ragged last block of rows) with K of one
    64-byte step (H = 40) or three (H = 130) and a ragged last block of states
    (300, 8200).  Logits and accumulators bit-exact and posteriors to 1e-4 on
    sampled utterances; the launch without taps writes the same posteriors."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(24, H, 1, states=S, seed=43 + H)
    x = np.random.default_rng(3).standard_normal((260, 127, 24)).astype(np.float32)
    utts = [0, 64, 126]
    g, o = _model_case(ql, orc, w, x, utts=utts, taps=True)
    assert np.array_equal(np_(g["acc_y"])[:, utts], o["acc_y"])
    assert np.array_equal(np_(g["logits"])[:, utts], o["logits"])
    p = np_(g["post"][:, :16]).astype(np.float64)
    assert np.max(np.abs(p.sum(-1) - 1.0)) < 1e-5
    # the same posteriors without taps (the launch that writes no logits)
    post = ql.acoustic_model_forward(ql.quantize_model(w), torch.from_numpy(x).cuda())["post"]
    assert torch.equal(post, g["post"])


def test_model_5x500_softmax8192_T500_B1(ql, orc):
    """Five 500-cell layers + 8192-way quantized softmax, T=500, batch 1, on the
    one-row layer wavefront (all five layers in one launch): every layer's
    input and recurrent int32 sums, codes, row params and fp32 h, the softmax
    sums and logits bit-exact, posteriors within 1e-4."""
    from paper_1607_04683_amd.workloads import LSTM5x500_S8192_T500_B1 as W_, model_weights, features
    w = model_weights(W_)[0]
    assert ql.stack_layers_per_launch(ql.quantize_model(w), W_.T, W_.B) == 5
    _model_case(ql, orc, w, features(W_), taps=True)


# Ten of the 64 utterances: the first row of each of the four 8-row quantizing
# workgroups in both 32-row batch slices, plus rows 45 and 63 (a wave other
# than the first of its workgroup; the last row).
B64_UTTS = [0, 8, 16, 24, 32, 40, 45, 48, 56, 63]


def test_model_5x500_softmax8192_T1000_B64_sampled(ql, orc):
    """Batch 64 x T=1000 on the batched layer wavefront (the benchmarked
    kernel); the oracle recomputes ten utterances (per-vector quantization
    makes utterances independent), and every tap of theirs is compared."""
    from paper_1607_04683_amd.workloads import LSTM5x500_S8192_T1000_B64 as W_, model_weights, features
    w = model_weights(W_)[0]
    assert ql.stack_layers_per_launch(ql.quantize_model(w), W_.T, W_.B) == 5
    assert ql.stack_layout(ql.quantize_model(w), W_.T, W_.B) == 1  # one XCD per layer
    _model_case(ql, orc, w, features(W_), utts=B64_UTTS, taps=True)


def test_model_4xlstmp2048_softmax16384_T800_B256_sampled(ql, orc):
    """4 x LSTMP(2048 cells, P=512), 640-dim input, 16384-way softmax, batch 256
    x T=800 on the GPU; the oracle recomputes four whole utterances (the first
    and the last among them); input, recurrent and projection sums, codes, h,
    softmax sums and logits bit-exact."""
    from paper_1607_04683_amd.workloads import (LSTMP4x2048P512_S16384_T800_B256 as W_,
                                                model_weights, features)
    _model_case(ql, orc, model_weights(W_)[0], features(W_), utts=[0, 77, 131, 255], taps=True)


def test_model_batch_invariance_and_determinism(ql):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 64, 2, states=500, seed=31)
    M = ql.quantize_model(w)
    x = torch.randn(12, 20, 40, device="cuda")
    full = ql.acoustic_model_forward(M, x)["post"]
    again = ql.acoustic_model_forward(M, x)["post"]
    assert torch.equal(full, again)
    for b in (0, 7, 19):
        one = ql.acoustic_model_forward(M, x[:, b:b + 1].contiguous())["post"]
        assert torch.equal(one[:, 0], full[:, b])


def test_lstm_recurrence_entry_equals_layer_forward(ql):
    """ql_lstm_recurrence on gx = R(Mult(Q(x), W_x')) + b (the per-row quantized
    product with bias) reproduces ql_lstm_layer_forward bit for bit."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(48, 40, 1, proj=16, seed=41)["layers"][0]
    L = ql.quantize_layer(w)
    x = torch.randn(9, 18, 48, device="cuda")
    ref = ql.lstm_layer_forward(L, x, taps=("acc_h", "h_codes"))
    gx, _ = ql.quantized_matmul(L.Wx, x.reshape(-1, 48), ql.QL_ACT_PER_ROW, L.bias)
    got = ql.lstm_recurrence(L, gx.reshape(9, 18, 4 * 40), taps=("acc_h", "h_codes"))
    assert torch.equal(got["h"], ref["h"])
    assert torch.equal(got["acc_h"], ref["acc_h"])
    assert torch.equal(got["h_codes"], ref["h_codes"])


def test_model_empty(ql):
    from paper_1607_04683_amd.workloads import random_model
    M = ql.quantize_model(random_model(8, 8, 1, states=5, seed=2))
    out = ql.acoustic_model_forward(M, torch.empty(0, 2, 8, device="cuda"))
    assert out["post"].shape == (0, 2, 5)


@pytest.mark.parametrize("layers,B", [(3, 5), (3, 37), (7, 1), (2, 1), (6, 20), (2, 12)])
def test_model_layer_wavefront(ql, orc, layers, B):
    """Layers sharing one width run several per launch (a wavefront); every
    tap of every layer (input and recurrent sums, codes, row params, fp32 h)
    stays bit-exact and posteriors within 1e-4.  One batch row per tile
    (tagged exchange) and 16-row tiles (counters, ragged last slice); more
    layers than fit one launch split into several launches.  At one row, tiles
    of 16 cells (3 per 48-cell layer) put each layer's tiles on an XCD of its
    own while a layer's B x 3 tiles fit one (32 CUs); 2 layers at B = 12 have
    36 tiles each and take the spread layout over all XCDs."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, 48, layers, states=64, seed=layers * 100 + B)
    x = np.random.default_rng(B).standard_normal((11, B, 40)).astype(np.float32)
    M = ql.quantize_model(w)
    assert ql.stack_layers_per_launch(M, 11, B) >= 2
    _model_case(ql, orc, w, x, taps=True)


@pytest.mark.parametrize("B", [1, 20])
def test_lstm_stack_forward_entry(ql, orc, B):
    """ql_lstm_stack_forward on the per-vector codes of x, from a given initial
    state (h0, c0 per layer): every layer's codes, sums, fp32 h and final
    state equal the oracle's layer-by-layer evaluation."""
    from paper_1607_04683_amd.workloads import random_model
    n, T, H = 3, 9, 48
    w = random_model(40, H, n, seed=7 + B)
    rng = np.random.default_rng(B + 3)
    x = rng.standard_normal((T, B, 40)).astype(np.float32)
    h0 = [(np.tanh(rng.standard_normal((B, H))) * 0.7).astype(np.float32) for _ in range(n)]
    c0 = [rng.standard_normal((B, H)).astype(np.float32) for _ in range(n)]
    layers = [ql.quantize_layer(L) for L in w["layers"]]
    xq = ql.quantize_activations(torch.from_numpy(x.reshape(T * B, 40)).cuda())
    s_in = [(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()) for a, b in zip(h0, c0)]
    s_out = [(torch.empty(B, H, device="cuda"), torch.empty(B, H, device="cuda")) for _ in range(n)]
    g = ql.lstm_stack_forward(layers, xq, T, B, want_h=True, taps=True, state_in=s_in,
                              state_out=s_out)
    cur = x
    for k in range(n):
        o = orc.lstm_layer_forward(orc.quantize_layer(w["layers"][k]), cur, h0[k], c0[k], taps=True)
        got = u8(g["codes"][k].codes)[:, :H].reshape(T, B, H)
        assert np.array_equal(got, o["h_codes"]), f"layer {k}"
        assert np.array_equal(np_(g["codes"][k].zero).reshape(T, B), o["h_zero"])
        for name in ("acc_x", "acc_h", "h_codes", "h_zero", "h_inv_q", "h"):
            got = np_(g["layers"][k][name])
            if name == "h_codes":
                got = got.view(np.uint8) ^ 0x80
            assert np.array_equal(got, o[name]), f"layer {k} {name}"
        assert np.array_equal(np_(s_out[k][0]), o["hT"]), f"layer {k} hT"
        assert np.array_equal(np_(s_out[k][1]), o["cT"]), f"layer {k} cT"
        cur = o["h"]
    assert np.array_equal(np_(g["h"]), cur)


def _stream(ql, M, x, cuts):
    """The forward of x [T][B][in] cut at frames `cuts`, chained through each
    chunk's final state (two state buffers used in turn)."""
    B = x.shape[1]
    bufs = [ql.empty_state(M, B), ql.empty_state(M, B)]
    state, posts, codes = None, [], []
    bounds = [0, *cuts, x.shape[0]]
    for i, (a, b) in enumerate(zip(bounds[:-1], bounds[1:])):
        out = bufs[i & 1]
        g = ql.acoustic_model_forward(M, x[a:b].contiguous(), taps=("h_codes",), state_in=state,
                                      state_out=out)
        posts.append(g["post"])
        codes.append([lt["h_codes"] for lt in g["layers"]])
        state = out
    return torch.cat(posts), [torch.cat([c[l] for c in codes]) for l in range(len(M.layers))]


@pytest.mark.parametrize("layers,H,P,B,cuts", [
    (3, 48, 0, 1, [1, 7, 8]),       # one-row wavefront, one-frame chunk
    (3, 48, 0, 20, [5, 11]),        # batched wavefront (counters)
    (3, 48, 16, 1, [4, 13]),        # projection wavefront
    (1, 40, 0, 3, [6]),             # one layer per launch
    (2, 40, 24, 5, [3, 9]),         # batched projection layers, one per launch
])
def test_model_stream_chunks_equal_one_call(ql, layers, H, P, B, cuts):
    """A stream cut into chunks and chained through (hT, cT) -> (h0, c0) gives
    the posteriors and codes of one call over the whole stream, bit for bit,
    on every path the model forward takes."""
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(40, H, layers, proj=P, states=64, seed=layers * 10 + B + P)
    M = ql.quantize_model(w)
    x = torch.from_numpy(np.random.default_rng(B).standard_normal((17, B, 40)).astype(np.float32)).cuda()
    full = ql.acoustic_model_forward(M, x, taps=("h_codes",))
    post, codes = _stream(ql, M, x, cuts)
    assert torch.equal(post, full["post"])
    for l in range(layers):
        assert torch.equal(codes[l], full["layers"][l]["h_codes"]), l


def test_model_5x500_stream_chunks_T500_B1(ql):
    """The 5 x 500 + softmax 8192 model at batch 1 (T = 500) fed as a live
    stream in chunks of 1 to 250 frames: bit-identical to one call."""
    from paper_1607_04683_amd.workloads import LSTM5x500_S8192_T500_B1 as W_, model_weights, features
    M = ql.quantize_model(model_weights(W_)[0])
    x = torch.from_numpy(features(W_)).cuda()
    full = ql.acoustic_model_forward(M, x, taps=("h_codes",))
    post, codes = _stream(ql, M, x, [1, 100, 250])
    assert torch.equal(post, full["post"])
    for l in range(5):
        assert torch.equal(codes[l], full["layers"][l]["h_codes"]), l
