"""Pins of the oracle's quantization-aware training step (Section 3.2,
Algorithm 1) against what does not depend on the oracle itself.

* The float training step (no quantization anywhere) against torch autograd
  in fp64 on nn.LSTM layers, a linear output layer and frame-level
  cross-entropy; and against central finite differences of the oracle's own
  loss.
* The quantization-aware step ('quant-all' and 'quant') against torch
  autograd on a graph whose forward values are those of the oracle's
  quantized inference (gate pre-activations, projected outputs and logits
  taken from the pinned inference oracle) while gradients flow through the
  float operations with the float parameters: the paper's backward pass, a
  float backward evaluated at the quantized forward pass's activations, with
  quantization itself not differentiated.
* The step's loss equals the cross-entropy of the inference oracle's
  posteriors, and the update is w - lr g in fp32.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

T, B, IN, H, S = 7, 3, 12, 10, 9


def _case(proj, seed):
    from paper_1607_04683_amd.workloads import random_model
    w = random_model(IN, H, 2, proj=proj, states=S, seed=seed)
    rng = np.random.default_rng(seed + 1)
    x = rng.standard_normal((T, B, IN)).astype(np.float32)
    y = rng.integers(0, S, (T, B)).astype(np.int32)
    return w, x, y


def _params(w):
    """fp64 leaf tensors of every parameter, in the oracle's layout."""
    P = {"layers": [], "Wy": torch.tensor(w["Wy"], dtype=torch.float64, requires_grad=True),
         "by": torch.tensor(w["by"], dtype=torch.float64, requires_grad=True)}
    for L in w["layers"]:
        P["layers"].append({k: None if L.get(k) is None else
                            torch.tensor(L[k], dtype=torch.float64, requires_grad=True)
                            for k in ("Wx", "Wh", "b", "Wr")})
    return P


def _grads_close(P, g, rtol):
    pairs = [(P["Wy"], g["Wy"], "Wy"), (P["by"], g["by"], "by")]
    for l, (Lp, Lg) in enumerate(zip(P["layers"], g["layers"])):
        for k in ("Wx", "Wh", "b", "Wr"):
            if Lp[k] is not None:
                pairs.append((Lp[k], Lg[k], f"layer {l} {k}"))
    worst = 0.0
    for t, o, name in pairs:
        ref = t.grad.numpy()
        scale = np.max(np.abs(ref))
        assert scale > 0, name
        err = np.max(np.abs(o.astype(np.float64) - ref)) / scale
        worst = max(worst, err)
        assert err <= rtol, (name, err)
    return worst


def _torch_float_loss(w, P, x, y):
    """nn.LSTM layers (fp64), then W_y h + b_y and mean cross-entropy."""
    cur = torch.from_numpy(x.astype(np.float64))
    for L, Lp in zip(w["layers"], P["layers"]):
        proj = 0 if L.get("Wr") is None else L["Wr"].shape[0]
        m = torch.nn.LSTM(L["Wx"].shape[1], H, proj_size=proj, dtype=torch.float64)
        # the module run on the leaves (its gate order is i, f, g, o too)
        params = {"weight_ih_l0": Lp["Wx"], "weight_hh_l0": Lp["Wh"], "bias_ih_l0": Lp["b"],
                  "bias_hh_l0": torch.zeros(4 * H, dtype=torch.float64)}
        if proj:
            params["weight_hr_l0"] = Lp["Wr"]
        cur, _ = torch.func.functional_call(m, params, (cur,))
    z = torch.nn.functional.linear(cur, P["Wy"], P["by"])
    return torch.nn.functional.cross_entropy(z.reshape(-1, S),
                                             torch.from_numpy(y.astype(np.int64)).reshape(-1))


@pytest.mark.parametrize("proj", [0, 6])
def test_float_step_gradients_equal_torch_autograd(orc, proj):
    w, x, y = _case(proj, seed=10 + proj)
    new, g, loss = orc.train_step(w, x, y, lr=0.5, quantize_layers=False, quantize_output=False)
    P = _params(w)
    ref = _torch_float_loss(w, P, x, y)
    ref.backward()
    assert abs(loss - ref.item()) < 1e-6
    _grads_close(P, g, rtol=2e-5)


def test_float_step_gradients_equal_finite_differences(orc):
    """Central differences of the oracle's own float loss at the largest
    gradient entries of every parameter (independent of torch); weights
    scaled up so that every gradient stands well above the fp32 forward
    pass's rounding."""
    w, x, y = _case(6, seed=3)
    for L in w["layers"]:
        for k in ("Wx", "Wh", "b", "Wr"):
            L[k] = (L[k] * 5).astype(np.float32)
    w["Wy"] = (w["Wy"] * 5).astype(np.float32)
    _, g, loss0 = orc.train_step(w, x, y, lr=0.0, quantize_layers=False, quantize_output=False)
    eps = 2e-2

    def loss_at(path, idx, delta):
        w2 = {"layers": [dict(L) for L in w["layers"]], "Wy": w["Wy"].copy(), "by": w["by"].copy()}
        if path[0] == "layers":
            arr = w2["layers"][path[1]][path[2]] = w["layers"][path[1]][path[2]].copy()
        else:
            arr = w2[path[0]]
        arr[idx] += delta
        return orc.train_step(w2, x, y, lr=0.0, quantize_layers=False, quantize_output=False)[2]

    paths = [("Wy",), ("by",)] + [("layers", l, k) for l in range(2) for k in ("Wx", "Wh", "b", "Wr")]
    for path in paths:
        gv = g[path[0]] if path[0] != "layers" else g["layers"][path[1]][path[2]]
        for flat in np.argsort(np.abs(gv).ravel())[-2:]:
            idx = np.unravel_index(flat, gv.shape)
            fd = (loss_at(path, idx, eps) - loss_at(path, idx, -eps)) / (2 * eps)
            assert abs(fd - gv[idx]) <= 0.03 * abs(gv[idx]) + 2e-6, (path, idx, fd, gv[idx])


def _torch_qat_loss(w, P, x, y, fwd, quantize_output):
    """Forward values from the quantized inference oracle (fwd), gradients
    through the float operations with the float parameters."""
    cur = torch.from_numpy(x.astype(np.float64))
    for L, Lp, lt in zip(w["layers"], P["layers"], fwd["layers"]):
        R = H if Lp["Wr"] is None else Lp["Wr"].shape[0]
        hp = torch.zeros(B, R, dtype=torch.float64)
        cp = torch.zeros(B, H, dtype=torch.float64)
        hs = []
        for t in range(T):
            a_f = cur[t] @ Lp["Wx"].T + Lp["b"] + hp @ Lp["Wh"].T
            a = a_f + (torch.from_numpy(lt["preact"][t].astype(np.float64)) - a_f).detach()
            i, f = torch.sigmoid(a[:, :H]), torch.sigmoid(a[:, H:2 * H])
            gg, o = torch.tanh(a[:, 2 * H:3 * H]), torch.sigmoid(a[:, 3 * H:])
            c = f * cp + i * gg
            m = o * torch.tanh(c)
            if Lp["Wr"] is not None:
                h_f = m @ Lp["Wr"].T
                h = h_f + (torch.from_numpy(lt["h"][t].astype(np.float64)) - h_f).detach()
            else:
                h = m
            hs.append(h)
            hp, cp = h, c
        cur = torch.stack(hs)
    z = torch.nn.functional.linear(cur, P["Wy"], P["by"])
    if quantize_output:
        z = z + (torch.from_numpy(fwd["logits"].astype(np.float64)) - z).detach()
    return torch.nn.functional.cross_entropy(z.reshape(-1, S),
                                             torch.from_numpy(y.astype(np.int64)).reshape(-1))


@pytest.mark.parametrize("proj", [0, 6])
@pytest.mark.parametrize("quantize_output", [True, False])
def test_qat_gradients_are_float_backprop_at_quantized_activations(orc, proj, quantize_output):
    w, x, y = _case(proj, seed=20 + proj)
    _, g, loss = orc.train_step(w, x, y, lr=0.1, quantize_layers=True,
                                quantize_output=quantize_output)
    fwd = orc.acoustic_model_forward(orc.quantize_model(w), x, taps=True)
    if not quantize_output:  # 'quant': float logits of the quantized layers' output
        hL = fwd["layers"][-1]["h"].astype(np.float64)
        fwd["logits"] = (hL @ w["Wy"].astype(np.float64).T + w["by"]).astype(np.float32)
    P = _params(w)
    ref = _torch_qat_loss(w, P, x, y, fwd, quantize_output)
    ref.backward()
    assert abs(loss - ref.item()) < 1e-6
    worst = _grads_close(P, g, rtol=2e-5)
    # the quantized forward moves the gradient far beyond that tolerance: the
    # pin tells the two steps apart
    _, gf, _ = orc.train_step(w, x, y, lr=0.1, quantize_layers=False, quantize_output=False)
    diff = max(np.max(np.abs(g["layers"][0][k] - gf["layers"][0][k])) /
               np.max(np.abs(gf["layers"][0][k])) for k in ("Wx", "Wh"))
    assert diff > 50 * max(worst, 1e-7)


def test_qat_loss_is_cross_entropy_of_inference_posteriors_and_update_is_sgd(orc):
    w, x, y = _case(6, seed=31)
    lr = 0.25
    new, g, loss = orc.train_step(w, x, y, lr=lr, gate_blocks=4)
    post = orc.acoustic_model_forward(orc.quantize_model(w), x)["post"]
    ref = -np.mean(np.log(np.take_along_axis(post, y[..., None].astype(np.int64), -1)
                          .astype(np.float64)))
    assert abs(loss - ref) < 1e-6
    lr32 = np.float32(lr)
    for L, Ln, Lg in zip(w["layers"], new["layers"], g["layers"]):
        for k in ("Wx", "Wh", "b", "Wr"):
            if L.get(k) is not None:
                assert np.array_equal(Ln[k], np.float32(L[k]) - lr32 * Lg[k]), k
    assert np.array_equal(new["Wy"], np.float32(w["Wy"]) - lr32 * g["Wy"])
    assert np.array_equal(new["by"], np.float32(w["by"]) - lr32 * g["by"])
    assert not np.array_equal(new["Wy"], w["Wy"])


def test_qat_gate_blocks_change_the_forward_only(orc):
    """Finer weight blocks change the quantized forward (so the gradient), and
    the float step ignores them."""
    w, x, y = _case(0, seed=41)
    _, g4, l4 = orc.train_step(w, x, y, lr=0.1, gate_blocks=4)
    _, g40, l40 = orc.train_step(w, x, y, lr=0.1, gate_blocks=40)
    assert l4 != l40
    _, f4, _ = orc.train_step(w, x, y, lr=0.1, gate_blocks=4, quantize_layers=False,
                              quantize_output=False)
    _, f40, _ = orc.train_step(w, x, y, lr=0.1, gate_blocks=40, quantize_layers=False,
                               quantize_output=False)
    assert np.array_equal(f4["Wy"], f40["Wy"])
