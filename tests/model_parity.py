"""Element-by-element comparison of a GPU model forward's taps with the
oracle's (helpers for the GPU parity tests; no test of its own).

Codes, zero points, recovery factors and int32 accumulators are compared bit
for bit; the fp32 h_t, gates, c_t and cell output of every layer too (every
float operation on the recurrent chain is elementwise and reproduced
exactly); logits bit for bit
(the softmax layer's recovery is elementwise as well); posteriors within
1e-4 absolute (the GPU's softmax sums in a different order)."""
import numpy as np
import torch

TOL = 1e-4
LAYER_TAPS = ("acc_x", "acc_h", "acc_r", "h_codes", "h_zero", "h_inv_q", "h", "gates", "c", "m")


def rows_of(t, utts):
    """The sampled utterances (dimension 1) of a [T][B]... tensor, gathered on
    the device before the copy to the host."""
    if utts is None:
        return t.cpu().numpy()
    idx = torch.tensor(list(utts), device=t.device)
    return t.index_select(1, idx).cpu().numpy()


def assert_model_taps(g, o, utts=None, names=LAYER_TAPS, logits=True):
    """g: GPU forward result (qlstm), o: oracle result on the same utterances
    (o's batch = len(utts) when utts is given)."""
    checked = 0
    for l, lt in enumerate(g["layers"]):
        for k in names:
            if lt.get(k) is None:
                continue
            got = rows_of(lt[k], utts)
            if k == "h_codes":
                got = got.view(np.uint8) ^ 0x80
            want = o["layers"][l][k]
            assert got.shape == want.shape, (l, k, got.shape, want.shape)
            if not np.array_equal(got, want):
                bad = np.argwhere(got != want)
                raise AssertionError(f"layer {l} {k}: {len(bad)} differ, first at {bad[0]}: "
                                     f"{got[tuple(bad[0])]} vs {want[tuple(bad[0])]}")
            checked += 1
    if logits and g.get("acc_y") is not None:
        assert np.array_equal(rows_of(g["acc_y"], utts), o["acc_y"]), "acc_y"
        assert np.array_equal(rows_of(g["logits"], utts), o["logits"]), "logits"
        checked += 2
    post = rows_of(g["post"], utts)
    err = float(np.max(np.abs(post - o["post"]))) if post.size else 0.0
    assert err <= TOL, err
    return checked
