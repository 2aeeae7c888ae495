"""Pins of the rejection-predictor oracle (Sec. 3.3, Sec. 4.1, App. B): closed forms of the
four draft-logit statistics, library definitions of entropy and softmax, and the MLP against
a hand-built network and against PyTorch's layers in float64."""
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

from oracle.predictor import draft_stats, reject_mlp


def test_uniform_and_two_level_rows_in_closed_form():
    V = 1000
    s = draft_stats(np.zeros((1, V), np.float32))[0]
    assert s[0] == pytest.approx(1 / V, rel=1e-12) and s[1] == pytest.approx(np.log(V), rel=1e-12)
    assert s[2] == pytest.approx(0.0, abs=1e-15) and s[3] == 0.0
    # one logit at a, the rest at 0: p1 = e^a / (e^a + V - 1), the others 1 / (e^a + V - 1)
    a = 3.0
    z = np.zeros((1, V), np.float32)
    z[0, 17] = a
    s = draft_stats(z)[0]
    Z = np.exp(a) + V - 1
    H = -(np.exp(a) / Z * np.log(np.exp(a) / Z) + (V - 1) / Z * np.log(1 / Z))
    assert s[0] == pytest.approx(np.exp(a) / Z, rel=1e-12)
    assert s[1] == pytest.approx(H, rel=1e-12)
    assert s[2] == pytest.approx((np.exp(a) - 1) / Z, rel=1e-12)
    assert s[3] == pytest.approx(a * np.sqrt(V - 1) / V, rel=1e-12)
    # temperature divides the logits; a repeated maximum has margin 0; one entry has margin 1
    s2 = draft_stats(2 * z, temperature=2.0)[0]
    assert np.allclose(s2, s, rtol=1e-12)
    z[0, 400] = a
    assert draft_stats(z)[0, 2] == pytest.approx(0.0, abs=1e-15)
    one = draft_stats(np.array([[5.0]], np.float32))[0]
    assert one[0] == 1.0 and one[1] == 0.0 and one[2] == 1.0 and one[3] == 0.0


def test_random_rows_against_library_definitions():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((6, 4099)) * rng.uniform(0.1, 8, (6, 1))).astype(np.float32)
    s = draft_stats(x, temperature=0.7)
    z = x.astype(np.float32) / np.float32(0.7)
    for r in range(6):
        p = scipy.special.softmax(z[r].astype(np.float64))
        q = np.sort(p)
        assert s[r, 0] == pytest.approx(q[-1], rel=1e-12)
        assert s[r, 1] == pytest.approx(scipy.stats.entropy(p), rel=1e-10)
        assert s[r, 2] == pytest.approx(q[-1] - q[-2], rel=1e-10, abs=1e-15)
        assert s[r, 3] == pytest.approx(np.std(z[r].astype(np.float64)), rel=1e-12)


def _params(rng, n_in):
    return {"mean": rng.standard_normal(n_in), "inv_std": rng.uniform(0.5, 2, n_in),
            "w1": rng.standard_normal((512, n_in)) * 0.5, "b1": rng.standard_normal(512) * 0.1,
            "w2": rng.standard_normal((128, 512)) / 16, "b2": rng.standard_normal(128) * 0.1,
            "w3": rng.standard_normal((64, 128)) / 8, "b3": rng.standard_normal(64) * 0.1,
            "w4": rng.standard_normal(64) / 8, "b4": 0.3}


def test_mlp_hand_built_network():
    # w1 passes feature 0 (x0 = (f0 - 1) * 2) to unit 0 and -x0 to unit 1; w2 and w3 copy units
    # 0 and 1 through; w4 = (1, -1): the output is sigmoid(relu(x0) - relu(-x0) + b4) =
    # sigmoid(x0 + b4)
    p = {k: np.zeros_like(v) for k, v in _params(np.random.default_rng(0), 4).items() if k != "b4"}
    p["mean"][:] = 1.0
    p["inv_std"][:] = 2.0
    p["w1"][0, 0], p["w1"][1, 0] = 1.0, -1.0
    p["w2"][0, 0] = p["w2"][1, 1] = 1.0
    p["w3"][0, 0] = p["w3"][1, 1] = 1.0
    p["w4"][0], p["w4"][1] = 1.0, -1.0
    p["b4"] = -0.25
    f = np.array([[1.5, 9, 9, 9], [0.25, -3, 0, 1]])
    x0 = (f[:, 0] - 1.0) * 2.0
    assert np.allclose(reject_mlp(p, f), 1 / (1 + np.exp(-(x0 - 0.25))), rtol=1e-15)


def test_mlp_against_torch_layers():
    rng = np.random.default_rng(5)
    for n_in in (4, 5):
        p = _params(rng, n_in)
        f = rng.standard_normal((17, n_in))
        net = torch.nn.Sequential(torch.nn.Linear(n_in, 512), torch.nn.ReLU(), torch.nn.Linear(512, 128),
                                  torch.nn.ReLU(), torch.nn.Linear(128, 64), torch.nn.ReLU(), torch.nn.Linear(64, 1),
                                  torch.nn.Sigmoid()).double()
        with torch.no_grad():
            for layer, (w, b) in zip([net[0], net[2], net[4]], [("w1", "b1"), ("w2", "b2"), ("w3", "b3")]):
                layer.weight.copy_(torch.from_numpy(p[w]))
                layer.bias.copy_(torch.from_numpy(p[b]))
            net[6].weight.copy_(torch.from_numpy(p["w4"])[None])
            net[6].bias.fill_(p["b4"])
            ref = net(torch.from_numpy((f - p["mean"]) * p["inv_std"]))[:, 0].numpy()
        assert np.allclose(reject_mlp(p, f), ref, rtol=1e-12, atol=1e-15)


def test_native_entry_points_reject_bad_arguments():
    import ctypes as C
    import paper_2601_11652_amd as W
    W.load_library()
    lib = W.load_library()
    ds = lib.wisp_draft_stats
    assert ds(None, 0, 10, 10, 1.0, None, None, 0, None) == W.WISP_OK          # nothing to do
    assert ds(None, 1, 10, 10, 0.0, None, None, 0, None) == W.WISP_E_INVALID   # T <= 0
    assert ds(None, 1, 10, 9, 1.0, None, None, 0, None) == W.WISP_E_INVALID    # ld < vocab
    assert ds(None, 1, 0, 9, 1.0, None, None, 0, None) == W.WISP_E_INVALID     # vocab < 1
    assert ds(None, 1, 10, 10, 1.0, None, None, 0, None) == W.WISP_E_INVALID   # NULL logits
    # partial records per chunk of every row: linear in rows, growing with the vocabulary
    n1 = lib.wisp_draft_stats_workspace_size(1, 1)
    big = lib.wisp_draft_stats_workspace_size(1, 128256)
    assert n1 > 0 and big >= n1 and lib.wisp_draft_stats_workspace_size(3, 128256) == 3 * big
    assert lib.wisp_draft_stats_workspace_size(1, 0) == 0
    m = W.wisp_reject_mlp()
    m.n_in = 9
    assert lib.wisp_reject_predict(C.byref(m), None, 1, None, None) == W.WISP_E_INVALID
    m.n_in = 4
    assert lib.wisp_reject_predict(C.byref(m), None, 0, None, None) == W.WISP_OK
    assert lib.wisp_reject_predict(C.byref(m), None, 1, None, None) == W.WISP_E_INVALID
