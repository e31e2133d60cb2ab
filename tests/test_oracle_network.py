"""Pins for the oracle's dense layers and the whole-network forward
(MobileNetV2 with gated stride-1 residual blocks).

Other side of each check: torch.nn.functional.conv2d in float64 on the CPU
(full 3x3 with stride and padding, grouped depthwise 3x3, 1x1), a torch
MobileNetV2 forward written from the same layer list, the gating identities
(all-ones masks give the dense network; all-zeros masks remove the gated
blocks)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_1912_03203_amd import inputs

ACTS = {0: lambda t: t, 1: torch.relu, 2: lambda t: torch.clamp(t, 0.0, 6.0)}


def T(a):
    return torch.from_numpy(np.asarray(a, np.float64))


@pytest.mark.parametrize("stride,H,W", [(1, 7, 9), (2, 8, 8), (2, 7, 5), (2, 1, 3), (1, 1, 1)])
def test_conv3x3_vs_torch(orc, stride, H, W):
    rng = np.random.default_rng(H * 10 + W)
    x = rng.normal(size=(2, 3, H, W))
    w, b = rng.normal(size=(5, 3, 3, 3)), rng.normal(size=5)
    for a in (0, 1, 2):
        got = orc.conv3x3(x, w, b, stride, a)
        ref = ACTS[a](F.conv2d(T(x), T(w), T(b), stride=stride, padding=1)).numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("stride,H,W", [(1, 6, 7), (2, 6, 7), (2, 9, 4), (2, 2, 2)])
def test_dwconv3x3_vs_torch(orc, stride, H, W):
    rng = np.random.default_rng(H * 7 + W)
    C = 6
    x = rng.normal(size=(2, C, H, W))
    w, b = rng.normal(size=(C, 9)), rng.normal(size=C)
    got = orc.dwconv3x3(x, w, b, stride, 2)
    ref = ACTS[2](F.conv2d(T(x), T(w).reshape(C, 1, 3, 3), T(b), stride=stride, padding=1, groups=C)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_conv1x1_vs_torch(orc):
    rng = np.random.default_rng(3)
    x = rng.normal(size=(2, 8, 3, 4))
    w, b = rng.normal(size=(12, 8)), rng.normal(size=12)
    got = orc.conv1x1(x, w, b, 2)
    ref = ACTS[2](F.conv2d(T(x), T(w).reshape(12, 8, 1, 1), T(b))).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def torch_mbv2(x, layers):
    """MobileNetV2 forward with torch ops, from the same layer list."""
    t = T(x)
    for L in layers:
        if L["kind"] == "conv3x3":
            t = ACTS[L["act"]](F.conv2d(t, T(L["w"]), T(L["b"]), stride=L["stride"], padding=1))
        elif L["kind"] == "conv1x1":
            O, C = L["w"].shape
            t = ACTS[L["act"]](F.conv2d(t, T(L["w"]).reshape(O, C, 1, 1), T(L["b"])))
        else:
            a1, a2, a3 = (ACTS[k] for k in L["acts"])
            h = t
            if L["w1"] is not None:
                E, C = L["w1"].shape
                h = a1(F.conv2d(h, T(L["w1"]).reshape(E, C, 1, 1), T(L["b1"])))
            E = h.shape[1]
            h = a2(F.conv2d(h, T(L["w2"]).reshape(E, 1, 3, 3), T(L["b2"]), stride=L["stride"], padding=1, groups=E))
            O = L["w3"].shape[0]
            f = a3(F.conv2d(h, T(L["w3"]).reshape(O, E, 1, 1), T(L["b3"])))
            t = t + f if (L["stride"] == 1 and t.shape[1] == O) else f
    return t.numpy()


@pytest.fixture(scope="module")
def net():
    x, layers, _ = inputs.make_network_inputs(0, 2, 32, 32, dtype="f32")
    return x, layers


def test_dense_network_vs_torch(orc, net):
    x, layers = net
    y, gates = orc.network_forward(x.transpose(0, 3, 1, 2), layers, None)
    assert gates == [] and y.shape == (2, 1280, 1, 1)
    np.testing.assert_allclose(y, torch_mbv2(x.transpose(0, 3, 1, 2), layers), rtol=1e-10, atol=1e-12)


def test_all_ones_masks_give_the_dense_network(orc, net):
    x, layers = net
    ng = sum(1 for L in layers if L.get("gated"))
    y1, gates = orc.network_forward(x.transpose(0, 3, 1, 2), layers, [np.inf] * ng)
    assert len(gates) == ng and all(g["G"].all() for g in gates)
    y, _ = orc.network_forward(x.transpose(0, 3, 1, 2), layers, None)
    np.testing.assert_allclose(y1, y, rtol=1e-12, atol=1e-12)


def test_all_zeros_masks_remove_the_gated_blocks(orc, net):
    x, layers = net
    ng = sum(1 for L in layers if L.get("gated"))
    y0, gates = orc.network_forward(x.transpose(0, 3, 1, 2), layers, [-np.inf] * ng)
    assert all(not g["G"].any() for g in gates)
    plain = [L for L in layers if not L.get("gated")]
    np.testing.assert_allclose(y0, torch_mbv2(x.transpose(0, 3, 1, 2), plain), rtol=1e-10, atol=1e-12)


def test_layer_list_is_mobilenetv2(net):
    """17 blocks with the (t, c, n, s) schedule, 10 of them gated (stride 1,
    equal widths); 224 x 224 maps to 7 x 7 x 1280."""
    _, layers = net
    blocks = [L for L in layers if L["kind"] == "block"]
    assert len(blocks) == 17
    assert sum(1 for L in blocks if L.get("gated")) == 10
    assert [L["stride"] for L in blocks].count(2) == 4
    assert layers[0]["kind"] == "conv3x3" and layers[-1]["w"].shape == (1280, 320)
