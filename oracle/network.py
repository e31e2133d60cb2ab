"""Dense layers of a whole MobileNetV2 feature extractor and the network
forward with gated stride-1 residual blocks (the paper's integration of
dynamic convolutions in MobileNetV2, Sec. 4.1.2 and Sec. 3.1.1: every
stride-1 residual block gets its own mask unit; strided and non-residual
blocks stay dense).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain numpy in fp64,
NCHW, written from the definitions: zero padding 1 for every 3x3 convolution,
output size (H - 1) // stride + 1, folded batch norm (weights and biases as
given).  The gated blocks use the package's pinned C oracle.
"""
from __future__ import annotations

import numpy as np

ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2


def act(a, kind):
    if kind == ACT_NONE:
        return a
    if kind == ACT_RELU:
        return np.maximum(a, 0.0)
    return np.minimum(np.maximum(a, 0.0), 6.0)


def conv3x3(x, w, b, stride, activation):
    """Full 3x3 convolution: out[n, o, i, j] = sum over c, kh, kw of
    w[o, c, kh, kw] * xpad[n, c, stride*i + kh, stride*j + kw] + b[o]."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    N, C, H, W = x.shape
    O = w.shape[0]
    Ho, Wo = (H - 1) // stride + 1, (W - 1) // stride + 1
    xp = np.zeros((N, C, H + 2, W + 2))
    xp[:, :, 1:H + 1, 1:W + 1] = x
    out = np.zeros((N, O, Ho, Wo))
    for kh in range(3):
        for kw in range(3):
            patch = xp[:, :, kh:kh + stride * (Ho - 1) + 1:stride, kw:kw + stride * (Wo - 1) + 1:stride]
            out += np.einsum("oc,nchw->nohw", w[:, :, kh, kw], patch)
    out += np.asarray(b, np.float64)[None, :, None, None]
    return act(out, activation)


def dwconv3x3(x, w, b, stride, activation):
    """Depthwise 3x3 convolution, w [C][9] with tap k = 3*kh + kw:
    out[n, c, i, j] = sum over kh, kw of w[c, 3kh+kw] * xpad[n, c, s*i+kh, s*j+kw] + b[c]."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64).reshape(-1, 9)
    N, C, H, W = x.shape
    Ho, Wo = (H - 1) // stride + 1, (W - 1) // stride + 1
    xp = np.zeros((N, C, H + 2, W + 2))
    xp[:, :, 1:H + 1, 1:W + 1] = x
    out = np.zeros((N, C, Ho, Wo))
    for kh in range(3):
        for kw in range(3):
            patch = xp[:, :, kh:kh + stride * (Ho - 1) + 1:stride, kw:kw + stride * (Wo - 1) + 1:stride]
            out += w[:, 3 * kh + kw][None, :, None, None] * patch
    out += np.asarray(b, np.float64)[None, :, None, None]
    return act(out, activation)


def conv1x1(x, w, b, activation, residual=None):
    """Pointwise convolution out[n, o] = act(sum_c w[o, c] x[n, c] + b[o]) (+ residual)."""
    x = np.asarray(x, np.float64)
    out = np.einsum("oc,nchw->nohw", np.asarray(w, np.float64), x)
    out += np.asarray(b, np.float64)[None, :, None, None]
    out = act(out, activation)
    if residual is not None:
        out = out + np.asarray(residual, np.float64)
    return out


def dense_block(x, layer):
    """A MobileNetV2 inverted-residual block on every position (Sec. 3.2,
    Eq. 1 with r = identity): optional 1x1 expansion (absent when the
    expansion factor is 1), depthwise 3x3 with the layer's stride, linear 1x1
    projection, plus x when the stride is 1 and the widths match."""
    acts = layer.get("acts", (ACT_RELU6, ACT_RELU6, ACT_NONE))
    h = x
    if layer.get("w1") is not None:
        h = conv1x1(h, layer["w1"], layer["b1"], acts[0])
    h = dwconv3x3(h, layer["w2"], layer["b2"], layer["stride"], acts[1])
    res = x if (layer["stride"] == 1 and np.asarray(x).shape[1] == np.asarray(layer["w3"]).shape[0]) else None
    return conv1x1(h, layer["w3"], layer["b3"], acts[2], residual=res)


def network_forward(x_nchw, layers, biases=None, round_to=None, keep_inputs=False):
    """Forward through a layer list.  Layer kinds:
      "conv3x3": w [O][C][3][3], b, stride, act
      "block":   w1/b1 (or w1 None), w2/b2, w3/b3, stride; gated blocks
                 (stride 1, equal widths) also carry w_m and get the mask
                 bias from `biases` (one per gated block, in order)
      "conv1x1": w [O][C], b, act
    Gated blocks run the pinned gated block (mask, dilation, dense block
    with masked output); with biases None every gated block runs dense.
    round_to(a) (optional) rounds each layer's output to the storage type
    before the next layer, as the device stores it.  Returns (y, gates) with
    gates a list of dicts (G, A, D, input x) per gated block; with
    keep_inputs, (y, gates, inputs) with every layer's input."""
    from . import block_forward

    x = np.asarray(x_nchw, np.float64)
    gates = []
    inputs_ = []
    gi = 0
    for layer in layers:
        inputs_.append(x)
        kind = layer["kind"]
        if kind == "conv3x3":
            x = conv3x3(x, layer["w"], layer["b"], layer["stride"], layer["act"])
        elif kind == "conv1x1":
            x = conv1x1(x, layer["w"], layer["b"], layer["act"])
        elif layer.get("gated"):
            if biases is None:
                x = dense_block(x, layer)
            else:
                r = block_forward(x, layer, layer["w_m"], biases[gi], 1)
                gates.append({"G": r["G"], "A": r["A"], "D": r["D"], "x": x})
                x = r["y"]
            gi += 1
        else:
            x = dense_block(x, layer)
        if round_to is not None:
            x = round_to(x)
    if keep_inputs:
        return x, gates, inputs_
    return x, gates
