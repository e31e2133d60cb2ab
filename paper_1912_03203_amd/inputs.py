"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module generates workloads only: feature maps, block weights, mask-unit
weights and the scalar mask bias that yields a chosen density.  It contains no
step of the gated block itself (no mask logits, no dilation, no convolution);
the bias helper only selects an order statistic from logits that the caller
computed with one of the two implementations.

Recipes (all from ``numpy.random.default_rng(seed)``):

* Blob features: every image is a sum of 4 Gaussian blobs with centre
  U[0,H) x U[0,W), width sigma ~ U[0.05, 0.2] * min(H, W) and a per-channel
  amplitude vector ~ N(0, 1), plus i.i.d. N(0, 0.05) noise.
* Ellipse ("person") features, standing in for the backbone output of a
  256x256 pose input at 64x64: a flat per-channel background ~ N(0, 0.3) with
  N(0, 0.05) noise; 1-2 ellipses, each covering U[0.15, 0.35] of the image,
  axis ratio U[0.3, 1] (taller than wide), rotation U[-30, 30] degrees, fully
  inside the image; the interior gets its own mean vector ~ N(0, 1) plus 3
  Gaussian texture blobs.
* Block weights: folded 1x1 / depthwise / 1x1 weights and biases ~ N(0, std)
  (std 0.1 unless stated), rounded once to the storage dtype; biases stay
  fp32.  Mask-unit weights ~ N(0, std) in fp32.
* ShuffleNetV2 units: blob features over all c channels; the branch weights
  as above on c/2 channels (hidden e), activations ReLU, none, ReLU; the mask
  unit reads the branch half.
* Mask bias for density d: b = -s_(k), where s are the bias-free fp32 logits
  of every position of the batch and s_(k) the k-th smallest (0-based),
  k = NHW - 1 - round(d * NHW).  With distinct logits exactly round(d * NHW)
  positions then satisfy s + b > 0.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

DTYPES = ("f32", "f16", "bf16")


@dataclass(frozen=True)
class Workload:
    """One benchmark / parity workload: a stack of stride-1 gated blocks."""

    name: str
    n: int
    h: int
    w: int
    c: int
    e: int
    dtype: str
    blocks: int
    densities: tuple
    features: str  # "blobs" or "ellipses"
    weight_std: float = 0.1
    # "mbv2": stride-1 inverted-residual blocks on all c channels;
    # "shufflenet": ShuffleNetV2 stride-1 units, c = both halves, the gated
    # branch (1x1, DW 3x3, 1x1 with ReLU, none, ReLU) on c/2 channels, hidden e
    unit: str = "mbv2"

    @property
    def branch_c(self) -> int:
        return self.c // 2 if self.unit == "shufflenet" else self.c

    @property
    def nhw(self) -> int:
        return self.n * self.h * self.w


WORKLOADS = {
    # fp32 parity block: 1 x 32x32x32, expansion 6, density 0.5.
    "mbv2_block_32x32x32_f32": Workload(
        "mbv2_block_32x32x32_f32", 1, 32, 32, 32, 192, "f32", 1, (0.5,), "blobs"),
    # MobileNetV2 stage-2 block: 32 x 56x56x24, hidden 144, fp16, density sweep.
    "mbv2_stage2_block_56x56x24_f16": Workload(
        "mbv2_stage2_block_56x56x24_f16", 32, 56, 56, 24, 144, "f16", 1,
        (0.1, 0.25, 0.5, 0.75, 0.9), "blobs"),
    # Pose-style stack: 8 stride-1 blocks at 32 x 64x64x32, hidden 192, fp16.
    "pose_stack8_64x64x32_f16": Workload(
        "pose_stack8_64x64x32_f16", 32, 64, 64, 32, 192, "f16", 8, (0.25,), "ellipses"),
    # ShuffleNetV2 1.0x stride-1 units, batch 64, bf16, density 0.3: one unit
    # at each stage shape (latency) and the stage repeats (throughput).
    "shufflenet_unit_28x28x116_bf16": Workload(
        "shufflenet_unit_28x28x116_bf16", 64, 28, 28, 116, 58, "bf16", 1, (0.3,), "blobs",
        unit="shufflenet"),
    "shufflenet_unit_14x14x232_bf16": Workload(
        "shufflenet_unit_14x14x232_bf16", 64, 14, 14, 232, 116, "bf16", 1, (0.3,), "blobs",
        unit="shufflenet"),
    "shufflenet_stage2_3units_28x28x116_bf16": Workload(
        "shufflenet_stage2_3units_28x28x116_bf16", 64, 28, 28, 116, 58, "bf16", 3, (0.3,), "blobs",
        unit="shufflenet"),
    "shufflenet_stage3_7units_14x14x232_bf16": Workload(
        "shufflenet_stage3_7units_14x14x232_bf16", 64, 14, 14, 232, 116, "bf16", 7, (0.3,), "blobs",
        unit="shufflenet"),
}

SHUFFLE_ACTS = (1, 0, 1)  # ReLU after both 1x1 convolutions, none after the depthwise


def rng_for(seed: int) -> np.random.Generator:
    return np.random.default_rng(seed)


def blob_features(rng, n, h, w, c, blobs=4, noise=0.05):
    """[n, h, w, c] float32 blob field (NHWC)."""
    hh = np.arange(h, dtype=np.float64)[:, None]
    ww = np.arange(w, dtype=np.float64)[None, :]
    out = np.zeros((n, h, w, c), np.float64)
    for i in range(n):
        for _ in range(blobs):
            ch, cw = rng.uniform(0, h), rng.uniform(0, w)
            sigma = rng.uniform(0.05, 0.2) * min(h, w)
            amp = rng.standard_normal(c)
            g = np.exp(-((hh - ch) ** 2 + (ww - cw) ** 2) / (2.0 * sigma * sigma))
            out[i] += g[:, :, None] * amp[None, None, :]
    out += rng.normal(0.0, noise, size=out.shape)
    return out.astype(np.float32)


def _ellipse_mask(rng, h, w):
    area = rng.uniform(0.15, 0.35) * h * w
    ratio = rng.uniform(0.3, 1.0)  # minor / major; major axis vertical before rotation
    theta = math.radians(rng.uniform(-30.0, 30.0))
    a = math.sqrt(area / (math.pi * ratio))  # semi-major (vertical)
    b = a * ratio
    # extent of the rotated ellipse, so it can be placed fully inside
    ext_h = math.sqrt((a * math.cos(theta)) ** 2 + (b * math.sin(theta)) ** 2)
    ext_w = math.sqrt((a * math.sin(theta)) ** 2 + (b * math.cos(theta)) ** 2)
    ext_h = min(ext_h, h / 2 - 0.5)
    ext_w = min(ext_w, w / 2 - 0.5)
    ch = rng.uniform(ext_h, h - ext_h)
    cw = rng.uniform(ext_w, w - ext_w)
    hh = np.arange(h, dtype=np.float64)[:, None] + 0.5 - ch
    ww = np.arange(w, dtype=np.float64)[None, :] + 0.5 - cw
    u = hh * math.cos(theta) + ww * math.sin(theta)
    v = -hh * math.sin(theta) + ww * math.cos(theta)
    return (u / a) ** 2 + (v / b) ** 2 <= 1.0


def ellipse_features(rng, n, h, w, c, noise=0.05):
    """Returns ([n, h, w, c] float32 NHWC features, [n, h, w] bool person labels)."""
    out = np.zeros((n, h, w, c), np.float64)
    labels = np.zeros((n, h, w), bool)
    hh = np.arange(h, dtype=np.float64)[:, None]
    ww = np.arange(w, dtype=np.float64)[None, :]
    for i in range(n):
        out[i] += rng.normal(0.0, 0.3, size=c)[None, None, :]
        for _ in range(int(rng.integers(1, 3))):
            m = _ellipse_mask(rng, h, w)
            labels[i] |= m
            inner = rng.standard_normal(c)
            tex = np.zeros((h, w, c))
            for _ in range(3):
                ch, cw = rng.uniform(0, h), rng.uniform(0, w)
                sigma = rng.uniform(0.03, 0.1) * min(h, w)
                amp = rng.standard_normal(c)
                g = np.exp(-((hh - ch) ** 2 + (ww - cw) ** 2) / (2.0 * sigma * sigma))
                tex += g[:, :, None] * amp[None, None, :]
            out[i][m] = inner[None, :] + tex[m]
    out += rng.normal(0.0, noise, size=out.shape)
    return out.astype(np.float32), labels


def ellipse_mask_weights(rng, x_nhwc, labels, blocks, jitter=0.02):
    """Per-block fp32 mask-unit weights pointing from background to person
    features: the normalised difference of the mean feature inside and outside
    the ellipses of the stack input, plus N(0, jitter) per block."""
    x = np.asarray(x_nhwc, np.float64)
    inside = x[labels].mean(axis=0)
    outside = x[~labels].mean(axis=0)
    d = inside - outside
    d = d / (np.linalg.norm(d) + 1e-12)
    return [(d + rng.normal(0.0, jitter, size=d.shape)).astype(np.float32) for _ in range(blocks)]


def person_mask_weights(rng, feats_nhwc, labels):
    """Mask-unit weights of one gated block of the pose network, pointing from
    the background to the people in the block's own input features: the
    [n, 256, 256] person labels are subsampled to the features' resolution
    (every step-th row and column) and passed to ellipse_mask_weights."""
    n, h, w, _ = np.asarray(feats_nhwc).shape
    step = labels.shape[1] // h
    lab = np.ascontiguousarray(labels[:, ::step, ::step][:, :h, :w])
    return ellipse_mask_weights(rng, feats_nhwc, lab, 1)[0]


def round_to_storage(a, dtype):
    """Round float values to the storage dtype (nearest even); returns float32
    values exactly representable in it.  fp32 and fp16 round once from the
    input precision; bf16 rounds through fp32."""
    a = np.asarray(a)
    if dtype == "f32":
        return np.ascontiguousarray(a, np.float32).copy()
    if dtype == "f16":
        return np.ascontiguousarray(a.astype(np.float16).astype(np.float32))
    if dtype == "bf16":
        import torch

        a32 = np.ascontiguousarray(a, np.float32)
        return torch.from_numpy(a32).to(torch.bfloat16).to(torch.float32).numpy()
    raise ValueError("unknown dtype %r" % (dtype,))


def block_weights(rng, c, e, co=None, dtype="f16", std=0.1, mask_std=0.1):
    """Folded inverted-residual weights in PyTorch layouts:
    w1 [e, c] (expand), w2 [e, 9] (depthwise taps, k = 3*(dh+1) + (dw+1)),
    w3 [co, e] (project); biases fp32; w_m [c] fp32 mask unit."""
    co = c if co is None else co
    w1 = rng.normal(0.0, std, size=(e, c))
    b1 = rng.normal(0.0, std, size=e)
    w2 = rng.normal(0.0, std, size=(e, 9))
    b2 = rng.normal(0.0, std, size=e)
    w3 = rng.normal(0.0, std, size=(co, e))
    b3 = rng.normal(0.0, std, size=co)
    w_m = rng.normal(0.0, mask_std, size=c)
    return {
        "w1": round_to_storage(w1, dtype),
        "b1": b1.astype(np.float32),
        "w2": round_to_storage(w2, dtype),
        "b2": b2.astype(np.float32),
        "w3": round_to_storage(w3, dtype),
        "b3": b3.astype(np.float32),
        "w_m": w_m.astype(np.float32),
    }


def density_count(density, total):
    """Number of active positions that the percentile bias targets."""
    return int(math.floor(density * total + 0.5))


def percentile_bias(pre_bias_logits, density):
    """Scalar fp32 mask bias giving round(density * NHW) active positions when
    the bias-free logits are distinct (selection only; logits are an input)."""
    s = np.ascontiguousarray(pre_bias_logits, np.float32).reshape(-1)
    total = s.size
    target = density_count(density, total)
    if target >= total:
        return np.float32(np.inf)
    k = total - 1 - target
    kth = np.partition(s, k)[k]
    return np.float32(-kth)


def make_block_inputs(workload: Workload, seed: int):
    """Feature map (storage-rounded float32, NHWC) and per-block weights.

    Returns (x_nhwc float32, [weights dict per block], labels or None)."""
    rng = rng_for(seed)
    wl = workload
    labels = None
    if wl.features == "ellipses":
        x, labels = ellipse_features(rng, wl.n, wl.h, wl.w, wl.c)
    else:
        x = blob_features(rng, wl.n, wl.h, wl.w, wl.c)
    x = round_to_storage(x, wl.dtype)
    blocks = [block_weights(rng, wl.branch_c, wl.e, dtype=wl.dtype, std=wl.weight_std)
              for _ in range(wl.blocks)]
    if wl.unit == "shufflenet":
        for blk in blocks:
            blk["acts"] = SHUFFLE_ACTS
    if labels is not None:
        for blk, wm in zip(blocks, ellipse_mask_weights(rng, x, labels, wl.blocks)):
            blk["w_m"] = wm
    return x, blocks, labels


# ------------------------------------------------------------------ whole networks
# MobileNetV2 1.0x: the stem, then (expansion t, width c, repeats n, stride s)
# per stage, then the final 1x1 convolution to 1280.
MBV2_STEM = 32
MBV2_STAGES = ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1), (6, 160, 3, 2),
               (6, 320, 1, 1))
MBV2_LAST = 1280


def mbv2_layers(rng, dtype="f16", std=0.05, mask_std=0.1, in_c=3, stages=MBV2_STAGES, last=MBV2_LAST):
    """Folded-BN weights of a MobileNetV2 feature extractor as a layer list
    (dicts; PyTorch layouts, storage-rounded weights, fp32 biases): the stem,
    the (t, c, n, s) stages, and a final 1x1 to `last` channels (none when
    last is None).  Every block with stride 1 and equal input and output
    widths is gated: it carries a mask unit w_m and "gated": True."""
    def wgt(*shape):
        return round_to_storage(rng.normal(0.0, std, size=shape), dtype)

    def bias(n):
        return rng.normal(0.0, std, size=n).astype(np.float32)

    layers = [{"kind": "conv3x3", "w": wgt(MBV2_STEM, in_c, 3, 3), "b": bias(MBV2_STEM), "stride": 2, "act": 2}]
    c_in = MBV2_STEM
    for t, c, n, s in stages:
        for i in range(n):
            stride = s if i == 0 else 1
            e = c_in * t
            layer = {"kind": "block", "stride": stride, "acts": (2, 2, 0),
                     "w1": wgt(e, c_in) if t != 1 else None, "b1": bias(e) if t != 1 else None,
                     "w2": wgt(e, 9), "b2": bias(e), "w3": wgt(c, e), "b3": bias(c)}
            if stride == 1 and c_in == c:
                layer["gated"] = True
                layer["w_m"] = rng.normal(0.0, mask_std, size=c_in).astype(np.float32)
            layers.append(layer)
            c_in = c
    if last is not None:
        layers.append({"kind": "conv1x1", "w": wgt(last, c_in), "b": bias(last), "act": 2})
    return layers


def make_network_inputs(seed, n, h, w, dtype="f16", density_range=(0.2, 0.6)):
    """Smooth random blob images (3 channels), the MobileNetV2 layer list and a
    target density per gated block ~ U[density_range]."""
    rng = rng_for(seed)
    x = round_to_storage(blob_features(rng, n, h, w, 3), dtype)
    layers = mbv2_layers(rng, dtype)
    ngated = sum(1 for l in layers if l.get("gated"))
    dens = rng.uniform(density_range[0], density_range[1], size=ngated)
    return x, layers, dens


# Pose-estimation network: a MobileNetV2 backbone from 256x256x3 to 64x64x32
# (stem, the t=1 block, the 24-channel stage, one 32-channel block), then 8
# stacked stride-1 blocks at 64x64x32 with hidden width 192.  Gated: the
# second 24-channel block and the 8 stacked blocks.
POSE_STAGES = ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 1, 1), (6, 32, 8, 1))


def make_pose_network_inputs(seed, n, dtype="f16", density_range=(0.2, 0.4)):
    """Ellipse "person" images (256x256x3: flat background, 1-2 textured
    ellipses), the pose layer list, a target density per gated block
    ~ U[density_range] and the [n, 256, 256] person labels (for mask units
    pointed at the people, see ellipse_mask_weights)."""
    rng = rng_for(seed)
    x, labels = ellipse_features(rng, n, 256, 256, 3)
    x = round_to_storage(x, dtype)
    layers = mbv2_layers(rng, dtype, stages=POSE_STAGES, last=None)
    ngated = sum(1 for l in layers if l.get("gated"))
    dens = rng.uniform(density_range[0], density_range[1], size=ngated)
    return x, layers, dens, labels
