"""Test helpers: layout conversion, error norms, and the oracle run over image
chunks in threads (the oracle's C functions release the GIL through ctypes;
images are independent, so chunked results equal one call on the batch)."""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
from paper_1912_03203_amd import inputs

TOL = {"f32": 1e-5, "f16": 2e-2, "bf16": 2e-2}
# unit roundoff of the storage types (round to nearest even)
UNIT_ROUNDOFF = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}


def workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def nchw(x_nhwc):
    return np.ascontiguousarray(np.transpose(np.asarray(x_nhwc), (0, 3, 1, 2)))


def nhwc(x_nchw):
    return np.ascontiguousarray(np.transpose(np.asarray(x_nchw), (0, 2, 3, 1)))


def normwise(got, want):
    """max |got - want| / max |want| over the tensor (0 when both are 0)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    scale = np.max(np.abs(want)) if want.size else 0.0
    err = np.max(np.abs(got - want)) if want.size else 0.0
    return 0.0 if err == 0 else err / (scale if scale > 0 else 1.0)


CANARY = 0xA5


class Guarded:
    """A device buffer of `numel` elements followed by `tail` guard bytes of
    0xA5: a kernel that writes past the end of an output, a list or a
    workspace changes them (checked with intact())."""

    def __init__(self, numel, dtype, fill=0, device="cuda", tail=1024):
        import torch

        elem = torch.empty((), dtype=dtype).element_size()
        self.nbytes = max(int(numel), 1) * elem
        self.raw = torch.full((self.nbytes + tail,), CANARY, dtype=torch.uint8, device=device)
        self.t = self.raw[:self.nbytes].view(dtype)[:int(numel)]
        if fill is not None:
            self.t.fill_(fill)

    def intact(self):
        return bool((self.raw[self.nbytes:] == CANARY).all())


def elementwise(got, want):
    """Diagnostic: max over elements of |got - want| / max(|want|, 1e-3 max|want|)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if not want.size:
        return 0.0
    floor = 1e-3 * np.max(np.abs(want))
    den = np.maximum(np.abs(want), floor if floor > 0 else 1.0)
    return float(np.max(np.abs(got - want) / den))


def oracle_block_dense_chunked(x_nchw, wts, G=None):
    """oracle.block_dense over chunks of images in a thread pool."""
    x = np.asarray(x_nchw, np.float64)
    N, C, H, W = x.shape
    nw = min(workers(), N)
    bounds = np.linspace(0, N, nw + 1).astype(int)
    plane = H * W

    def run(i):
        a, b = bounds[i], bounds[i + 1]
        g = None if G is None else np.asarray(G)[a * plane:b * plane]
        y, _, _ = oracle.block_dense(x[a:b], wts, G=g)
        return y

    with ThreadPoolExecutor(nw) as ex:
        parts = list(ex.map(run, range(nw)))
    return np.concatenate(parts, axis=0)


def oracle_mask_chunked(x_nchw, w_m, b_m):
    x = np.asarray(x_nchw, np.float32)
    N = x.shape[0]
    nw = min(workers(), N)
    bounds = np.linspace(0, N, nw + 1).astype(int)

    def run(i):
        return oracle.mask(x[bounds[i]:bounds[i + 1]], w_m, b_m)

    with ThreadPoolExecutor(nw) as ex:
        parts = list(ex.map(run, range(nw)))
    return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])


def oracle_calibrated_block(x_nhwc_f32, wts, density, dtype, dilate=1):
    """Oracle run of one gated block on storage-rounded input: the mask bias
    comes from the oracle's own bias-free logits (percentile recipe).
    Returns dict: b_m, G, A, D, nbr, logits, y_nhwc (fp64), y_store (f32 values
    rounded to the storage dtype)."""
    x = nchw(x_nhwc_f32)
    N, C, H, W = x.shape
    _, s = oracle_mask_chunked(x, wts["w_m"], 0.0)
    b_m = inputs.percentile_bias(s, density)
    G, logits = oracle_mask_chunked(x, wts["w_m"], b_m)
    Gd = oracle.dilate(G, N, H, W, dilate)
    A, D, nbr = oracle.indices(G, Gd, N, H, W)
    y = oracle_block_dense_chunked(x.astype(np.float64), wts, G)
    y_nhwc = nhwc(y)
    return {"b_m": b_m, "G": G, "A": A, "D": D, "nbr": nbr, "logits": logits, "y": y_nhwc,
            "y_store": inputs.round_to_storage(y_nhwc, dtype)}


def oracle_calibrated_shuffle(x_nhwc_f32, wts, density, dtype):
    """Oracle run of one ShuffleNetV2 unit (oracle.shuffle_unit_forward, with
    the branch block run in chunks): the mask bias comes from the oracle's
    bias-free logits of the branch half.  Returns the branch's dict plus
    y (NHWC fp64, the shuffled unit output)."""
    x = np.asarray(x_nhwc_f32, np.float32)
    cb = x.shape[-1] // 2
    r = oracle_calibrated_block(np.ascontiguousarray(x[..., cb:]), wts, density, dtype)
    y = oracle.channel_shuffle2(np.concatenate([nchw(x[..., :cb]).astype(np.float64), nchw(r["y"])], axis=1))
    out = dict(r)
    out["y"] = nhwc(y)
    return out
