"""Pins for the oracle's mask dilation and index maps (Sec. 3.2: mask
dilation, masked gather rank rule, neighbour lookup of the modified depthwise
convolution).  Library routines (scipy's binary dilation, numpy's flatnonzero
and searchsorted) and closed forms stand on the other side."""
import itertools

import numpy as np
import pytest
from scipy import ndimage


def all_masks(H, W):
    """Every binary H x W mask, one per image: [2**(H*W), H, W]."""
    k = H * W
    ids = np.arange(2 ** k, dtype=np.int64)
    bits = (ids[:, None] >> np.arange(k)[None, :]) & 1
    return bits.reshape(-1, H, W).astype(np.uint8)


def scipy_dilate(G, r):
    st = np.ones((2 * r + 1, 2 * r + 1), bool)
    return np.stack([ndimage.binary_dilation(g.astype(bool), structure=st) for g in G]).astype(np.uint8)


def library_indices(G, Gd, N, H, W):
    g = G.reshape(-1)
    gd = Gd.reshape(-1)
    A = np.flatnonzero(g).astype(np.int32)
    D = np.flatnonzero(gd).astype(np.int32)
    nbr = np.full((A.size, 9), -1, np.int32)
    n, h, w = A // (H * W), (A // W) % H, A % W
    for dh, dw in itertools.product((-1, 0, 1), (-1, 0, 1)):
        k = 3 * (dh + 1) + (dw + 1)
        hh, ww = h + dh, w + dw
        ok = (hh >= 0) & (hh < H) & (ww >= 0) & (ww < W)
        lin = (n * H + hh) * W + ww
        pos = np.searchsorted(D, lin)
        pos_c = np.minimum(pos, max(D.size - 1, 0))
        hit = ok & (D.size > 0) & (D[pos_c] == lin) if D.size else np.zeros_like(ok)
        nbr[hit, k] = pos_c[hit]
    return A, D, nbr


@pytest.mark.parametrize("H,W", [(1, 1), (1, 5), (2, 2), (3, 3), (3, 4), (4, 3), (2, 6), (1, 12)])
def test_dilation_exhaustive_vs_scipy(orc, H, W):
    G = all_masks(H, W)
    N = G.shape[0]
    Gd = orc.dilate(G.reshape(-1), N, H, W, 1).reshape(N, H, W)
    np.testing.assert_array_equal(Gd, scipy_dilate(G, 1))


@pytest.mark.parametrize("r", [0, 2, 3])
def test_dilation_other_radii_vs_scipy(orc, r):
    rng = np.random.default_rng(r)
    G = (rng.random((5, 9, 11)) < 0.08).astype(np.uint8)
    Gd = orc.dilate(G.reshape(-1), 5, 9, 11, r).reshape(5, 9, 11)
    want = G if r == 0 else scipy_dilate(G, r)
    np.testing.assert_array_equal(Gd, want)


@pytest.mark.parametrize("H,W", [(2, 3), (3, 3), (3, 4), (4, 3)])
def test_indices_exhaustive_vs_numpy(orc, H, W):
    """All masks as one batch: raster order across images, per-image
    neighbourhoods, lists identical to flatnonzero / searchsorted."""
    G = all_masks(H, W)
    N = G.shape[0]
    Gd = orc.dilate(G.reshape(-1), N, H, W, 1)
    A, D, nbr = orc.indices(G.reshape(-1), Gd, N, H, W)
    A2, D2, nbr2 = library_indices(G, Gd, N, H, W)
    np.testing.assert_array_equal(A, A2)
    np.testing.assert_array_equal(D, D2)
    np.testing.assert_array_equal(nbr, nbr2)


def test_indices_invariants_random(orc):
    rng = np.random.default_rng(5)
    N, H, W = 4, 17, 23
    G = (rng.random(N * H * W) < 0.2).astype(np.uint8)
    Gd = orc.dilate(G, N, H, W, 1)
    A, D, nbr = orc.indices(G, Gd, N, H, W)
    assert np.all(np.diff(A) > 0) and np.all(np.diff(D) > 0)
    assert np.all(np.isin(A, D))
    np.testing.assert_array_equal(D[nbr[:, 4]], A)  # centre tap is the pixel itself
    # with dilation radius 1 every in-image neighbour of an active pixel is in D
    n, h, w = A // (H * W), (A // W) % H, A % W
    for k in range(9):
        dh, dw = k // 3 - 1, k % 3 - 1
        inside = (h + dh >= 0) & (h + dh < H) & (w + dw >= 0) & (w + dw < W)
        assert np.all((nbr[:, k] >= 0) == inside)
        lin = (n * H + h + dh) * W + w + dw
        np.testing.assert_array_equal(D[nbr[inside, k]], lin[inside])


@pytest.mark.parametrize("pos,expect", [((3, 3), 9), ((0, 3), 6), ((3, 0), 6), ((6, 3), 6),
                                        ((0, 0), 4), ((6, 6), 4), ((0, 6), 4)])
def test_single_pixel_closed_forms(orc, pos, expect):
    H = W = 7
    G = np.zeros((1, H, W), np.uint8)
    G[0, pos[0], pos[1]] = 1
    Gd = orc.dilate(G.reshape(-1), 1, H, W, 1)
    A, D, nbr = orc.indices(G.reshape(-1), Gd, 1, H, W)
    assert A.tolist() == [pos[0] * W + pos[1]]
    assert D.size == expect
    assert int((nbr[0] >= 0).sum()) == expect


def test_all_ones_and_all_zeros(orc):
    N, H, W = 2, 5, 6
    ones = np.ones(N * H * W, np.uint8)
    A, D, nbr = orc.indices(ones, orc.dilate(ones, N, H, W, 1), N, H, W)
    np.testing.assert_array_equal(A, np.arange(N * H * W))
    np.testing.assert_array_equal(D, np.arange(N * H * W))
    zeros = np.zeros(N * H * W, np.uint8)
    A, D, nbr = orc.indices(zeros, orc.dilate(zeros, N, H, W, 1), N, H, W)
    assert A.size == 0 and D.size == 0 and nbr.shape == (0, 9)


def test_dilate_zero_gives_active_list(orc):
    rng = np.random.default_rng(9)
    N, H, W = 3, 8, 9
    G = (rng.random(N * H * W) < 0.3).astype(np.uint8)
    Gd = orc.dilate(G, N, H, W, 0)
    np.testing.assert_array_equal(Gd, G)
    A, D, _ = orc.indices(G, Gd, N, H, W)
    np.testing.assert_array_equal(A, D)


def test_batch_lists_concatenate_per_image(orc):
    """Batch independence: each image's lists, offset by n*H*W, concatenate
    to the batch lists (raster order is image-major)."""
    rng = np.random.default_rng(12)
    N, H, W = 3, 6, 7
    G = (rng.random(N * H * W) < 0.25).astype(np.uint8)
    Gd = orc.dilate(G, N, H, W, 1)
    A, D, nbr = orc.indices(G, Gd, N, H, W)
    As, Ds, nbrs, doff = [], [], [], 0
    for n in range(N):
        g = G[n * H * W:(n + 1) * H * W]
        a, d, nb = orc.indices(g, orc.dilate(g, 1, H, W, 1), 1, H, W)
        As.append(a + n * H * W)
        Ds.append(d + n * H * W)
        nbrs.append(np.where(nb >= 0, nb + doff, -1))
        doff += d.size
    np.testing.assert_array_equal(A, np.concatenate(As))
    np.testing.assert_array_equal(D, np.concatenate(Ds))
    np.testing.assert_array_equal(nbr, np.concatenate(nbrs))
