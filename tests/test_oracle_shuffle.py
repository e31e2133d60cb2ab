"""Pins for the oracle's ShuffleNetV2 stride-1 unit with a gated residual
branch (Sec. 4.1.2; the branch is the gated block of Eq. 3).

Other side of each check: torch's channel_shuffle and a float64 conv2d chain
on the CPU (the all-ones mask gives the dense unit), the channel permutation
alone (the all-zeros mask), and the mask unit applied to the branch half."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from tests.test_oracle_block import torch_block, weights

SHUFFLE_ACTS = (1, 0, 1)  # ReLU after both 1x1 convolutions, none after the depthwise


def torch_unit(x, w):
    """Dense unit: concat(x1, x2 + F(x2)) through torch's channel_shuffle."""
    C = x.shape[1]
    x1, x2 = x[:, : C // 2], x[:, C // 2:]
    b, _ = torch_block(x2, w)
    z = torch.cat([torch.from_numpy(np.asarray(x1, np.float64)), torch.from_numpy(b)], dim=1)
    return F.channel_shuffle(z, 2).numpy()


@pytest.mark.parametrize("C", [2, 6, 116, 232])
def test_channel_shuffle_is_torch_channel_shuffle(orc, C):
    x = np.random.default_rng(C).normal(size=(2, C, 3, 2))
    got = orc.channel_shuffle2(x)
    ref = F.channel_shuffle(torch.from_numpy(x), 2).numpy()
    assert got.tobytes() == np.ascontiguousarray(ref).tobytes()


def test_all_zeros_mask_is_the_shuffled_input_bitwise(orc):
    rng = np.random.default_rng(3)
    N, C, H, W = 2, 12, 5, 7
    x = rng.normal(0, 1, (N, C, H, W)).astype(np.float32).astype(np.float64)
    x[0, C // 2, 0, 0] = -0.0
    w = weights(rng, C // 2, C // 2, acts=SHUFFLE_ACTS)
    w_m = rng.normal(0, 1, C // 2).astype(np.float32)
    r = orc.shuffle_unit_forward(x, w, w_m, -np.inf)
    assert r["G"].sum() == 0
    ref = F.channel_shuffle(torch.from_numpy(x), 2).numpy()
    assert r["y"].tobytes() == np.ascontiguousarray(ref).tobytes()


@pytest.mark.parametrize("N,C,E,H,W", [(1, 12, 6, 6, 5), (2, 116, 58, 4, 4), (1, 10, 16, 3, 8)])
def test_all_ones_mask_is_the_dense_unit_vs_torch(orc, N, C, E, H, W):
    rng = np.random.default_rng(C + E)
    x = rng.normal(0, 1, (N, C, H, W)).astype(np.float32).astype(np.float64)
    w = weights(rng, C // 2, E, acts=SHUFFLE_ACTS)
    w_m = rng.normal(0, 1, C // 2).astype(np.float32)
    r = orc.shuffle_unit_forward(x, w, w_m, np.inf)
    assert r["G"].all()
    np.testing.assert_allclose(r["y"], torch_unit(x, w), rtol=1e-12, atol=1e-12)


def test_partial_mask_comes_from_the_branch_half(orc):
    """The mask unit reads x2: the decisions equal the mask oracle on x2 (and
    differ from it on x1 for these inputs); the output is the dense unit at
    active positions, the shuffled input elsewhere, and the pass-through
    channels (even outputs) are x1 everywhere, bit for bit."""
    rng = np.random.default_rng(11)
    N, C, H, W = 2, 16, 6, 6
    cb = C // 2
    x = rng.normal(0, 1, (N, C, H, W)).astype(np.float32).astype(np.float64)
    w = weights(rng, cb, 12, acts=SHUFFLE_ACTS)
    w_m = rng.normal(0, 1, cb).astype(np.float32)
    r = orc.shuffle_unit_forward(x, w, w_m, 0.1)
    G2, _ = orc.mask(x[:, cb:].astype(np.float32), w_m, 0.1)
    G1, _ = orc.mask(x[:, :cb].astype(np.float32), w_m, 0.1)
    assert 0 < r["G"].sum() < N * H * W
    assert np.array_equal(r["G"], G2) and not np.array_equal(r["G"], G1)
    dense = torch_unit(x, w)
    plain = F.channel_shuffle(torch.from_numpy(x), 2).numpy()
    act = r["G"].reshape(N, 1, H, W).astype(bool)
    np.testing.assert_allclose(np.where(act, r["y"], 0), np.where(act, dense, 0), rtol=1e-12, atol=1e-12)
    assert np.where(act, 0, r["y"]).tobytes() == np.where(act, 0, plain).tobytes()
    assert r["y"][:, 0::2].tobytes() == np.ascontiguousarray(x[:, :cb]).tobytes()


def test_chunked_helper_equals_the_unit_oracle(orc):
    """The tests' chunked ShuffleNet helper reproduces shuffle_unit_forward."""
    from paper_1912_03203_amd import inputs
    from tests import util

    rng = np.random.default_rng(5)
    x = inputs.round_to_storage(inputs.blob_features(rng, 2, 7, 9, 20), "bf16")
    w = inputs.block_weights(rng, 10, 16, dtype="bf16")
    w["acts"] = SHUFFLE_ACTS
    got = util.oracle_calibrated_shuffle(x, w, 0.4, "bf16")
    ref = orc.shuffle_unit_forward(util.nchw(x), w, w["w_m"], got["b_m"])
    assert np.array_equal(got["G"], ref["G"])
    np.testing.assert_allclose(got["y"], util.nhwc(ref["y"]), rtol=1e-13, atol=1e-13)
