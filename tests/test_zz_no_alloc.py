"""dynconv_stack_forward_noalloc (the stack on the library's static
per-device scratch array) against dynconv_stack_forward (a caller
workspace): bitwise equal outputs, masks and counts on two calls in a row,
the second on a smaller input, and a clear error for a stack whose
workspace exceeds the array."""
import numpy as np
import pytest
import torch

from paper_1912_03203_amd import dynconv as dc
from paper_1912_03203_amd import inputs
from tests import util

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dc.load()


def _case(seed, N, H, W, C, E, nb, dtype, density):
    rng = inputs.rng_for(seed)
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, C), dtype)
    blocks = [inputs.block_weights(rng, C, E, dtype=dtype) for _ in range(nb)]
    _, s = util.oracle_mask_chunked(util.nchw(x), blocks[0]["w_m"], 0.0)
    b0 = float(inputs.percentile_bias(s, density))
    t = dc.NAME_TO_DTYPE[dtype]
    bw = [dc.BlockWeights.from_arrays(w, t, b_mask=b0) for w in blocks]
    xd = torch.from_numpy(np.ascontiguousarray(x)).to(DEV).to(t)
    return xd, bw


def _run(fn, xd, bw, flags):
    n, h, w, _ = xd.shape
    masks = torch.full((len(bw), n * h * w), 7, dtype=torch.uint8, device=DEV)
    counts = torch.full((len(bw), 2), -5, dtype=torch.int32, device=DEV)
    y = torch.full_like(xd, float("nan"))
    fn(xd, y, bw, flags=flags, masks=masks, counts=counts)
    torch.cuda.synchronize()
    return y, masks, counts


@pytest.mark.parametrize("flags", [0, dc.STACK_DENSE])
def test_noalloc_matches_workspace_call_twice_smaller_second(flags):
    # the pose stack's shape first, then a smaller ragged one: the second
    # call reuses the array with the first call's contents still in it
    cases = [(41, 32, 64, 64, 32, 192, 8, "f16", 0.25), (42, 3, 17, 29, 24, 96, 3, "f16", 0.3)]
    assert dc.stack_noalloc_max_workspace_bytes() == 16 << 20
    for seed, N, H, W, C, E, nb, dtype, d in cases:
        print("noalloc case N=%d H=%d W=%d C=%d E=%d blocks=%d flags=%d" % (N, H, W, C, E, nb, flags), flush=True)
        xd, bw = _case(seed, N, H, W, C, E, nb, dtype, d)
        need = dc.stack_workspace_bytes(dc.shape_of(xd), bw, xd.dtype, flags)
        assert 0 < need <= dc.stack_noalloc_max_workspace_bytes()
        ref = _run(dc.stack_forward, xd, bw, flags)
        got = _run(dc.stack_forward_noalloc, xd, bw, flags)
        for a, b in zip(ref, got):
            assert torch.equal(a, b)


def test_noalloc_rejects_stack_beyond_the_array():
    # the multi-kernel chain's workspace at this size exceeds 16 MiB
    xd, bw = _case(43, 32, 56, 56, 24, 144, 1, "f16", 0.25)
    need = dc.stack_workspace_bytes(dc.shape_of(xd), bw, xd.dtype, dc.STACK_UNFUSED)
    assert need > dc.stack_noalloc_max_workspace_bytes()
    y = torch.zeros_like(xd)
    with pytest.raises(dc.DynconvError, match="workspace"):
        dc.stack_forward_noalloc(xd, y, bw, flags=dc.STACK_UNFUSED)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(y)) == 0  # nothing was enqueued
