"""Parity of the one-launch block kernel (the stack's execution for at most
64 channels) with the CPU oracle, and its agreement with the
multi-kernel chain.  Same tolerances as the per-block calls: masks and counts
bit-exact, outputs within 1e-5 (fp32) / 2e-2 (fp16, bf16) normwise, inactive
positions untouched."""
import numpy as np
import pytest
import torch

from paper_1912_03203_amd import dynconv as dc
from paper_1912_03203_amd import inputs
from tests import util
from tests.test_gpu_parity import DEV, check_block_output, check_stack_end_to_end, host, log, oracle_stack, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dc.load()


def run_stack(x_np, blocks_np, biases, dtype, flags=0, in_place=False):
    dt = dc.NAME_TO_DTYPE[dtype]
    bw = [dc.BlockWeights.from_arrays(w, dt, b_mask=b) for w, b in zip(blocks_np, biases)]
    n, h, w, c = x_np.shape
    nb = len(bw)
    # every buffer the call writes is followed by guard bytes
    xg = util.Guarded(n * h * w * c, dc.NAME_TO_DTYPE[dtype], fill=None)
    x = xg.t.view(n, h, w, c)
    x.copy_(to_dev(x_np, dtype))
    mg = util.Guarded(nb * n * h * w, torch.uint8, fill=7)
    cg = util.Guarded(nb * 2, torch.int32, fill=-5)
    masks, counts = mg.t.view(nb, n * h * w), cg.t.view(nb, 2)
    yg = xg if in_place else util.Guarded(x.numel(), x.dtype, fill=float("nan"))
    y = x if in_place else yg.t.view(x.shape)
    wsg = util.Guarded(dc.stack_workspace_bytes(dc.shape_of(x), bw, x.dtype, flags), torch.uint8, fill=None)
    stack = dc.Stack(x, y, bw, flags=flags, masks=masks, counts=counts, ws=wsg.t)
    stack()
    torch.cuda.synchronize()
    assert all(g.intact() for g in (xg, mg, cg, yg, wsg)), "a buffer written past its end"
    if not in_place:
        assert host(x).tobytes() == np.asarray(x_np, np.float32).tobytes()  # input untouched
    return {"y": y, "masks": masks, "counts": counts, "names": stack.launch_names()}


def uses_cells(dtype, C, E):
    """Narrow 16-bit blocks run the work-balanced cell kernel, the others the
    patch kernel."""
    return dtype != "f32" and C <= 32 and E <= 192


def expected_launches(dtype, C, E, blocks=1):
    if uses_cells(dtype, C, E):
        return ["k_mask_cells"] + ["k_block_cells"] * blocks + ["k_band_counts"]
    return ["k_block_fused"] * blocks + ["k_band_counts"]


FUSED_CASES = [
    # name, dtype, (N, H, W, C, E), density, seed
    ("fp32_parity_block", "f32", (1, 32, 32, 32, 192), 0.5, 0),
    ("stage2_d0.10", "f16", (32, 56, 56, 24, 144), 0.10, 0),
    ("stage2_d0.25", "f16", (32, 56, 56, 24, 144), 0.25, 0),
    ("stage2_d0.50", "f16", (32, 56, 56, 24, 144), 0.50, 1),
    ("stage2_d0.75", "f16", (32, 56, 56, 24, 144), 0.75, 19),
    ("stage2_d0.90", "f16", (32, 56, 56, 24, 144), 0.90, 3),
    ("pose_d0.25", "f16", (32, 64, 64, 32, 192), 0.25, 2),
    ("ragged_bf16_c40", "bf16", (3, 7, 11, 40, 80), 0.3, 4),
    ("c64_e384_f16", "f16", (2, 9, 64, 64, 384), 0.4, 5),
    ("width1_f16", "f16", (2, 300, 1, 16, 48), 0.3, 6),
    ("width7_f32", "f32", (3, 20, 7, 8, 16), 0.6, 7),
    ("height1_bf16", "bf16", (5, 1, 50, 24, 96), 0.5, 8),
    ("wide_w100_f16", "f16", (2, 9, 100, 32, 96), 0.3, 9),
    ("wide_w130_bf16", "bf16", (1, 7, 130, 24, 48), 0.5, 10),
    ("fp32_c48", "f32", (2, 10, 20, 48, 96), 0.4, 11),
    ("fp32_c64_w33", "f32", (1, 6, 33, 64, 64), 0.6, 12),
    ("c96_e576_f16", "f16", (4, 14, 14, 96, 576), 0.4, 13),   # 16-bit, 65-128 channels
    ("c128_bf16_w40", "bf16", (2, 10, 40, 128, 256), 0.3, 14),
    ("c72_f16_h1", "f16", (3, 1, 30, 72, 144), 0.5, 15),
    ("c120_bf16_w1", "bf16", (2, 70, 1, 120, 128), 0.4, 16),
    ("c128_f16_w23", "f16", (2, 9, 23, 128, 272), 0.3, 18),
    # cell kernel: ragged cells, a single cell, hidden widths with a partial
    # last slice, more cells than the persistent grid's waves
    ("cells_ragged_bf16", "bf16", (3, 7, 11, 24, 96), 0.4, 20),
    ("cells_one_cell_f16", "f16", (1, 3, 5, 8, 16), 0.5, 21),
    ("cells_e80_f16", "f16", (4, 13, 21, 16, 80), 0.3, 22),
    ("cells_e176_bf16_w70", "bf16", (2, 9, 70, 32, 176), 0.35, 24),
    ("cells_many_f16", "f16", (96, 64, 64, 32, 192), 0.25, 23),
    # the pose shape nearly dense (about 32 active cells per workgroup, two
    # or more per wave) and very sparse (most workgroups with 0-2 cells)
    ("pose_d0.90_bf16", "bf16", (32, 64, 64, 32, 192), 0.90, 25),
    ("pose_d0.05_f16", "f16", (32, 64, 64, 32, 192), 0.05, 26),
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=[c[0] for c in FUSED_CASES])
def test_fused_block_parity(case):
    name, dtype, (N, H, W, C, E), density, seed = case
    log("fused block %s" % name)
    rng = inputs.rng_for(2000 + seed)
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, C), dtype)
    wts = inputs.block_weights(rng, C, E, dtype=dtype)
    o = util.oracle_calibrated_block(x, wts, density, dtype)
    g = run_stack(x, [wts], [o["b_m"]], dtype)
    assert g["names"] == expected_launches(dtype, C, E)
    assert g["masks"][0].cpu().numpy().tobytes() == o["G"].tobytes()
    assert tuple(int(v) for v in g["counts"][0].cpu()) == (o["A"].size, o["D"].size)
    check_block_output(host(g["y"]), x, o["y"], o["G"], dtype)
    # the same arithmetic as the kernel chain, bit for bit
    chain = run_stack(x, [wts], [o["b_m"]], dtype, flags=dc.STACK_UNFUSED)
    assert torch.equal(g["y"], chain["y"])


def test_cells_schedule_concentrated_work():
    """All active positions in one image of a 16-image batch: the cell
    kernel's equal-work shares put that image's cells on many workgroups and
    leave the others' shares to the empty cells; masks, counts and output as
    the oracle, over a two-block stack (the second block's shares come from
    the first block's per-cell counts)."""
    rng = inputs.rng_for(55)
    N, H, W, C, E = 16, 64, 64, 32, 192
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, C), "f16")
    x[1:] = 0.0
    blocks = [inputs.block_weights(rng, C, E, dtype="f16") for _ in range(2)]
    xs, outs = oracle_stack(x, blocks, 0.3 / N, "f16")
    for o in outs:
        assert o["G"].reshape(N, -1)[1:].sum() == 0 and o["G"].sum() > 0
    biases = [o["b_m"] for o in outs]
    g = run_stack(x, blocks, biases, "f16")
    assert g["names"] == expected_launches("f16", C, E, blocks=2)
    check_stack_end_to_end(x, blocks, biases, g["masks"].cpu().numpy(), g["counts"].cpu().numpy(),
                           host(g["y"]), "f16")
    assert host(g["y"])[1:].tobytes() == x[1:].tobytes()


@pytest.mark.parametrize("bias", [-np.inf, np.inf])
def test_fused_empty_and_full_masks(bias):
    rng = inputs.rng_for(9)
    N, H, W, C, E = 4, 12, 40, 24, 144
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, C), "f16")
    wts = inputs.block_weights(rng, C, E, dtype="f16")
    g = run_stack(x, [wts], [bias], "f16")
    P, Pd = (int(v) for v in g["counts"][0].cpu())
    if bias < 0:
        assert (P, Pd) == (0, 0)
        assert host(g["y"]).tobytes() == x.tobytes()
    else:
        assert (P, Pd) == (N * H * W, N * H * W)
        dense = run_stack(x, [wts], [0.0], "f16", flags=dc.STACK_DENSE)
        assert torch.equal(g["y"], dense["y"])


@pytest.mark.parametrize("dtype,shape,nb", [("f16", (32, 64, 64, 32, 192), 8),
                                            # 81,920 cells: 5 count words per thread of the
                                            # cell kernel's schedule (its search over them)
                                            ("f16", (320, 64, 64, 32, 192), 2),
                                            ("bf16", (5, 11, 19, 24, 144), 3),
                                            ("bf16", (4, 20, 28, 48, 96), 3),
                                            ("f32", (2, 16, 16, 16, 96), 2),
                                            ("f16", (2, 12, 90, 64, 128), 2),
                                            ("f32", (1, 9, 40, 40, 80), 3),
                                            ("f16", (4, 14, 14, 96, 576), 2),
                                            ("bf16", (2, 9, 33, 120, 128), 2)])
def test_fused_stack_matches_kernel_chain(dtype, shape, nb):
    """One-launch blocks (out of place and in place, which takes the extra copy
    for an odd block count) and the multi-kernel chain give the same masks,
    counts and outputs bit for bit: same operand fragments, same summation
    order, same roundings."""
    N, H, W, C, E = shape
    rng = inputs.rng_for(31)
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, C), dtype)
    blocks = [inputs.block_weights(rng, C, E, dtype=dtype) for _ in range(nb)]
    _, s = util.oracle_mask_chunked(util.nchw(x), blocks[0]["w_m"], 0.0)
    b0 = inputs.percentile_bias(s, 0.3)
    biases = [b0] + [b0 * 0.5] * (nb - 1)  # later densities drift; not calibrated here
    ref = run_stack(x, blocks, biases, dtype, flags=dc.STACK_UNFUSED, in_place=True)
    assert ref["names"][0] == "k_mask" and "k_block_fused" not in ref["names"]
    for in_place in (False, True):
        g = run_stack(x, blocks, biases, dtype, in_place=in_place)
        assert ("k_block_cells" if uses_cells(dtype, C, E) else "k_block_fused") in g["names"]
        assert torch.equal(g["masks"], ref["masks"])
        assert torch.equal(g["counts"], ref["counts"])
        assert torch.equal(g["y"], ref["y"])


def test_fused_pose_stack_teacher_forced_and_end_to_end():
    """Every block of the 8-block pose stack as a one-launch block fed the
    oracle's input; then the whole fused stack end to end."""
    wl = inputs.WORKLOADS["pose_stack8_64x64x32_f16"]
    x0, blocks, _ = inputs.make_block_inputs(wl, 0)
    xs, outs = oracle_stack(x0, blocks, 0.25, wl.dtype)
    for b in range(wl.blocks):
        g = run_stack(xs[b], [blocks[b]], [outs[b]["b_m"]], wl.dtype)
        assert g["masks"][0].cpu().numpy().tobytes() == outs[b]["G"].tobytes()
        check_block_output(host(g["y"]), xs[b], outs[b]["y"], outs[b]["G"], wl.dtype)
    biases = [o["b_m"] for o in outs]
    g = run_stack(x0, blocks, biases, wl.dtype)
    check_stack_end_to_end(x0, blocks, biases, g["masks"].cpu().numpy(), g["counts"].cpu().numpy(),
                           host(g["y"]), wl.dtype)


def test_fused_stack_in_graph_replays():
    """The stack captured in a HIP graph: several replays, with eager work and
    synchronisation between them, each equal to the eager result."""
    wl = inputs.WORKLOADS["pose_stack8_64x64x32_f16"]
    x0, blocks, _ = inputs.make_block_inputs(wl, 3)
    dt = dc.NAME_TO_DTYPE[wl.dtype]
    _, s = util.oracle_mask_chunked(util.nchw(x0), blocks[0]["w_m"], 0.0)
    b0 = float(inputs.percentile_bias(s, 0.25))
    bw = [dc.BlockWeights.from_arrays(w, dt, b_mask=b0) for w in blocks]
    x = to_dev(x0, wl.dtype)
    counts = torch.zeros(wl.blocks, 2, dtype=torch.int32, device=DEV)
    for flags in (0, dc.STACK_DENSE):
        y = torch.empty_like(x)
        stack = dc.Stack(x, y, bw, flags=flags, counts=counts)
        stack()
        torch.cuda.synchronize()
        eager = y.clone()
        eager_counts = counts.clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            stack()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            stack()
        for _ in range(4):
            y.fill_(0)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, eager)
            if flags == 0:
                assert torch.equal(counts, eager_counts)
