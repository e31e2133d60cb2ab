"""Whole MobileNetV2 feature extractors (dynconv_network_forward) against
the oracle: each layer kind fed the oracle's input (masks bit-exact at gated
blocks, outputs within 1e-5 fp32 / 2e-2 fp16-bf16 normwise), the dense
network end to end (also on sampled images of the 64-image batch), the
network call equal to its layers called one by one, and the gated network
end to end (mask flips only next to the threshold)."""
import numpy as np
import pytest
import torch

from paper_1912_03203_amd import dynconv as dc
from paper_1912_03203_amd import inputs
from tests import util
from tests.test_gpu_parity import DEV, host, log, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dc.load()


def run_net(x_np, layers, dtype, biases=None, flags=0, masks=False):
    dt = dc.NAME_TO_DTYPE[dtype]
    net = dc.NetworkWeights(layers, dt, biases=biases)
    x = to_dev(x_np, dtype)
    out = dc.network_output_shape(dc.shape_of(x), net)
    y = torch.full((out.n, out.h, out.w, out.c), float("nan"), dtype=dt, device=DEV)
    ng = sum(1 for L in layers if L.get("gated"))
    mk = counts = None
    if masks and ng:
        total, cur = 0, (x.shape[1], x.shape[2])
        # masks of every gated block at its resolution (layer by layer shapes)
        sh = dc.shape_of(x)
        for i, L in enumerate(layers):
            if L.get("gated"):
                total += sh.n * sh.h * sh.w
            one = dc.NetworkWeights([L], dt, biases=[0.0] if L.get("gated") else None)
            sh = dc.network_output_shape(sh, one)
        mk = torch.full((total,), 7, dtype=torch.uint8, device=DEV)
        counts = torch.full((ng, 2), -1, dtype=torch.int32, device=DEV)
    call = dc.Network(x, y, net, flags=flags, masks=mk, counts=counts)
    call()
    torch.cuda.synchronize()
    return host(y), (None if mk is None else mk.cpu().numpy()), (None if counts is None else counts.cpu().numpy())


def rounder(dtype):
    return lambda a: util.nchw(inputs.round_to_storage(util.nhwc(a), dtype)).astype(np.float64)


@pytest.fixture(scope="module")
def net_f16():
    x, layers, dens = inputs.make_network_inputs(5, 2, 224, 224, dtype="f16")
    return x, layers, dens


def oracle_biases(x, layers, dens, dtype, labels=None):
    """Per gated block, the percentile bias of its oracle input (in order).
    With person labels (the pose network), each gated block's mask weights
    are first pointed at the people in its oracle input, as the benchmark's
    calibration does on the device's features."""
    import oracle
    biases = []
    cur = util.nchw(x).astype(np.float64)
    rnd = rounder(dtype)
    gi = 0
    rng = np.random.default_rng(11)
    for L in layers:
        if L.get("gated"):
            if labels is not None:
                L["w_m"] = inputs.person_mask_weights(rng, util.nhwc(cur), labels)
            _, s = util.oracle_mask_chunked(cur, L["w_m"], 0.0)
            b = float(inputs.percentile_bias(s, dens[gi]))
            biases.append(b)
            cur = rnd(oracle.block_forward(cur, L, L["w_m"], b)["y"])
            gi += 1
        else:
            cur, _ = oracle.network_forward(cur, [L], None, round_to=rnd)
    return biases


@pytest.mark.parametrize("dtype", ["f16", "f32", "bf16"])
def test_each_layer_teacher_forced(dtype):
    """Every layer of a 2 x 96x96 network on the oracle's input of that layer."""
    import oracle
    x, layers, dens = inputs.make_network_inputs(6, 2, 96, 96, dtype=dtype)
    biases = oracle_biases(x, layers, dens, dtype)
    _, gates, ins = oracle.network_forward(util.nchw(x), layers, biases, round_to=rounder(dtype), keep_inputs=True)
    gi = 0
    for i, L in enumerate(layers):
        xin = inputs.round_to_storage(util.nhwc(ins[i]), dtype)
        if L.get("gated"):
            o = oracle.block_forward(util.nchw(xin), L, L["w_m"], biases[gi])
            y, m, c = run_net(xin, [L], dtype, biases=[biases[gi]], masks=True)
            assert m.tobytes() == o["G"].tobytes(), "layer %d mask" % i
            assert tuple(c[0]) == (o["A"].size, o["D"].size)
            want = util.nhwc(o["y"])
            gi += 1
        else:
            y, _, _ = run_net(xin, [L], dtype)
            want = util.nhwc(oracle.network_forward(util.nchw(xin), [L], None)[0])
        err = util.normwise(y, want)
        log("  layer %2d %-8s %s err %.2e" % (i, L["kind"], y.shape, err))
        assert err <= util.TOL[dtype], "layer %d" % i


def test_dense_network_end_to_end(net_f16):
    import oracle
    x, layers, _ = net_f16
    y, _, _ = run_net(x, layers, "f16", flags=dc.STACK_DENSE)
    want, _ = oracle.network_forward(util.nchw(x), layers, None, round_to=rounder("f16"))
    err = util.normwise(y, util.nhwc(want))
    log("  dense network 2 x 224x224 -> %s, err %.2e" % (y.shape, err))
    assert err <= util.TOL["f16"]


def test_dense_network_full_batch_sampled_images():
    """The 64-image batch of the benchmark; images 0 and 63 against the
    oracle run on those images alone (images are independent)."""
    import oracle
    x, layers, _ = inputs.make_network_inputs(0, 64, 224, 224, dtype="f16")
    y, _, _ = run_net(x, layers, "f16", flags=dc.STACK_DENSE)
    for i in (0, 63):
        want, _ = oracle.network_forward(util.nchw(x[i:i + 1]), layers, None, round_to=rounder("f16"))
        err = util.normwise(y[i:i + 1], util.nhwc(want))
        log("  image %d err %.2e" % (i, err))
        assert err <= util.TOL["f16"]


def test_network_equals_layer_calls(net_f16):
    """The network call equals its layers called one at a time, bit for bit
    (gated and dense)."""
    x, layers, dens = net_f16
    biases = [0.05 * (i + 1) for i in range(sum(1 for L in layers if L.get("gated")))]
    for flags in (0, dc.STACK_DENSE):
        y, _, _ = run_net(x, layers, "f16", biases=biases, flags=flags)
        cur, gi = x, 0
        for L in layers:
            b = None
            if L.get("gated"):
                b = [biases[gi]]
                gi += 1
            cur, _, _ = run_net(cur, [L], "f16", biases=b, flags=flags)
        assert cur.tobytes() == y.tobytes()


def test_gated_network_end_to_end(net_f16):
    """Gated network with the oracle's biases.  The device's gated blocks see
    inputs computed in fp16 by the device, so decisions next to the threshold
    may differ from the oracle's.  Checked as in the parity reading for
    stacks: the oracle runs the network with the device's masks forced; at
    every gated block, a decision that differs from the oracle's own on the
    oracle's input has |m| <= ||w_m||_1 * 2e-2 * max|x| (the input's error
    envelope); the output is within 2e-2 of the forced-mask oracle."""
    import oracle
    x, layers, dens = net_f16
    biases = oracle_biases(x, layers, dens, "f16")
    y, m, c = run_net(x, layers, "f16", biases=biases, masks=True)
    rnd = rounder("f16")
    cur = util.nchw(x).astype(np.float64)
    off, gi, flips = 0, 0, []
    for L in layers:
        if L.get("gated"):
            N, C, H, W = cur.shape
            G = m[off:off + N * H * W]
            off += N * H * W
            Go, mo = oracle.mask(cur.astype(np.float32), L["w_m"], biases[gi])
            d = G != Go
            envelope = np.abs(L["w_m"]).sum() * util.TOL["f16"] * np.abs(cur).max()
            assert (np.abs(mo[d]) <= envelope).all(), "gated block %d" % gi
            flips.append(int(d.sum()))
            assert int(c[gi][0]) == int(G.sum())
            cur = rnd(oracle.block_dense(cur, L, G)[0])
            gi += 1
        else:
            cur, _ = oracle.network_forward(cur, [L], None, round_to=rnd)
    log("  decisions differing from the oracle's own, per gated block: %s" % flips)
    err = util.normwise(y, util.nhwc(cur))
    log("  gated network vs forced-mask oracle: err %.2e" % err)
    assert err <= util.TOL["f16"]


def test_gated_network_full_batch_sampled_images():
    """The benchmark's launch configuration: the gated network on the 64-image
    batch (224x224x3, fp16), with mask biases set by the oracle on images 0
    and 63.  Images are independent, so those two images are checked as in
    test_gated_network_end_to_end against the oracle run on them alone."""
    import oracle
    x, layers, dens = inputs.make_network_inputs(0, 64, 224, 224, dtype="f16")
    pick = [0, 63]
    xs = np.ascontiguousarray(x[pick])
    biases = oracle_biases(xs, layers, dens, "f16")
    y, m, _ = run_net(x, layers, "f16", biases=biases, masks=True)
    rnd = rounder("f16")
    cur = util.nchw(xs).astype(np.float64)
    off, gi, flips = 0, 0, []
    for L in layers:
        if L.get("gated"):
            _, _, H, W = cur.shape
            hw = H * W
            G = np.concatenate([m[off + i * hw: off + (i + 1) * hw] for i in pick])
            off += 64 * hw
            Go, mo = oracle.mask(cur.astype(np.float32), L["w_m"], biases[gi])
            d = G != Go
            envelope = np.abs(L["w_m"]).sum() * util.TOL["f16"] * np.abs(cur).max()
            assert (np.abs(mo[d]) <= envelope).all(), "gated block %d" % gi
            flips.append(int(d.sum()))
            cur = rnd(oracle.block_dense(cur, L, G)[0])
            gi += 1
        else:
            cur, _ = oracle.network_forward(cur, [L], None, round_to=rnd)
    log("  decisions differing from the oracle's own, per gated block: %s" % flips)
    err = util.normwise(y[pick], util.nhwc(cur))
    log("  images 0 and 63 of the gated 64-image batch vs forced-mask oracle: err %.2e" % err)
    assert err <= util.TOL["f16"]


def test_pose_network_end_to_end():
    """The pose network (256x256x3 ellipse images -> MobileNetV2 backbone ->
    8 stacked gated blocks at 64x64x32) on 2 images, in the benchmark's
    configuration: every gated block's mask unit pointed at the people in its
    input (concentrated masks, cells fully active on the people), the
    oracle's biases; checked as in test_gated_network_end_to_end."""
    import oracle
    x, layers, dens, labels = inputs.make_pose_network_inputs(7, 2, dtype="f16")
    biases = oracle_biases(x, layers, dens, "f16", labels=labels)
    y, m, c = run_net(x, layers, "f16", biases=biases, masks=True)
    assert y.shape == (2, 64, 64, 32)
    rnd = rounder("f16")
    cur = util.nchw(x).astype(np.float64)
    off, gi, flips = 0, 0, []
    for L in layers:
        if L.get("gated"):
            N, C, H, W = cur.shape
            G = m[off:off + N * H * W]
            off += N * H * W
            Go, mo = oracle.mask(cur.astype(np.float32), L["w_m"], biases[gi])
            d = G != Go
            envelope = np.abs(L["w_m"]).sum() * util.TOL["f16"] * np.abs(cur).max()
            assert (np.abs(mo[d]) <= envelope).all(), "gated block %d" % gi
            flips.append(int(d.sum()))
            assert int(c[gi][0]) == int(G.sum())
            cur = rnd(oracle.block_dense(cur, L, G)[0])
            gi += 1
        else:
            cur, _ = oracle.network_forward(cur, [L], None, round_to=rnd)
    log("  pose network: decisions differing from the oracle's own, per gated block: %s" % flips)
    err = util.normwise(y, util.nhwc(cur))
    log("  pose network vs forced-mask oracle: err %.2e" % err)
    assert err <= util.TOL["f16"]


POINTWISE_CASES = [
    # dtype, (N, H, W), C, O: every output-range width (2..12 tiles of 16),
    # contraction chunks of 1..8 steps of 32 and several chunks, one partial
    # 64-position tile, and large position counts
    ("f16", (16, 112, 112), 16, 96),
    ("f16", (4, 56, 56), 24, 144),
    ("bf16", (64, 7, 7), 960, 320),
    ("f16", (64, 7, 7), 320, 1280),
    ("f16", (2, 3, 5), 576, 160),
    ("f32", (3, 9, 11), 40, 200),
    ("f32", (64, 7, 7), 960, 320),
    ("bf16", (1, 1, 1), 8, 8),
    ("f16", (8, 14, 14), 136, 72),
]


@pytest.mark.parametrize("dtype,nhw,C,O", POINTWISE_CASES)
def test_pointwise_layer(dtype, nhw, C, O):
    """A network of one 1x1 convolution against the oracle's conv1x1."""
    import oracle.network as onet
    N, H, W = nhw
    rng = inputs.rng_for(4000 + C + O)
    x = inputs.round_to_storage(rng.normal(0.0, 1.0, size=(N, H, W, C)), dtype)
    L = {"kind": "conv1x1", "w": inputs.round_to_storage(rng.normal(0.0, 0.05, size=(O, C)), dtype),
         "b": rng.normal(0.0, 0.05, size=O).astype(np.float32), "act": 2}
    y, _, _ = run_net(x, [L], dtype)
    want = util.nhwc(onet.conv1x1(util.nchw(x), L["w"], L["b"], L["act"]))
    err = util.normwise(y, want)
    log("  pointwise %s %s C=%d O=%d err %.2e" % (dtype, nhw, C, O, err))
    assert err <= util.TOL[dtype]


@pytest.mark.parametrize("dtype,nhw,stride,c,co,e", [
    ("f16", (2, 9, 7), 2, 16, 24, 96), ("bf16", (3, 1, 13), 2, 24, 32, 48), ("f32", (2, 11, 5), 1, 8, 16, 40),
    ("f16", (1, 2, 2), 2, 32, 64, 1792), ("bf16", (4, 17, 30), 1, 40, 16, 40)])
def test_strided_and_widening_blocks(dtype, nhw, stride, c, co, e):
    """Ungated blocks of odd sizes, both strides, widening outputs (no
    residual), a 1792-channel hidden layer and expansion factor 1."""
    import oracle.network as onet
    N, H, W = nhw
    rng = inputs.rng_for(4200 + c + e)
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, c), dtype)

    def wgt(*shape):
        return inputs.round_to_storage(rng.normal(0.0, 0.1, size=shape), dtype)

    t1 = e != c
    L = {"kind": "block", "stride": stride, "acts": (2, 2, 0),
         "w1": wgt(e, c) if t1 else None, "b1": rng.normal(0, 0.1, e).astype(np.float32) if t1 else None,
         "w2": wgt(e, 9), "b2": rng.normal(0, 0.1, e).astype(np.float32),
         "w3": wgt(co, e), "b3": rng.normal(0, 0.1, co).astype(np.float32)}
    y, _, _ = run_net(x, [L], dtype)
    want = util.nhwc(onet.dense_block(util.nchw(x), L))
    assert y.shape == want.shape
    err = util.normwise(y, want)
    log("  block %s %s s%d %d->%d (E %d) err %.2e" % (dtype, nhw, stride, c, co, e, err))
    assert err <= util.TOL[dtype]


@pytest.mark.parametrize("dtype,nhw,stride,c,co,e", [
    ("bf16", (260, 19, 19), 2, 24, 32, 40),   # 4 output tiles per image (ragged), 2 slices (last partial)
    ("f16", (54, 30, 33), 1, 64, 64, 144),    # two contraction steps, 4.5 slices, residual
    ("f16", (64, 56, 56), 2, 16, 24, 96)])    # MobileNetV2's second block at batch 64
def test_expand_depthwise_one_launch(dtype, nhw, stride, c, co, e):
    """Ungated blocks with enough 8x8 output tiles run the expansion and the
    depthwise in one launch (k_expand_dw); against the oracle's dense block."""
    import oracle.network as onet
    N, H, W = nhw
    rng = inputs.rng_for(4400 + c + e)
    x = inputs.round_to_storage(inputs.blob_features(rng, N, H, W, c), dtype)

    def wgt(*shape):
        return inputs.round_to_storage(rng.normal(0.0, 0.1, size=shape), dtype)

    L = {"kind": "block", "stride": stride, "acts": (2, 2, 0),
         "w1": wgt(e, c), "b1": rng.normal(0, 0.1, e).astype(np.float32),
         "w2": wgt(e, 9), "b2": rng.normal(0, 0.1, e).astype(np.float32),
         "w3": wgt(co, e), "b3": rng.normal(0, 0.1, co).astype(np.float32)}
    net = dc.NetworkWeights([L], dc.NAME_TO_DTYPE[dtype])
    xd = to_dev(x, dtype)
    out = dc.network_output_shape(dc.shape_of(xd), net)
    y = torch.empty((out.n, out.h, out.w, out.c), dtype=xd.dtype, device=DEV)
    names = dc.Network(xd, y, net).launch_names()
    assert names == ["k_expand_dw", "k_conv1x1"], names
    yg, _, _ = run_net(x, [L], dtype)
    want = util.nhwc(onet.dense_block(util.nchw(x), L))
    err = util.normwise(yg, want)
    log("  expand+dw %s %s s%d %d->%d (E %d) err %.2e" % (dtype, nhw, stride, c, co, e, err))
    assert err <= util.TOL[dtype]


@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_ungated_residual_block(dtype):
    """A stride-1 block of equal widths without a mask unit runs dense and
    adds its input (the projection's residual operand)."""
    import oracle.network as onet
    rng = inputs.rng_for(4100)
    C, E = 24, 144
    x = inputs.round_to_storage(inputs.blob_features(rng, 3, 20, 17, C), dtype)
    w = inputs.block_weights(rng, C, E, dtype=dtype)
    L = {"kind": "block", "stride": 1, "acts": (2, 2, 0), "w1": w["w1"], "b1": w["b1"], "w2": w["w2"],
         "b2": w["b2"], "w3": w["w3"], "b3": w["b3"]}
    y, _, _ = run_net(x, [L], dtype)
    want = util.nhwc(onet.dense_block(util.nchw(x), L))
    err = util.normwise(y, want)
    log("  ungated residual block %s err %.2e" % (dtype, err))
    assert err <= util.TOL[dtype]


@pytest.mark.parametrize("dtype,nhw,ci,co,stride", [
    ("f16", (2, 17, 23), 3, 32, 2), ("bf16", (1, 9, 8), 16, 40, 1), ("f32", (3, 5, 7), 1, 8, 2),
    ("f16", (1, 1, 1), 4, 72, 1), ("f16", (2, 30, 3), 8, 200, 2), ("bf16", (3, 31, 29), 7, 8, 2),
    ("f16", (2, 40, 37), 11, 24, 1)])
def test_full_conv3x3_layer(dtype, nhw, ci, co, stride):
    """A network of one full 3x3 convolution (the stem's kind) against the
    oracle's conv3x3: odd sizes, both strides, output counts that are not
    multiples of 32, 1-16 input channels (1-5 contraction steps of 32 on the
    matrix cores in 16-bit storage; fp32 on the VALU)."""
    import oracle.network as onet
    N, H, W = nhw
    rng = inputs.rng_for(4300 + ci + co)
    x = inputs.round_to_storage(rng.normal(0.0, 1.0, size=(N, H, W, ci)), dtype)
    L = {"kind": "conv3x3", "w": inputs.round_to_storage(rng.normal(0.0, 0.1, size=(co, ci, 3, 3)), dtype),
         "b": rng.normal(0.0, 0.1, size=co).astype(np.float32), "stride": stride, "act": 2}
    y, _, _ = run_net(x, [L], dtype)
    want = util.nhwc(onet.conv3x3(util.nchw(x), L["w"], L["b"], stride, L["act"]))
    assert y.shape == want.shape
    err = util.normwise(y, want)
    log("  conv3x3 %s %s %d->%d s%d err %.2e" % (dtype, nhw, ci, co, stride, err))
    assert err <= util.TOL[dtype]
