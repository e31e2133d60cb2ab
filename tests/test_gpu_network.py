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


def oracle_biases(x, layers, dens, dtype):
    """Per gated block, the percentile bias of its oracle input (in order)."""
    import oracle
    biases = []
    cur = util.nchw(x).astype(np.float64)
    rnd = rounder(dtype)
    gi = 0
    for L in layers:
        if L.get("gated"):
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
