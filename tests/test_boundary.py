"""The C-ABI library: it loads, exports every entry point that
include/dynconv.h declares, sizes workspaces on the host, and rejects invalid
arguments before anything is enqueued.  Runs without a GPU: every call here
fails host-side validation, so no HIP call is made."""
import ctypes
import os
import re

import pytest

from paper_1912_03203_amd import dynconv as dc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dynconv.h")

OK, ERR_NULL, ERR_SHAPE, ERR_DTYPE, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_ALIGN, ERR_WORKSPACE, \
    ERR_HIP, ERR_ARG = range(10)

FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dynconv_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    # the sanitizer tests point this at an instrumented host-only build
    override = os.environ.get("DYNCONV_TEST_LIB")
    if override:
        return dc.load(override)
    if not os.path.exists(dc.LIB_PATH):
        from paper_1912_03203_amd import build

        build.build()
    return dc.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(dc.EXPORTED) == set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings_and_version(lib):
    for code in range(10):
        s = dc.status_str(code)
        assert s and s != "unknown status"
    assert dc.status_str(99) == "unknown status"
    assert b"gfx950" in lib.dynconv_version()


def fake_block(C=32, E=192, Co=None, acts=(2, 2, 0), **over):
    Co = C if Co is None else Co
    b = dc.Block(C, E, Co, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, acts[0], acts[1], acts[2], FAKE, 0.0)
    for k, v in over.items():
        setattr(b, k, v)
    return b


@pytest.mark.parametrize("entry", ["dynconv_mask", "dynconv_mask_gsoftmax"])
def test_mask_validation(lib, entry):
    s = dc.Shape(2, 8, 8, 32)
    f = getattr(lib, entry)
    assert f(None, s, 1, FAKE, 0.0, FAKE, None, None) == ERR_NULL
    assert f(FAKE, s, 1, None, 0.0, FAKE, None, None) == ERR_NULL
    assert f(FAKE, s, 1, FAKE, 0.0, None, None, None) == ERR_NULL
    assert f(FAKE, s, 7, FAKE, 0.0, FAKE, None, None) == ERR_DTYPE
    assert f(FAKE, dc.Shape(0, 8, 8, 32), 1, FAKE, 0.0, FAKE, None, None) == ERR_SHAPE
    assert f(FAKE, dc.Shape(2, -1, 8, 32), 1, FAKE, 0.0, FAKE, None, None) == ERR_SHAPE
    assert f(FAKE, dc.Shape(2, 8, 8, 0), 1, FAKE, 0.0, FAKE, None, None) == ERR_SHAPE
    assert f(FAKE, dc.Shape(2, 8, 8, 12), 1, FAKE, 0.0, FAKE, None, None) == ERR_UNSUPPORTED
    assert f(FAKE, dc.Shape(2, 8, 8, 264), 1, FAKE, 0.0, FAKE, None, None) == ERR_UNSUPPORTED
    assert f(FAKE, dc.Shape(1, 1, 4097, 32), 1, FAKE, 0.0, FAKE, None, None) == ERR_UNSUPPORTED
    # N*H*W*9 would overflow int32 indices
    assert f(FAKE, dc.Shape(4096, 4096, 16, 8), 1, FAKE, 0.0, FAKE, None, None) == ERR_SHAPE
    assert f(FAKE + 8, s, 1, FAKE, 0.0, FAKE, None, None) == ERR_ALIGN


def test_build_indices_validation(lib):
    s = dc.Shape(2, 8, 8, 0)
    need = lib.dynconv_indices_workspace_bytes(s)
    assert need == 256 + 256 + 256  # 16 rows of int2 counts, 17 of offsets, 16 mask words; 256-aligned
    idx = dc.Indices(FAKE, FAKE, FAKE, FAKE, 128)
    f = lib.dynconv_build_indices
    assert f(None, s, 1, ctypes.byref(idx), FAKE, need, None) == ERR_NULL
    assert f(FAKE, s, 1, None, FAKE, need, None) == ERR_NULL
    bad = dc.Indices(FAKE, None, FAKE, FAKE, 128)
    assert f(FAKE, s, 1, ctypes.byref(bad), FAKE, need, None) == ERR_NULL
    assert f(FAKE, s, -1, ctypes.byref(idx), FAKE, need, None) == ERR_ARG
    assert f(FAKE, s, 4, ctypes.byref(idx), FAKE, need, None) == ERR_ARG
    small = dc.Indices(FAKE, FAKE, FAKE, FAKE, 127)
    assert f(FAKE, s, 1, ctypes.byref(small), FAKE, need, None) == ERR_CAPACITY
    assert f(FAKE, s, 1, ctypes.byref(idx), FAKE, need - 1, None) == ERR_WORKSPACE
    assert f(FAKE, s, 1, ctypes.byref(idx), None, need, None) == ERR_WORKSPACE
    assert f(FAKE, dc.Shape(2, 0, 8, 0), 1, ctypes.byref(idx), FAKE, need, None) == ERR_SHAPE


def test_block_validation(lib):
    s = dc.Shape(2, 8, 8, 32)
    b = fake_block()
    need = lib.dynconv_block_workspace_bytes(s, ctypes.byref(b), 1)
    # hidden tensor: N*H*W rows plus one zero row, x 192 channels x fp16, 256-aligned
    assert need == (2 * 8 * 8 * 192 * 2 + 192 * 2 + 255) // 256 * 256
    f = lib.dynconv_block_forward

    def call(x=FAKE, y=FAKE, shape=s, dt=1, blk=b, idx=None, ws=FAKE, nbytes=need):
        return f(x, y, shape, dt, ctypes.byref(blk) if blk is not None else None,
                 ctypes.byref(idx) if idx is not None else None, ws, nbytes, None)

    assert call(x=None) == ERR_NULL
    assert call(blk=None) == ERR_NULL
    assert call(blk=fake_block(w_dw=None)) == ERR_NULL
    assert call(dt=3) == ERR_DTYPE
    assert call(blk=fake_block(C=24)) == ERR_SHAPE  # block channels differ from the map's
    assert call(blk=fake_block(Co=16)) == ERR_UNSUPPORTED  # no identity path
    assert call(blk=fake_block(E=152)) == ERR_UNSUPPORTED
    assert call(blk=fake_block(E=1552)) == ERR_UNSUPPORTED
    assert call(blk=fake_block(acts=(2, 3, 0))) == ERR_ARG
    assert call(blk=fake_block(w_project=FAKE + 4)) == ERR_ALIGN
    assert call(y=FAKE + 64) == ERR_SHAPE  # partial overlap with x
    assert call(idx=dc.Indices(FAKE, FAKE, FAKE, FAKE, 127)) == ERR_CAPACITY
    assert call(idx=dc.Indices(FAKE, FAKE, None, FAKE, 128)) == ERR_NULL
    assert call(nbytes=need - 1) == ERR_WORKSPACE
    assert call(ws=None) == ERR_WORKSPACE


def test_stack_validation(lib):
    s = dc.Shape(4, 16, 16, 32)
    blocks = (dc.Block * 3)(fake_block(), fake_block(E=96), fake_block())
    npos = 4 * 16 * 16
    rows = 4 * 16

    def up(v):
        return (v + 255) // 256 * 256

    # 16-bit blocks of at most 32 channels and 192 hidden: the cell kernel's
    # ping-pong copy of x, two masks, counts, per-cell counts (2 x 8 cells:
    # 16 per 16 x 16 image) and two per-cell active-count buffers
    fused = lib.dynconv_stack_workspace_bytes(s, blocks, 3, 1, 0)
    ncells = 4 * 8 * 2
    assert fused == up(npos * 32 * 2) + 2 * up(npos) + up(8 * 3) + up(8 * 3 * ncells) + 2 * up(ncells)
    # fp32: the patch kernel's ping-pong copy, two masks, counts, per-patch
    # counts (16 x 16 images give one patch per image at full height; a batch
    # this small gets patches of one row, 64 in all)
    assert lib.dynconv_stack_workspace_bytes(s, blocks, 3, 0, 0) == \
        up(npos * 32 * 4) + 2 * up(npos) + up(8 * 3) + up(8 * 3 * 64)
    # a hidden width above 192 leaves the cell kernel for the patch kernel
    e384 = (dc.Block * 1)(fake_block(E=384))
    assert lib.dynconv_stack_workspace_bytes(s, e384, 1, 1, 0) == \
        up(npos * 32 * 2) + 2 * up(npos) + up(8) + up(8 * 64)
    # kernel chain: mask, lists, counts, row scratch, hidden tensor of the widest block
    need = lib.dynconv_stack_workspace_bytes(s, blocks, 3, 1, 2)
    assert need == (npos + 4 * npos + 4 * npos + 36 * npos + up(8 * 3) + up(8 * rows)
                    + up(8 * (rows + 1)) + up(8 * rows) + up((npos + 1) * 192 * 2))
    # more than 64 channels in fp32, more than 128 in 16-bit, take the kernel chain
    for dt, c in ((0, 72), (1, 136)):
        wide_c = dc.Shape(1, 4, 100, c)
        blk = (dc.Block * 1)(fake_block(C=c))
        assert lib.dynconv_stack_workspace_bytes(wide_c, blk, 1, dt, 0) == \
            lib.dynconv_stack_workspace_bytes(wide_c, blk, 1, dt, 2)
    # 16-bit up to 128 channels stays on the one-launch path (64-position patches)
    c96 = dc.Shape(2, 14, 14, 96)
    blk96 = (dc.Block * 1)(fake_block(C=96, E=576))
    assert lib.dynconv_stack_workspace_bytes(c96, blk96, 1, 1, 0) != \
        lib.dynconv_stack_workspace_bytes(c96, blk96, 1, 1, 2)
    # wide images stay on the one-launch paths: 26 cells of 2 x 8; for the
    # patch kernel (fp32) column strips of 25 and, for a batch this small,
    # row strips of 1 (16 patches)
    wide = dc.Shape(1, 4, 100, 32)
    assert lib.dynconv_stack_workspace_bytes(wide, blocks, 3, 1, 0) == \
        up(400 * 32 * 2) + 2 * up(400) + up(8 * 3) + up(8 * 3 * 26) + 2 * up(26)
    assert lib.dynconv_stack_workspace_bytes(wide, blocks, 3, 0, 0) == \
        up(400 * 32 * 4) + 2 * up(400) + up(8 * 3) + up(8 * 3 * 16)
    f = lib.dynconv_stack_forward
    assert f(None, FAKE, s, 1, blocks, 3, 0, None, None, FAKE, need, None) == ERR_NULL
    assert f(FAKE, None, s, 1, blocks, 3, 0, None, None, FAKE, need, None) == ERR_NULL
    assert f(FAKE, FAKE, s, 1, blocks, 0, 0, None, None, FAKE, need, None) == ERR_ARG
    assert f(FAKE, FAKE, s, 1, blocks, 1025, 0, None, None, FAKE, need, None) == ERR_ARG
    assert f(FAKE, FAKE, s, 1, blocks, 3, 8, None, None, FAKE, need, None) == ERR_ARG
    assert f(FAKE, FAKE, s, 1, blocks, 3, 2, None, None, FAKE, need - 1, None) == ERR_WORKSPACE
    assert f(FAKE, FAKE, s, 1, blocks, 3, 0, None, None, FAKE, fused - 1, None) == ERR_WORKSPACE
    assert f(FAKE, FAKE + 64, s, 1, blocks, 3, 0, None, None, FAKE, fused, None) == ERR_SHAPE
    nomask = (dc.Block * 1)(fake_block(w_mask=None))
    need1 = lib.dynconv_stack_workspace_bytes(s, nomask, 1, 1, 0)
    assert f(FAKE, FAKE, s, 1, nomask, 1, 0, None, None, FAKE, need1, None) == ERR_NULL
    assert lib.dynconv_stack_workspace_bytes(s, blocks, 0, 1, 0) == 0
    pf = lib.dynconv_stack_forward_profiled
    ev = (ctypes.c_void_p * 6)(*([FAKE] * 6))
    # the first block's mask unit, 3 block launches and the count reduction need 10 events
    assert pf(FAKE, FAKE, s, 1, blocks, 3, 0, None, None, FAKE, fused, None, ev, 6) == ERR_ARG
    assert pf(FAKE, FAKE, s, 1, blocks, 3, 0, None, None, FAKE, fused, None, None, 8) == ERR_NULL


def test_stack_launch_plans(lib):
    s = dc.Shape(32, 64, 64, 32)
    arr = (dc.Block * 8)(*([fake_block()] * 8))

    def names(flags, in_place, shape=s, n=8):
        total = lib.dynconv_stack_launch_names(shape, arr, n, 1, flags, in_place, None, 0)
        out = (ctypes.c_char_p * total)()
        lib.dynconv_stack_launch_names(shape, arr, n, 1, flags, in_place, out, total)
        return [x.decode() for x in out]

    assert names(0, 0) == ["k_mask_cells"] + ["k_block_cells"] * 8 + ["k_band_counts"]
    assert names(1, 1) == ["k_block_cells"] * 8
    assert names(0, 1, n=3) == ["k_copy16", "k_mask_cells"] + ["k_block_cells"] * 3 + ["k_band_counts"]
    assert names(5, 0) == ["k_block_cells"] * 8  # dense wins over G-Softmax: no mask units
    wide_e = (dc.Block * 2)(*([fake_block(E=256)] * 2))
    total = lib.dynconv_stack_launch_names(s, wide_e, 2, 1, 0, 0, None, 0)
    out = (ctypes.c_char_p * total)()
    lib.dynconv_stack_launch_names(s, wide_e, 2, 1, 0, 0, out, total)
    assert [x.decode() for x in out] == ["k_block_fused"] * 2 + ["k_band_counts"]
    assert names(2, 1) == ["k_mask", "k_rowcount", "k_rowscan", "k_compact", "k_expand",
                           "k_dw_project"] * 8
    assert names(3, 0) == ["k_copy16"] + ["k_expand", "k_dw_project"] * 8
    assert names(0, 1, shape=dc.Shape(2, 8, 300, 32), n=2) == \
        ["k_mask_cells"] + ["k_block_cells"] * 2 + ["k_band_counts"]
    # the cell kernel's share bounds are 32-bit: with cells x workgroups past
    # 2^32 (a 1x1 image is one cell; 10^8 cells on any GPU of 43 CUs or more)
    # the stack takes the patch kernel
    assert names(0, 0, shape=dc.Shape(100_000_000, 1, 1, 32), n=2) == ["k_block_fused"] * 2 + ["k_band_counts"]
    arr136 = (dc.Block * 2)(*([fake_block(C=136)] * 2))
    total = lib.dynconv_stack_launch_names(dc.Shape(2, 8, 8, 136), arr136, 2, 1, 0, 1, None, 0)
    out = (ctypes.c_char_p * total)()
    lib.dynconv_stack_launch_names(dc.Shape(2, 8, 8, 136), arr136, 2, 1, 0, 1, out, total)
    assert [x.decode() for x in out][:7] == [
        "k_mask", "k_rowcount", "k_rowscan", "k_compact", "k_expand", "k_dw_project", "k_mask"]
    assert lib.dynconv_stack_launch_names(s, arr, 0, 1, 0, 0, None, 0) == -1


def test_shuffle_stack_validation_and_plans(lib):
    """ShuffleNetV2 units: 116 channels split 58 | 58, the branch padded to 64
    channels (hidden 64); bf16."""
    s = dc.Shape(2, 28, 28, 116)
    br = (dc.Block * 3)(*([fake_block(C=64, E=64, acts=(1, 0, 1))] * 3))
    npos = 2 * 28 * 28

    def up(v):
        return (v + 255) // 256 * 256

    ws = lib.dynconv_shuffle_stack_workspace_bytes(s, br, 3, 2, 0)
    inner = lib.dynconv_stack_workspace_bytes(dc.Shape(2, 28, 28, 64), br, 3, 2, 0)
    # the one-launch branch reads and writes full rows: one full-row buffer
    # (more than one unit) and the block stack's scratch
    assert ws == up(npos * 116 * 2) + inner
    one = lib.dynconv_shuffle_stack_workspace_bytes(s, br, 1, 2, 0)
    assert one == lib.dynconv_stack_workspace_bytes(dc.Shape(2, 28, 28, 64), br, 1, 2, 0)
    # the kernel chain runs on two compact branch-row buffers
    chain = lib.dynconv_shuffle_stack_workspace_bytes(s, br, 3, 2, 2)
    assert chain == 2 * up(npos * 64 * 2) + up(npos * 116 * 2) + \
        lib.dynconv_stack_workspace_bytes(dc.Shape(2, 28, 28, 64), br, 3, 2, 2)
    f = lib.dynconv_shuffle_stack_forward
    assert f(None, FAKE, s, 2, br, 3, 0, None, None, FAKE, ws, None) == ERR_NULL
    assert f(FAKE, FAKE + (1 << 30), s, 2, br, 0, 0, None, None, FAKE, ws, None) == ERR_ARG
    assert f(FAKE, FAKE + (1 << 30), s, 2, br, 3, 8, None, None, FAKE, ws, None) == ERR_ARG
    assert f(FAKE, FAKE, s, 2, br, 3, 0, None, None, FAKE, ws, None) == ERR_SHAPE        # y == x
    assert f(FAKE, FAKE + 4096, s, 2, br, 3, 0, None, None, FAKE, ws, None) == ERR_SHAPE  # overlap
    assert f(FAKE, FAKE + (1 << 30), dc.Shape(2, 28, 28, 115), 2, br, 3, 0, None, None, FAKE, ws,
             None) == ERR_SHAPE                                                          # odd channels
    narrow = (dc.Block * 1)(fake_block(C=56, E=64))
    assert f(FAKE, FAKE + (1 << 30), s, 2, narrow, 1, 0, None, None, FAKE, ws, None) == ERR_SHAPE  # cp < cb
    mixed = (dc.Block * 2)(fake_block(C=64, E=64), fake_block(C=72, E=64))
    assert f(FAKE, FAKE + (1 << 30), s, 2, mixed, 2, 0, None, None, FAKE, ws, None) == ERR_SHAPE
    assert f(FAKE, FAKE + (1 << 30), s, 2, br, 3, 0, None, None, FAKE, ws - 1, None) == ERR_WORKSPACE

    def names(flags, n=3, shape=s, arr=br):
        total = lib.dynconv_shuffle_stack_launch_names(shape, arr, n, 2, flags, None, 0)
        out = (ctypes.c_char_p * total)()
        lib.dynconv_shuffle_stack_launch_names(shape, arr, n, 2, flags, out, total)
        return [x.decode() for x in out]

    assert names(0) == ["k_block_fused"] * 3 + ["k_band_counts"]
    assert names(1, n=1) == ["k_block_fused"]
    # 9-channel bf16 halves are not whole 4-byte words: compact branch rows
    odd = (dc.Block * 2)(*([fake_block(C=16, E=16, acts=(1, 0, 1))] * 2))
    assert names(0, n=2, shape=dc.Shape(1, 6, 6, 18), arr=odd) == [
        "k_shuffle_split", "k_block_fused", "k_shuffle_merge", "k_block_fused", "k_shuffle_merge",
        "k_band_counts"]
    assert names(2, n=1) == ["k_shuffle_split", "k_mask", "k_rowcount", "k_rowscan", "k_compact",
                             "k_expand", "k_dw_project", "k_shuffle_merge"]
    # 116-channel halves run as 120-channel branches on the one-launch path (16-bit)
    wide = (dc.Block * 2)(*([fake_block(C=120, E=128, acts=(1, 0, 1))] * 2))
    assert names(1, n=2, shape=dc.Shape(2, 14, 14, 232), arr=wide) == ["k_block_fused"] * 2
    # 140-channel halves (144-channel branches) take compact rows and the kernel chain
    wider = (dc.Block * 2)(*([fake_block(C=144, E=144, acts=(1, 0, 1))] * 2))
    assert names(1, n=2, shape=dc.Shape(2, 14, 14, 280), arr=wider) == [
        "k_shuffle_split", "k_expand", "k_dw_project", "k_shuffle_merge", "k_expand", "k_dw_project",
        "k_shuffle_merge"]
    assert lib.dynconv_shuffle_stack_launch_names(s, br, 0, 2, 0, None, 0) == -1


def net_layers(over=None):
    """stem 3x3 s2 (3 -> 32), an ungated block s2 (32 -> 24, hidden 96), a
    1x1 (24 -> 64); overrides as {(layer index, field): value}."""
    stem = dc.Layer(dc.LAYER_CONV3X3, 2, 0, 3, 32, FAKE, FAKE, 2)
    blk = dc.Layer(dc.LAYER_BLOCK, 2, 0, 0, 0, 0, 0, 0, fake_block(C=32, E=96, Co=24, w_mask=None))
    last = dc.Layer(dc.LAYER_CONV1X1, 1, 0, 24, 64, FAKE, FAKE, 2)
    arr = (dc.Layer * 3)(stem, blk, last)
    for (i, field), v in (over or {}).items():
        if field.startswith("blk."):
            setattr(arr[i].blk, field[4:], v)
        else:
            setattr(arr[i], field, v)
    return arr


def test_network_validation(lib):
    s = dc.Shape(2, 9, 11, 3)
    out = dc.Shape()

    def shape(arr, n=3, sh=s):
        return lib.dynconv_network_output_shape(sh, arr, n, ctypes.byref(out))

    assert shape(net_layers()) == OK
    assert (out.n, out.h, out.w, out.c) == (2, 3, 3, 64)  # (9-1)//2+1 = 5 -> 3; 11 -> 6 -> 3
    assert lib.dynconv_network_workspace_bytes(s, net_layers(), 3, 1, 0) > 0
    cap = 16
    names = (ctypes.c_char_p * cap)()
    n = lib.dynconv_network_launch_names(s, net_layers(), 3, 1, 0, 0, names, cap)
    assert [names[i].decode() for i in range(n)] == ["k_conv3x3", "k_conv1x1", "k_dwconv3x3", "k_conv1x1",
                                                     "k_conv1x1"]
    # widths, strides, kinds, activations and pointers are checked layer by layer
    assert shape(net_layers({(0, "c_in"): 17}), sh=dc.Shape(2, 9, 11, 17)) == ERR_SHAPE
    assert shape(net_layers({(0, "c_out"): 36})) == ERR_UNSUPPORTED
    assert shape(net_layers({(0, "stride"): 3})) == ERR_ARG
    assert shape(net_layers({(0, "act"): 3})) == ERR_ARG
    assert shape(net_layers({(0, "w"): None})) == ERR_NULL
    assert shape(net_layers({(1, "blk.c_in"): 24})) == ERR_SHAPE
    assert shape(net_layers({(1, "blk.c_hidden"): 1800})) == ERR_UNSUPPORTED
    assert shape(net_layers({(1, "gated"): 1})) == ERR_UNSUPPORTED   # gated needs stride 1, equal widths
    assert shape(net_layers({(1, "kind"): 7})) == ERR_ARG
    assert shape(net_layers({(2, "c_in"): 32})) == ERR_SHAPE
    assert shape(net_layers({(2, "c_out"): 4104})) == ERR_UNSUPPORTED
    assert shape(net_layers({(2, "w"): FAKE + 8})) == ERR_ALIGN
    assert shape(net_layers(), n=0) == ERR_ARG
    assert lib.dynconv_network_workspace_bytes(s, net_layers({(0, "stride"): 3}), 3, 1, 0) == 0
    assert lib.dynconv_network_launch_names(s, net_layers(), 3, 1, 8, 0, None, 0) == -1
    f = lib.dynconv_network_forward
    need = lib.dynconv_network_workspace_bytes(s, net_layers(), 3, 1, 0)
    assert f(FAKE, FAKE + (1 << 30), s, 1, net_layers(), 3, 0, None, None, FAKE, need - 1, None) == ERR_WORKSPACE
    assert f(FAKE, FAKE, s, 1, net_layers(), 3, 0, None, None, FAKE, need, None) == ERR_SHAPE  # y overlaps x
    assert f(None, FAKE, s, 1, net_layers(), 3, 0, None, None, FAKE, need, None) == ERR_NULL
    assert f(FAKE, FAKE + (1 << 30), s, 5, net_layers(), 3, 0, None, None, FAKE, need, None) == ERR_DTYPE
