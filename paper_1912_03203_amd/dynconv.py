"""Python binding of the C ABI in include/dynconv.h (argument marshalling only).

Every computation happens in the HIP library ``libdynconv.so`` built next to
this file; this module passes device pointers of torch tensors, sizes and the
current HIP stream through ctypes.  There is no fallback: if the library is
missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdynconv.so")

F32, F16, BF16 = 0, 1, 2
ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
STACK_DENSE, STACK_UNFUSED, STACK_GSOFTMAX = 1, 2, 4

_TORCH_DTYPE = {F32: torch.float32, F16: torch.float16, BF16: torch.bfloat16}
_CODE = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
NAME_TO_DTYPE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

EXPORTED = (
    "dynconv_status_str", "dynconv_version", "dynconv_mask", "dynconv_mask_gsoftmax",
    "dynconv_indices_workspace_bytes",
    "dynconv_build_indices", "dynconv_block_workspace_bytes", "dynconv_block_forward",
    "dynconv_stack_workspace_bytes", "dynconv_stack_forward", "dynconv_stack_launch_names",
    "dynconv_stack_forward_profiled", "dynconv_shuffle_stack_workspace_bytes",
    "dynconv_shuffle_stack_forward", "dynconv_shuffle_stack_launch_names",
    "dynconv_shuffle_stack_forward_profiled", "dynconv_network_output_shape",
    "dynconv_network_workspace_bytes", "dynconv_network_forward", "dynconv_network_launch_names",
    "dynconv_network_forward_profiled", "dynconv_stack_noalloc_max_workspace_bytes",
    "dynconv_stack_forward_noalloc",
)


class Shape(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c", ctypes.c_int32)]


class Block(ctypes.Structure):
    _fields_ = [
        ("c_in", ctypes.c_int32), ("c_hidden", ctypes.c_int32), ("c_out", ctypes.c_int32),
        ("w_expand", ctypes.c_void_p), ("b_expand", ctypes.c_void_p),
        ("w_dw", ctypes.c_void_p), ("b_dw", ctypes.c_void_p),
        ("w_project", ctypes.c_void_p), ("b_project", ctypes.c_void_p),
        ("act_expand", ctypes.c_int32), ("act_dw", ctypes.c_int32), ("act_project", ctypes.c_int32),
        ("w_mask", ctypes.c_void_p), ("b_mask", ctypes.c_float),
    ]


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("stride", ctypes.c_int32), ("gated", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32), ("w", ctypes.c_void_p),
                ("b", ctypes.c_void_p), ("act", ctypes.c_int32), ("blk", Block)]


LAYER_CONV3X3, LAYER_BLOCK, LAYER_CONV1X1 = 0, 1, 2


class Indices(ctypes.Structure):
    _fields_ = [("active", ctypes.c_void_p), ("dilated", ctypes.c_void_p),
                ("nbr", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("capacity", ctypes.c_int64)]


class DynconvError(RuntimeError):
    pass


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise DynconvError("libdynconv.so is not built (%s); run __graft_entry__.build()" % path)
    lib = ctypes.CDLL(path)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    lib.dynconv_status_str.argtypes = [ctypes.c_int]
    lib.dynconv_status_str.restype = ctypes.c_char_p
    lib.dynconv_version.argtypes = []
    lib.dynconv_version.restype = ctypes.c_char_p
    lib.dynconv_mask.argtypes = [vp, Shape, ctypes.c_int, vp, ctypes.c_float, vp, vp, vp]
    lib.dynconv_mask.restype = ctypes.c_int
    lib.dynconv_mask_gsoftmax.argtypes = [vp, Shape, ctypes.c_int, vp, ctypes.c_float, vp, vp, vp]
    lib.dynconv_mask_gsoftmax.restype = ctypes.c_int
    lib.dynconv_indices_workspace_bytes.argtypes = [Shape]
    lib.dynconv_indices_workspace_bytes.restype = sz
    lib.dynconv_build_indices.argtypes = [vp, Shape, i32, ctypes.POINTER(Indices), vp, sz, vp]
    lib.dynconv_build_indices.restype = ctypes.c_int
    lib.dynconv_block_workspace_bytes.argtypes = [Shape, ctypes.POINTER(Block), ctypes.c_int]
    lib.dynconv_block_workspace_bytes.restype = sz
    lib.dynconv_block_forward.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Block),
                                          ctypes.POINTER(Indices), vp, sz, vp]
    lib.dynconv_block_forward.restype = ctypes.c_int
    lib.dynconv_stack_workspace_bytes.argtypes = [Shape, ctypes.POINTER(Block), i32, ctypes.c_int,
                                                  i32]
    lib.dynconv_stack_workspace_bytes.restype = sz
    lib.dynconv_stack_forward.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Block), i32,
                                          i32, vp, vp, vp, sz, vp]
    lib.dynconv_stack_forward.restype = ctypes.c_int
    lib.dynconv_stack_launch_names.argtypes = [Shape, ctypes.POINTER(Block), i32, ctypes.c_int, i32,
                                               i32, ctypes.POINTER(ctypes.c_char_p), i32]
    lib.dynconv_stack_launch_names.restype = i32
    lib.dynconv_stack_forward_profiled.argtypes = [vp, vp, Shape, ctypes.c_int,
                                                   ctypes.POINTER(Block), i32, i32, vp, vp, vp, sz,
                                                   vp, ctypes.POINTER(ctypes.c_void_p), i32]
    lib.dynconv_stack_forward_profiled.restype = ctypes.c_int
    lib.dynconv_stack_noalloc_max_workspace_bytes.argtypes = []
    lib.dynconv_stack_noalloc_max_workspace_bytes.restype = sz
    lib.dynconv_stack_forward_noalloc.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Block), i32,
                                                  i32, vp, vp, vp]
    lib.dynconv_stack_forward_noalloc.restype = ctypes.c_int
    lib.dynconv_shuffle_stack_workspace_bytes.argtypes = [Shape, ctypes.POINTER(Block), i32,
                                                          ctypes.c_int, i32]
    lib.dynconv_shuffle_stack_workspace_bytes.restype = sz
    lib.dynconv_shuffle_stack_forward.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Block),
                                                  i32, i32, vp, vp, vp, sz, vp]
    lib.dynconv_shuffle_stack_forward.restype = ctypes.c_int
    lib.dynconv_shuffle_stack_launch_names.argtypes = [Shape, ctypes.POINTER(Block), i32, ctypes.c_int,
                                                       i32, ctypes.POINTER(ctypes.c_char_p), i32]
    lib.dynconv_shuffle_stack_launch_names.restype = i32
    lib.dynconv_shuffle_stack_forward_profiled.argtypes = [vp, vp, Shape, ctypes.c_int,
                                                           ctypes.POINTER(Block), i32, i32, vp, vp, vp,
                                                           sz, vp, ctypes.POINTER(ctypes.c_void_p), i32]
    lib.dynconv_shuffle_stack_forward_profiled.restype = ctypes.c_int
    lib.dynconv_network_output_shape.argtypes = [Shape, ctypes.POINTER(Layer), i32, ctypes.POINTER(Shape)]
    lib.dynconv_network_output_shape.restype = ctypes.c_int
    lib.dynconv_network_workspace_bytes.argtypes = [Shape, ctypes.POINTER(Layer), i32, ctypes.c_int, i32]
    lib.dynconv_network_workspace_bytes.restype = sz
    lib.dynconv_network_forward.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Layer), i32, i32, vp,
                                            vp, vp, sz, vp]
    lib.dynconv_network_forward.restype = ctypes.c_int
    lib.dynconv_network_launch_names.argtypes = [Shape, ctypes.POINTER(Layer), i32, ctypes.c_int, i32, i32,
                                                 ctypes.POINTER(ctypes.c_char_p), i32]
    lib.dynconv_network_launch_names.restype = i32
    lib.dynconv_network_forward_profiled.argtypes = [vp, vp, Shape, ctypes.c_int, ctypes.POINTER(Layer), i32,
                                                     i32, vp, vp, vp, sz, vp, ctypes.POINTER(ctypes.c_void_p),
                                                     i32]
    lib.dynconv_network_forward_profiled.restype = ctypes.c_int
    _lib = lib
    return lib


def status_str(code: int) -> str:
    return load().dynconv_status_str(code).decode()


def _check(code: int, what: str):
    if code != 0:
        raise DynconvError("%s failed: %s (status %d)" % (what, status_str(code), code))


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def dtype_code(dtype) -> int:
    return _CODE[dtype]


def shape_of(x: torch.Tensor) -> Shape:
    n, h, w, c = x.shape
    return Shape(n, h, w, c)


# ------------------------------------------------------------------ weights
@dataclass
class BlockWeights:
    """Device copies of one block's folded weights plus the C struct that
    points at them (the tensors must outlive every call that uses it)."""

    w_expand: torch.Tensor
    b_expand: torch.Tensor
    w_dw: torch.Tensor
    b_dw: torch.Tensor
    w_project: torch.Tensor
    b_project: torch.Tensor
    w_mask: torch.Tensor
    b_mask: float
    acts: tuple = (ACT_RELU6, ACT_RELU6, ACT_NONE)

    @classmethod
    def from_arrays(cls, wts: dict, dtype, device="cuda", b_mask=0.0, acts=None):
        def dev(a, dt):
            return torch.as_tensor(a).to(device=device, dtype=dt).contiguous()

        return cls(dev(wts["w1"], dtype), dev(wts["b1"], torch.float32),
                   dev(wts["w2"], dtype).reshape(-1, 9).contiguous(), dev(wts["b2"], torch.float32),
                   dev(wts["w3"], dtype), dev(wts["b3"], torch.float32),
                   dev(wts["w_m"], torch.float32), float(b_mask),
                   tuple(acts) if acts is not None else tuple(wts.get("acts", (2, 2, 0))))

    def struct(self) -> Block:
        E, C = self.w_expand.shape
        Co = self.w_project.shape[0]
        return Block(C, E, Co, self.w_expand.data_ptr(), self.b_expand.data_ptr(),
                     self.w_dw.data_ptr(), self.b_dw.data_ptr(), self.w_project.data_ptr(),
                     self.b_project.data_ptr(), self.acts[0], self.acts[1], self.acts[2],
                     self.w_mask.data_ptr(), float(self.b_mask))


@dataclass
class IndexBuffers:
    active: torch.Tensor
    dilated: torch.Tensor
    nbr: torch.Tensor
    counts: torch.Tensor

    @classmethod
    def alloc(cls, npos: int, device="cuda"):
        z = dict(device=device, dtype=torch.int32)
        return cls(torch.empty(max(npos, 1), **z), torch.empty(max(npos, 1), **z),
                   torch.empty(max(npos, 1) * 9, **z), torch.zeros(2, **z))

    def struct(self) -> Indices:
        return Indices(self.active.data_ptr(), self.dilated.data_ptr(), self.nbr.data_ptr(),
                       self.counts.data_ptr(), self.active.numel())


# ------------------------------------------------------------------ calls
def mask(x: torch.Tensor, w_mask: torch.Tensor, b_mask: float, out=None, logits=None, stream=None,
         gsoftmax=False):
    """Hard mask of one block (uint8 [N*H*W]); optional fp32 logits.  With
    gsoftmax the G-Softmax decision (dynconv_mask_gsoftmax) is taken."""
    lib = load()
    n, h, w, _ = x.shape
    if out is None:
        out = torch.empty(n * h * w, dtype=torch.uint8, device=x.device)
    fn = lib.dynconv_mask_gsoftmax if gsoftmax else lib.dynconv_mask
    _check(fn(_ptr(x), shape_of(x), dtype_code(x.dtype), _ptr(w_mask), ctypes.c_float(b_mask), _ptr(out),
              _ptr(logits), _stream(stream)), "dynconv_mask")
    return out


def indices_workspace_bytes(shape: Shape) -> int:
    return load().dynconv_indices_workspace_bytes(shape)


def build_indices(mask_t: torch.Tensor, shape: Shape, dilate: int, idx: IndexBuffers,
                  ws: torch.Tensor, stream=None):
    lib = load()
    s = idx.struct()
    _check(lib.dynconv_build_indices(_ptr(mask_t), shape, int(dilate), ctypes.byref(s), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream(stream)),
           "dynconv_build_indices")


def block_workspace_bytes(shape: Shape, blk: BlockWeights, dtype) -> int:
    s = blk.struct()
    return load().dynconv_block_workspace_bytes(shape, ctypes.byref(s), dtype_code(dtype))


def block_forward(x: torch.Tensor, y: torch.Tensor, blk: BlockWeights, idx, ws: torch.Tensor,
                  stream=None):
    lib = load()
    s = blk.struct()
    ids = idx.struct() if idx is not None else None
    _check(lib.dynconv_block_forward(_ptr(x), _ptr(y), shape_of(x), dtype_code(x.dtype),
                                     ctypes.byref(s), ctypes.byref(ids) if ids is not None else None,
                                     _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "dynconv_block_forward")
    return y


def round_up(v: int, m: int) -> int:
    return (v + m - 1) // m * m


def padded_branch_arrays(wts: dict) -> dict:
    """A ShuffleNetV2 branch's weights (cb channels, hidden E) zero-padded to
    the channel counts the library takes: cp = round_up(cb, 8) inputs and
    outputs, round_up(E, 16) hidden channels.  Padded hidden channels have
    zero weights and biases (their activations are 0 for NONE, RELU, RELU6),
    padded outputs are discarded by the unit, padded inputs are zero."""
    import numpy as np

    E, cb = np.asarray(wts["w1"]).shape
    cp, ep = round_up(cb, 8), round_up(E, 16)

    def pad(a, shape):
        a = np.asarray(a, np.float32)
        out = np.zeros(shape, np.float32)
        out[tuple(slice(0, n) for n in a.shape)] = a
        return out

    out = dict(wts)
    out.update(w1=pad(wts["w1"], (ep, cp)), b1=pad(wts["b1"], (ep,)), w2=pad(wts["w2"], (ep, 9)),
               b2=pad(wts["b2"], (ep,)), w3=pad(wts["w3"], (cp, ep)), b3=pad(wts["b3"], (cp,)),
               w_m=pad(wts["w_m"], (cp,)))
    return out


def _blocks_array(blocks):
    arr = (Block * len(blocks))()
    for i, b in enumerate(blocks):
        arr[i] = b.struct()
    return arr


def stack_workspace_bytes(shape: Shape, blocks, dtype, flags=0) -> int:
    arr = _blocks_array(blocks)
    return load().dynconv_stack_workspace_bytes(shape, arr, len(blocks), dtype_code(dtype), flags)


class Stack:
    """A prepared stack call y = blocks(x): the block array and pointers are
    marshalled once, so repeated launches (a timed loop, a graph capture) cost
    a single ctypes call.  y may be x (in place)."""

    def __init__(self, x: torch.Tensor, y: torch.Tensor, blocks, flags=0, masks=None, counts=None,
                 ws=None):
        self.lib = load()
        self.x, self.y = x, y
        self.blocks = list(blocks)
        self.arr = _blocks_array(self.blocks)
        self.shape = shape_of(x)
        self.dtype = dtype_code(x.dtype)
        self.flags = int(flags)
        need = self.lib.dynconv_stack_workspace_bytes(self.shape, self.arr, len(self.blocks),
                                                      self.dtype, self.flags)
        if need == 0:
            raise DynconvError("dynconv_stack_workspace_bytes rejected the stack")
        if ws is None:
            ws = torch.empty(need, dtype=torch.uint8, device=x.device)
        self.ws = ws
        self.masks = masks
        self.counts = counts

    def launch_names(self):
        lib = self.lib
        args = (self.shape, self.arr, len(self.blocks), self.dtype, self.flags,
                1 if self.x.data_ptr() == self.y.data_ptr() else 0)
        total = lib.dynconv_stack_launch_names(*args, None, 0)
        if total < 0:
            raise DynconvError("dynconv_stack_launch_names rejected the stack")
        names = (ctypes.c_char_p * total)()
        lib.dynconv_stack_launch_names(*args, names, total)
        return [n.decode() for n in names]

    def _args(self, stream):
        return (_ptr(self.x), _ptr(self.y), self.shape, self.dtype, self.arr, len(self.blocks),
                self.flags, _ptr(self.masks), _ptr(self.counts), _ptr(self.ws),
                self.ws.numel() * self.ws.element_size(), _stream(stream))

    def __call__(self, stream=None):
        _check(self.lib.dynconv_stack_forward(*self._args(stream)), "dynconv_stack_forward")
        return self.y

    def profiled(self, events, stream=None):
        """Same call, with launch i timed by the raw HIP events
        (events[2i], events[2i+1]); len(events) >= 2 * number of launches."""
        arr = (ctypes.c_void_p * len(events))(*events)
        _check(self.lib.dynconv_stack_forward_profiled(*self._args(stream), arr, len(events)),
               "dynconv_stack_forward_profiled")
        return self.y


def stack_forward(x: torch.Tensor, y: torch.Tensor, blocks, flags=0, masks=None, counts=None,
                  ws=None, stream=None):
    return Stack(x, y, blocks, flags, masks, counts, ws)(stream)


def stack_noalloc_max_workspace_bytes() -> int:
    return int(load().dynconv_stack_noalloc_max_workspace_bytes())


def stack_forward_noalloc(x: torch.Tensor, y: torch.Tensor, blocks, flags=0, masks=None, counts=None,
                          stream=None):
    """dynconv_stack_forward_noalloc: the stack call on the library's static
    per-device scratch array instead of a caller workspace."""
    lib = load()
    arr = _blocks_array(blocks)
    _check(lib.dynconv_stack_forward_noalloc(_ptr(x), _ptr(y), shape_of(x), dtype_code(x.dtype), arr,
                                             len(blocks), int(flags), _ptr(masks), _ptr(counts),
                                             _stream(stream)),
           "dynconv_stack_forward_noalloc")
    return y


class ShuffleStack:
    """A prepared ShuffleNetV2 unit stack y = units(x) (dynconv_shuffle_stack_forward);
    `branches` are BlockWeights on the padded channel counts (padded_branch_arrays).
    x and y must not overlap."""

    def __init__(self, x: torch.Tensor, y: torch.Tensor, branches, flags=0, masks=None, counts=None,
                 ws=None):
        self.lib = load()
        self.x, self.y = x, y
        self.branches = list(branches)
        self.arr = _blocks_array(self.branches)
        self.shape = shape_of(x)
        self.dtype = dtype_code(x.dtype)
        self.flags = int(flags)
        need = self.lib.dynconv_shuffle_stack_workspace_bytes(self.shape, self.arr, len(self.branches),
                                                              self.dtype, self.flags)
        if need == 0:
            raise DynconvError("dynconv_shuffle_stack_workspace_bytes rejected the units")
        if ws is None:
            ws = torch.empty(need, dtype=torch.uint8, device=x.device)
        self.ws = ws
        self.masks = masks
        self.counts = counts

    def launch_names(self):
        lib = self.lib
        args = (self.shape, self.arr, len(self.branches), self.dtype, self.flags)
        total = lib.dynconv_shuffle_stack_launch_names(*args, None, 0)
        if total < 0:
            raise DynconvError("dynconv_shuffle_stack_launch_names rejected the units")
        names = (ctypes.c_char_p * total)()
        lib.dynconv_shuffle_stack_launch_names(*args, names, total)
        return [n.decode() for n in names]

    def _args(self, stream):
        return (_ptr(self.x), _ptr(self.y), self.shape, self.dtype, self.arr, len(self.branches),
                self.flags, _ptr(self.masks), _ptr(self.counts), _ptr(self.ws),
                self.ws.numel() * self.ws.element_size(), _stream(stream))

    def __call__(self, stream=None):
        _check(self.lib.dynconv_shuffle_stack_forward(*self._args(stream)), "dynconv_shuffle_stack_forward")
        return self.y

    def profiled(self, events, stream=None):
        arr = (ctypes.c_void_p * len(events))(*events)
        _check(self.lib.dynconv_shuffle_stack_forward_profiled(*self._args(stream), arr, len(events)),
               "dynconv_shuffle_stack_forward_profiled")
        return self.y


class NetworkWeights:
    """Device copies of a layer list (dicts as paper_1912_03203_amd.inputs
    builds them) and the C layer array pointing at them; gated blocks get
    their mask biases from `biases` (one per gated block, in order)."""

    def __init__(self, layers, dtype, biases=None, device="cuda"):
        self.keep = []
        self.arr = (Layer * len(layers))()
        gi = 0

        def dev(a, dt):
            t = torch.as_tensor(a).to(device=device, dtype=dt).contiguous()
            self.keep.append(t)
            return t

        for i, L in enumerate(layers):
            if L["kind"] in ("conv3x3", "conv1x1"):
                w = dev(L["w"], dtype)
                b = dev(L["b"], torch.float32)
                kind = LAYER_CONV3X3 if L["kind"] == "conv3x3" else LAYER_CONV1X1
                self.arr[i] = Layer(kind, int(L.get("stride", 1)), 0, int(w.shape[1]), int(w.shape[0]),
                                    w.data_ptr(), b.data_ptr(), int(L["act"]), Block())
                continue
            acts = L.get("acts", (ACT_RELU6, ACT_RELU6, ACT_NONE))
            w2 = dev(L["w2"], dtype).reshape(-1, 9).contiguous()
            self.keep.append(w2)
            b2 = dev(L["b2"], torch.float32)
            w3 = dev(L["w3"], dtype)
            b3 = dev(L["b3"], torch.float32)
            E = int(w2.shape[0])
            c_out = int(w3.shape[0])
            if L.get("w1") is not None:
                w1 = dev(L["w1"], dtype)
                b1 = dev(L["b1"], torch.float32)
                c_in, w1p, b1p = int(w1.shape[1]), w1.data_ptr(), b1.data_ptr()
            else:
                c_in, w1p, b1p = E, None, None
            gated = 1 if L.get("gated") else 0
            wm_p, bm = None, 0.0
            if gated:
                wm = dev(L["w_m"], torch.float32)
                wm_p = wm.data_ptr()
                bm = float(biases[gi]) if biases is not None else 0.0
                gi += 1
            blk = Block(c_in, E, c_out, w1p, b1p, w2.data_ptr(), b2.data_ptr(), w3.data_ptr(), b3.data_ptr(),
                        int(acts[0]), int(acts[1]), int(acts[2]), wm_p, bm)
            self.arr[i] = Layer(LAYER_BLOCK, int(L["stride"]), gated, c_in, c_out, None, None, 0, blk)
        self.n = len(layers)
        self.ngated = gi if biases is not None else sum(1 for L in layers if L.get("gated"))

    def set_bias(self, gated_index, value):
        gi = 0
        for i in range(self.n):
            if self.arr[i].gated:
                if gi == gated_index:
                    self.arr[i].blk.b_mask = float(value)
                    return
                gi += 1
        raise IndexError(gated_index)


def network_output_shape(shape: Shape, net: NetworkWeights) -> Shape:
    out = Shape()
    _check(load().dynconv_network_output_shape(shape, net.arr, net.n, ctypes.byref(out)),
           "dynconv_network_output_shape")
    return out


class Network:
    """A prepared whole-network call y = layers(x) (dynconv_network_forward).
    x and y must not overlap; y has the shape network_output_shape gives."""

    def __init__(self, x: torch.Tensor, y: torch.Tensor, net: NetworkWeights, flags=0, masks=None, counts=None,
                 ws=None):
        self.lib = load()
        self.x, self.y, self.net = x, y, net
        self.shape = shape_of(x)
        self.dtype = dtype_code(x.dtype)
        self.flags = int(flags)
        need = self.lib.dynconv_network_workspace_bytes(self.shape, net.arr, net.n, self.dtype, self.flags)
        if need == 0:
            raise DynconvError("dynconv_network_workspace_bytes rejected the network")
        self.ws = torch.empty(need, dtype=torch.uint8, device=x.device) if ws is None else ws
        self.masks = masks
        self.counts = counts

    def launch_names(self):
        args = (self.shape, self.net.arr, self.net.n, self.dtype, self.flags, 1 if self.counts is not None else 0)
        total = self.lib.dynconv_network_launch_names(*args, None, 0)
        if total < 0:
            raise DynconvError("dynconv_network_launch_names rejected the network")
        names = (ctypes.c_char_p * total)()
        self.lib.dynconv_network_launch_names(*args, names, total)
        return [n.decode() for n in names]

    def _args(self, stream):
        return (_ptr(self.x), _ptr(self.y), self.shape, self.dtype, self.net.arr, self.net.n, self.flags,
                _ptr(self.masks), _ptr(self.counts), _ptr(self.ws), self.ws.numel() * self.ws.element_size(),
                _stream(stream))

    def __call__(self, stream=None):
        _check(self.lib.dynconv_network_forward(*self._args(stream)), "dynconv_network_forward")
        return self.y

    def profiled(self, events, stream=None):
        arr = (ctypes.c_void_p * len(events))(*events)
        _check(self.lib.dynconv_network_forward_profiled(*self._args(stream), arr, len(events)),
               "dynconv_network_forward_profiled")
        return self.y
