"""ctypes binding of libpalq.so (include/palq.h).

Argument marshalling only: every step of the path runs in the HIP library.
torch supplies device memory and the stream.  Importing this module loads the
library and raises ImportError if it has not been built
(python -m paper_2208_01944_amd.build).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpalq.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2208_01944_amd.build`")

# torch ships its own HIP runtime under the same soname (libamdhip64.so.7).
# Loading torch first makes the library bind to that runtime, so the process
# has one HIP runtime that both use (loaded the other way round, the
# library's context creation fails on the GPU machine).
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

c_i32, c_i64, c_p, c_f = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float

OK, ERR_ARG, ERR_UNSUPPORTED, ERR_OVERFLOW, ERR_DEVICE, ERR_NOMEM = 0, -1, -2, -3, -4, -5
OP_CONV, OP_MAXPOOL, OP_AVGSUM, OP_FC, OP_SHUFFLE_MODULE, OP_CHANNEL_SHUFFLE = 1, 2, 3, 4, 5, 6
NET_KEEP_ALL, NET_TIMING, NET_GRAPH, NET_PIXEL_LAYOUT = 1, 2, 4, 8
LAYOUT_PIXEL, LAYOUT_GROUP = 0, 1


class Act(ctypes.Structure):
    _fields_ = [("n", c_i32), ("h", c_i32), ("w", c_i32), ("groups", c_i32),
                ("ch_per_group", c_i32), ("bits", c_i32), ("is_signed", c_i32), ("layout", c_i32),
                ("data", c_p)]


class Filter(ctypes.Structure):
    _fields_ = [("groups", c_i32), ("cout_pg", c_i32), ("cin_pg", c_i32), ("kh", c_i32),
                ("kw", c_i32), ("bits", c_i32), ("data", c_p)]


class Requant(ctypes.Structure):
    _fields_ = [("mult", c_p), ("shift", c_p), ("bias", c_p), ("out_bits", c_i32)]


class Residual(ctypes.Structure):
    _fields_ = [("identity", ctypes.POINTER(Act)), ("res_mult", c_p),
                ("proj_in", ctypes.POINTER(Act)), ("proj_w", ctypes.POINTER(Filter)),
                ("proj_stride", c_i32)]


class Layer(ctypes.Structure):
    _fields_ = [("op", c_i32), ("src", c_i32), ("dst", c_i32), ("w", Filter), ("stride", c_i32),
                ("pad", c_i32), ("mult", c_p), ("shift", c_p), ("bias", c_p), ("out_bits", c_i32),
                ("shuffle_steps", c_i32), ("res_src", c_i32), ("res_mult", c_p),
                ("proj_src", c_i32), ("proj_w", Filter), ("proj_stride", c_i32),
                ("pool_k", c_i32), ("pool_stride", c_i32), ("pool_pad", c_i32), ("fc_w", c_p),
                ("fc_out", c_i32)]


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


P_ACT, P_FIL = ctypes.POINTER(Act), ctypes.POINTER(Filter)
_create = _sig("palq_create", c_i32, c_i32, c_p, ctypes.POINTER(c_p))
_destroy = _sig("palq_destroy", None, c_p)
_set_stream = _sig("palq_set_stream", c_i32, c_p, c_p)
_sync = _sig("palq_sync", c_i32, c_p)
_set_conv_fp4 = _sig("palq_set_conv_fp4", c_i32, c_p, c_i32)
_set_conv_bitdecomp = _sig("palq_set_conv_bitdecomp", c_i32, c_p, c_i32)
_last_error = _sig("palq_last_error", ctypes.c_char_p, c_p)
_version = _sig("palq_version", ctypes.c_char_p)
_row_bytes = _sig("palq_row_bytes", c_i64, c_i32, c_i32)
_act_bytes = _sig("palq_act_bytes", c_i64, P_ACT)
_pack = _sig("palq_pack", c_i32, c_p, c_p, P_ACT)
_unpack = _sig("palq_unpack", c_i32, c_p, P_ACT, c_p)
_quantize = _sig("palq_quantize", c_i32, c_p, c_p, c_f, c_f, P_ACT, c_p)
_group_conv = _sig("palq_group_conv", c_i32, c_p, P_ACT, P_FIL, c_i32, c_i32,
                   ctypes.POINTER(Requant), ctypes.POINTER(Residual), c_i32, P_ACT, c_p)
_group_conv_noalloc = _sig("palq_group_conv_noalloc", c_i32, c_p, P_ACT, P_FIL, c_i32, c_i32,
                           ctypes.POINTER(Requant), ctypes.POINTER(Residual), c_i32, P_ACT, c_p)
NOALLOC_SCRATCH_BYTES = 16 << 20
_conv_plan_create = _sig("palq_conv_plan_create", c_i32, c_p, P_ACT, P_FIL, c_i32, c_i32, ctypes.POINTER(Requant),
                         ctypes.POINTER(Residual), c_i32, P_ACT, ctypes.POINTER(c_p))
_conv_run = _sig("palq_conv_run", c_i32, c_p, c_p, c_p, c_p, c_p, c_p)
_conv_plan_destroy = _sig("palq_conv_plan_destroy", None, c_p)
_conv_plan_kernels = _sig("palq_conv_plan_kernels", ctypes.c_char_p, c_p)
_shuffle = _sig("palq_cyclic_shuffle", c_i32, c_p, P_ACT, c_i32, P_ACT)
_channel_shuffle = _sig("palq_channel_shuffle", c_i32, c_p, P_ACT, P_ACT)
_shuffle_module = _sig("palq_shuffle_module", c_i32, c_p, P_ACT, P_FIL, ctypes.POINTER(Requant), c_p, P_ACT)
_maxpool = _sig("palq_maxpool", c_i32, c_p, P_ACT, c_i32, c_i32, c_i32, P_ACT)
_avgsum = _sig("palq_avgsum", c_i32, c_p, P_ACT, c_p)
_fc = _sig("palq_fc", c_i32, c_p, c_p, c_i32, c_i32, c_p, c_i32, c_p)
_net_create = _sig("palq_net_create", c_i32, c_p, P_ACT, ctypes.POINTER(Layer), c_i32, c_i32,
                   ctypes.POINTER(c_p))
_net_destroy = _sig("palq_net_destroy", None, c_p)
_forward = _sig("palq_forward", c_i32, c_p, c_p, c_p, c_p)
_forward_image = _sig("palq_forward_image", c_i32, c_p, c_p, c_p, c_f, c_f, c_p)
_net_tensor = _sig("palq_net_tensor", c_i32, c_p, c_i32, P_ACT)
_net_ops = _sig("palq_net_ops", c_i64, c_p)
_net_layer_kernels = _sig("palq_net_layer_kernels", ctypes.c_char_p, c_p, c_i32, c_i32)
_net_layer_times = _sig("palq_net_layer_times", c_i32, c_p, ctypes.POINTER(c_f), ctypes.POINTER(c_i32))
_net_reset_times = _sig("palq_net_reset_times", c_i32, c_p)

EXPORTS = ["palq_create", "palq_destroy", "palq_set_stream", "palq_set_conv_fp4", "palq_set_conv_bitdecomp", "palq_sync", "palq_last_error",
           "palq_version", "palq_row_bytes", "palq_act_bytes", "palq_pack", "palq_unpack",
           "palq_quantize", "palq_group_conv", "palq_group_conv_noalloc", "palq_conv_plan_create",
           "palq_conv_run", "palq_conv_plan_destroy", "palq_conv_plan_kernels", "palq_shuffle_module", "palq_cyclic_shuffle",
           "palq_channel_shuffle", "palq_maxpool",
           "palq_avgsum", "palq_fc", "palq_net_create", "palq_net_destroy", "palq_forward",
           "palq_forward_image", "palq_net_tensor", "palq_net_ops", "palq_net_layer_kernels", "palq_net_layer_times",
           "palq_net_reset_times"]


class PalqError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"palq status {status}: {msg}")
        self.status = status


def row_bytes(codes: int, bits: int) -> int:
    return int(_row_bytes(codes, bits))


def version() -> str:
    return _version().decode()


def make_act(n, h, w, groups, cpg, bits, signed=False, data=0, layout=LAYOUT_PIXEL) -> Act:
    return Act(n, h, w, groups, cpg, bits, int(bool(signed)), layout, data)


def act_bytes(a: Act) -> int:
    return int(_act_bytes(ctypes.byref(a)))


def _ptr(t):
    if t is None:
        return None
    return t.data_ptr()


class Tensor:
    """A packed code tensor in device memory: a torch uint8 buffer + its Act."""

    def __init__(self, buf, act: Act):
        self.buf = buf
        self.act = act

    @property
    def shape(self):
        a = self.act
        return (a.n, a.h, a.w, a.groups * a.ch_per_group)


class Context:
    """One palq context on a device (or -1: validate only)."""

    def __init__(self, device: int = 0, stream=None):
        self.device = device
        if device >= 0:
            import torch
            self.torch = torch
            self.dev = torch.device("cuda", device)
            if stream is None:
                stream = torch.cuda.current_stream(self.dev).cuda_stream
        else:
            self.torch = None
        h = c_p()
        st = _create(device, stream or 0, ctypes.byref(h))
        if st != OK:
            raise PalqError(st, f"palq_create(device={device}) failed")
        self.h = h

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            _destroy(h)
            self.h = None

    def _check(self, st):
        if st != OK:
            raise PalqError(st, _last_error(self.h).decode())

    def last_error(self) -> str:
        return _last_error(self.h).decode()

    def sync(self):
        self._check(_sync(self.h))

    def set_stream(self, stream):
        """palq_set_stream: later calls enqueue on `stream` (a torch stream)."""
        self._check(_set_stream(self.h, stream.cuda_stream))

    def set_conv_fp4(self, enable: bool):
        """FP4 (2-bit) and FP6 (3-bit) matrix cores for exact layers (True) or
        int8 only."""
        self._check(_set_conv_fp4(self.h, int(bool(enable))))

    def set_conv_bitdecomp(self, enable: bool):
        """Wide (4/6/8-bit) layers as the Eq. 4 bit decomposition on FP4
        matrix cores (True) or directly on int8 (False, the default)."""
        self._check(_set_conv_bitdecomp(self.h, int(bool(enable))))

    # ----------------------------------------------------------- memory
    def empty_act(self, n, h, w, groups, cpg, bits, signed=False, layout=LAYOUT_PIXEL) -> Tensor:
        a = make_act(n, h, w, groups, cpg, bits, signed, layout=layout)
        nb = act_bytes(a)
        if nb < 0:
            raise PalqError(ERR_ARG, "invalid activation descriptor")
        buf = self.torch.empty(max(nb, 16), dtype=self.torch.uint8, device=self.dev)
        a.data = buf.data_ptr()
        return Tensor(buf, a)

    def upload(self, arr, dtype=None):
        t = self.torch.from_numpy(np.ascontiguousarray(arr if dtype is None else arr.astype(dtype)))
        return t.to(self.dev)

    # ----------------------------------------------------------- layout
    def pack(self, codes, groups, bits, signed=False, layout=LAYOUT_PIXEL) -> Tensor:
        """codes: numpy [n, h, w, groups*cpg] integer codes -> packed device tensor."""
        n, h, w, c = codes.shape
        out = self.empty_act(n, h, w, groups, c // groups, bits, signed, layout=layout)
        dt = np.int8 if signed else np.uint8
        src = self.upload(np.asarray(codes).astype(dt))
        self._check(_pack(self.h, src.data_ptr(), ctypes.byref(out.act)))
        return out

    def pack_filter(self, w_codes, bits) -> tuple:
        """w_codes: numpy [G, Co, kh, kw, Ci] signed codes -> (device buffer, Filter)."""
        g, co, kh, kw, ci = w_codes.shape
        t = self.pack(np.asarray(w_codes).reshape(g * co, kh, kw, ci), 1, bits, signed=True)
        f = Filter(g, co, ci, kh, kw, bits, t.act.data)
        return t, f

    def unpack(self, t: Tensor) -> np.ndarray:
        a = t.act
        n = a.n * a.h * a.w * a.groups * a.ch_per_group
        out = self.torch.empty(max(n, 1), dtype=self.torch.uint8, device=self.dev)
        self._check(_unpack(self.h, ctypes.byref(a), out.data_ptr()))
        arr = out[:n].cpu().numpy()
        arr = arr.view(np.int8) if a.is_signed else arr
        return arr.reshape(a.n, a.h, a.w, a.groups * a.ch_per_group).astype(np.int64)

    # ----------------------------------------------------------- ops
    def quantize(self, x, l, u, out: Tensor, range_out=None):
        self._check(_quantize(self.h, _ptr(x), l, u, ctypes.byref(out.act), _ptr(range_out)))

    def group_conv(self, x: Tensor, w: Filter, stride, pad, mult, shift, bias, out: Tensor,
                   shuffle=0, identity: Tensor = None, res_mult=None, proj_in: Tensor = None,
                   proj_w: Filter = None, proj_stride=1, acc_dump=None, noalloc=False):
        """palq_group_conv (noalloc: palq_group_conv_noalloc)."""
        rq = Requant(_ptr(mult), _ptr(shift), _ptr(bias), out.act.bits)
        res = None
        if identity is not None or proj_in is not None:
            res = Residual()
            if identity is not None:
                res.identity = ctypes.pointer(identity.act)
                res.res_mult = _ptr(res_mult)
            if proj_in is not None:
                res.proj_in = ctypes.pointer(proj_in.act)
                res.proj_w = ctypes.pointer(proj_w)
                res.proj_stride = proj_stride
        fn = _group_conv_noalloc if noalloc else _group_conv
        self._check(fn(self.h, ctypes.byref(x.act), ctypes.byref(w), stride, pad,
                       ctypes.byref(rq), ctypes.byref(res) if res is not None else None,
                       shuffle, ctypes.byref(out.act), _ptr(acc_dump)))

    def shuffle_module(self, x: Tensor, w: Filter, mult, shift, bias, res_mult, out: Tensor):
        rq = Requant(_ptr(mult), _ptr(shift), _ptr(bias), out.act.bits)
        self._check(_shuffle_module(self.h, ctypes.byref(x.act), ctypes.byref(w), ctypes.byref(rq),
                                    _ptr(res_mult), ctypes.byref(out.act)))

    def channel_shuffle(self, x: Tensor, out: Tensor):
        self._check(_channel_shuffle(self.h, ctypes.byref(x.act), ctypes.byref(out.act)))

    def cyclic_shuffle(self, x: Tensor, steps, out: Tensor):
        self._check(_shuffle(self.h, ctypes.byref(x.act), steps, ctypes.byref(out.act)))

    def maxpool(self, x: Tensor, k, stride, pad, out: Tensor):
        self._check(_maxpool(self.h, ctypes.byref(x.act), k, stride, pad, ctypes.byref(out.act)))

    def avgsum(self, x: Tensor, out):
        self._check(_avgsum(self.h, ctypes.byref(x.act), _ptr(out)))

    def fc(self, x, n, cin, w, cout, logits):
        self._check(_fc(self.h, _ptr(x), n, cin, _ptr(w), cout, _ptr(logits)))


class ConvPlan:
    """A planned layer (palq_conv_plan_create): the filter, requant arrays
    and shortcut scale are consumed at creation; run() takes tensors of the
    planned shapes."""

    def __init__(self, ctx: Context, x: Tensor, w: Filter, stride, pad, mult, shift, bias, out: Tensor,
                 shuffle=0, identity: Tensor = None, res_mult=None, proj_in: Tensor = None,
                 proj_w: Filter = None, proj_stride=1):
        self.ctx = ctx
        rq = Requant(_ptr(mult), _ptr(shift), _ptr(bias), out.act.bits)
        res = None
        if identity is not None or proj_in is not None:
            res = Residual()
            if identity is not None:
                res.identity = ctypes.pointer(identity.act)
                res.res_mult = _ptr(res_mult)
            if proj_in is not None:
                res.proj_in = ctypes.pointer(proj_in.act)
                res.proj_w = ctypes.pointer(proj_w)
                res.proj_stride = proj_stride
        h = c_p()
        ctx._check(_conv_plan_create(ctx.h, ctypes.byref(x.act), ctypes.byref(w), stride, pad, ctypes.byref(rq),
                                     ctypes.byref(res) if res is not None else None, shuffle,
                                     ctypes.byref(out.act), ctypes.byref(h)))
        self.h = h

    @property
    def kernels(self) -> str:
        return _conv_plan_kernels(self.h).decode()

    def run(self, x: Tensor, out: Tensor, res_in: Tensor = None, acc_dump=None):
        self.ctx._check(_conv_run(self.ctx.h, self.h, x.act.data, res_in.act.data if res_in is not None else None,
                                  out.act.data, _ptr(acc_dump)))

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            _conv_plan_destroy(h)
            self.h = None


class Net:
    """A network built from the layer-spec list of paper_2208_01944_amd.inputs."""

    def __init__(self, ctx: Context, spec, flags=0):
        self.ctx = ctx
        self.spec = spec
        self._keep = []  # device copies alive until palq_net_create has copied them
        x = spec["x"]
        n, h, w, c = x.shape
        self.input_act = make_act(n, h, w, 1, c, 8, True)
        layers = (Layer * len(spec["layers"]))()
        i32 = lambda a: self._dev(np.asarray(a, np.int32))
        for i, L in enumerate(spec["layers"]):
            d = layers[i]
            d.src, d.dst = L["src"], L["dst"]
            d.res_src = -1
            d.proj_src = -1
            if L["op"] == "conv":
                d.op = OP_CONV
                wb = int(L["w_bits"])
                wt, d.w = ctx.pack_filter(L["w"], wb)
                self._keep.append(wt)
                d.stride, d.pad = L["stride"], L["pad"]
                d.mult, d.shift = i32(L["mult"]), i32(L["shift"])
                d.bias = i32(L["bias"]) if L.get("bias") is not None else None
                d.out_bits = L["out_bits"]
                d.shuffle_steps = L.get("shuffle", 0)
                if L.get("res", -1) >= 0:
                    d.res_src = L["res"]
                    d.res_mult = i32(L["res_mult"])
                if L.get("proj_src", -1) >= 0:
                    d.proj_src = L["proj_src"]
                    pt, d.proj_w = ctx.pack_filter(L["proj_w"], wb)
                    self._keep.append(pt)
                    d.proj_stride = L["proj_stride"]
            elif L["op"] == "shuffle_module":
                d.op = OP_SHUFFLE_MODULE
                wt, d.w = ctx.pack_filter(L["w"], int(L["w_bits"]))
                self._keep.append(wt)
                d.mult, d.shift = i32(L["mult"]), i32(L["shift"])
                d.bias = i32(L["bias"]) if L.get("bias") is not None else None
                d.out_bits = L["out_bits"]
                d.res_mult = i32(L["res_mult"])
            elif L["op"] == "channel_shuffle":
                d.op = OP_CHANNEL_SHUFFLE
            elif L["op"] == "maxpool":
                d.op = OP_MAXPOOL
                d.pool_k, d.pool_stride, d.pool_pad = L["k"], L["stride"], L["pad"]
            elif L["op"] == "avgsum":
                d.op = OP_AVGSUM
            elif L["op"] == "fc":
                d.op = OP_FC
                d.fc_w = self._dev(np.asarray(L["w"], np.int8))
                d.fc_out = L["w"].shape[0]
            else:
                raise ValueError(L["op"])
        self.n_layers = len(spec["layers"])
        self.classes = spec["layers"][-1]["w"].shape[0]
        h = c_p()
        ctx._check(_net_create(ctx.h, ctypes.byref(self.input_act), layers, len(spec["layers"]),
                               flags, ctypes.byref(h)))
        self.h = h
        self._keep = []

    def _dev(self, arr):
        t = self.ctx.upload(arr)
        self._keep.append(t)
        return t.data_ptr()

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            _net_destroy(h)
            self.h = None

    @property
    def ops(self) -> int:
        return int(_net_ops(self.h))

    @staticmethod
    def _require(t, nbytes, what):
        """The C calls take plain pointers: refuse a torch tensor smaller than
        the network's batch needs before handing it over."""
        if hasattr(t, "numel") and t.numel() * t.element_size() < nbytes:
            raise PalqError(ERR_ARG, f"{what} holds fewer bytes than the network's batch needs")

    def forward(self, x_packed, logits):
        a = self.input_act
        self._require(x_packed, act_bytes(a), "input")
        self._require(logits, 4 * a.n * self.classes, "logits")
        self.ctx._check(_forward(self.ctx.h, self.h, _ptr(x_packed), _ptr(logits)))

    def forward_image(self, x_f32, l, u, logits):
        """palq_forward_image: quantise an fp32 [n][h][w][3] image (Eq. 2,
        fixed l, u) and run the network on it."""
        a = self.input_act
        self._require(x_f32, 4 * a.n * a.h * a.w * a.ch_per_group, "input")
        self._require(logits, 4 * a.n * self.classes, "logits")
        self.ctx._check(_forward_image(self.ctx.h, self.h, _ptr(x_f32), float(l), float(u), _ptr(logits)))

    def tensor(self, tid) -> Tensor:
        a = Act()
        st = _net_tensor(self.h, tid, ctypes.byref(a))
        if st != OK:
            raise PalqError(st, f"no tensor {tid}")
        return Tensor(None, a)

    def layer_kernels(self, image=False):
        """The kernels each layer launches in palq_forward (or, image=True,
        palq_forward_image), as the library's selection picked them."""
        out = []
        for i in range(self.n_layers):
            r = _net_layer_kernels(self.h, i, int(bool(image)))
            if r is None:
                raise PalqError(ERR_ARG, f"palq_net_layer_kernels({i})")
            out.append(r.decode())
        return out

    def input_kernel(self):
        """palq_forward_image's own quantiser pass ("" when the stem's
        bordered input takes the codes directly)."""
        return _net_layer_kernels(self.h, -1, 1).decode()

    def layer_times(self):
        ms = (c_f * self.n_layers)()
        fw = c_i32()
        self.ctx._check(_net_layer_times(self.h, ms, ctypes.byref(fw)))
        return np.array(ms[:], dtype=np.float64), fw.value

    def reset_times(self):
        self.ctx._check(_net_reset_times(self.h))
