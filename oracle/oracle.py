"""PalQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct reference for what the PalQuant inference path
computes.  Only the parity tests, the GPU smoke check and the benchmark's CPU
baseline leg may import this module.  It imports nothing from the product
package and the product imports nothing from here.

Tensors are UNPACKED integer codes in numpy arrays, channels last: an
activation is [N, H, W, C] with C = G * C^ and channel g * C^ + j belonging
to group g (the [N, G, C^, H, W] reshape of the cyclic permutation section,
stored NHWC).  Floating point follows the paper's fp32 quantiser; all integer
work is int64 (Python ints where noted).

Sections of the paper this file follows:
  * uniform quantiser, Section 3.2 Eq. 2 (+ de-quantiser Eq. 3);
  * the layer product Y = X W^T, Section 3.1 Eq. 1, done per group
    (parallel low-precision quantisation, Section 4.1);
  * the cyclic permutation pi(i) = (i+1) mod G and Y[:, pi(i)] = X[:, i],
    Section 4.2 Eq. 6-8;
  * the cyclic-shuffle module Z = X + Conv1x1(pi(X)), Section 4.2 Eq. 9-10;
  * BitOps, Appendix B.
The paper fixes no integer requantisation, residual scale, stem/FC format or
tie rule; the readings used here are listed where they are applied.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libpalq_oracle.so")
        src = os.path.join(_HERE, "palq_oracle.c")
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(src):
            from . import build as _build  # compile the checker on first use
            _build.build()
        lib = ctypes.CDLL(path)
        i64 = ctypes.c_int64
        p = ctypes.c_void_p
        lib.palq_oracle_group_conv.argtypes = [p, i64, i64, i64, i64, i64, p, i64, i64, i64, i64, i64, p]
        lib.palq_oracle_group_conv.restype = ctypes.c_int
        lib.palq_oracle_threads.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def threads() -> int:
    """OpenMP team size the C conv loop runs with."""
    return int(_lib().palq_oracle_threads())


# ---------------------------------------------------------------------------
# Section 3.2, Eq. 2: uniform quantiser.
# ---------------------------------------------------------------------------
def quantize(x, l, u, bits: int, signed: bool = False) -> np.ndarray:
    """Eq. 2: x_n = clip((x - l) / (u - l), 0, 1); x_q = round((2^b - 1) x_n).

    Readings (the paper gives no op order or tie rule):
      * every operation in IEEE fp32 with correct rounding, in the order
        d = x - l, r = u - l, t = d / r, clip (t > 1 -> 1, then not(t >= 0) -> 0,
        so NaN -> 0), y = t * (2^b - 1), q = round-half-to-even(y);
      * signed codes are x_q - 2^(b-1) (two's complement b-bit range).
    Returns int32 codes.
    """
    f = np.float32
    x = np.asarray(x, dtype=np.float32)
    l = f(l)
    u = f(u)
    d = x - l
    r = u - l
    t = d / r
    t = np.where(t > f(1.0), f(1.0), t)
    t = np.where(t >= f(0.0), t, f(0.0))
    y = t * f((1 << bits) - 1)
    q = np.rint(y).astype(np.int32)
    if signed:
        q = q - np.int32(1 << (bits - 1))
    return q


def calibrate_range(x):
    """Per-tensor lower/upper bound when none is given: min and max of the
    non-NaN values (l and u are per-layer scalars in Section 3.2)."""
    x = np.asarray(x, dtype=np.float32)
    return np.float32(np.nanmin(x)), np.float32(np.nanmax(x))


def dequantize(q, bits: int, kind: str) -> np.ndarray:
    """Eq. 3, with the two cases as the surrounding prose states them
    (weights land in [-1, 1], activations are non-negative); the printed
    formula has the cases the other way round.  Unsigned codes in, fp64 out.
    """
    q = np.asarray(q, dtype=np.float64)
    s = float((1 << bits) - 1)
    if kind == "activation":
        return q / s
    if kind == "weight":
        return 2.0 * (q / s - 0.5)
    raise ValueError(kind)


# ---------------------------------------------------------------------------
# Section 3.1 Eq. 1 per group (Section 4.1): grouped convolution, int64.
# ---------------------------------------------------------------------------
def out_size(h: int, k: int, stride: int, pad: int) -> int:
    return (h + 2 * pad - k) // stride + 1


def group_conv(x, w, stride: int, pad: int) -> np.ndarray:
    """acc[n, oy, ox, g*Co + k] = sum_{ky,kx,c} x[n, oy*s-p+ky, ox*s-p+kx, g*Ci + c]
    * w[g, k, ky, kx, c]; taps outside the image contribute 0.

    x: [N, H, W, G*Ci] integer codes; w: [G, Co, kh, kw, Ci] integer codes.
    Returns int64 [N, Ho, Wo, G*Co].
    """
    x = np.ascontiguousarray(x, dtype=np.int32)
    w = np.ascontiguousarray(w, dtype=np.int32)
    n, h, wd, c = x.shape
    g, co, kh, kw, ci = w.shape
    if c != g * ci:
        raise ValueError(f"input has {c} channels, filter expects {g}x{ci}")
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    acc = np.zeros((n, ho, wo, g * co), dtype=np.int64)
    if n == 0:
        return acc
    rc = _lib().palq_oracle_group_conv(x.ctypes.data, n, h, wd, g, ci, w.ctypes.data, co, kh, kw,
                                       stride, pad, acc.ctypes.data)
    if rc != 0:
        raise ValueError("bad convolution geometry")
    return acc


# ---------------------------------------------------------------------------
# Section 4.2 Eq. 6-8: cyclic permutation at group level.
# ---------------------------------------------------------------------------
def cyclic_permute(x, groups: int, steps: int = 1) -> np.ndarray:
    """Y[..., pi^s(i), :] = X[..., i, :] with pi(i) = (i + 1) mod G, on the
    channel axis viewed as [G, C^].  steps may be any integer (pi^G = id)."""
    x = np.asarray(x)
    c = x.shape[-1]
    if c % groups:
        raise ValueError("channels not divisible by groups")
    v = x.reshape(x.shape[:-1] + (groups, c // groups))
    y = np.empty_like(v)
    for i in range(groups):
        y[..., (i + steps) % groups, :] = v[..., i, :]
    return y.reshape(x.shape)


# ---------------------------------------------------------------------------
# Fixed-point requantisation (the paper has none; reading of this build).
# ---------------------------------------------------------------------------
def requant(t, mult, shift, out_bits: int) -> np.ndarray:
    """q = clamp(floor((t * M + 2^(sh-1)) / 2^sh), 0, 2^b_out - 1).

    The clamp at 0 is the fused ReLU.  The learned output scale alpha and any
    folded batch-norm scale live in the per-channel multiplier M (Section 3.2
    introduces alpha as a per-layer output multiplier).  out_bits == 32 means
    no requantisation: the int32 value t itself.
    """
    t = np.asarray(t, dtype=np.int64)
    if out_bits == 32:
        return t.astype(np.int64)
    m = np.asarray(mult, dtype=np.int64)
    sh = np.asarray(shift, dtype=np.int64)
    num = t * m + (np.int64(1) << (sh - 1))
    q = num >> sh  # arithmetic shift == floor division by 2^sh
    return np.clip(q, 0, (1 << out_bits) - 1)


# ---------------------------------------------------------------------------
# One PalQuant convolution layer with its epilogue.
# ---------------------------------------------------------------------------
def conv_layer(x, w, stride, pad, mult, shift, bias, out_bits, shuffle=0,
               res=None, res_mult=None, proj_x=None, proj_w=None, proj_stride=1):
    """A B-bit grouped conv followed by requantisation and the cyclic
    permutation, returning (codes, acc) with both in output (destination)
    channel order: step 1 below, then layer_epilogue (steps 2-4).

    Steps, in order:
      1. acc = group_conv(x, w)  (source group g, channel k);
      2. the conv branch value acc + bias and its per-channel parameters are
         cyclically permuted by `shuffle` steps (Eq. 8): source group g lands
         in group (g + s) mod G;
      3. the shortcut is added at the destination: res_mult * res (identity
         codes, per-channel scale travelling with the branch channel) or the
         raw int64 accumulator of a 1x1 projection conv of the block input
         (same groups, destination indexing);
      4. requant with the branch channel's M and shift (ReLU in the clamp).
    Reading: permuting the branch before the residual add mirrors the
    module Z = X + Conv(pi(X)) (Eq. 9-10) so that groups mix; permuting after
    the add would only relabel groups.
    The returned acc is everything the contraction sums into each output
    channel: the permuted conv accumulator plus the projection accumulator.
    """
    acc = group_conv(x, w, stride, pad)
    return layer_epilogue(acc, w.shape[0], mult, shift, bias, out_bits, shuffle, res=res,
                          res_mult=res_mult, proj_x=proj_x, proj_w=proj_w, proj_stride=proj_stride)


def layer_epilogue(acc, groups, mult, shift, bias, out_bits, shuffle=0, res=None, res_mult=None,
                   proj_x=None, proj_w=None, proj_stride=1):
    """Steps 2-4 of conv_layer on the layer's accumulator acc (source channel
    order, as group_conv returns it); returns (codes, acc_d) like conv_layer.
    With shuffle, res and proj_x the same, conv_layer(x, w, ...) equals
    layer_epilogue(group_conv(x, w, ...), G, ...)."""
    g = groups
    acc_d = cyclic_permute(acc, g, shuffle)
    bias = np.zeros(acc.shape[-1], np.int64) if bias is None else np.asarray(bias, np.int64)
    bias_d = cyclic_permute(bias, g, shuffle)
    mult_d = cyclic_permute(np.asarray(mult, np.int64), g, shuffle)
    shift_d = cyclic_permute(np.asarray(shift, np.int64), g, shuffle)
    if proj_x is not None:
        acc_d = acc_d + group_conv(proj_x, proj_w, proj_stride, 0)
    t = acc_d + bias_d
    if res is not None:
        rm_d = cyclic_permute(np.asarray(res_mult, np.int64), g, shuffle)
        t = t + rm_d * np.asarray(res, np.int64)
    return requant(t, mult_d, shift_d, out_bits), acc_d


def centring_bias(acc_d, groups, shuffle=0, res=None, res_mult=None):
    """The centred variant's conv bias (a test-input recipe, not part of the
    method): bias_d[c] = -round_half_up(mean over all positions of
    (acc_d + residual)[c]) at destination channel c, computed exactly with
    Python integers, returned indexed by the source channel (the permutation
    undone) as an int32 array.  acc_d: the layer's destination-order
    accumulator (conv_layer's second result, which already holds any
    projection accumulator); res/res_mult: the identity shortcut, if any."""
    from fractions import Fraction
    t = np.asarray(acc_d, np.int64)
    if res is not None:
        rm_d = cyclic_permute(np.asarray(res_mult, np.int64), groups, shuffle)
        t = t + rm_d * np.asarray(res, np.int64)
    cnt = int(np.prod(t.shape[:-1]))
    sums = t.reshape(-1, t.shape[-1]).sum(axis=0)
    bias_d = np.array([-int((Fraction(int(s), cnt) + Fraction(1, 2)).__floor__()) for s in sums],
                      dtype=np.int64)
    return cyclic_permute(bias_d, groups, -shuffle).astype(np.int32)


def channel_shuffle(x, groups: int) -> np.ndarray:
    """Channel shuffle (Section 4.3, Table 3): the channel axis viewed as a
    [G, C^] matrix is transposed to [C^, G] and flattened again, so output
    channel o = c * G + g holds input channel g * C^ + c."""
    x = np.asarray(x)
    c = x.shape[-1]
    if c % groups:
        raise ValueError("channels not divisible by groups")
    v = x.reshape(x.shape[:-1] + (groups, c // groups))
    return np.swapaxes(v, -1, -2).reshape(x.shape)


# ---------------------------------------------------------------------------
# Section 4.2 Eq. 9-10: the cyclic shuffle module.
# ---------------------------------------------------------------------------
def shuffle_module(x, w, mult, shift, bias, res_mult, out_bits):
    """Z = X + Conv1x1(Y) with Y = CyclicPermute(X) (Eq. 9-10), as an integer
    layer: the 1x1 B-bit group conv runs on the permuted input Y (Eq. 8, one
    step), the shortcut X enters unpermuted, scaled by res_mult (the same
    shortcut scale as an identity residual), and the sum is requantised.
    Every per-channel array is indexed by the module's output channel.
    Returns (codes, acc) with acc the 1x1 accumulator of each output channel.
    """
    w = np.asarray(w)
    G = w.shape[0]
    if w.shape[2:4] != (1, 1) or w.shape[1] != w.shape[4]:
        raise ValueError("the module's conv is 1x1 with as many outputs as inputs per group")
    y = cyclic_permute(x, G, 1)
    acc = group_conv(y, w, 1, 0)
    bias = np.zeros(acc.shape[-1], np.int64) if bias is None else np.asarray(bias, np.int64)
    t = acc + bias + np.asarray(res_mult, np.int64) * np.asarray(x, np.int64)
    return requant(t, mult, shift, out_bits), acc


# ---------------------------------------------------------------------------
# Network glue (stem/FC stay high precision, Section 5 "first and last
# layer are not quantized"; here they are 8-bit integer).
# ---------------------------------------------------------------------------
def maxpool(x, k: int, stride: int, pad: int) -> np.ndarray:
    """Max over the in-image part of each k x k window (codes are >= 0, and
    every window holds at least one in-image pixel when pad < k)."""
    x = np.asarray(x, dtype=np.int64)
    n, h, w, c = x.shape
    ho, wo = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    out = np.empty((n, ho, wo, c), dtype=np.int64)
    for oy in range(ho):
        y0, y1 = max(oy * stride - pad, 0), min(oy * stride - pad + k, h)
        for ox in range(wo):
            x0, x1 = max(ox * stride - pad, 0), min(ox * stride - pad + k, w)
            out[:, oy, ox, :] = x[:, y0:y1, x0:x1, :].max(axis=(1, 2))
    return out


def avgsum(x) -> np.ndarray:
    """Global average pool kept as its exact integer sum over H x W."""
    return np.asarray(x, dtype=np.int64).sum(axis=(1, 2))


def fc(x, w) -> np.ndarray:
    """logits[n, o] = sum_c x[n, c] * w[o, c] (Eq. 1, int64)."""
    x = np.asarray(x, dtype=np.int64)
    w = np.asarray(w, dtype=np.int64)
    return x @ w.T


def run_net(net, x, keep=False):
    """Runs a layer list (see the spec format of the input generators) on
    input codes x.  Returns the logits, and with keep=True also the dict of
    every tensor id -> codes and conv id -> acc."""
    tensors = {0: np.asarray(x, dtype=np.int64)}
    accs = {}
    out = None
    for L in net["layers"]:
        op = L["op"]
        src = tensors[L["src"]]
        if op == "conv":
            res = tensors[L["res"]] if L.get("res", -1) >= 0 else None
            px = tensors[L["proj_src"]] if L.get("proj_src", -1) >= 0 else None
            q, acc = conv_layer(src, L["w"], L["stride"], L["pad"], L["mult"], L["shift"],
                                L.get("bias"), L["out_bits"], L.get("shuffle", 0),
                                res=res, res_mult=L.get("res_mult"),
                                proj_x=px, proj_w=L.get("proj_w"),
                                proj_stride=L.get("proj_stride", 1))
            accs[L["dst"]] = acc
            out = q
        elif op == "shuffle_module":
            q, acc = shuffle_module(src, L["w"], L["mult"], L["shift"], L.get("bias"),
                                    L["res_mult"], L["out_bits"])
            accs[L["dst"]] = acc
            out = q
        elif op == "channel_shuffle":
            out = channel_shuffle(src, L["groups"])
        elif op == "maxpool":
            out = maxpool(src, L["k"], L["stride"], L["pad"])
        elif op == "avgsum":
            out = avgsum(src)
        elif op == "fc":
            out = fc(src, L["w"])
        else:
            raise ValueError(op)
        tensors[L["dst"]] = out
    if keep:
        return out, tensors, accs
    return out


def calibrate_centring(net, x, return_logits=False):
    """Returns a copy of `net` whose conv biases centre every layer's
    pre-requant value: bias[c] = -round_half_up(mean over positions of
    (acc + residual)[c]) (centring_bias), computed exactly in layer order on
    the oracle's own forward pass over x.  Used only to build non-degenerate
    test inputs; the biases are then ordinary inputs to both sides.  With
    return_logits the oracle's output of the centred network on x (the
    last layer's result, equal to run_net(centred, x)) is returned too."""
    import copy

    net = copy.deepcopy(net)
    tensors = {0: np.asarray(x, dtype=np.int64)}
    out = None
    for L in net["layers"]:
        src = tensors[L["src"]]
        if L["op"] == "conv":
            g = L["w"].shape[0]
            res = tensors[L["res"]] if L.get("res", -1) >= 0 else None
            px = tensors[L["proj_src"]] if L.get("proj_src", -1) >= 0 else None
            acc = group_conv(src, L["w"], L["stride"], L["pad"])
            kw = dict(res=res, res_mult=L.get("res_mult"), proj_x=px, proj_w=L.get("proj_w"),
                      proj_stride=L.get("proj_stride", 1))
            _, acc_d = layer_epilogue(acc, g, L["mult"], L["shift"], None, L["out_bits"],
                                      L.get("shuffle", 0), **kw)
            L["bias"] = centring_bias(acc_d, g, L.get("shuffle", 0), res=res,
                                      res_mult=L.get("res_mult"))
            out, _ = layer_epilogue(acc, g, L["mult"], L["shift"], L["bias"], L["out_bits"],
                                    L.get("shuffle", 0), **kw)
        elif L["op"] == "shuffle_module":
            _, acc = shuffle_module(src, L["w"], L["mult"], L["shift"], None, L["res_mult"],
                                    L["out_bits"])
            t = acc + np.asarray(L["res_mult"], np.int64) * src
            L["bias"] = centring_bias(t, L["w"].shape[0])
            out, _ = shuffle_module(src, L["w"], L["mult"], L["shift"], L["bias"],
                                    L["res_mult"], L["out_bits"])
        elif L["op"] == "channel_shuffle":
            out = channel_shuffle(src, L["groups"])
        elif L["op"] == "maxpool":
            out = maxpool(src, L["k"], L["stride"], L["pad"])
        elif L["op"] == "avgsum":
            out = avgsum(src)
        elif L["op"] == "fc":
            out = fc(src, L["w"])
        tensors[L["dst"]] = out
    if return_logits:
        return net, out
    return net


# ---------------------------------------------------------------------------
# Appendix B: BitOps = b_w * b_a * t * c * k * k * h * w per conv/FC layer.
# ---------------------------------------------------------------------------
def layer_macs(cin_total, cout_total, groups, k, ho, wo) -> int:
    """MACs of a (grouped) conv: t kernels of size (c/G) x k x k at h x w
    output positions; a grouped layer's t kernels each see c/G channels."""
    return cout_total * (cin_total // groups) * k * k * ho * wo


def bitops(macs: int, b_w: int, b_a: int) -> int:
    return b_w * b_a * macs
