"""Seeded synthetic inputs for PalQuant layers and networks.

This module draws random codes and parameters and lays out network
topologies; it contains none of the method's arithmetic (no convolution,
requantisation or permutation).  Both the GPU path's tests/benchmark and the
CPU oracle consume what it returns.

Random source: numpy Generator(PCG64(seed)); codes are drawn with
integers(lo, hi, endpoint=True).  Default seed = 220801944 + config index.

Layer spec (a dict per layer, list order = execution order; tensor id 0 is
the network input):
  conv    : src, dst, w [G, Co, kh, kw, Ci] int8 codes, stride, pad,
            in_bits, in_signed, w_bits, out_bits, mult/shift/bias int32
            [G*Co] (indexed by the conv's own output channel), shuffle
            (cyclic steps), res (tensor id or -1) + res_mult int32 [G*Co],
            proj_src (tensor id or -1) + proj_w [G, Co, 1, 1, Cp] + proj_stride
  maxpool : src, dst, k, stride, pad
  avgsum  : src, dst
  fc      : src, dst, w [O, C] int8
"""
from __future__ import annotations

import math
import os

import numpy as np

SEED_BASE = 220801944


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def code_range(bits: int, signed: bool):
    if signed:
        return -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    return 0, (1 << bits) - 1


def codes(g: np.random.Generator, shape, bits: int, signed: bool) -> np.ndarray:
    """Uniform b-bit codes (unsigned [0, 2^b-1] or signed [-2^(b-1), 2^(b-1)-1])."""
    lo, hi = code_range(bits, signed)
    dt = np.int8 if bits <= 7 or signed else np.uint8
    return g.integers(lo, hi, size=shape, endpoint=True).astype(dt)


def _moments(bits: int, signed: bool):
    lo, hi = code_range(bits, signed)
    v = np.arange(lo, hi + 1, dtype=np.float64)
    return v.mean(), (v * v).mean()


def default_shift(k_total: int, in_bits: int, in_signed: bool, w_bits: int, out_bits: int) -> int:
    """Shift that maps one standard deviation of a uniform-code accumulator
    to about one output step for a multiplier in [2^14, 2^15):
    sh = 16 + round(log2 sigma) - out_bits, sigma^2 = K Var(a w)."""
    ea, ea2 = _moments(in_bits, in_signed)
    ew, ew2 = _moments(w_bits, True)
    var = ea2 * ew2 - (ea * ew) ** 2
    sigma = math.sqrt(k_total * var)
    return int(16 + round(math.log2(sigma)) - out_bits)


def conv_params(g, groups, cout, out_bits, shift, residual: bool):
    """Per-channel multiplier M in [2^14, 2^15), constant shift, zero bias and,
    for identity shortcuts, res_mult in [2^(sh-15), 2^(sh-14)) (about one
    output code per residual code)."""
    c = groups * cout
    mult = g.integers(1 << 14, (1 << 15) - 1, size=c, endpoint=True).astype(np.int32)
    shift_a = np.full(c, shift, dtype=np.int32)
    bias = np.zeros(c, dtype=np.int32)
    res_mult = None
    if residual:
        lo = 1 << max(shift - 15, 0)
        hi = max((1 << max(shift - 14, 0)) - 1, lo)
        res_mult = g.integers(lo, hi, size=c, endpoint=True).astype(np.int32)
    return mult, shift_a, bias, res_mult


def conv_layer_spec(g, *, src, dst, groups, cin, cout, k, stride, pad, in_bits, in_signed,
                    w_bits, out_bits, shuffle=0, res=-1, proj_src=-1, proj_cin=0,
                    proj_stride=1, shift=None):
    w = codes(g, (groups, cout, k, k, cin), w_bits, True)
    if shift is None:
        shift = default_shift(k * k * cin, in_bits, in_signed, w_bits, out_bits)
    mult, shift_a, bias, res_mult = conv_params(g, groups, cout, out_bits, shift, res >= 0)
    L = dict(op="conv", src=src, dst=dst, w=w, stride=stride, pad=pad, in_bits=in_bits,
             in_signed=in_signed, w_bits=w_bits, out_bits=out_bits, mult=mult, shift=shift_a,
             bias=bias, shuffle=shuffle, res=res, res_mult=res_mult, proj_src=proj_src,
             proj_w=None, proj_stride=proj_stride)
    if proj_src >= 0:
        L["proj_w"] = codes(g, (groups, cout, 1, 1, proj_cin), w_bits, True)
    return L


def shuffle_module_spec(g, *, src, dst, groups, ch, bits, shift=None):
    """A cyclic shuffle module (Eq. 9-10) on a G x ch tensor of b-bit codes:
    1x1 b-bit group filter [G][ch][1][1][ch], per-output-channel M, shift,
    zero bias and an identity-shortcut scale res_mult (reading A10)."""
    w = codes(g, (groups, ch, 1, 1, ch), bits, True)
    if shift is None:
        shift = default_shift(ch, bits, False, bits, bits)
    mult, shift_a, bias, res_mult = conv_params(g, groups, ch, bits, shift, True)
    return dict(op="shuffle_module", src=src, dst=dst, w=w, in_bits=bits, w_bits=bits,
                out_bits=bits, mult=mult, shift=shift_a, bias=bias, res_mult=res_mult)


# ---------------------------------------------------------------------------
# Single-layer cases
# ---------------------------------------------------------------------------
def single_layer(seed, *, n, h, w, groups, cin, cout, k=3, stride=1, pad=1, bits=2,
                 w_bits=None, out_bits=None, shuffle=1, shift=None, residual=None):
    """One grouped conv layer with its input.  residual: None | "identity" |
    "projection" (the projection input is a second tensor of cin channels
    at the layer's input resolution)."""
    g = rng(seed)
    w_bits = bits if w_bits is None else w_bits
    out_bits = bits if out_bits is None else out_bits
    x = codes(g, (n, h, w, groups * cin), bits, False)
    ho = (h + 2 * pad - k) // stride + 1
    wo = (w + 2 * pad - k) // stride + 1
    res_id = -1
    proj_id = -1
    extra = {}
    if residual == "identity":
        extra[1] = codes(g, (n, ho, wo, groups * cout), out_bits, False)
        res_id = 1
    elif residual == "projection":
        extra[1] = codes(g, (n, h, w, groups * cin), bits, False)
        proj_id = 1
    L = conv_layer_spec(g, src=0, dst=2, groups=groups, cin=cin, cout=cout, k=k, stride=stride,
                        pad=pad, in_bits=bits, in_signed=False, w_bits=w_bits, out_bits=out_bits,
                        shuffle=shuffle, res=res_id, proj_src=proj_id, proj_cin=cin,
                        proj_stride=stride, shift=shift)
    return dict(x=x, extra=extra, layer=L)


def config_c1(seed=SEED_BASE + 1):
    """N=1, 56x56, G=2 groups of 64 -> 64, 3x3/s1/p1, 2-bit codes, shift 20,
    ReLU, one cyclic step."""
    return single_layer(seed, n=1, h=56, w=56, groups=2, cin=64, cout=64, shuffle=1, shift=20)


C2_LAYERS = [(56, 64), (28, 128), (14, 256), (7, 512)]


def config_c2(i, seed=None, n=32):
    """ResNet-18 stage i's 3x3 conv shape at G=4, batch 32, 2-bit."""
    hw, c = C2_LAYERS[i]
    seed = SEED_BASE + 2 if seed is None else seed
    return single_layer(seed * 10 + i, n=n, h=hw, w=hw, groups=4, cin=c, cout=c, shuffle=1)


def config_c4(groups, bits, seed=None, n=128):
    """ResNet-18 stage-3 layer (14x14, 256 per group, 3x3) at G groups, b bits."""
    seed = SEED_BASE + 4 if seed is None else seed
    return single_layer(seed * 100 + groups * 10 + bits, n=n, h=14, w=14, groups=groups,
                        cin=256, cout=256, bits=bits, shuffle=1)


# ---------------------------------------------------------------------------
# Networks
# ---------------------------------------------------------------------------
def _stem(g, layers, groups, bits, width=64):
    """8-bit signed input x 8-bit signed weights, 7x7/s2/p3, 3 -> width*G,
    requantised to b bits, then 3x3/s2/p1 max pool."""
    layers.append(conv_layer_spec(g, src=0, dst=1, groups=1, cin=3, cout=width * groups, k=7,
                                  stride=2, pad=3, in_bits=8, in_signed=True, w_bits=8,
                                  out_bits=bits))
    layers.append(dict(op="maxpool", src=1, dst=2, k=3, stride=2, pad=1))
    return 2, 3


def resnet18(n=64, groups=4, bits=2, hw=224, classes=1000, seed=SEED_BASE + 3, stages=(2, 2, 2, 2),
             modules=False, channel_shuffle=False, width_mult=1):
    """ResNet-18 topology with every 3x3 conv a G-group b-bit conv at the
    original width per group; conv2 of each basic block adds the shortcut in
    int32 before requantisation and writes its branch one cyclic step on;
    stage-first blocks take a 1x1/s2 grouped projection shortcut.  modules:
    a cyclic shuffle module (Eq. 9-10) at the start of stages 2-4, after the
    stage's first (strided) conv, at the stage's width and resolution
    (Section 4.3 places the module at the beginning of each stage).
    channel_shuffle: the per-stage channel shuffle (Section 4.3, Table 3) at
    the end of the first block of stages 2-4.  width_mult scales every
    stage width (and the stem's output), e.g. for the dense workload of the
    bit-decomposition baseline (Eq. 4: G^2 B-bit products of full width)."""
    g = rng(seed)
    x = codes(g, (n, hw, hw, 3), 8, True)
    layers = []
    cur, nid = _stem(g, layers, groups, bits, width=64 * width_mult)
    ch = 64 * width_mult
    for si, (width, nblk) in enumerate(zip((64 * width_mult, 128 * width_mult, 256 * width_mult,
                                           512 * width_mult), stages)):
        for b in range(nblk):
            s = 2 if (si > 0 and b == 0) else 1
            t1 = nid
            nid += 1
            layers.append(conv_layer_spec(g, src=cur, dst=t1, groups=groups, cin=ch, cout=width, k=3,
                                          stride=s, pad=1, in_bits=bits, in_signed=False,
                                          w_bits=bits, out_bits=bits))
            if modules and si > 0 and b == 0:
                layers.append(shuffle_module_spec(g, src=t1, dst=nid, groups=groups, ch=width,
                                                  bits=bits))
                t1 = nid
                nid += 1
            t2 = nid
            nid += 1
            proj = (s != 1 or ch != width)
            layers.append(conv_layer_spec(g, src=t1, dst=t2, groups=groups, cin=width, cout=width,
                                          k=3, stride=1, pad=1, in_bits=bits, in_signed=False,
                                          w_bits=bits, out_bits=bits, shuffle=1,
                                          res=-1 if proj else cur, proj_src=cur if proj else -1,
                                          proj_cin=ch, proj_stride=s))
            cur, ch = t2, width
            if channel_shuffle and si > 0 and b == 0:
                layers.append(dict(op="channel_shuffle", src=cur, dst=nid, groups=groups))
                cur = nid
                nid += 1
    layers.append(dict(op="avgsum", src=cur, dst=nid))
    layers.append(dict(op="fc", src=nid, dst=nid + 1, w=codes(g, (classes, ch * groups), 8, True)))
    return dict(name=f"resnet18_palq_g{groups}_b{bits}" + ("_mod" if modules else "") +
                ("_cs" if channel_shuffle else ""), n=n, hw=hw,
                groups=groups, bits=bits, x=x, layers=layers, classes=classes)


def resnet50(n=128, groups=2, bits=2, hw=224, classes=1000, seed=SEED_BASE + 5,
             stages=(3, 4, 6, 3)):
    """ResNet-50 (v1.5: stride on the 3x3) bottleneck topology at G groups of
    the original width; the first 1x1's output goes one cyclic step on; the
    last 1x1 adds the shortcut (identity or 1x1/s projection) in int32."""
    g = rng(seed)
    x = codes(g, (n, hw, hw, 3), 8, True)
    layers = []
    cur, nid = _stem(g, layers, groups, bits)
    ch = 64
    for si, (width, nblk) in enumerate(zip((64, 128, 256, 512), stages)):
        for b in range(nblk):
            s = 2 if (si > 0 and b == 0) else 1
            out_c = 4 * width
            t1, t2, t3 = nid, nid + 1, nid + 2
            nid += 3
            common = dict(groups=groups, in_bits=bits, in_signed=False, w_bits=bits, out_bits=bits)
            layers.append(conv_layer_spec(g, src=cur, dst=t1, cin=ch, cout=width, k=1, stride=1,
                                          pad=0, shuffle=1, **common))
            layers.append(conv_layer_spec(g, src=t1, dst=t2, cin=width, cout=width, k=3, stride=s,
                                          pad=1, **common))
            proj = (s != 1 or ch != out_c)
            layers.append(conv_layer_spec(g, src=t2, dst=t3, cin=width, cout=out_c, k=1, stride=1,
                                          pad=0, res=-1 if proj else cur,
                                          proj_src=cur if proj else -1, proj_cin=ch,
                                          proj_stride=s, **common))
            cur, ch = t3, out_c
    layers.append(dict(op="avgsum", src=cur, dst=nid))
    layers.append(dict(op="fc", src=nid, dst=nid + 1, w=codes(g, (classes, ch * groups), 8, True)))
    return dict(name=f"resnet50_palq_g{groups}_b{bits}", n=n, hw=hw, groups=groups, bits=bits,
                x=x, layers=layers, classes=classes)


def image_fp32(seed, n, hw=224, c=3):
    """Synthetic fp32 image batch (standard-normal pixels, NHWC) for the
    quantiser in front of the stem."""
    return rng(seed).standard_normal((n, hw, hw, c), dtype=np.float32)


# ---------------------------------------------------------------------------
# Benchmark workloads (fp32 image batches in front of the 8-bit stem) and
# their centred variants
# ---------------------------------------------------------------------------
# Images: standard-normal fp32 pixels quantised over [-3, 3] (Eq. 2) to
# signed 8-bit codes by the network's first step.
IMAGE_RANGE = (-3.0, 3.0)
GOLDEN_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden")


def workload(name):
    """(spec, fp32 images, images the centring is calibrated on) of a
    benchmark network: "resnet18_g4_b2" (ResNet-18 topology, G=4, 2-bit,
    batch 64, 224x224), "resnet18_g4_b2_shuffles" (the same with the cyclic
    shuffle modules and channel shuffles) or "resnet50_g2_b2" (ResNet-50
    v1.5 bottlenecks, G=2, 2-bit, batch 128, 224x224)."""
    if name == "resnet18_g4_b2":
        return resnet18(n=64, groups=4, bits=2), image_fp32(SEED_BASE + 30, 64), [0, 63]
    if name == "resnet50_g2_b2":
        return resnet50(n=128, groups=2, bits=2), image_fp32(SEED_BASE + 50, 128), [0, 127]
    if name == "resnet18_g4_b2_shuffles":
        # the same network with a cyclic shuffle module at the start of stages
        # 2-4 and the per-stage channel shuffle (Section 4.3, Table 3)
        return (resnet18(n=64, groups=4, bits=2, modules=True, channel_shuffle=True),
                image_fp32(SEED_BASE + 30, 64), [0, 63])
    raise ValueError(name)


def centred_path(name):
    return os.path.join(GOLDEN_DIR, f"centred_bias_{name}.npz")


def with_stored_biases(spec, name):
    """A copy of `spec` whose conv biases are the stored centred ones of
    workload `name` (tests/golden/centred_bias_<name>.npz, written by
    tests/golden/make_centred_bias.py from the oracle's calibration on the
    workload's calibration images): layer i's bias is array "layer<i>"."""
    import copy
    spec = copy.deepcopy(spec)
    with np.load(centred_path(name), allow_pickle=False) as z:
        for i, L in enumerate(spec["layers"]):
            if L["op"] in ("conv", "shuffle_module"):
                b = z[f"layer{i}"]
                if b.shape != (L["w"].shape[0] * L["w"].shape[1],):
                    raise ValueError(f"stored bias of layer {i} has shape {b.shape}")
                L["bias"] = b.astype(np.int32)
    spec["name"] = spec["name"] + "_centred"
    return spec


# Single-layer benchmark cases: C1 (the 56x56 G=2 layer at batch 1), the
# four ResNet-18 stage layers at G=4 and batch 32, and the G x B sweep on the
# stage-3 layer at batch 128.
SINGLE_WORKLOADS = ["c1"] + [f"c2_l{i}" for i in range(4)] + \
    [f"c4_g{g}_b{b}" for g in (1, 2, 4) for b in (2, 3, 4)]


def single_workload(name):
    if name == "c1":
        return config_c1()
    if name.startswith("c2_l"):
        return config_c2(int(name[4:]))
    if name.startswith("c4_g"):
        g, b = name[4:].split("_b")
        return config_c4(int(g), int(b))
    raise ValueError(name)


def single_stored_bias(name):
    """The stored centred bias of single-layer case `name`
    (tests/golden/centred_bias_single.npz, array `name`)."""
    with np.load(os.path.join(GOLDEN_DIR, "centred_bias_single.npz"), allow_pickle=False) as z:
        return z[name].astype(np.int32)
