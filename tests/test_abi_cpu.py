"""Host-only checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments (validate-only context, no GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

from tests import packref

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def P():
    from paper_2208_01944_amd import palq
    return palq


@pytest.fixture(scope="module")
def vctx(P):
    return P.Context(-1)


def test_exports_every_declared_symbol(P):
    hdr = open(os.path.join(ROOT, "include", "palq.h")).read()
    declared = set(re.findall(r"\b(palq_[a-z_0-9]+)\s*\(", hdr))
    assert declared, "no declarations found"
    lib = ctypes.CDLL(P.LIB_PATH)
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared == set(P.EXPORTS)
    assert "gfx950" in P.version()


def test_row_bytes_matches_reference(P):
    for bits in (2, 3, 4, 8):
        for c in (1, 3, 15, 16, 17, 31, 32, 33, 63, 64, 96, 100, 256, 512):
            assert P.row_bytes(c, bits) == packref.row_bytes(c, bits)
    assert P.row_bytes(4, 5) == -1 and P.row_bytes(0, 2) == -1


def test_packref_golden_bytes():
    # code j at bits [b*j, b*j+b): [1,2,3,0] at 2 bits is 0b00_11_10_01
    assert packref.pack_row([1, 2, 3, 0], 2) == bytes([0x39, 0, 0, 0])
    assert packref.pack_row([-2, 1], 2) == bytes([0b0110, 0, 0, 0])
    assert packref.pack_row([0xA, 0x5, 0xF], 4) == bytes([0x5A, 0x0F, 0, 0])
    assert packref.pack_row([-128, 127, 3], 8) == bytes([0x80, 0x7F, 0x03, 0])
    # 3-bit: code 5 (0b101) at j=0 -> low bits 01 at bit 0, bit 2 at hi bit 0
    b = packref.pack_row([5] + [0] * 31, 3)
    assert b[0] == 1 and b[8] == 1 and sum(b) == 2
    b = packref.pack_row([0] * 17 + [4] + [0] * 14, 3)  # j=17: hi bit 2*(17 & 15) + 1 = 3
    assert int.from_bytes(b[8:12], "little") == 1 << 3 and sum(b[:8]) == 0
    b = packref.pack_row([0] * 5 + [4] + [0] * 25 + [4], 3)  # j=5: hi bit 10; j=31: hi bit 31
    assert int.from_bytes(b[8:12], "little") == (1 << 10) | (1 << 31) and sum(b[:8]) == 0


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_packref_round_trip(bits):
    g = np.random.default_rng(bits)
    for signed in (False, True):
        lo, hi = (-(1 << (bits - 1)), (1 << (bits - 1)) - 1) if signed else (0, (1 << bits) - 1)
        x = g.integers(lo, hi + 1, (2, 3, 2, 3 * 37))
        buf = packref.pack(x, 3, bits)
        assert buf.size == 2 * 3 * 2 * 3 * packref.row_bytes(37, bits)
        np.testing.assert_array_equal(packref.unpack(buf, x.shape, 3, bits, signed), x)


def _fake(i):
    return 0x100000000 * (i + 1)


def _act(P, n=1, h=8, w=8, g=2, c=64, bits=2, signed=False, slot=0):
    return P.make_act(n, h, w, g, c, bits, signed, _fake(slot))


def _conv(P, vctx, **over):
    x = over.pop("x", _act(P))
    f = over.pop("f", P.Filter(2, 32, 64, 3, 3, 2, _fake(10)))
    out = over.pop("out", _act(P, c=32, slot=20))
    rq = over.pop("rq", P.Requant(_fake(30), _fake(31), None, 2))
    res = over.pop("res", None)
    stride, pad = over.pop("stride", 1), over.pop("pad", 1)
    return P._group_conv(vctx.h, ctypes.byref(x), ctypes.byref(f), stride, pad, ctypes.byref(rq),
                         ctypes.byref(res) if res is not None else None, 1, ctypes.byref(out), None)


def test_validate_only_group_conv_errors(P, vctx):
    assert _conv(P, vctx) == P.OK
    assert _conv(P, vctx, x=_act(P, bits=5)) == P.ERR_ARG
    assert _conv(P, vctx, x=_act(P, g=3)) == P.ERR_ARG                    # groups mismatch
    assert _conv(P, vctx, x=_act(P, c=32)) == P.ERR_ARG                   # cin mismatch
    assert _conv(P, vctx, out=_act(P, h=7, c=32, slot=20)) == P.ERR_ARG   # wrong out shape
    assert _conv(P, vctx, out=_act(P, c=32, bits=3, slot=20)) == P.ERR_ARG  # bits != out_bits
    assert _conv(P, vctx, out=_act(P, c=32, slot=0)) == P.ERR_ARG          # aliases the input
    assert _conv(P, vctx, rq=P.Requant(None, _fake(31), None, 2)) == P.ERR_ARG
    assert _conv(P, vctx, rq=P.Requant(_fake(30) + 4, _fake(31), None, 2)) == P.ERR_ARG  # misaligned
    assert _conv(P, vctx, stride=0) == P.ERR_ARG
    # unsigned 6- and 8-bit inputs (the dense baselines) with weights of their width
    for b in (6, 8):
        assert _conv(P, vctx, x=_act(P, bits=b), f=P.Filter(2, 32, 64, 3, 3, b, _fake(10))) == P.OK
    assert _conv(P, vctx, x=_act(P, bits=4, signed=True)) == P.ERR_UNSUPPORTED  # signed input below 8 bits
    assert P.row_bytes(10, 6) == 12 and P.row_bytes(10, 5) == -1  # 6-bit codes one per byte
    # signed 8-bit input is the stem format
    assert _conv(P, vctx, x=_act(P, bits=8, signed=True), f=P.Filter(2, 32, 64, 3, 3, 8, _fake(10))) == P.OK
    # accumulator bound: K * 255... 8-bit weights with a huge K
    big = P.Filter(1, 32, 8192, 3, 3, 8, _fake(10))
    assert _conv(P, vctx, x=_act(P, g=1, c=8192, bits=8, signed=True), f=big,
                 out=_act(P, g=1, c=32, slot=20)) == P.ERR_OVERFLOW
    assert "2^30" in vctx.last_error()
    # 2-bit inputs (the int8 path scales their accumulator by 16): 2^26
    wide = 1 << 22
    assert _conv(P, vctx, x=_act(P, g=1, c=wide), f=P.Filter(1, 32, wide, 3, 3, 2, _fake(10)),
                 out=_act(P, g=1, c=32, slot=20)) == P.ERR_OVERFLOW
    assert "2^26" in vctx.last_error()


def test_validate_only_residual_errors(P, vctx):
    ident = _act(P, c=32, slot=40)
    res = P.Residual(ctypes.pointer(ident), _fake(41), None, None, 1)
    assert _conv(P, vctx, res=res) == P.OK
    res.res_mult = None
    assert _conv(P, vctx, res=res) == P.ERR_ARG
    bad = _act(P, c=16, slot=40)
    assert _conv(P, vctx, res=P.Residual(ctypes.pointer(bad), _fake(41), None, None, 1)) == P.ERR_ARG
    pin = _act(P, h=16, w=16, c=64, slot=50)
    pw = P.Filter(2, 32, 64, 1, 1, 2, _fake(51))
    res = P.Residual(None, None, ctypes.pointer(pin), ctypes.pointer(pw), 2)
    assert _conv(P, vctx, res=res) == P.OK
    res.proj_stride = 1                       # 16x16 at stride 1 is not 8x8
    assert _conv(P, vctx, res=res) == P.ERR_ARG
    res = P.Residual(ctypes.pointer(ident), _fake(41), ctypes.pointer(pin), ctypes.pointer(pw), 2)
    assert _conv(P, vctx, res=res) == P.ERR_ARG  # both kinds


def test_validate_only_other_calls(P, vctx):
    a = _act(P)
    b = _act(P, slot=5)
    assert P._shuffle(vctx.h, ctypes.byref(a), 3, ctypes.byref(b)) == P.OK
    assert P._shuffle(vctx.h, ctypes.byref(a), 1, ctypes.byref(a)) == P.ERR_ARG  # in == out
    c = _act(P, bits=3, slot=5)
    assert P._shuffle(vctx.h, ctypes.byref(a), 1, ctypes.byref(c)) == P.ERR_ARG
    q = _act(P, slot=6)
    assert P._quantize(vctx.h, _fake(7), 0.0, 1.0, ctypes.byref(q), None) == P.OK
    assert P._quantize(vctx.h, _fake(7), 1.0, 1.0, ctypes.byref(q), None) == P.ERR_ARG
    assert P._quantize(vctx.h, _fake(7), 0.0, float("inf"), ctypes.byref(q), None) == P.ERR_ARG
    assert P._quantize(vctx.h, _fake(7), float("nan"), 1.0, ctypes.byref(q), None) == P.OK
    assert P._quantize(vctx.h, None, 0.0, 1.0, ctypes.byref(q), None) == P.ERR_ARG
    pooled = _act(P, h=4, w=4, slot=8)
    assert P._maxpool(vctx.h, ctypes.byref(a), 3, 2, 1, ctypes.byref(pooled)) == P.OK
    assert P._maxpool(vctx.h, ctypes.byref(a), 3, 2, 3, ctypes.byref(pooled)) == P.ERR_ARG
    assert P._avgsum(vctx.h, ctypes.byref(a), _fake(9)) == P.OK
    assert P._fc(vctx.h, _fake(9), 4, 128, _fake(11), 10, _fake(12)) == P.OK
    assert P._fc(vctx.h, _fake(9), 4, 0, _fake(11), 10, _fake(12)) == P.ERR_ARG
    assert P._pack(vctx.h, None, ctypes.byref(a)) == P.ERR_ARG
    # layouts: either is taken, any other value is an argument error
    g = _act(P, slot=13)
    g.layout = P.LAYOUT_GROUP
    assert P._shuffle(vctx.h, ctypes.byref(a), 3, ctypes.byref(g)) == P.OK
    assert P._maxpool(vctx.h, ctypes.byref(g), 3, 2, 1, ctypes.byref(pooled)) == P.OK
    g.layout = 2
    assert P._shuffle(vctx.h, ctypes.byref(a), 3, ctypes.byref(g)) == P.ERR_ARG
    assert "layout" in vctx.last_error()
    assert P._avgsum(vctx.h, ctypes.byref(g), _fake(9)) == P.ERR_ARG
    assert P._set_conv_fp4(vctx.h, 0) == P.OK
    assert P._set_conv_fp4(vctx.h, 1) == P.OK
    assert P._set_conv_fp4(vctx.h, 2) == P.ERR_ARG
    assert P._set_conv_fp4(None, 1) == P.ERR_ARG


def _layer(P, **kw):
    L = P.Layer()
    L.res_src = -1
    L.proj_src = -1
    for k, v in kw.items():
        setattr(L, k, v)
    return L


def test_validate_only_net_create(P, vctx):
    inp = P.make_act(2, 16, 16, 1, 3, 8, True, 0)
    Ls = (P.Layer * 5)()
    Ls[0] = _layer(P, op=P.OP_CONV, src=0, dst=1, w=P.Filter(1, 128, 3, 3, 3, 8, _fake(1)), stride=2,
                   pad=1, mult=_fake(2), shift=_fake(3), out_bits=2)
    Ls[1] = _layer(P, op=P.OP_MAXPOOL, src=1, dst=2, pool_k=3, pool_stride=2, pool_pad=1)
    Ls[2] = _layer(P, op=P.OP_CONV, src=2, dst=3, w=P.Filter(2, 64, 64, 3, 3, 2, _fake(4)), stride=1,
                   pad=1, mult=_fake(5), shift=_fake(6), out_bits=2, shuffle_steps=1, res_src=2,
                   res_mult=_fake(7))
    Ls[3] = _layer(P, op=P.OP_AVGSUM, src=3, dst=4)
    Ls[4] = _layer(P, op=P.OP_FC, src=4, dst=5, fc_w=_fake(8), fc_out=10)
    h = ctypes.c_void_p()
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.OK
    # 2 * MACs: 2*(2*8*8*128*27) + 2*(2*4*4*128*576) + 2*(2*128*10)
    assert P._net_ops(h) == 2 * (2 * 8 * 8 * 128 * 27) + 2 * (2 * 4 * 4 * 128 * 576) + 2 * (2 * 128 * 10)
    # kernel names: nothing is planned on a validate-only network; bad indices give NULL
    assert [P._net_layer_kernels(h, i, 0) for i in range(5)] == [b""] * 5
    assert P._net_layer_kernels(h, -1, 1) == b"" and P._net_layer_kernels(h, -1, 0) == b""
    assert P._net_layer_kernels(h, 5, 0) is None and P._net_layer_kernels(h, -2, 0) is None
    assert P._net_layer_kernels(h, 0, 2) is None and P._net_layer_kernels(None, 0, 0) is None
    P._net_destroy(h)
    # FC not last / wrong input / reused id
    Ls[4] = _layer(P, op=P.OP_FC, src=3, dst=5, fc_w=_fake(8), fc_out=10)
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.ERR_ARG
    Ls[4] = _layer(P, op=P.OP_FC, src=4, dst=4, fc_w=_fake(8), fc_out=10)
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.ERR_ARG
    Ls[4] = _layer(P, op=P.OP_FC, src=4, dst=5, fc_w=_fake(8), fc_out=10)
    Ls[2].w = P.Filter(4, 64, 64, 3, 3, 2, _fake(4))  # 4 x 64 != 128 input channels
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.ERR_ARG
    assert "layer 2" in vctx.last_error()


def test_validate_only_net_tensor_layouts(P, vctx):
    """Which tensors a network stores group by group: outputs of several
    groups whose every reader keeps those groups; a tensor that a reader
    re-splits, a one-group tensor and, with PALQ_NET_PIXEL_LAYOUT, every
    tensor stay in the pixel layout."""
    inp = P.make_act(2, 16, 16, 1, 3, 8, True, 0)
    Ls = (P.Layer * 8)()
    Ls[0] = _layer(P, op=P.OP_CONV, src=0, dst=1, w=P.Filter(1, 128, 3, 3, 3, 8, _fake(1)), stride=2,
                   pad=1, mult=_fake(2), shift=_fake(3), out_bits=2)
    Ls[1] = _layer(P, op=P.OP_MAXPOOL, src=1, dst=2, pool_k=3, pool_stride=2, pool_pad=1)
    Ls[2] = _layer(P, op=P.OP_CONV, src=2, dst=3, w=P.Filter(2, 64, 64, 3, 3, 2, _fake(4)), stride=1,
                   pad=1, mult=_fake(5), shift=_fake(6), out_bits=2)
    Ls[3] = _layer(P, op=P.OP_CONV, src=3, dst=4, w=P.Filter(2, 64, 64, 3, 3, 2, _fake(7)), stride=1,
                   pad=1, mult=_fake(8), shift=_fake(9), out_bits=2, res_src=3, res_mult=_fake(10))
    Ls[4] = _layer(P, op=P.OP_CHANNEL_SHUFFLE, src=4, dst=5)
    Ls[5] = _layer(P, op=P.OP_CONV, src=5, dst=6, w=P.Filter(4, 32, 32, 3, 3, 2, _fake(11)), stride=1,
                   pad=1, mult=_fake(12), shift=_fake(13), out_bits=2)
    Ls[6] = _layer(P, op=P.OP_AVGSUM, src=6, dst=7)
    Ls[7] = _layer(P, op=P.OP_FC, src=7, dst=8, fc_w=_fake(14), fc_out=10)
    want = {1: P.LAYOUT_PIXEL,   # one group
            2: P.LAYOUT_PIXEL,   # one group (the next conv re-splits it)
            3: P.LAYOUT_GROUP,   # conv input and identity shortcut, both with its 2 groups
            4: P.LAYOUT_GROUP,   # read by the channel shuffle
            5: P.LAYOUT_PIXEL,   # re-split into 4 groups by the next conv
            6: P.LAYOUT_GROUP}   # read by the global sum
    for flags, expect in ((0, want), (P.NET_PIXEL_LAYOUT, {t: P.LAYOUT_PIXEL for t in want})):
        h = ctypes.c_void_p()
        assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 8, flags, ctypes.byref(h)) == P.OK, vctx.last_error()
        for t, lay in expect.items():
            d = P.Act()
            assert P._net_tensor(h, t, ctypes.byref(d)) == P.OK
            assert d.layout == lay, (flags, t, d.layout)
        P._net_destroy(h)


def test_validate_only_forward_image(P, vctx):
    """palq_forward_image: image-input networks only, finite l < u, non-null
    aligned pointers (validate-only: no device work)."""
    inp = P.make_act(2, 16, 16, 1, 3, 8, True, 0)
    Ls = (P.Layer * 3)()
    Ls[0] = _layer(P, op=P.OP_CONV, src=0, dst=1, w=P.Filter(1, 128, 3, 7, 7, 8, _fake(1)), stride=2,
                   pad=3, mult=_fake(2), shift=_fake(3), out_bits=2)
    Ls[1] = _layer(P, op=P.OP_AVGSUM, src=1, dst=2)
    Ls[2] = _layer(P, op=P.OP_FC, src=2, dst=3, fc_w=_fake(8), fc_out=10)
    h = ctypes.c_void_p()
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 3, 0, ctypes.byref(h)) == P.OK
    fi = P._forward_image
    assert fi(vctx.h, h, _fake(20), -3.0, 3.0, _fake(21)) == P.OK
    assert fi(vctx.h, h, _fake(20), 3.0, 3.0, _fake(21)) == P.ERR_ARG          # u == l
    assert fi(vctx.h, h, _fake(20), float("nan"), 3.0, _fake(21)) == P.ERR_ARG  # no calibration here
    assert fi(vctx.h, h, _fake(20), -3.0, float("inf"), _fake(21)) == P.ERR_ARG
    assert fi(vctx.h, h, None, -3.0, 3.0, _fake(21)) == P.ERR_ARG
    assert fi(vctx.h, h, _fake(20) + 2, -3.0, 3.0, _fake(21)) == P.ERR_ARG      # misaligned
    P._net_destroy(h)
    # a network whose input is not an 8-bit 3-channel image
    inp2 = P.make_act(2, 16, 16, 2, 64, 2, False, 0)
    Ls2 = (P.Layer * 3)()
    Ls2[0] = _layer(P, op=P.OP_CONV, src=0, dst=1, w=P.Filter(2, 64, 64, 3, 3, 2, _fake(1)), stride=1,
                    pad=1, mult=_fake(2), shift=_fake(3), out_bits=2)
    Ls2[1] = _layer(P, op=P.OP_AVGSUM, src=1, dst=2)
    Ls2[2] = _layer(P, op=P.OP_FC, src=2, dst=3, fc_w=_fake(8), fc_out=10)
    assert P._net_create(vctx.h, ctypes.byref(inp2), Ls2, 3, 0, ctypes.byref(h)) == P.OK
    assert fi(vctx.h, h, _fake(20), -3.0, 3.0, _fake(21)) == P.ERR_ARG
    assert "image" in vctx.last_error()
    P._net_destroy(h)
    # graph replay is a network flag; not together with per-layer timing
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 3, P.NET_GRAPH, ctypes.byref(h)) == P.OK
    P._net_destroy(h)
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 3, P.NET_GRAPH | P.NET_TIMING, ctypes.byref(h)) == P.ERR_ARG
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 3, 16, ctypes.byref(h)) == P.ERR_ARG  # unknown flag


def test_validate_only_shuffle_module(P, vctx):
    x = _act(P, c=64)
    out = _act(P, c=64, slot=20)
    f = P.Filter(2, 64, 64, 1, 1, 2, _fake(10))
    rq = P.Requant(_fake(30), _fake(31), None, 2)

    def mod(x=x, f=f, rq=rq, rm=_fake(40), out=out):
        return P._shuffle_module(vctx.h, ctypes.byref(x), ctypes.byref(f), ctypes.byref(rq), rm,
                                 ctypes.byref(out))
    assert mod() == P.OK
    assert mod(f=P.Filter(2, 64, 64, 3, 3, 2, _fake(10))) == P.ERR_ARG   # not 1x1
    assert mod(f=P.Filter(2, 32, 64, 1, 1, 2, _fake(10))) == P.ERR_ARG   # cout != cin
    assert mod(rm=None) == P.ERR_ARG
    assert mod(out=_act(P, c=64, slot=0)) == P.ERR_ARG                    # out aliases in
    assert mod(out=_act(P, h=4, c=64, slot=20)) == P.ERR_ARG              # wrong shape
    assert mod(x=_act(P, c=64, g=3), f=P.Filter(3, 64, 64, 1, 1, 2, _fake(10)),
               out=_act(P, c=64, g=3, slot=20)) == P.OK


def test_validate_only_net_with_shuffle_module(P, vctx):
    inp = P.make_act(2, 16, 16, 1, 3, 8, True, 0)
    Ls = (P.Layer * 5)()
    Ls[0] = _layer(P, op=P.OP_CONV, src=0, dst=1, w=P.Filter(1, 128, 3, 3, 3, 8, _fake(1)), stride=2,
                   pad=1, mult=_fake(2), shift=_fake(3), out_bits=2)
    Ls[1] = _layer(P, op=P.OP_SHUFFLE_MODULE, src=1, dst=2, w=P.Filter(2, 64, 64, 1, 1, 2, _fake(4)),
                   mult=_fake(5), shift=_fake(6), out_bits=2, res_mult=_fake(7))
    Ls[2] = _layer(P, op=P.OP_CONV, src=2, dst=3, w=P.Filter(2, 64, 64, 3, 3, 2, _fake(8)), stride=1,
                   pad=1, mult=_fake(9), shift=_fake(10), out_bits=2)
    Ls[3] = _layer(P, op=P.OP_AVGSUM, src=3, dst=4)
    Ls[4] = _layer(P, op=P.OP_FC, src=4, dst=5, fc_w=_fake(11), fc_out=10)
    h = ctypes.c_void_p()
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.OK
    # 2 * MACs: stem + module (1x1, 64 per group) + 3x3 + FC
    assert P._net_ops(h) == 2 * (2 * 8 * 8 * 128 * 27) + 2 * (2 * 8 * 8 * 128 * 64) + \
        2 * (2 * 8 * 8 * 128 * 576) + 2 * (2 * 128 * 10)
    P._net_destroy(h)
    Ls[1].w = P.Filter(2, 64, 64, 3, 3, 2, _fake(4))
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.ERR_ARG
    assert "layer 1" in vctx.last_error()
    Ls[1].w = P.Filter(2, 64, 64, 1, 1, 2, _fake(4))
    Ls[1].res_mult = None
    assert P._net_create(vctx.h, ctypes.byref(inp), Ls, 5, 0, ctypes.byref(h)) == P.ERR_ARG


def test_validate_only_channel_shuffle(P, vctx):
    a = _act(P, g=4, c=37, bits=3)
    b = _act(P, g=4, c=37, bits=3, slot=5)
    assert P._channel_shuffle(vctx.h, ctypes.byref(a), ctypes.byref(b)) == P.OK
    assert P._channel_shuffle(vctx.h, ctypes.byref(a), ctypes.byref(a)) == P.ERR_ARG      # overlap
    c = _act(P, g=4, c=37, bits=2, slot=5)
    assert P._channel_shuffle(vctx.h, ctypes.byref(a), ctypes.byref(c)) == P.ERR_ARG      # bits differ
    d = _act(P, g=2, c=74, bits=3, slot=5)
    assert P._channel_shuffle(vctx.h, ctypes.byref(a), ctypes.byref(d)) == P.ERR_ARG      # grouping differs


def test_validate_only_group_conv_noalloc(P, vctx):
    """palq_group_conv_noalloc takes palq_group_conv's arguments and checks;
    a layer whose prepacked filter and requant constants exceed the static
    buffer is refused on the host (nothing enqueued)."""
    def call(x, f, out):
        rq = P.Requant(_fake(30), _fake(31), None, 2)
        return P._group_conv_noalloc(vctx.h, ctypes.byref(x), ctypes.byref(f), 1, 1, ctypes.byref(rq), None, 1,
                                     ctypes.byref(out), None)
    assert call(_act(P), P.Filter(2, 32, 64, 3, 3, 2, _fake(10)), _act(P, c=32, slot=20)) == P.OK
    assert call(_act(P, bits=5), P.Filter(2, 32, 64, 3, 3, 2, _fake(10)), _act(P, c=32, slot=20)) == P.ERR_ARG
    # ResNet-18's largest 3x3 at G = 4 (512 -> 512 per group) fits: int8 + FP4 slabs of 72 K-blocks
    big_ok = P.Filter(4, 512, 512, 3, 3, 2, _fake(10))
    assert call(_act(P, g=4, c=512), big_ok, _act(P, g=4, c=512, slot=20)) == P.OK
    # twice the groups does not: 8 x 512 x 72 x 96 bytes > 16 MiB
    too_big = P.Filter(8, 512, 512, 3, 3, 2, _fake(10))
    assert call(_act(P, g=8, c=512), too_big, _act(P, g=8, c=512, slot=20)) == P.ERR_UNSUPPORTED
    assert "static buffer" in vctx.last_error()
    assert P.NOALLOC_SCRATCH_BYTES == 16 << 20


def test_validate_only_conv_plan(P, vctx):
    """palq_conv_plan_create checks like palq_group_conv; palq_conv_run checks
    pointers against the plan (validate-only: nothing runs)."""
    x, f, out = _act(P), P.Filter(2, 32, 64, 3, 3, 2, _fake(10)), _act(P, c=32, slot=20)
    rq = P.Requant(_fake(30), _fake(31), None, 2)
    h = ctypes.c_void_p()
    assert P._conv_plan_create(vctx.h, ctypes.byref(x), ctypes.byref(f), 1, 1, ctypes.byref(rq), None, 1,
                               ctypes.byref(out), ctypes.byref(h)) == P.OK
    assert P._conv_run(vctx.h, h, _fake(1), None, _fake(40), None) == P.OK
    assert P._conv_plan_kernels(h) == b"" and P._conv_plan_kernels(None) is None
    assert P._conv_run(vctx.h, h, None, None, _fake(40), None) == P.ERR_ARG           # null input
    assert P._conv_run(vctx.h, h, _fake(1) + 8, None, _fake(40), None) == P.ERR_ARG   # misaligned
    assert P._conv_run(vctx.h, h, _fake(1), _fake(3), _fake(40), None) == P.ERR_ARG   # no shortcut planned
    assert P._conv_run(vctx.h, h, _fake(1), None, _fake(1), None) == P.ERR_ARG        # out aliases in
    other = P.Context(-1)
    assert P._conv_run(other.h, h, _fake(1), None, _fake(40), None) == P.ERR_ARG      # another context
    P._conv_plan_destroy(h)
    # the layer's own checks apply at plan time
    bad = _act(P, c=32, bits=3, slot=20)
    assert P._conv_plan_create(vctx.h, ctypes.byref(x), ctypes.byref(f), 1, 1, ctypes.byref(rq), None, 1,
                               ctypes.byref(bad), ctypes.byref(h)) == P.ERR_ARG
    assert "plan:" in vctx.last_error()
    # a planned identity shortcut needs its input at run time
    res = P.Residual()
    ident = _act(P, c=32, slot=50)
    res.identity = ctypes.pointer(ident)
    res.res_mult = _fake(32)
    assert P._conv_plan_create(vctx.h, ctypes.byref(x), ctypes.byref(f), 1, 1, ctypes.byref(rq), ctypes.byref(res), 1,
                               ctypes.byref(out), ctypes.byref(h)) == P.OK
    assert P._conv_run(vctx.h, h, _fake(1), None, _fake(40), None) == P.ERR_ARG
    assert P._conv_run(vctx.h, h, _fake(1), _fake(3), _fake(40), None) == P.OK
    P._conv_plan_destroy(h)
