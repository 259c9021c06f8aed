"""GPU parity of the single-op entry points against the CPU oracle.

Every case draws seeded inputs (paper_2208_01944_amd.inputs), runs the HIP
library through its C ABI and compares with oracle/ element by element:
codes and int32 accumulators bit-exact.
"""
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2208_01944_amd import inputs as I
from tests import packref

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    from paper_2208_01944_amd import palq
    return palq.Context(0)


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


# ---------------------------------------------------------------- layout
def group_major(packed, pixels, groups):
    """Pixel-layout packed bytes [pixels][groups][row] reordered to the group
    layout [groups][pixels][row]."""
    return np.asarray(packed).reshape(pixels, groups, -1).transpose(1, 0, 2).reshape(-1)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("cpg", [1, 5, 16, 37, 64, 96])
@pytest.mark.parametrize("layout", [0, 1])
def test_pack_bytes_match_reference(ctx, bits, cpg, layout):
    say(f"pack bits={bits} cpg={cpg} layout={layout}")
    g = np.random.default_rng(bits * 100 + cpg)
    for signed in (False, True):
        x = I.codes(g, (2, 3, 5, 3 * cpg), bits, signed).astype(np.int64)
        t = ctx.pack(x, 3, bits, signed, layout=layout)
        got = t.buf[:packref.row_bytes(cpg, bits) * 2 * 3 * 5 * 3].cpu().numpy()
        ref = packref.pack(x, 3, bits)
        np.testing.assert_array_equal(got, group_major(ref, 2 * 3 * 5, 3) if layout else ref)
        np.testing.assert_array_equal(ctx.unpack(t), x)


# ---------------------------------------------------------------- quantiser
@pytest.mark.parametrize("bits,signed", [(2, False), (3, False), (4, False), (8, True), (2, True)])
@pytest.mark.parametrize("layout", [0, 1])
def test_quantize_matches_oracle(ctx, torch, bits, signed, layout):
    say(f"quantize bits={bits} signed={signed} layout={layout}")
    g = np.random.default_rng(bits)
    x = g.normal(0, 1.5, (3, 17, 11, 2 * 21)).astype(np.float32)
    x.flat[::97] = np.nan
    x.flat[5::211] = np.inf
    x.flat[7::233] = -np.inf
    # exact ties of Eq. 2 for l=0, u=3 at 2 bits
    x.flat[:3] = [0.5, 1.5, 2.5]
    xd = ctx.upload(x)
    out = ctx.empty_act(3, 17, 11, 2, 21, bits, signed, layout=layout)
    rng = torch.empty(2, dtype=torch.float32, device=ctx.dev)
    ctx.quantize(xd, -2.0, 3.0, out, rng)
    np.testing.assert_array_equal(ctx.unpack(out), O.quantize(x, -2.0, 3.0, bits, signed))
    np.testing.assert_array_equal(rng.cpu().numpy(), np.array([-2.0, 3.0], np.float32))
    # calibrated range (NaN bounds): min/max of the finite... non-NaN values
    x2 = np.where(np.isinf(x), 0.0, x).astype(np.float32)
    ctx.quantize(ctx.upload(x2), float("nan"), float("nan"), out, rng)
    l, u = O.calibrate_range(x2)
    np.testing.assert_array_equal(rng.cpu().numpy(), np.array([l, u], np.float32))
    np.testing.assert_array_equal(ctx.unpack(out), O.quantize(x2, l, u, bits, signed))


# ---------------------------------------------------------------- conv
def run_conv(ctx, torch, case, centred=False, layout=(0, 0, 0)):
    """Runs a single_layer() case on the GPU; returns (codes, acc, ref_codes,
    ref_acc).  layout: the (input, output, shortcut input) tensor layouts."""
    L = case["layer"]
    x = case["x"]
    G, co, kh, kw, ci = L["w"].shape
    res = case["extra"].get(1) if L["res"] >= 0 else None
    px = case["extra"].get(1) if L["proj_src"] >= 0 else None
    bias = L["bias"]
    if centred:
        _, acc0 = O.conv_layer(x, L["w"], L["stride"], L["pad"], L["mult"], L["shift"], None,
                               L["out_bits"], L["shuffle"], res=res, res_mult=L["res_mult"],
                               proj_x=px, proj_w=L["proj_w"], proj_stride=L["proj_stride"])
        t = acc0
        if res is not None:
            t = t + O.cyclic_permute(np.asarray(L["res_mult"], np.int64), G, L["shuffle"]) * res
        mean = np.floor(t.reshape(-1, t.shape[-1]).mean(axis=0) + 0.5).astype(np.int64)
        bias = O.cyclic_permute(-mean, G, -L["shuffle"]).astype(np.int32)
    ref_q, ref_acc = O.conv_layer(x, L["w"], L["stride"], L["pad"], L["mult"], L["shift"], bias,
                                  L["out_bits"], L["shuffle"], res=res, res_mult=L["res_mult"],
                                  proj_x=px, proj_w=L["proj_w"], proj_stride=L["proj_stride"])
    in_signed = bool(L["in_signed"])
    xt = ctx.pack(x, G, L["in_bits"], in_signed, layout=layout[0])
    wt, wf = ctx.pack_filter(L["w"], L["w_bits"])
    n, h, w, _ = x.shape
    ho = (h + 2 * L["pad"] - kh) // L["stride"] + 1
    wo = (w + 2 * L["pad"] - kw) // L["stride"] + 1
    out = ctx.empty_act(n, ho, wo, G, co, L["out_bits"], layout=layout[1])
    dump = torch.zeros(max(n * ho * wo * G * co, 4), dtype=torch.int32, device=ctx.dev)
    i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
    kw_ = {}
    if res is not None:
        kw_["identity"] = ctx.pack(res, G, L["out_bits"], layout=layout[2])
        kw_["res_mult"] = i32(L["res_mult"])
    if px is not None:
        kw_["proj_in"] = ctx.pack(px, G, L["in_bits"], layout=layout[2])
        pt, kw_["proj_w"] = ctx.pack_filter(L["proj_w"], L["w_bits"])
        kw_["proj_stride"] = L["proj_stride"]
    # without the accumulator dump (the kernels' common-case epilogue) ...
    ctx.group_conv(xt, wf, L["stride"], L["pad"], i32(L["mult"]), i32(L["shift"]), i32(bias), out,
                   shuffle=L["shuffle"], **kw_)
    ctx.sync()
    q_plain = ctx.unpack(out)
    # ... and with it (the general epilogue)
    ctx.group_conv(xt, wf, L["stride"], L["pad"], i32(L["mult"]), i32(L["shift"]), i32(bias), out,
                   shuffle=L["shuffle"], acc_dump=dump, **kw_)
    ctx.sync()
    acc = dump[:n * ho * wo * G * co].cpu().numpy().astype(np.int64).reshape(ref_acc.shape)
    q = ctx.unpack(out)
    np.testing.assert_array_equal(q_plain, q)
    return q, acc, ref_q, ref_acc


def check_conv(ctx, torch, case, centred=False, spread=False, layout=(0, 0, 0)):
    q, acc, rq, racc = run_conv(ctx, torch, case, centred, layout)
    np.testing.assert_array_equal(acc, racc)
    np.testing.assert_array_equal(q, rq)
    if spread:  # the centred variant must exercise every output code
        hist = np.bincount(rq.reshape(-1), minlength=1 << case["layer"]["out_bits"])
        assert np.all(hist > 0), hist


def test_conv_c1_stated_and_centred(ctx, torch):
    say("conv C1 (N=1, 56x56, G=2, 64->64, 2-bit, shift 20)")
    case = I.config_c1()
    check_conv(ctx, torch, case)
    check_conv(ctx, torch, case, centred=True, spread=True)


CONV_CASES = [
    # several tiles + ragged tail, MFMA path
    dict(n=2, h=13, w=13, groups=3, cin=64, cout=64, k=3, stride=1, pad=1, bits=2),
    dict(n=2, h=15, w=15, groups=2, cin=64, cout=96, k=3, stride=2, pad=1, bits=2),
    dict(n=3, h=9, w=11, groups=2, cin=128, cout=64, k=1, stride=1, pad=0, bits=2),
    dict(n=2, h=10, w=10, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=3),
    dict(n=2, h=10, w=10, groups=2, cin=64, cout=128, k=3, stride=1, pad=1, bits=4),
    dict(n=1, h=7, w=7, groups=4, cin=192, cout=32, k=3, stride=1, pad=1, bits=2),
    dict(n=2, h=6, w=5, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=2, out_bits=8),
    dict(n=2, h=6, w=5, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=2, out_bits=3),
    dict(n=2, h=6, w=5, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=2, out_bits=4),
    dict(n=2, h=8, w=8, groups=4, cin=64, cout=64, k=3, stride=1, pad=1, bits=2, residual="identity"),
    dict(n=2, h=9, w=9, groups=4, cin=64, cout=64, k=3, stride=2, pad=1, bits=2, residual="projection"),
    dict(n=2, h=8, w=8, groups=3, cin=64, cout=64, k=3, stride=1, pad=1, bits=3, residual="identity"),
    # direct path: odd channel counts, mixed widths, 5x5
    dict(n=2, h=7, w=6, groups=3, cin=5, cout=7, k=3, stride=1, pad=1, bits=2),
    dict(n=1, h=9, w=9, groups=2, cin=16, cout=40, k=5, stride=2, pad=2, bits=4),
    dict(n=2, h=6, w=6, groups=2, cin=20, cout=20, k=3, stride=1, pad=0, bits=3, residual="identity"),
    dict(n=2, h=7, w=7, groups=2, cin=24, cout=32, k=3, stride=2, pad=1, bits=2, residual="projection"),
    dict(n=2, h=6, w=6, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=2, w_bits=4),
    # unsigned 8- and 6-bit codes (the dense baselines): int8 matrix cores with the flipped-byte operand
    dict(n=2, h=10, w=10, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=8),
    dict(n=2, h=9, w=9, groups=1, cin=64, cout=128, k=3, stride=2, pad=1, bits=6),
    dict(n=2, h=8, w=8, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=8, residual="identity"),
    dict(n=2, h=9, w=9, groups=1, cin=64, cout=64, k=3, stride=2, pad=1, bits=8, residual="projection"),
    dict(n=2, h=7, w=6, groups=2, cin=20, cout=24, k=3, stride=1, pad=1, bits=8),  # direct path
    dict(n=2, h=7, w=7, groups=2, cin=64, cout=64, k=3, stride=1, pad=1, bits=6, residual="identity"),
]


@pytest.mark.parametrize("i", range(len(CONV_CASES)))
@pytest.mark.parametrize("shuffle", [0, 1, -1, 7])
def test_conv_cases(ctx, torch, i, shuffle):
    p = dict(CONV_CASES[i])
    say(f"conv case {i} {p} shuffle={shuffle}")
    case = I.single_layer(1000 + i, shuffle=shuffle, **p)
    check_conv(ctx, torch, case, centred=(shuffle == 1))


@pytest.mark.parametrize("i", range(len(CONV_CASES)))
@pytest.mark.parametrize("layout", [(1, 1, 1), (0, 1, 0), (1, 0, 1)])
def test_conv_cases_group_layout(ctx, torch, i, layout):
    """Every conv case with its tensors in the group layout (and mixed)."""
    p = dict(CONV_CASES[i])
    say(f"conv case {i} {p} layouts={layout}")
    case = I.single_layer(1000 + i, shuffle=1, **p)
    check_conv(ctx, torch, case, centred=True, layout=layout)


@pytest.mark.parametrize("i", [0, 1, 2, 3, 5, 9, 10])
def test_conv_cases_int8_matrix_cores(ctx, torch, i):
    """The 2-bit cases (and the 3-bit one) with the FP4 / FP6 matrix cores
    switched off (int8 only)."""
    p = dict(CONV_CASES[i])
    say(f"conv case {i} {p} int8 only")
    case = I.single_layer(1000 + i, shuffle=1, **p)
    ctx.set_conv_fp4(False)
    try:
        check_conv(ctx, torch, case, centred=True)
    finally:
        ctx.set_conv_fp4(True)


def test_conv_stem_shape(ctx, torch):
    """8-bit signed input, 3 channels, 7x7/s2/p3 (the network's first layer)."""
    say("conv stem 8-bit 7x7/s2")
    g = I.rng(77)
    x = I.codes(g, (2, 23, 21, 3), 8, True)
    L = I.conv_layer_spec(g, src=0, dst=1, groups=1, cin=3, cout=64, k=7, stride=2, pad=3,
                          in_bits=8, in_signed=True, w_bits=8, out_bits=2)
    check_conv(ctx, torch, dict(x=x, extra={}, layer=L), centred=True)


def test_conv_empty_batch(ctx, torch):
    say("conv n=0")
    case = I.single_layer(5, n=0, h=8, w=8, groups=2, cin=64, cout=64)
    q, acc, rq, racc = run_conv(ctx, torch, case)
    assert q.size == 0 and racc.size == 0


def _residual_args(ctx, case):
    """The layer's shortcut as palq keyword arguments (identity codes with
    their multipliers, or the projection input and filter), {} if none."""
    L = case["layer"]
    G = L["w"].shape[0]
    i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
    if L["res"] >= 0:
        return dict(identity=ctx.pack(case["extra"][1], G, L["out_bits"]), res_mult=i32(L["res_mult"]))
    if L["proj_src"] >= 0:
        pt, pw = ctx.pack_filter(L["proj_w"], L["w_bits"])
        return dict(proj_in=ctx.pack(case["extra"][1], G, L["in_bits"]), proj_w=pw,
                    proj_stride=L["proj_stride"], _keep=pt)
    return {}


def run_conv_full(ctx, torch, case, bias):
    """GPU only (no oracle), the layer with its shortcut: codes of the whole
    batch from palq_group_conv, then from a plan of the layer (the launch
    networks and the benchmark use) without and with the accumulator dump
    (the same kernel family with its dump build).  Returns (group_conv
    codes, plan codes, plan dump-build codes, dumped accumulators)."""
    from paper_2208_01944_amd import palq
    L = case["layer"]
    x = case["x"]
    G, co, kh, kw, ci = L["w"].shape
    xt = ctx.pack(x, G, L["in_bits"])
    wt, wf = ctx.pack_filter(L["w"], L["w_bits"])
    n, h, w, _ = x.shape
    ho = (h + 2 * L["pad"] - kh) // L["stride"] + 1
    wo = (w + 2 * L["pad"] - kw) // L["stride"] + 1
    out = ctx.empty_act(n, ho, wo, G, co, L["out_bits"])
    dump = torch.zeros(n * ho * wo * G * co, dtype=torch.int32, device=ctx.dev)
    i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
    res = _residual_args(ctx, case)
    keep = res.pop("_keep", None)
    args = (xt, wf, L["stride"], L["pad"], i32(L["mult"]), i32(L["shift"]), i32(bias), out)
    ctx.group_conv(*args, shuffle=L["shuffle"], **res)
    ctx.sync()
    q_direct = ctx.unpack(out)
    plan = palq.ConvPlan(ctx, *args, shuffle=L["shuffle"], **res)
    res_in = res.get("identity", res.get("proj_in"))
    out.buf.fill_(0)
    plan.run(xt, out, res_in)
    ctx.sync()
    q_plain = ctx.unpack(out)
    dump.fill_(-1)
    plan.run(xt, out, res_in, acc_dump=dump)
    ctx.sync()
    del keep
    acc = dump.cpu().numpy().astype(np.int64).reshape(n, ho, wo, G * co)
    return q_direct, q_plain, ctx.unpack(out), acc


def oracle_full(case):
    """The oracle on the whole batch, accumulator once: (acc_d, stated codes,
    centred bias, centred codes), shortcut included (acc_d holds a fused
    projection's accumulator, not an identity shortcut).  The centred bias
    (reading A14) is the oracle's centring over the positions whose window
    lies inside the image (stride-1 layers): border pixels, with fewer taps,
    then saturate while the interior spreads over every code (centring over
    all positions leaves 7x7 and 14x14 maps with almost no middle codes)."""
    L = case["layer"]
    G = L["w"].shape[0]
    acc = O.group_conv(case["x"], L["w"], L["stride"], L["pad"])
    res = case["extra"].get(1) if L["res"] >= 0 else None
    px = case["extra"].get(1) if L["proj_src"] >= 0 else None
    sc = dict(res=res, res_mult=L["res_mult"] if res is not None else None, proj_x=px,
              proj_w=L["proj_w"] if px is not None else None, proj_stride=L["proj_stride"])
    q_stated, acc_d = O.layer_epilogue(acc, G, L["mult"], L["shift"], L["bias"], L["out_bits"], L["shuffle"], **sc)
    p = L["pad"] if L["stride"] == 1 else 0
    crop = lambda a: a[:, p:a.shape[1] - p, p:a.shape[2] - p] if a is not None else None
    bias_c = O.centring_bias(crop(acc_d), G, L["shuffle"], res=crop(res), res_mult=sc["res_mult"])
    q_centred, _ = O.layer_epilogue(acc, G, L["mult"], L["shift"], bias_c, L["out_bits"], L["shuffle"], **sc)
    return acc_d, q_stated, bias_c, q_centred


def check_full(ctx, torch, case, fp4_modes=(True, False), all_codes=True):
    """Every image of a full-size single-layer case, stated and centred, in
    the launch the benchmark uses (FP4 matrix cores for 2-bit layers) and
    with int8 matrix cores only: accumulators (from the dump build of the
    same kernel) and codes of both builds bit-exact; every output code
    occurs in the centred codes (all_codes; else at least half of them, for
    the wide codes of the dense baselines, whose upper tail is thin)."""
    L = case["layer"]
    acc_d, q_stated, bias_c, q_centred = oracle_full(case)
    hist = np.bincount(q_centred.reshape(-1), minlength=1 << L["out_bits"])
    if all_codes:
        assert np.all(hist >= 0.01 * q_centred.size / len(hist)), hist  # every output code occurs
    else:
        assert np.count_nonzero(hist) >= len(hist) // 2, hist
    for fp4 in fp4_modes:
        ctx.set_conv_fp4(fp4)
        try:
            for name, bias, want in (("centred", bias_c, q_centred), ("stated", L["bias"], q_stated)):
                say(f"  fp4={fp4} {name}")
                q_direct, q_plain, q_dump, acc = run_conv_full(ctx, torch, case, bias)
                np.testing.assert_array_equal(acc, acc_d, err_msg=f"acc fp4={fp4} {name}")
                np.testing.assert_array_equal(q_dump, want, err_msg=f"codes (dump build) fp4={fp4} {name}")
                np.testing.assert_array_equal(q_plain, want, err_msg=f"codes fp4={fp4} {name}")
                np.testing.assert_array_equal(q_direct, want, err_msg=f"codes (palq_group_conv) fp4={fp4} {name}")
        finally:
            ctx.set_conv_fp4(True)


@pytest.mark.parametrize("layer", range(4))
def test_conv_c2_full_batch_every_image(ctx, torch, layer):
    """Each ResNet-18 stage shape at G=4, batch 32: every image, every
    output code and accumulator."""
    say(f"conv C2 layer {layer} batch 32 (every image)")
    check_full(ctx, torch, I.config_c2(layer))


@pytest.mark.parametrize("groups", [1, 2, 4])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_conv_c4_sweep_every_image(ctx, torch, groups, bits):
    """The G x B sweep on the 14x14 / 256-channel layer at batch 128: every
    image, on the FP4 (2-bit) and FP6 (3-bit) matrix cores and on int8
    (4-bit layers have only the int8 path)."""
    say(f"conv C4 G={groups} b={bits} batch 128 (every image)")
    check_full(ctx, torch, I.config_c4(groups, bits), (True, False) if bits in (2, 3) else (True,))


@pytest.mark.parametrize("pb4", [False, True])
def test_conv_tile_chunked_xcd_order_centred(ctx, torch, pb4):
    """Small centred cases that reach the tiled kernel's chunked tile order
    (the packed input outweighs the filter by 7x, so 32 pixel chunks) and,
    with pb4, its 2 x 4 accumulator blocks (256-pixel tiles on 128-channel
    layers, chosen when they do not lengthen the busiest CU's share)."""
    if pb4:
        # M = 16384 pixels per group: 64 tiles of 256 pixels x 4 groups = 256 (one per CU)
        case = I.single_layer(2201, n=16, h=32, w=32, groups=4, cin=128, cout=128, shuffle=1)
    else:
        case = I.single_layer(2202, n=8, h=28, w=28, groups=4, cin=64, cout=64, shuffle=3)
    say(f"conv tiled chunk order pb4={pb4} {case['x'].shape}")
    check_full(ctx, torch, case)


FP6_CASES = {
    # 64-channel build in the chunked tile order (the packed input outweighs the filter 7x)
    "c64_chunked": dict(n=8, h=28, w=28, groups=4, cin=64, cout=64, shuffle=3),
    # 128-channel build, ragged last tile, 128-channel input (two K-blocks per tap)
    "c128_ragged": dict(n=3, h=11, w=13, groups=2, cin=128, cout=128, shuffle=1),
    # strided 1x1 layer, three groups
    "c64_1x1_s2": dict(n=4, h=16, w=16, groups=3, cin=64, cout=192, k=1, stride=2, pad=0, shuffle=-1),
}


@pytest.mark.parametrize("name", sorted(FP6_CASES))
def test_conv_fp6_builds(ctx, torch, name):
    """3-bit layers on the FP6 (E2M3) matrix cores: the layer's plan names
    conv_fp6_kernel (conv_grouped_kernel with the low-precision formats
    switched off), and every image's accumulators (dump build) and codes,
    stated and centred, equal the oracle's on both paths."""
    from paper_2208_01944_amd import palq
    case = I.single_layer(2300 + sorted(FP6_CASES).index(name), bits=3, **FP6_CASES[name])
    L = case["layer"]
    say(f"conv FP6 {name} {case['x'].shape}")
    for fp, want in ((True, "conv_fp6_kernel"), (False, "conv_grouped_kernel")):
        ctx.set_conv_fp4(fp)
        try:
            t = _layer_tensors(ctx, case, L["bias"])
            plan = palq.ConvPlan(ctx, t["x"], t["w"], L["stride"], L["pad"], t["mult"], t["shift"], t["bias"],
                                 t["out"], shuffle=L["shuffle"])
            assert plan.kernels == want, plan.kernels
        finally:
            ctx.set_conv_fp4(True)
    check_full(ctx, torch, case)


BD_DEFAULT = dict(shuffle=0)
BD_CASES = {
    # 128-channel tiles, ragged last tile
    "c128": dict(n=2, h=13, w=11, groups=1, cin=64, cout=128),
    # 64-channel tiles, two groups, 128 input channels (two K-blocks per tap), shuffled
    "c64_g2": dict(n=2, h=9, w=9, groups=2, cin=128, cout=64, shuffle=1),
    "stride2": dict(n=3, h=15, w=15, groups=1, cin=64, cout=128, stride=2),
    "identity": dict(n=2, h=10, w=10, groups=1, cin=64, cout=64, residual="identity"),
    "projection": dict(n=2, h=11, w=11, groups=1, cin=64, cout=128, stride=2, residual="projection"),
}


@pytest.mark.parametrize("bits", [4, 6, 8])
@pytest.mark.parametrize("name", sorted(BD_CASES))
def test_conv_bitdecomp(ctx, torch, name, bits):
    """M-bit layers run as the Eq. 4 bit decomposition (palq_set_conv_bitdecomp):
    (M/2)^2 2-bit chunk products per MAC on FP4 matrix cores with 4^(i+j)
    block scales.  The plan names conv_bitdecomp_kernel, and every image's
    accumulators (dump build) and codes, stated and centred, equal the
    oracle's direct M-bit result."""
    from paper_2208_01944_amd import palq
    p = dict(BD_DEFAULT, **BD_CASES[name])
    case = I.single_layer(2400 + 10 * bits + sorted(BD_CASES).index(name), bits=bits, **p)
    L = case["layer"]
    say(f"conv Eq. 4 {name} M={bits} {case['x'].shape}")
    ctx.set_conv_bitdecomp(True)
    try:
        t = _layer_tensors(ctx, case, L["bias"])
        plan = palq.ConvPlan(ctx, t["x"], t["w"], L["stride"], L["pad"], t["mult"], t["shift"], t["bias"],
                             t["out"], shuffle=L["shuffle"], **t["kw"])
        assert plan.kernels == "conv_bitdecomp_kernel", plan.kernels
        del plan
        check_full(ctx, torch, case, (True,), all_codes=False)
    finally:
        ctx.set_conv_bitdecomp(False)


FEW_TILE_CASES = {
    # 27 K-blocks (3 per tap), 16 tiles
    "odd_kblocks": dict(n=2, h=14, w=14, groups=4, cin=192, cout=128, shuffle=1),
    "identity": dict(n=2, h=14, w=14, groups=4, cin=128, cout=128, shuffle=1, residual="identity"),
    "projection": dict(n=2, h=15, w=15, groups=4, cin=128, cout=128, stride=2, shuffle=3, residual="projection"),
}


@pytest.mark.parametrize("name", sorted(FEW_TILE_CASES))
def test_conv_fp4_c128_few_tiles(ctx, torch, name):
    """128-channel FP4 layers with few tiles and long K-loops (an odd
    K-block count, identity and projection shortcuts): every image's
    accumulators (dump build) and codes, stated and centred, equal the
    oracle's, also on int8 matrix cores."""
    case = I.single_layer(2500 + sorted(FEW_TILE_CASES).index(name), **FEW_TILE_CASES[name])
    say(f"conv FP4 few tiles {name} {case['x'].shape}")
    check_full(ctx, torch, case)


SHORT_K_CASES = {
    # 1 x 1 layers with one or two K-blocks (the bottleneck 1 x 1 convs of
    # ResNet-50's first two stages): 64-channel tiles, 128-channel tiles with
    # an identity shortcut, and a projection that adds its own K-block
    "c64_kb1": dict(n=2, h=13, w=14, groups=2, cin=64, cout=64, k=1, pad=0, shuffle=1),
    "c256_kb1_identity": dict(n=2, h=14, w=14, groups=2, cin=64, cout=256, k=1, pad=0, shuffle=0,
                              residual="identity"),
    "c256_kb2_projection": dict(n=2, h=14, w=14, groups=2, cin=64, cout=256, k=1, pad=0, shuffle=0,
                                residual="projection"),
    "c512_kb2_identity": dict(n=2, h=7, w=9, groups=2, cin=128, cout=512, k=1, pad=0, shuffle=1,
                              residual="identity", shift=18),  # one below the A13 shift: every code occurs
    "c128_kb3_s2": dict(n=3, h=15, w=15, groups=3, cin=192, cout=128, k=1, stride=2, pad=0, shuffle=-1),
}


@pytest.mark.parametrize("name", sorted(SHORT_K_CASES))
def test_conv_fp4_short_k(ctx, torch, name):
    """2-bit layers with fewer K-blocks than the ring has stages run on the
    FP4 kernel (the plan names conv_fp4_kernel, conv_grouped_kernel with
    FP4 switched off); every image's accumulators (dump build) and codes,
    stated and centred, equal the oracle's on both paths."""
    from paper_2208_01944_amd import palq
    case = I.single_layer(2700 + sorted(SHORT_K_CASES).index(name), **SHORT_K_CASES[name])
    L = case["layer"]
    say(f"conv FP4 short K {name} {case['x'].shape}")
    for fp, want in ((True, "conv_fp4_kernel"), (False, "conv_grouped_kernel")):
        ctx.set_conv_fp4(fp)
        try:
            t = _layer_tensors(ctx, case, L["bias"])
            plan = palq.ConvPlan(ctx, t["x"], t["w"], L["stride"], L["pad"], t["mult"], t["shift"], t["bias"],
                                 t["out"], shuffle=L["shuffle"], **t["kw"])
            assert plan.kernels == want, plan.kernels
        finally:
            ctx.set_conv_fp4(True)
    check_full(ctx, torch, case)


@pytest.mark.parametrize("kind", ["shift23", "big_bias"])
def test_conv_fp4_requant_outside_fp32_bounds(ctx, torch, kind):
    """FP4 layers whose requant leaves the fp32 epilogue's bounds (a shift
    of 23; biases of magnitude 2^24 on some channels, with an identity
    shortcut) run the fp64 epilogue of the same kernel in a plan: every
    image's codes and accumulators, stated and centred, equal the oracle's."""
    if kind == "shift23":
        case = I.single_layer(2800, n=2, h=14, w=14, groups=4, cin=64, cout=64, shuffle=1, shift=23)
    else:
        case = I.single_layer(2801, n=2, h=14, w=14, groups=2, cin=128, cout=128, shuffle=1, residual="identity")
        b = np.array(case["layer"]["bias"], np.int64)
        b[::7] = 1 << 24
        b[3::7] = -(1 << 24)
        case["layer"]["bias"] = b.astype(np.int32)
    say(f"conv FP4 requant outside the fp32 bounds: {kind}")
    check_full(ctx, torch, case, fp4_modes=(True,), all_codes=False)


def test_conv_deterministic(ctx, torch):
    say("conv determinism")
    case = I.config_c2(1, n=4)
    a = run_conv_full(ctx, torch, case, case["layer"]["bias"])
    b = run_conv_full(ctx, torch, case, case["layer"]["bias"])
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


# ---------------------------------------------------------------- shuffle & glue
@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("layout", [(0, 0), (1, 1), (1, 0)])
def test_cyclic_shuffle(ctx, bits, layout):
    say(f"shuffle bits={bits} layouts={layout}")
    g = np.random.default_rng(bits)
    x = I.codes(g, (2, 5, 4, 4 * 40), bits, False).astype(np.int64)
    t = ctx.pack(x, 4, bits, layout=layout[0])
    out = ctx.empty_act(2, 5, 4, 4, 40, bits, layout=layout[1])
    for s in (0, 1, 3, 4, -1, 9):
        ctx.cyclic_shuffle(t, s, out)
        np.testing.assert_array_equal(ctx.unpack(out), O.cyclic_permute(x, 4, s))


@pytest.mark.parametrize("bits,cpg", [(2, 48), (2, 21), (3, 48), (4, 48), (4, 7)])
@pytest.mark.parametrize("layout", [(0, 0), (1, 1), (0, 1)])
def test_maxpool_avgsum_fc(ctx, torch, bits, cpg, layout):
    say(f"maxpool/avgsum/fc bits={bits} cpg={cpg} layouts={layout}")
    g = np.random.default_rng(bits)
    x = I.codes(g, (3, 13, 12, 2 * cpg), bits, False).astype(np.int64)
    t = ctx.pack(x, 2, bits, layout=layout[0])
    out = ctx.empty_act(3, 7, 6, 2, cpg, bits, layout=layout[1])
    ctx.maxpool(t, 3, 2, 1, out)
    np.testing.assert_array_equal(ctx.unpack(out), O.maxpool(x, 3, 2, 1))
    got = out.buf.cpu().numpy()[:3 * 7 * 6 * 2 * packref.row_bytes(cpg, bits)]
    ref = packref.pack(O.maxpool(x, 3, 2, 1), 2, bits)
    np.testing.assert_array_equal(got, group_major(ref, 3 * 7 * 6, 2) if layout[1] else ref)  # zero padding
    C = 2 * cpg
    sums = torch.empty(3 * C, dtype=torch.int32, device=ctx.dev)
    ctx.avgsum(t, sums)
    ref_s = O.avgsum(x)
    np.testing.assert_array_equal(sums.cpu().numpy().reshape(3, C), ref_s)
    w = I.codes(g, (10, C), 8, True)
    logits = torch.empty(30, dtype=torch.int32, device=ctx.dev)
    ctx.fc(sums, 3, C, ctx.upload(w), 10, logits)
    ctx.sync()
    np.testing.assert_array_equal(logits.cpu().numpy().reshape(3, 10), O.fc(ref_s, w))


@pytest.mark.parametrize("cpg,h,w", [(64, 9, 9), (16, 5, 17), (128, 7, 7), (64, 12, 11), (48, 7, 7), (512, 3, 5), (2048, 2, 2), (4096, 1, 3)])
@pytest.mark.parametrize("layout", [0, 1])
def test_maxpool_avgsum_2bit_vector_paths(ctx, torch, cpg, h, w, layout):
    """2-bit rows of a multiple of 16 bytes take the vector max pool; at
    most 85 pixels take the byte-lane global sum (85 x 3 = 255 is the
    largest sum a byte holds; 12 x 11 = 132 pixels takes the other path)."""
    say(f"2-bit maxpool/avgsum cpg={cpg} {h}x{w} layout={layout}")
    g = np.random.default_rng(cpg + h)
    x = I.codes(g, (3, h, w, 2 * cpg), 2, False).astype(np.int64)
    x[1] = 3  # every code at its maximum: sums reach 3 * h * w
    t = ctx.pack(x, 2, 2, layout=layout)
    ho, wo = O.out_size(h, 3, 2, 1), O.out_size(w, 3, 2, 1)
    out = ctx.empty_act(3, ho, wo, 2, cpg, 2, layout=layout)
    ctx.maxpool(t, 3, 2, 1, out)
    np.testing.assert_array_equal(ctx.unpack(out), O.maxpool(x, 3, 2, 1))
    sums = torch.empty(3 * 2 * cpg, dtype=torch.int32, device=ctx.dev)
    ctx.avgsum(t, sums)
    ctx.sync()
    np.testing.assert_array_equal(sums.cpu().numpy().reshape(3, 2 * cpg), O.avgsum(x))


@pytest.mark.parametrize("n,cin,cout", [(37, 96, 70), (3, 40, 5), (64, 2048, 1000)])
def test_fc_full_range_modular(ctx, torch, n, cin, cout):
    """Features over the whole int32 range (the matrix-core path splits them
    into signed byte digits when cin % 32 == 0): logits equal the exact sum
    reduced modulo 2^32."""
    say(f"fc full range {n}x{cin}->{cout}")
    g = np.random.default_rng(cin)
    x = g.integers(-2**31, 2**31, (n, cin), dtype=np.int64)
    x[0, :] = -2**31
    x[-1, :] = 2**31 - 1
    w = I.codes(g, (cout, cin), 8, True)
    logits = torch.empty(n * cout, dtype=torch.int32, device=ctx.dev)
    ctx.fc(ctx.upload(x.astype(np.int32)), n, cin, ctx.upload(w), cout, logits)
    ctx.sync()
    ref = O.fc(x, w)
    ref32 = ((np.asarray(ref, dtype=object) % 2**32).astype(np.int64)).astype(np.uint32).view(np.int32)
    np.testing.assert_array_equal(logits.cpu().numpy().reshape(n, cout), ref32)


def test_fc_large(ctx, torch):
    """The network's FC shape (64 x 2048 -> 1000) with several K slices."""
    say("fc 64x2048->1000")
    g = np.random.default_rng(5)
    x = g.integers(0, 148, (64, 2048)).astype(np.int32)
    w = I.codes(g, (1000, 2048), 8, True)
    logits = torch.empty(64 * 1000, dtype=torch.int32, device=ctx.dev)
    ctx.fc(ctx.upload(x), 64, 2048, ctx.upload(w), 1000, logits)
    ctx.sync()
    np.testing.assert_array_equal(logits.cpu().numpy().reshape(64, 1000), O.fc(x, w))


# ---------------------------------------------------------------- shuffle module
@pytest.mark.parametrize("G,C,bits,n,h,w", [
    (2, 64, 2, 2, 9, 7),      # grouped MFMA kernel
    (4, 128, 2, 2, 6, 5),
    (3, 64, 3, 1, 5, 9),      # 3-bit codes
    (2, 64, 4, 2, 5, 5),      # 4-bit codes
    (4, 32, 2, 2, 4, 4),      # direct kernel (32 channels per group)
    (2, 256, 2, 1, 7, 7),     # long enough K for the tiled kernel
])
def test_shuffle_module_matches_oracle(ctx, torch, G, C, bits, n, h, w):
    say(f"shuffle module G={G} C={C} b={bits} {n}x{h}x{w}")
    g = I.rng(500 + G * 7 + C + bits)
    x = I.codes(g, (n, h, w, G * C), bits, False)
    L = I.shuffle_module_spec(g, src=0, dst=1, groups=G, ch=C, bits=bits)
    # centred bias so that every output code occurs (reading A14)
    _, acc = O.shuffle_module(x, L["w"], L["mult"], L["shift"], None, L["res_mult"], bits)
    t = acc + np.asarray(L["res_mult"], np.int64) * x
    mean = t.reshape(-1, G * C).sum(axis=0) / t.reshape(-1, G * C).shape[0]
    bias = (-np.floor(mean + 0.5)).astype(np.int32)
    ref, _ = O.shuffle_module(x, L["w"], L["mult"], L["shift"], bias, L["res_mult"], bits)
    xt = ctx.pack(x, G, bits)
    wt, wf = ctx.pack_filter(L["w"], bits)
    out = ctx.empty_act(n, h, w, G, C, bits)
    i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
    ctx.shuffle_module(xt, wf, i32(L["mult"]), i32(L["shift"]), i32(bias), i32(L["res_mult"]), out)
    ctx.sync()
    got = ctx.unpack(out)
    np.testing.assert_array_equal(got, ref)
    hist = np.bincount(ref.reshape(-1), minlength=1 << bits)
    assert np.count_nonzero(hist) >= 2, hist


# (bits, G, C, image shape): the word-level build takes b in {2, 4, 8}, G in
# {2, 4, 8, 16}, unpadded rows and whole 16-byte stores per pixel; the rest
# (3-bit, G = 3, padded rows, a pixel that is not whole stores) takes the
# per-chunk build.  The 28 x 28 case spans many workgroups with a ragged tail.
CHANNEL_SHUFFLE_CASES = [
    (2, 4, 64, (2, 5, 3)), (2, 2, 37, (2, 5, 3)), (3, 3, 48, (2, 5, 3)), (4, 4, 128, (2, 5, 3)),
    (8, 2, 40, (2, 5, 3)), (2, 4, 512, (2, 5, 3)), (2, 8, 32, (2, 5, 3)), (2, 16, 16, (2, 5, 3)),
    (2, 2, 16, (2, 5, 3)), (4, 8, 16, (2, 5, 3)), (8, 16, 4, (2, 5, 3)), (4, 2, 24, (2, 5, 3)),
    (2, 8, 8, (2, 5, 3)), (2, 4, 32, (4, 28, 28)), (8, 4, 16, (3, 7, 9)),
]


@pytest.mark.parametrize("bits,G,C,shape", CHANNEL_SHUFFLE_CASES)
@pytest.mark.parametrize("layout", [(0, 0), (1, 1), (1, 0)])
def test_channel_shuffle_matches_oracle(ctx, bits, G, C, shape, layout):
    say(f"channel shuffle b={bits} G={G} C={C} shape={shape} layouts={layout}")
    g = np.random.default_rng(bits * 100 + G * 10 + C)
    x = I.codes(g, shape + (G * C,), bits, False).astype(np.int64)
    xt = ctx.pack(x, G, bits, layout=layout[0])
    out = ctx.empty_act(*shape, G, C, bits, layout=layout[1])
    ctx.channel_shuffle(xt, out)
    ctx.sync()
    np.testing.assert_array_equal(ctx.unpack(out), O.channel_shuffle(x, G))


def test_channel_shuffle_full_size(ctx):
    """The stage-2 channel shuffle of the batch-64 ResNet-18 G = 4 2-bit
    network with shuffles (64 x 56 x 56 pixels, 4 groups of 64 channels),
    every code against the oracle's transposition."""
    say("channel shuffle full size 64x56x56 G=4 C=64 b=2")
    g = np.random.default_rng(2208)
    x = I.codes(g, (64, 56, 56, 256), 2, False)
    xt = ctx.pack(x, 4, 2)
    out = ctx.empty_act(64, 56, 56, 4, 64, 2)
    ctx.channel_shuffle(xt, out)
    ctx.sync()
    np.testing.assert_array_equal(ctx.unpack(out).reshape(x.shape), O.channel_shuffle(x, 4))


@pytest.mark.parametrize("big_bias", [False, True])
def test_conv_filter_longer_than_lds(ctx, torch, big_bias):
    """A 2-bit layer whose filter (K = 9 x 1024) is too long for the general
    build's filter-in-LDS: the tiled kernel takes it; the accumulator dump and
    (big_bias: the int64 requant fallback) go to the direct kernel."""
    say(f"conv K=9x1024 G=1 big_bias={big_bias}")
    case = I.single_layer(77, n=1, h=7, w=7, groups=1, cin=1024, cout=128, shuffle=0)
    if big_bias:
        L = case["layer"]
        L["mult"] = np.full_like(L["mult"], 1 << 23)
        L["shift"] = np.full_like(L["shift"], 40)
        L["bias"] = np.full_like(L["mult"], 1 << 29)
    q, acc, rq, racc = run_conv(ctx, torch, case, centred=not big_bias)
    np.testing.assert_array_equal(acc, racc)
    np.testing.assert_array_equal(q, rq)


@pytest.mark.parametrize("signed", [True, False])
@pytest.mark.parametrize("calibrate", [False, True])
def test_quantize_image_path(ctx, torch, signed, calibrate):
    """The 3-channel 8-bit image input (the four-pixels-per-thread path), with
    NaN/inf and exact ties, fixed and calibrated ranges."""
    say(f"quantize image 8-bit signed={signed} calibrate={calibrate}")
    g = np.random.default_rng(31 + signed)
    x = g.normal(0, 1.2, (2, 9, 14, 3)).astype(np.float32)
    x.flat[::61] = np.nan
    if not calibrate:
        x.flat[5::97] = np.inf
        x.flat[7::113] = -np.inf
    x.flat[1:4] = [-3.0 + 6.0 * 0.5 / 255.0, 0.0, 3.0]
    out = ctx.empty_act(2, 9, 14, 1, 3, 8, signed)
    if calibrate:
        ctx.quantize(ctx.upload(x), float("nan"), float("nan"), out)
        l, u = O.calibrate_range(x)
    else:
        l, u = -3.0, 3.0
        ctx.quantize(ctx.upload(x), l, u, out)
    ctx.sync()
    np.testing.assert_array_equal(ctx.unpack(out), O.quantize(x, l, u, 8, signed))


# ---------------------------------------------------------------- planned layers
def _layer_tensors(ctx, case, bias):
    L = case["layer"]
    G, co, kh, kw, ci = L["w"].shape
    n, h, w, _ = case["x"].shape
    ho = (h + 2 * L["pad"] - kh) // L["stride"] + 1
    wo = (w + 2 * L["pad"] - kw) // L["stride"] + 1
    i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
    t = dict(x=ctx.pack(case["x"], G, L["in_bits"]), out=ctx.empty_act(n, ho, wo, G, co, L["out_bits"]),
             mult=i32(L["mult"]), shift=i32(L["shift"]), bias=i32(bias), shape=(n, ho, wo, G * co))
    t["wt"], t["w"] = ctx.pack_filter(L["w"], L["w_bits"])
    if L["res"] >= 0:
        t["res_in"] = ctx.pack(case["extra"][1], G, L["out_bits"])
        t["kw"] = dict(identity=t["res_in"], res_mult=i32(L["res_mult"]))
    elif L["proj_src"] >= 0:
        t["res_in"] = ctx.pack(case["extra"][1], G, L["in_bits"])
        pt, pw = ctx.pack_filter(L["proj_w"], L["w_bits"])
        t["kw"] = dict(proj_in=t["res_in"], proj_w=pw, proj_stride=L["proj_stride"])
        t["pt"] = pt
    else:
        t["res_in"], t["kw"] = None, {}
    return t


@pytest.mark.parametrize("kind", ["plain", "identity", "projection", "bits3"])
def test_conv_plan_runs(ctx, torch, kind):
    """A planned layer run on two inputs after its parameter arrays are gone,
    with and without the accumulator dump, and captured into a HIP graph
    (capture fails on any allocation or synchronisation) replayed with other
    work between replays: every result equals the oracle's."""
    from paper_2208_01944_amd import palq
    say(f"conv plan {kind}")
    p = dict(n=2, h=14, w=14, groups=4, cin=128, cout=128, shuffle=1)
    if kind == "identity":
        p.update(residual="identity")
    elif kind == "projection":
        p.update(residual="projection", stride=2, h=15, w=15)
    elif kind == "bits3":
        p.update(bits=3, cin=64, cout=64, groups=3)
    cases = [I.single_layer(4100 + s, **p) for s in range(2)]
    for c in cases[1:]:  # the second input shares the first case's filter and parameters
        c["layer"] = cases[0]["layer"]
    L = cases[0]["layer"]
    refs = []
    for c in cases:
        res = c["extra"].get(1) if L["res"] >= 0 else None
        px = c["extra"].get(1) if L["proj_src"] >= 0 else None
        refs.append(O.conv_layer(c["x"], L["w"], L["stride"], L["pad"], L["mult"], L["shift"], L["bias"],
                                 L["out_bits"], L["shuffle"], res=res, res_mult=L["res_mult"], proj_x=px,
                                 proj_w=L["proj_w"], proj_stride=L["proj_stride"]))
    t0 = _layer_tensors(ctx, cases[0], L["bias"])
    plan = palq.ConvPlan(ctx, t0["x"], t0["w"], L["stride"], L["pad"], t0["mult"], t0["shift"], t0["bias"],
                         t0["out"], shuffle=L["shuffle"], **t0["kw"])
    for k in ("mult", "shift", "bias", "wt", "pt"):
        t0.pop(k, None)  # the plan holds its own copies
    torch.cuda.synchronize()
    tens = [t0, _layer_tensors(ctx, cases[1], L["bias"])]
    for t, (rq, racc) in zip(tens, refs):
        dump = torch.full((int(np.prod(t["shape"])),), -7, dtype=torch.int32, device=ctx.dev)
        plan.run(t["x"], t["out"], t["res_in"])
        ctx.sync()
        np.testing.assert_array_equal(ctx.unpack(t["out"]), rq)
        plan.run(t["x"], t["out"], t["res_in"], acc_dump=dump)
        ctx.sync()
        np.testing.assert_array_equal(dump.cpu().numpy().astype(np.int64).reshape(t["shape"]), racc)
        np.testing.assert_array_equal(ctx.unpack(t["out"]), rq)
    # graph capture and replays of the second input's run
    t = tens[1]
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        ctx.set_stream(side)
        graph.capture_begin()
        plan.run(t["x"], t["out"], t["res_in"])
        graph.capture_end()
    ctx.set_stream(torch.cuda.current_stream())
    for r in range(3):
        t["out"].buf.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(ctx.unpack(t["out"]), refs[1][0], err_msg=f"replay {r}")
        plan.run(tens[0]["x"], tens[0]["out"], tens[0]["res_in"])  # other work between replays
        ctx.sync()


def test_set_stream_orders_context_scratch(ctx, torch):
    """Two group_conv calls with different filters on two streams: the
    second call's prepack reuses the context's scratch, so the new stream
    must wait for the first call (palq_set_stream orders them)."""
    say("set_stream ordering")
    cases = [I.single_layer(4200 + s, n=16, h=28, w=28, groups=4, cin=128, cout=128, shuffle=1) for s in range(2)]
    refs = [O.conv_layer(c["x"], c["layer"]["w"], 1, 1, c["layer"]["mult"], c["layer"]["shift"], c["layer"]["bias"],
                         2, 1)[0] for c in cases]
    tens = [_layer_tensors(ctx, c, c["layer"]["bias"]) for c in cases]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for rep in range(3):
        for t, s in zip(tens, streams):
            ctx.set_stream(s)
            ctx.group_conv(t["x"], t["w"], 1, 1, t["mult"], t["shift"], t["bias"], t["out"], shuffle=1)
        ctx.set_stream(torch.cuda.current_stream())
        torch.cuda.synchronize()
        for t, r in zip(tens, refs):
            np.testing.assert_array_equal(ctx.unpack(t["out"]), r, err_msg=f"round {rep}")
