"""GPU parity of palq_forward (whole networks) against the CPU oracle."""
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2208_01944_amd import inputs as I

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


def gpu_forward(ctx, torch, spec, keep=False):
    from paper_2208_01944_amd import palq
    net = palq.Net(ctx, spec, flags=palq.NET_KEEP_ALL if keep else 0)
    x = spec["x"]
    xt = ctx.pack(x, 1, 8, signed=True)
    logits = torch.empty(x.shape[0] * net.classes, dtype=torch.int32, device=ctx.dev)
    net.forward(xt.buf, logits)
    ctx.sync()
    return net, logits.cpu().numpy().astype(np.int64).reshape(x.shape[0], net.classes)


def compare_tensors(ctx, net, spec, tensors, images):
    for L in spec["layers"]:
        d = L["dst"]
        if L["op"] in ("conv", "maxpool", "shuffle_module", "channel_shuffle"):
            got = ctx.unpack(net.tensor(d))[images]
            np.testing.assert_array_equal(got, tensors[d], err_msg=f"tensor {d} ({L['op']})")


@pytest.mark.parametrize("variant", ["stated", "centred"])
def test_resnet18_small_all_tensors(ctx, torch, variant):
    say(f"resnet18 hw=64 n=2 G=4 b=2 {variant}")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=11)
    if variant == "centred":
        spec = O.calibrate_centring(spec, spec["x"])
    net, logits = gpu_forward(ctx, torch, spec, keep=True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


def test_resnet18_group_layout_matches_pixel_layout(ctx, torch):
    """The network stores a conv output of several groups that every reader
    takes with those groups in the group layout (default); with
    PALQ_NET_PIXEL_LAYOUT it keeps the pixel layout.  Both give the oracle's
    tensors and logits."""
    from paper_2208_01944_amd import palq
    say("resnet18 hw=64 n=2 G=4 b=2 centred, group vs pixel layout")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=12)
    spec = O.calibrate_centring(spec, spec["x"])
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    xt = ctx.pack(spec["x"], 1, 8, signed=True)
    for flags, want in ((palq.NET_KEEP_ALL, palq.LAYOUT_GROUP),
                        (palq.NET_KEEP_ALL | palq.NET_PIXEL_LAYOUT, palq.LAYOUT_PIXEL)):
        net = palq.Net(ctx, spec, flags=flags)
        logits = torch.empty(2 * net.classes, dtype=torch.int32, device=ctx.dev)
        net.forward(xt.buf, logits)
        ctx.sync()
        for L in spec["layers"]:
            if L["op"] == "conv" and L["w"].shape[0] > 1:
                assert net.tensor(L["dst"]).act.layout == want, (flags, L["dst"])
        compare_tensors(ctx, net, spec, tensors, slice(None))
        np.testing.assert_array_equal(logits.cpu().numpy().astype(np.int64).reshape(2, -1), ref)


def test_forward_refuses_buffers_smaller_than_the_batch(ctx, torch):
    """The binding checks the input and logits tensors against the network's
    batch before the C call (which takes plain pointers): a short buffer
    raises, nothing is launched."""
    from paper_2208_01944_amd import palq
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=13)
    net = palq.Net(ctx, spec)
    x = torch.zeros(2 * 64 * 64 * 3, dtype=torch.float32, device=ctx.dev)
    logits = torch.empty(2 * net.classes, dtype=torch.int32, device=ctx.dev)
    with pytest.raises(palq.PalqError):
        net.forward_image(x[: 64 * 64 * 3], -1.0, 1.0, logits)
    with pytest.raises(palq.PalqError):
        net.forward_image(x, -1.0, 1.0, logits[: net.classes])
    xt = ctx.pack(spec["x"], 1, 8, signed=True)
    with pytest.raises(palq.PalqError):
        net.forward(xt.buf[: xt.buf.numel() // 2], logits)
    net.forward_image(x, -1.0, 1.0, logits)
    ctx.sync()


def test_resnet18_small_int8_matrix_cores(ctx, torch):
    say("resnet18 hw=64 n=2 G=4 b=2 centred, int8 only")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=14)
    spec = O.calibrate_centring(spec, spec["x"])
    ctx.set_conv_fp4(False)
    try:
        net, logits = gpu_forward(ctx, torch, spec, keep=True)
    finally:
        ctx.set_conv_fp4(True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


@pytest.mark.parametrize("fp4", [True, False])
def test_resnet18_with_shuffle_modules_all_tensors(ctx, torch, fp4):
    say(f"resnet18 + cyclic shuffle modules hw=64 n=2 G=4 b=2 centred fp4={fp4}")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=15, modules=True)
    assert sum(L["op"] == "shuffle_module" for L in spec["layers"]) == 3
    spec = O.calibrate_centring(spec, spec["x"])
    ctx.set_conv_fp4(fp4)
    try:
        net, logits = gpu_forward(ctx, torch, spec, keep=True)
    finally:
        ctx.set_conv_fp4(True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


def test_resnet18_with_modules_and_channel_shuffle(ctx, torch):
    say("resnet18 + cyclic shuffle modules + per-stage channel shuffle hw=64 n=2 G=4 b=2 centred")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=16, modules=True,
                      channel_shuffle=True)
    assert sum(L["op"] == "channel_shuffle" for L in spec["layers"]) == 3
    spec = O.calibrate_centring(spec, spec["x"])
    net, logits = gpu_forward(ctx, torch, spec, keep=True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


def stem_pool_spec(n, hw, groups, seed):
    """The stem (7x7/s2 8-bit conv to 64 G channels, 2-bit output) and its
    3x3/s2 max pool, then the global sum and a small FC."""
    g = I.rng(seed)
    x = I.codes(g, (n, hw, hw, 3), 8, True)
    layers = []
    cur, nid = I._stem(g, layers, groups, 2)
    layers.append(dict(op="avgsum", src=cur, dst=nid))
    layers.append(dict(op="fc", src=nid, dst=nid + 1, w=I.codes(g, (10, 64 * groups), 8, True)))
    return dict(name="stem_pool", n=n, hw=hw, groups=groups, bits=2, x=x, layers=layers, classes=10)


@pytest.mark.parametrize("n,hw,groups", [(3, 64, 4), (2, 50, 2), (1, 250, 4), (2, 33, 8), (1, 9, 2)])
def test_stem_with_max_pool(ctx, torch, n, hw, groups):
    """Without NET_KEEP_ALL the stem and its max pool run as one launch that
    pools the accumulators; the pooled tensor (its buffer is not reused by the
    sum or the FC) and the logits must match the oracle's.  Sizes cover even
    and odd conv outputs (25, 125, 17, 3 rows), up to 125 columns, and 128-,
    256- and 512-channel stems."""
    say(f"stem + max pool n={n} hw={hw} G={groups}")
    spec = stem_pool_spec(n, hw, groups, seed=40 + hw)
    spec = O.calibrate_centring(spec, spec["x"])
    net, logits = gpu_forward(ctx, torch, spec)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    got = ctx.unpack(net.tensor(2))
    np.testing.assert_array_equal(got, tensors[2])
    np.testing.assert_array_equal(logits, ref)
    assert len(np.unique(tensors[2])) == 4  # every code occurs


@pytest.mark.parametrize("stem_pad,hw", [(3, 64), (0, 64), (3, 50)])
def test_forward_image_matches_quantize_then_forward(ctx, torch, stem_pad, hw):
    """palq_forward_image (quantise into the stem's zero-border copy, or, for
    a stem without padding, into a buffer of its own) gives the logits of
    palq_quantize + palq_forward and of the oracle, on fp32 images with
    NaN, infinities and values outside [l, u]."""
    from paper_2208_01944_amd import palq
    say(f"forward_image stem pad={stem_pad} hw={hw}")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=hw, classes=100, seed=17)
    if stem_pad == 0:
        st = dict(spec["layers"][0])
        st["pad"] = 0
        spec["layers"][0] = st
    g = np.random.default_rng(70 + stem_pad)
    x = g.normal(0, 1.3, (2, hw, hw, 3)).astype(np.float32)
    x.flat[::97] = np.nan
    x.flat[3::89] = np.inf
    x.flat[5::101] = -np.inf
    l, u = -3.0, 3.0
    codes = O.quantize(x, l, u, 8, True)
    spec = O.calibrate_centring(spec, codes)
    ref = O.run_net(spec, codes)
    net = palq.Net(ctx, spec)
    xd = ctx.upload(x)
    out1 = torch.empty(2 * 100, dtype=torch.int32, device=ctx.dev)
    out2 = torch.empty_like(out1)
    net.forward_image(xd, l, u, out1)
    xt = ctx.empty_act(2, hw, hw, 1, 3, 8, True)
    ctx.quantize(xd, l, u, xt)
    net.forward(xt.buf, out2)
    net.forward_image(xd, l, u, out1)  # again, after the other path used the buffers
    ctx.sync()
    a = out1.cpu().numpy().astype(np.int64).reshape(2, 100)
    b = out2.cpu().numpy().astype(np.int64).reshape(2, 100)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(a, ref)


def test_graph_replay_matches_eager(ctx, torch):
    """PALQ_NET_GRAPH: replays of the captured forward (same input buffer,
    its contents changed between calls, eager work and synchronisations in
    between) give the eager network's logits every time; a new input pointer
    or the image entry point captures again."""
    from paper_2208_01944_amd import palq
    say("graph replay resnet18 hw=64 n=2")
    spec = I.resnet18(n=2, groups=4, bits=2, hw=64, classes=100, seed=18)
    spec = O.calibrate_centring(spec, spec["x"])
    g = np.random.default_rng(81)
    x2 = I.codes(g, spec["x"].shape, 8, True)
    net_e = palq.Net(ctx, spec)
    net_g = palq.Net(ctx, spec, flags=palq.NET_GRAPH)
    xa, xb = ctx.pack(spec["x"], 1, 8, signed=True), ctx.pack(x2, 1, 8, signed=True)
    buf = ctx.pack(spec["x"], 1, 8, signed=True)
    ref = {}
    for name, xt in (("a", xa), ("b", xb)):
        out = torch.empty(200, dtype=torch.int32, device=ctx.dev)
        net_e.forward(xt.buf, out)
        ctx.sync()
        ref[name] = out.cpu().numpy().astype(np.int64).reshape(2, 100)
    np.testing.assert_array_equal(ref["a"], O.run_net(spec, spec["x"]))
    out = torch.empty(200, dtype=torch.int32, device=ctx.dev)
    scratch = torch.empty(200, dtype=torch.int32, device=ctx.dev)
    for it in range(6):
        name = "ab"[it % 2]
        buf.buf.copy_((xa if name == "a" else xb).buf)
        net_g.forward(buf.buf, out)        # it 0 eager, 1 capture, then replays
        net_e.forward(xb.buf, scratch)     # eager work on the same stream
        ctx.sync()
        np.testing.assert_array_equal(out.cpu().numpy().astype(np.int64).reshape(2, 100), ref[name],
                                      err_msg=f"call {it}")
    net_g.forward(xb.buf, out)             # another input pointer: captured again
    ctx.sync()
    np.testing.assert_array_equal(out.cpu().numpy().astype(np.int64).reshape(2, 100), ref["b"])
    # the image entry point through the graph, twice
    xf = g.normal(0, 1.3, (2, 64, 64, 3)).astype(np.float32)
    xd = ctx.upload(xf)
    codes = ctx.empty_act(2, 64, 64, 1, 3, 8, True)
    ctx.quantize(xd, -3.0, 3.0, codes)
    net_e.forward(codes.buf, scratch)
    ctx.sync()
    want = scratch.cpu().numpy().copy()
    for _ in range(2):
        net_g.forward_image(xd, -3.0, 3.0, out)
        ctx.sync()
        np.testing.assert_array_equal(out.cpu().numpy(), want)


def test_resnet50_small_all_tensors(ctx, torch):
    say("resnet50 hw=64 n=2 G=2 b=2 centred")
    spec = I.resnet50(n=2, groups=2, bits=2, hw=64, classes=50, seed=12)
    spec = O.calibrate_centring(spec, spec["x"])
    net, logits = gpu_forward(ctx, torch, spec, keep=True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


@pytest.mark.parametrize("bits", [6, 8])
def test_resnet18_dense_wide_codes(ctx, torch, bits):
    """The dense (G = 1) M-bit network of the Table 2 baselines at M = 6 and
    8: unsigned codes of M bits throughout (8-bit projections included),
    every tensor and the logits equal the oracle's."""
    say(f"resnet18 hw=32 n=2 G=1 b={bits} centred")
    spec = I.resnet18(n=2, groups=1, bits=bits, hw=32, classes=10, seed=15 + bits)
    spec = O.calibrate_centring(spec, spec["x"])
    net, logits = gpu_forward(ctx, torch, spec, keep=True)
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_resnet18_dense_bitdecomp(ctx, torch, bits):
    """The dense M-bit network run with every grouped layer as the Eq. 4 bit
    decomposition on FP4 matrix cores: each of those layers launches
    conv_bitdecomp_kernel, and every tensor and the logits equal the
    oracle's (which computes the M-bit products directly)."""
    say(f"resnet18 hw=32 n=2 G=1 b={bits} Eq. 4")
    spec = I.resnet18(n=2, groups=1, bits=bits, hw=32, classes=10, seed=25 + bits)
    spec = O.calibrate_centring(spec, spec["x"])
    ctx.set_conv_bitdecomp(True)
    try:
        net, logits = gpu_forward(ctx, torch, spec, keep=True)
    finally:
        ctx.set_conv_bitdecomp(False)
    convs = [i for i, L in enumerate(spec["layers"]) if L["op"] == "conv" and not L["in_signed"]]
    kernels = net.layer_kernels()
    assert all(kernels[i] == "conv_bitdecomp_kernel" for i in convs), kernels
    ref, tensors, _ = O.run_net(spec, spec["x"], keep=True)
    compare_tensors(ctx, net, spec, tensors, slice(None))
    np.testing.assert_array_equal(logits, ref)


def test_resnet18_bits3_g3(ctx, torch):
    say("resnet18 hw=32 n=3 G=3 b=3 centred")
    spec = I.resnet18(n=3, groups=3, bits=3, hw=32, classes=10, seed=13)
    spec = O.calibrate_centring(spec, spec["x"])
    _, logits = gpu_forward(ctx, torch, spec)
    np.testing.assert_array_equal(logits, O.run_net(spec, spec["x"]))


def full_size_run(ctx, torch, name):
    """The benchmark's network (stored centred biases, default flags) on
    the workload's whole fp32 image batch through palq_forward_image, as
    bench.py times it: (centred spec, the batch's 8-bit codes (oracle's
    quantiser), GPU logits, the kernels each layer launched)."""
    from paper_2208_01944_amd import palq
    spec, x, _ = I.workload(name)
    spec = I.with_stored_biases(spec, name)
    l, u = I.IMAGE_RANGE
    net = palq.Net(ctx, spec)
    logits = torch.empty(x.shape[0] * net.classes, dtype=torch.int32, device=ctx.dev)
    net.forward_image(ctx.upload(x), l, u, logits)
    ctx.sync()
    got = logits.cpu().numpy().astype(np.int64).reshape(x.shape[0], net.classes)
    kernels = net.layer_kernels(image=True)
    del net
    return spec, O.quantize(x, l, u, 8, signed=True), got, kernels


@pytest.fixture(scope="module")
def c3_run(ctx, torch):
    say("C3 resnet18 n=64 224x224 G=4 b=2 centred: GPU forward_image of the whole batch")
    return full_size_run(ctx, torch, "resnet18_g4_b2")


@pytest.fixture(scope="module")
def c5_run(ctx, torch):
    say("C5 resnet50 n=128 224x224 G=2 b=2 centred: GPU forward_image of the whole batch")
    return full_size_run(ctx, torch, "resnet50_g2_b2")


def test_c3_launches_the_benchmark_kernels(c3_run):
    """The full-size network runs the kernels the benchmark reports: the
    fused stem + max pool and the 2-bit grouped layers on FP4 matrix cores."""
    kernels = c3_run[3]
    assert kernels[0] == "quantize_pad4_kernel + stem_pool_kernel", kernels[0]
    assert kernels[1] == "", kernels[1]
    assert kernels.count("conv_fp4_kernel") == 16, kernels
    assert kernels[-2:] == ["avgsum2_wg_kernel", "fc_mfma_kernel"], kernels[-2:]


@pytest.mark.parametrize("chunk", range(8))
def test_c3_full_size_every_image(c3_run, chunk):
    """C3 at full size: the logits of every image of the batch (8 per test)
    against the oracle's forward of the same centred network."""
    spec, codes, got, _ = c3_run
    sl = slice(8 * chunk, 8 * chunk + 8)
    say(f"C3 oracle images {sl.start}..{sl.stop - 1}")
    ref = O.run_net(spec, codes[sl])
    np.testing.assert_array_equal(got[sl], ref)
    assert len(np.unique(ref)) > 100  # logits are not degenerate


@pytest.mark.parametrize("chunk", range(16))
def test_c5_full_size_every_image(c5_run, chunk):
    """C5 (ResNet-50, G=2, 2-bit, batch 128) at full size: every image's
    logits (8 per test) against the oracle."""
    spec, codes, got, kernels = c5_run
    if chunk == 0:
        assert kernels.count("conv_fp4_kernel") >= 40, kernels
    sl = slice(8 * chunk, 8 * chunk + 8)
    say(f"C5 oracle images {sl.start}..{sl.stop - 1}")
    ref = O.run_net(spec, codes[sl])
    np.testing.assert_array_equal(got[sl], ref)
    assert len(np.unique(ref)) > 100
