"""GPU checks of palq_group_conv_noalloc (the grouped conv whose prepacked
filter and requant constants live in the library's static per-GPU buffer):
bit-exact against palq_group_conv (and the oracle) on two calls in a row,
the second with a smaller input and another filter, and inside a captured
HIP graph replayed several times."""
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2208_01944_amd import inputs as I

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def centred(case):
    L = case["layer"]
    G = L["w"].shape[0]
    res = case["extra"].get(1) if L["res"] >= 0 else None
    acc = O.group_conv(case["x"], L["w"], L["stride"], L["pad"])
    _, acc_d = O.layer_epilogue(acc, G, L["mult"], L["shift"], None, L["out_bits"], L["shuffle"],
                                res=res, res_mult=L["res_mult"])
    bias = O.centring_bias(acc_d, G, L["shuffle"], res=res, res_mult=L["res_mult"])
    q, _ = O.layer_epilogue(acc, G, L["mult"], L["shift"], bias, L["out_bits"], L["shuffle"],
                            res=res, res_mult=L["res_mult"])
    return bias, q, acc_d


class Layer:
    """Device copies of one single_layer() case for repeated calls."""

    def __init__(self, ctx, torch, case, bias, layout=0):
        L = case["layer"]
        self.ctx, self.case, self.layout = ctx, case, layout
        G, co, kh, kw, ci = L["w"].shape
        n, h, w, _ = case["x"].shape
        self.ho = (h + 2 * L["pad"] - kh) // L["stride"] + 1
        self.wo = (w + 2 * L["pad"] - kw) // L["stride"] + 1
        self.xt = ctx.pack(case["x"], G, L["in_bits"], layout=layout)
        self.wt, self.wf = ctx.pack_filter(L["w"], L["w_bits"])
        i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
        self.rq = (i32(L["mult"]), i32(L["shift"]), i32(bias))
        self.kw = {}
        if L["res"] >= 0:
            self.kw["identity"] = ctx.pack(case["extra"][1], G, L["out_bits"], layout=layout)
            self.kw["res_mult"] = i32(L["res_mult"])
        self.shape = (n, self.ho, self.wo, G * co)
        self.nout = n * self.ho * self.wo * G * co
        self.G, self.co = G, co

    def outputs(self, torch):
        L = self.case["layer"]
        out = self.ctx.empty_act(self.shape[0], self.ho, self.wo, self.G, self.co, L["out_bits"],
                                 layout=self.layout)
        dump = torch.full((self.nout,), -7, dtype=torch.int32, device=self.ctx.dev)
        return out, dump

    def run(self, out, dump, noalloc):
        L = self.case["layer"]
        self.ctx.group_conv(self.xt, self.wf, L["stride"], L["pad"], *self.rq, out, shuffle=L["shuffle"],
                            acc_dump=dump, noalloc=noalloc, **self.kw)

    def read(self, out, dump):
        self.ctx.sync()
        return self.ctx.unpack(out), dump.cpu().numpy().astype(np.int64).reshape(self.shape)


@pytest.mark.parametrize("layout", [0, 1])
def test_noalloc_matches_group_conv_two_calls(layout):
    """Two no-alloc calls in a row, the second with a smaller input (and
    another filter, so the static buffer's previous contents would show):
    codes and accumulators equal palq_group_conv's and the oracle's, with
    the tensors in the pixel (0) and the group (1) layout."""
    import torch
    from paper_2208_01944_amd import palq
    ctx = palq.Context(0)
    cases = [I.single_layer(3101, n=8, h=28, w=28, groups=4, cin=128, cout=128, shuffle=1),
             I.single_layer(3102, n=2, h=14, w=14, groups=4, cin=64, cout=64, shuffle=3, residual="identity")]
    for i, case in enumerate(cases):
        say(f"no-alloc call {i}: x {case['x'].shape} layout {layout}")
        bias, q_ref, acc_ref = centred(case)
        lay = Layer(ctx, torch, case, bias, layout)
        out_n, dump_n = lay.outputs(torch)
        lay.run(out_n, dump_n, noalloc=True)
        q_n, acc_n = lay.read(out_n, dump_n)
        out_g, dump_g = lay.outputs(torch)
        lay.run(out_g, dump_g, noalloc=False)
        q_g, acc_g = lay.read(out_g, dump_g)
        np.testing.assert_array_equal(q_n, q_g)
        np.testing.assert_array_equal(acc_n, acc_g)
        np.testing.assert_array_equal(q_n, q_ref)
        np.testing.assert_array_equal(acc_n, acc_ref)
        assert len(np.unique(q_ref)) == 4


def test_noalloc_rejects_layers_beyond_its_buffer():
    """A layer whose prepacked filter exceeds the static buffer is refused
    before anything is enqueued (the output keeps its contents)."""
    import torch
    from paper_2208_01944_amd import palq
    ctx = palq.Context(0)
    # G = 8 groups of 512 -> 512 3x3: 8 * 512 * 72 K-blocks * 96 B of prepacked slabs > 16 MiB
    case = I.single_layer(3103, n=1, h=3, w=3, groups=8, cin=512, cout=512, shuffle=1)
    lay = Layer(ctx, torch, case, case["layer"]["bias"])
    out, dump = lay.outputs(torch)
    out.buf.fill_(0x5A)
    with pytest.raises(palq.PalqError) as err:
        lay.run(out, dump, noalloc=True)
    assert err.value.status == palq.ERR_UNSUPPORTED
    ctx.sync()
    assert bool((out.buf == 0x5A).all())


def test_noalloc_in_captured_graph_replays():
    """The no-alloc call captured into a HIP graph (capture fails on any
    allocation or synchronisation) and replayed several times with other
    work between the replays: every replay equals the eager palq_group_conv."""
    import torch
    from paper_2208_01944_amd import palq
    ctx = palq.Context(0)
    case = I.single_layer(3104, n=4, h=14, w=14, groups=4, cin=256, cout=256, shuffle=1)
    bias, q_ref, acc_ref = centred(case)
    lay = Layer(ctx, torch, case, bias)
    out_e, dump_e = lay.outputs(torch)
    lay.run(out_e, dump_e, noalloc=False)
    q_e, acc_e = lay.read(out_e, dump_e)
    np.testing.assert_array_equal(q_e, q_ref)
    np.testing.assert_array_equal(acc_e, acc_ref)
    out, dump = lay.outputs(torch)
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        ctx.set_stream(side)
        graph.capture_begin()
        lay.run(out, dump, noalloc=True)
        graph.capture_end()
    ctx.set_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    other = I.single_layer(3105, n=2, h=7, w=7, groups=2, cin=64, cout=64, shuffle=1)
    olay = Layer(ctx, torch, other, other["layer"]["bias"])
    for r in range(4):
        out.buf.fill_(0)
        dump.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        q, acc = lay.read(out, dump)
        np.testing.assert_array_equal(q, q_e, err_msg=f"replay {r}")
        np.testing.assert_array_equal(acc, acc_e, err_msg=f"replay {r}")
        o2, d2 = olay.outputs(torch)
        olay.run(o2, d2, noalloc=True)  # eager no-alloc work on the same buffer between replays
        ctx.sync()
