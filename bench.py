"""Benchmark: PalQuant ResNet-18 (G=4 parallel 2-bit groups) forward, batch 64.

One step = quantise the fp32 224x224x3 input batch to 8-bit codes (Eq. 2,
fixed l/u) + the whole network through palq_forward: 8-bit stem, max pool,
16 grouped 2-bit 3x3 convs with int32 residual adds and the cyclic
permutation fused into each block's second conv, 3 fused 1x1 projections,
integer global sum and the 8-bit FC to int32 logits.  Inputs are resident in
HBM before the timed region.

Prints one JSON line (see the keys below).  --gpus above 1 is refused: this
build runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective int TOPS + images/s, ResNet-18-shaped G=4 2-bit fwd, batch 64"
INT8_MFMA_PEAK_TOPS = 5000.0   # MI355X dense int8 MFMA, 5.0 POP/s
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="wall-clock budget of the oracle sample")
    return ap.parse_args()


def cpu_baseline(spec, x_f32, l, u, budget_s):
    """The oracle (as it stands) on a bounded sample of the same workload:
    whole images (quantise + forward), one at a time, until the budget is
    spent; reported in images/s."""
    from oracle import oracle as O
    t0 = time.perf_counter()
    done = 0
    while done < spec["n"]:
        codes = O.quantize(x_f32[done:done + 1], l, u, 8, signed=True)
        O.run_net(spec, codes)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "images/s", "cores": O.threads(), "kind": "oracle",
            "sample": f"{done} of {spec['n']} images of the same batch, quantise + full forward, "
                      f"{dt:.1f} s wall"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq

    n = args.batch
    spec = I.resnet18(n=n, groups=4, bits=2)
    x_f32 = I.image_fp32(I.SEED_BASE + 30, n)
    l, u = -3.0, 3.0

    ctx = palq.Context(0)
    stream = torch.cuda.current_stream()
    net = palq.Net(ctx, spec)
    net_t = palq.Net(ctx, spec, flags=palq.NET_TIMING)
    xd = ctx.upload(x_f32)
    codes = ctx.empty_act(n, 224, 224, 1, 3, 8, signed=True)
    logits = torch.empty(n * net.classes, dtype=torch.int32, device=ctx.dev)

    def step(nn):
        ctx.quantize(xd, l, u, codes)
        nn.forward(codes.buf, logits)

    for _ in range(args.warmup):
        step(net)
        step(net_t)
    torch.cuda.synchronize()

    # timed region: K whole steps
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(net)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps

    # per-layer device time (HIP events on the library's stream) over K steps
    net_t.reset_times()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(args.steps):
        step(net_t)
    torch.cuda.synchronize()
    wall_t = time.perf_counter() - t1
    layer_ms, fw = net_t.layer_times()
    layer_ms = layer_ms / max(fw, 1)

    # algorithmic work per layer (2 x MACs) and which kernel runs it
    conv_ops, conv_ms, other_ms = 0, 0.0, 0.0
    shapes = {0: (224, 224, 3)}
    per_layer = []
    for i, L in enumerate(spec["layers"]):
        s = shapes[L["src"]]
        if L["op"] == "conv":
            g, co, k, _, ci = L["w"].shape
            ho = (s[0] + 2 * L["pad"] - k) // L["stride"] + 1
            kk = k * k * ci + (L["proj_w"].shape[-1] if L.get("proj_w") is not None else 0)
            ops = 2 * n * ho * ho * g * co * kk
            shapes[L["dst"]] = (ho, ho, g * co)
            stem = L["in_bits"] == 8 and L["in_signed"] and L["w_bits"] == 8 and ci <= 4 and k <= 8
            mfma = co % 32 == 0 and (stem or (ci % 64 == 0 and L["in_bits"] == L["w_bits"]
                                               and not L["in_signed"]))
            per_layer.append(dict(layer=i, op="conv", kernel="mfma" if mfma else "direct",
                                  ops=ops, ms=float(layer_ms[i])))
            if mfma:
                conv_ops += ops
                conv_ms += layer_ms[i]
            else:
                other_ms += layer_ms[i]
        else:
            if L["op"] == "maxpool":
                ho = (s[0] + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                shapes[L["dst"]] = (ho, ho, s[2])
            else:
                shapes[L["dst"]] = (1, 1, s[2])
            per_layer.append(dict(layer=i, op=L["op"], ms=float(layer_ms[i])))
            other_ms += layer_ms[i]

    total_ops = net.ops
    img_s = n / (ms_per_step / 1e3)
    tops = total_ops / (ms_per_step / 1e3) / 1e12
    achieved = conv_ops / (conv_ms / 1e3) / 1e12 if conv_ms > 0 else 0.0
    res = {
        "metric": METRIC,
        "value": img_s,
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded uniform codes and random fp32 images, random weights)",
        "config": {"workload": "resnet18_palq_G4_b2_224_fwd", "global_batch": n, "image": [224, 224, 3],
                   "groups": 4, "bits": 2, "step": "quantize fp32 input + palq_forward"},
        "effective_tops": tops,
        "int_ops_per_step": total_ops,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": INT8_MFMA_PEAK_TOPS,
                     "unit": "TFLOP/s", "frac": achieved / INT8_MFMA_PEAK_TOPS, "traffic": None,
                     "kernel": "conv_mfma_kernel (all MFMA conv launches of one step)",
                     "kernel_ms_per_step": conv_ms, "kernel_int_ops_per_step": conv_ops},
        "timing_pass_ms_per_step": wall_t * 1e3 / args.steps,
        "layers": per_layer,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(spec, x_f32, l, u, args.cpu_seconds)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
