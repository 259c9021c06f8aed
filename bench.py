"""Benchmark: PalQuant ResNet-18 (G=4 parallel 2-bit groups) forward, batch 64.

One step = palq_forward_image: quantise the fp32 224x224x3 input batch to
8-bit codes (Eq. 2, fixed l/u; written straight into the stem's zero-border
input) + the whole network: 8-bit stem fused with its max pool,
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
FP4_MFMA_PEAK_TFLOPS = 10100.0  # MI355X dense FP4 MFMA, 10.1 PFLOP/s
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true", help="replay the forward from a captured HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="wall-clock budget of the oracle sample")
    ap.add_argument("--summarize-profile", metavar="DIR", default=None,
                    help="only turn the rocprofv3 outputs under DIR (kt/, fetch/, write/, cfetch/, "
                         "cwrite/ and bench.json, made by the commands written into the summaries) "
                         "into the text summaries under profiles/ and exit")
    ap.add_argument("--table2", action="store_true",
                    help="only run the Table 2 analogue (PalQuant against the dense M-bit network and "
                         "the bit-decomposition workload, forward only, batch --batch) and exit")
    ap.add_argument("--hbm-copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (the calibration "
                         "kernel for the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_tile_kernel_fp4_resnet18_g4_b2_bs64_traffic.txt")
DOMINANT = "conv_tile_kernel[fp4]"
KERNEL_SOURCE = os.path.join(ROOT, "paper_2208_01944_amd", "csrc", "k_conv_mfma.hip")


def measured_traffic():
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary, or None when the kernel source has changed since the counters
    were taken (the summary records the source's sha256)."""
    import hashlib
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith((" ", "#", "|")):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    if kv.get("kernel_source_sha256") != src or "hbm_bytes_per_launch" not in kv:
        return None
    return float(kv["hbm_bytes_per_launch"])


PROFILE_CMDS = {
    "kt": "rocprofv3 --kernel-trace --stats --output-format csv -d DIR/kt -o run -- "
          "python3 bench.py --steps 20 --warmup 2 --no-cpu-baseline",
    "fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/fetch -o run -- "
             "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline",
    "write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/write -o run -- "
             "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline",
    "cfetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/cfetch -o run -- "
              "python3 bench.py --hbm-copy-probe 1024",
    "cwrite": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/cwrite -o run -- "
              "python3 bench.py --hbm-copy-probe 1024",
    "bench": "python3 bench.py --steps 50 --warmup 5 --no-cpu-baseline > DIR/bench.json",
}


def _short(name):
    return name.replace("void ", "").replace("palq::(anonymous namespace)::", "").split("(")[0]


def family(short):
    """Kernel family of a demangled kernel name: the tiled convolution splits
    by its template arguments (CB, PB, WN, WM, RB, STEM, stages, FP4) into the
    stem, the grouped FP4 and the grouped int8 builds."""
    base = short.split("<")[0]
    if base != "conv_tile_kernel" or "<" not in short:
        return base
    args = [t.strip() for t in short[short.index("<") + 1:short.rindex(">")].split(",")]
    if args[5] == "true":
        return "conv_tile_kernel[stem]"
    return "conv_tile_kernel[fp4]" if len(args) > 7 and args[7] == "true" else "conv_tile_kernel[int8]"


def summarize_profile(d):
    """Writes the kernel-time and HBM-traffic summaries of one profiling
    session (rocprofv3 csv output) under profiles/."""
    import csv
    import hashlib
    bench = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
    head = ["# commands (run from the repository root, on one MI355X, `cd /tmp && export TMPDIR=/tmp` first;",
            "# DIR is any output folder)"]
    # ---- kernel time
    rows = list(csv.DictReader(open(os.path.join(d, "kt", "run_kernel_stats.csv"))))
    out = head + ["#   " + PROFILE_CMDS["kt"], "#   " + PROFILE_CMDS["bench"], "",
                  "Kernel time, rocprofv3 --kernel-trace --stats (all launches of the profiled run:",
                  "create-time weight prepack, 2+20 steps of the plain network and of the HIP-event-timed one)", "",
                  "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    fam = {}
    for r in rows:
        k = _short(r["Name"])
        out.append(f"| {k} | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {int(r['MinNs']) / 1e3:.1f} | {int(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
        f = fam.setdefault(family(k), [0, 0])
        f[0] += int(r["Calls"])
        f[1] += int(r["TotalDurationNs"])
    g = fam[DOMINANT]
    rf = bench["roofline"]
    out += ["", "%s, all instantiations: %d calls, average %.1f us per launch" % (DOMINANT, g[0], g[1] / g[0] / 1e3),
            "bench.py HIP events on the library stream, same kernel: average %.1f us per launch over %d launches/step"
            % (rf["avg_launch_us"], rf["launches_per_step"]),
            "bench.py (plain timed region): %.1f images/s, %.4f ms/step; roofline frac %.4f (%.0f of %.0f %s)"
            % (bench["value"], bench["ms_per_step"], rf["frac"], rf["achieved"], rf["peak"], rf["unit"]), "",
            "Per layer (bench.py HIP events, us per launch):", ""]
    out += ["| layer | op | kernel | us | int ops | alg. bytes |", "|---|---|---|---|---|---|"]
    for L in bench["layers"]:
        out.append(f"| {L['layer']} | {L['op']} | {L.get('kernel', '')} | {L['ms'] * 1e3:.1f} | "
                   f"{L.get('ops', 0):.3e} | {L.get('bytes', 0):.3e} |")
    open(os.path.join(ROOT, "profiles", "resnet18_g4_b2_bs64_kernel_stats.md"), "w").write("\n".join(out) + "\n")

    # ---- traffic
    def load(sub):
        return [(_short(r["Kernel_Name"]), float(r["Counter_Value"]))
                for r in csv.DictReader(open(os.path.join(d, sub, "run_counter_collection.csv")))]
    cf = [v for k, v in load("cfetch") if "copyBuffer" in k]
    cw = [v for k, v in load("cwrite") if "copyBuffer" in k]
    probe_kib = 1024 * 1024
    ff, fw = probe_kib / (sum(cf) / len(cf)), probe_kib / (sum(cw) / len(cw))
    F, W = load("fetch"), load("write")
    assert [k for k, _ in F] == [k for k, _ in W]
    gl = [(f * ff * 1024, w * fw * 1024) for (k, f), (_, w) in zip(F, W) if family(k) == DOMINANT]
    layers = [L for L in bench["layers"] if L.get("kernel") == DOMINANT]
    nl = len(layers)
    assert len(gl) % nl == 0
    nf = len(gl) // nl
    per_launch = sum(a + b for a, b in gl) / len(gl)
    src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    out = head + ["#   " + PROFILE_CMDS[k] for k in ("fetch", "write", "cfetch", "cwrite")] + [
        "",
        "HBM traffic of %s, ResNet-18 PalQuant G=4 2-bit, batch 64 (%d forwards x %d launches)"
        % (DOMINANT, nf, nl), "",
        "copy calibration (1 GiB device copy): FETCH_SIZE reads %.1f KiB per launch for 1048576 KiB copied"
        % (sum(cf) / len(cf)),
        "  -> fetch factor %.4f; WRITE_SIZE reads %.1f KiB -> write factor %.4f" % (ff, sum(cw) / len(cw), fw), "",
        "| layer | alg. MB | HBM read MB | HBM write MB | (read+write)/alg |", "|---|---|---|---|---|"]
    for i, L in enumerate(layers):
        r = sum(gl[j * nl + i][0] for j in range(nf)) / nf
        w = sum(gl[j * nl + i][1] for j in range(nf)) / nf
        out.append(f"| {L['layer']} | {L['bytes'] / 1e6:.2f} | {r / 1e6:.2f} | {w / 1e6:.2f} | "
                   f"{(r + w) / L['bytes']:.2f} |")
    out += ["", "kernel: " + DOMINANT,
            "kernel_source_sha256: " + src,
            "hbm_bytes_per_launch: %.0f" % per_launch,
            "algorithmic_bytes_per_launch: %.0f" % rf["algorithmic_bytes_per_launch"]]
    open(TRAFFIC_FILE, "w").write("\n".join(out) + "\n")
    print("wrote", TRAFFIC_FILE)


def copy_probe(mib):
    import torch
    n = mib << 18                      # int32 elements
    src = torch.full((n,), 7, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "launches": 3}))


def conv_kernel(L, ci, co, k):
    """Which kernel family the library's selection rules give a conv layer of
    this workload (the stem and 2-bit grouped layers take the tiled kernel;
    2-bit layers run on FP4 matrix cores unless PALQ_CONV_FP4=0)."""
    stem = L["in_bits"] == 8 and L["in_signed"] and L["w_bits"] == 8 and ci <= 4 and k <= 8
    if stem:
        tiled = co % 128 == 0 and L.get("res", -1) < 0 and L["out_bits"] == 2
        return "conv_tile_kernel[stem]" if tiled else "conv_stem_kernel"
    grouped = co % 32 == 0 and ci % 64 == 0 and L["in_bits"] == L["w_bits"] and not L["in_signed"]
    if not grouped:
        return "conv_direct_kernel"
    tiled = L["in_bits"] == 2 and co % 64 == 0 and L["out_bits"] == 2
    if not tiled:
        return "conv_grouped_kernel"
    bound = k * k * ci * 3 * 2 + (L["proj_w"].shape[-1] * 3 * 2 if L.get("proj_w") is not None else 0)
    fp4 = os.environ.get("PALQ_CONV_FP4", "1") != "0" and bound < (1 << 23)
    return "conv_tile_kernel[fp4]" if fp4 else "conv_tile_kernel[int8]"


def table2(args):
    """On-GPU analogue of the paper's Table 2 for M = 2G bits at B = 2: the
    PalQuant ResNet-18 (G groups of 2-bit convs), the dense M-bit network of
    the original width (G = 1, only M = 4 is a supported code width), and the
    workload of the Eq. 4 bit-decomposition (G^2 2-bit products of the full
    width, run as a dense 2-bit network with G-fold widths: the same MACs
    and operand bytes, without the final shift-add).  One JSON line per G."""
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq

    ctx = palq.Context(0)
    n = args.batch

    def timed(spec):
        net = palq.Net(ctx, spec)
        x = ctx.pack(spec["x"], 1, 8, signed=True)
        logits = torch.empty(n * net.classes, dtype=torch.int32, device=ctx.dev)
        for _ in range(max(args.warmup, 1)):
            net.forward(x.buf, logits)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            net.forward(x.buf, logits)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        return {"images_per_s": n / dt, "ms_per_forward": dt * 1e3, "int_ops": net.ops}

    for G in (2, 3, 4):
        row = {"table2": f"ResNet-18, M = {2 * G} bits as G = {G} x B = 2", "batch": n}
        row["palquant"] = timed(I.resnet18(n=n, groups=G, bits=2))
        row["dense_m_bit"] = (timed(I.resnet18(n=n, groups=1, bits=4)) if 2 * G == 4
                              else f"not run: {2 * G}-bit codes are outside the supported widths (2, 3, 4)")
        row["bit_decomposition_workload"] = timed(I.resnet18(n=n, groups=1, bits=2, width_mult=G))
        for k in ("dense_m_bit", "bit_decomposition_workload"):
            if isinstance(row[k], dict):
                row[f"speedup_vs_{k}"] = row["palquant"]["images_per_s"] / row[k]["images_per_s"]
        print(json.dumps(row), flush=True)


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
    if args.summarize_profile:
        summarize_profile(args.summarize_profile)
        return
    if args.hbm_copy_probe:
        copy_probe(args.hbm_copy_probe)
        return
    if args.table2:
        table2(args)
        return
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq

    n = args.batch
    spec = I.resnet18(n=n, groups=4, bits=2)
    x_f32 = I.image_fp32(I.SEED_BASE + 30, n)
    l, u = -3.0, 3.0

    ctx = palq.Context(0)
    stream = torch.cuda.current_stream()
    # eager launches (--graph: replay from a captured HIP graph, which
    # measured about 1.5 % slower for this network)
    net = palq.Net(ctx, spec, flags=palq.NET_GRAPH if args.graph else 0)
    net_t = palq.Net(ctx, spec, flags=palq.NET_TIMING)
    xd = ctx.upload(x_f32)
    logits = torch.empty(n * net.classes, dtype=torch.int32, device=ctx.dev)

    def step(nn):
        # quantise the fp32 batch (Eq. 2) straight into the stem's padded
        # input and run the network: palq_forward_image
        nn.forward_image(xd, l, u, logits)

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

    # algorithmic work per layer (2 x MACs, and the bytes a launch must move
    # at least once: packed input codes, packed weights, packed output codes,
    # the residual / projection input and the per-channel requant arrays) and
    # which kernel runs it
    def act_bytes(h, w, c, bits):
        return n * h * w * c * bits / 8

    kern = {}
    shapes = {0: (224, 224, 3, 8)}
    per_layer = []
    for i, L in enumerate(spec["layers"]):
        s = shapes[L["src"]]
        if L["op"] == "conv":
            g, co, k, _, ci = L["w"].shape
            ho = (s[0] + 2 * L["pad"] - k) // L["stride"] + 1
            kk = k * k * ci + (L["proj_w"].shape[-1] if L.get("proj_w") is not None else 0)
            ops = 2 * n * ho * ho * g * co * kk
            shapes[L["dst"]] = (ho, ho, g * co, L["out_bits"])
            nbytes = act_bytes(s[0], s[1], s[2], s[3]) + g * co * k * k * ci * L["w_bits"] / 8 \
                + act_bytes(ho, ho, g * co, L["out_bits"]) + 3 * 4 * g * co
            if L.get("res", -1) >= 0:
                r = shapes[L["res"]]
                nbytes += act_bytes(r[0], r[1], r[2], r[3]) + 4 * g * co
            if L.get("proj_src", -1) >= 0:
                r = shapes[L["proj_src"]]
                nbytes += act_bytes(r[0], r[1], r[2], r[3]) + L["proj_w"].size * L["w_bits"] / 8
            kname = conv_kernel(L, ci, co, k)
            nxt = spec["layers"][i + 1] if i + 1 < len(spec["layers"]) else {}
            fused_pool = (kname == "conv_tile_kernel[stem]" and nxt.get("op") == "maxpool" and
                          nxt.get("src") == L["dst"] and (nxt["k"], nxt["stride"], nxt["pad"]) == (3, 2, 1) and
                          ho <= 127)
            if fused_pool:  # the stem and its max pool run as one launch (its time includes the quantiser)
                kname = "quantize_pad4_kernel + stem_pool_kernel"
            per_layer.append(dict(layer=i, op="conv", kernel=kname, ops=ops, bytes=nbytes,
                                  ms=float(layer_ms[i])))
        else:
            if L["op"] == "maxpool":
                ho = (s[0] + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                shapes[L["dst"]] = (ho, ho, s[2], s[3])
                prev = per_layer[-1] if per_layer else {}
                kname = ("fused into layer %d (no launch)" % prev["layer"]
                         if prev.get("kernel", "").endswith("stem_pool_kernel") else "maxpool_kernel")
            else:
                shapes[L["dst"]] = (1, 1, s[2], 32)
                # this workload's paths: the per-image sum kernel (which also
                # writes the FC's digit planes) and the matrix-core FC
                kname = "avgsum2_wg_kernel" if L["op"] == "avgsum" else "fc_mfma_kernel"
            per_layer.append(dict(layer=i, op=L["op"], kernel=kname, ms=float(layer_ms[i])))
        K = kern.setdefault(kname, dict(launches=0, ops=0, bytes=0.0, ms=0.0))
        K["launches"] += 1
        K["ms"] += float(layer_ms[i])
        K["ops"] += per_layer[-1].get("ops", 0)
        K["bytes"] += per_layer[-1].get("bytes", 0.0)

    total_ops = net.ops
    img_s = n / (ms_per_step / 1e3)
    tops = total_ops / (ms_per_step / 1e3) / 1e12
    # the dominant kernel: the grouped 2-bit conv (3x3 convs of the residual
    # blocks, projections fused), 16 launches per step, on FP4 matrix cores
    # (int8 with PALQ_CONV_FP4=0); its peak is that of the format it runs on
    dom = DOMINANT if DOMINANT in kern else "conv_tile_kernel[int8]"
    D = kern[dom]
    peak = FP4_MFMA_PEAK_TFLOPS if dom == DOMINANT else INT8_MFMA_PEAK_TOPS
    launch_ms = D["ms"] / D["launches"]
    ops_per_launch = D["ops"] / D["launches"]
    achieved = ops_per_launch / (launch_ms / 1e3) / 1e12
    traffic = measured_traffic() if dom == DOMINANT else None
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
        "dtype": "fp4+int8" if dom == DOMINANT else "int8",
        "data": "synthetic (seeded uniform codes and random fp32 images, random weights)",
        "config": {"workload": "resnet18_palq_G4_b2_224_fwd", "global_batch": n, "image": [224, 224, 3],
                   "groups": 4, "bits": 2, "step": "palq_forward_image (quantize fp32 input + forward)"},
        "effective_tops": tops,
        "int_ops_per_step": total_ops,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak, "traffic": traffic,
                     "kernel": dom, "launches_per_step": D["launches"],
                     "avg_launch_us": launch_ms * 1e3, "int_ops_per_launch": ops_per_launch,
                     "algorithmic_bytes_per_launch": D["bytes"] / D["launches"],
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"},
        "kernels": {k: dict(v, avg_launch_us=v["ms"] * 1e3 / v["launches"]) for k, v in kern.items()},
        "timing_pass_ms_per_step": wall_t * 1e3 / args.steps,
        "layers": per_layer,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(spec, x_f32, l, u, args.cpu_seconds)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
