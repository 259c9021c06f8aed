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
FP4_MFMA_PEAK_TFLOPS = 10100.0  # MI355X dense FP4 (and FP6) MFMA, 10.1 PFLOP/s
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=64, help="batch of the --table2 networks")
    ap.add_argument("--workload", default="resnet18_g4_b2",
                    help="resnet18_g4_b2 (the default: ResNet-18 G=4 2-bit, batch 64), "
                         "resnet18_g4_b2_shuffles (the same with cyclic shuffle modules and channel "
                         "shuffles), resnet50_g2_b2 (ResNet-50 G=2 2-bit, batch 128), or single layers: c1, c2 "
                         "(its four layers c2_l0..c2_l3), c4 (its nine cells c4_g<G>_b<B>) or "
                         "layers (all of them); one JSON line per network or layer")
    ap.add_argument("--no-histograms", action="store_true",
                    help="skip the per-layer output-code histograms (an untimed extra forward)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true", help="replay the forward from a captured HIP graph")
    ap.add_argument("--pixel-layout", action="store_true",
                    help="keep every intermediate tensor in the pixel layout (the network stores "
                         "conv outputs group by group by default)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="wall-clock budget of the oracle sample")
    ap.add_argument("--summarize-profile", metavar="DIR", default=None,
                    help="only turn the rocprofv3 outputs under DIR (kt/, fetch/, write/, cfetch/, "
                         "cwrite/ and bench.json, made by the commands written into the summaries) "
                         "into the text summaries under profiles/ and exit")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="only turn the counter passes under DIR (p1/ .. p5/ and bench.json) into "
                         "profiles/<workload>_sq_counters.md and exit")
    ap.add_argument("--table2", action="store_true",
                    help="only run the Table 2 analogue (PalQuant against the dense M-bit network and "
                         "the bit-decomposition workload, forward only, batch --batch) and exit")
    ap.add_argument("--hbm-copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (the calibration "
                         "kernel for the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_fp4_kernel_resnet18_g4_b2_traffic.txt")
DOMINANT = "conv_fp4_kernel"
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
          "python3 bench.py --workload W --steps 20 --warmup 2 --no-cpu-baseline --no-histograms",
    "fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/fetch -o run -- "
             "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-histograms",
    "write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/write -o run -- "
             "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-histograms",
    "cfetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/cfetch -o run -- "
              "python3 bench.py --hbm-copy-probe 1024",
    "cwrite": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/cwrite -o run -- "
              "python3 bench.py --hbm-copy-probe 1024",
    "bench": "python3 bench.py --workload W --steps 50 --warmup 5 --no-cpu-baseline > DIR/bench.json",
}


def _short(name):
    return name.replace("void ", "").replace("palq::(anonymous namespace)::", "").split("(")[0]


def family(short):
    """Kernel family of a demangled kernel name: the tiled convolution
    (conv_tile_kernel) splits by its template arguments (CB, PB, WN, WM, RB,
    STEM, stages, FP4, DUMP) into the stem, the grouped FP4 and the grouped
    int8 builds; other kernels are their base name (conv_fp4_kernel: the
    2-bit grouped layers on FP4 matrix cores)."""
    base = short.split("<")[0]
    if base != "conv_tile_kernel" or "<" not in short:
        return base
    args = [t.strip() for t in short[short.index("<") + 1:short.rindex(">")].split(",")]
    if args[5] == "true":
        return "conv_tile_kernel[stem]"
    return "conv_tile_kernel[fp4]" if len(args) > 7 and args[7] == "true" else "conv_tile_kernel[int8]"


def summarize_single_profile(d, workload):
    """Kernel-time summary of one single-layer bench session (rocprofv3 csv
    under DIR/kt, the bench's JSON lines in DIR/bench.json, one per layer or
    sweep cell) written to profiles/<workload>_kernel_stats.md."""
    import csv
    import hashlib
    lines = [json.loads(x) for x in open(os.path.join(d, "bench.json")).read().splitlines() if x.startswith("{")]
    rows = list(csv.DictReader(open(os.path.join(d, "kt", "run_kernel_stats.csv"))))
    out = ["# commands (run from the repository root, on one MI355X, `cd /tmp && export TMPDIR=/tmp` first;",
           "# DIR is any output folder, W = " + workload + ")",
           "#   rocprofv3 --kernel-trace --stats --output-format csv -d DIR/kt -o run -- "
           "python3 bench.py --workload W --steps 50 --warmup 5 --no-cpu-baseline",
           "#   python3 bench.py --workload W --steps 50 --warmup 5 --no-cpu-baseline > DIR/bench.json",
           "#   python3 bench.py --workload W --summarize-profile DIR", "",
           "Kernel time, rocprofv3 --kernel-trace --stats (all launches of the profiled run: plan-time",
           "prepack and requant constants, warm-up and timed launches of every layer of the workload)", "",
           "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {_short(r['Name'])} | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {int(r['MinNs']) / 1e3:.1f} | {int(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
    out += ["", "bench.py (HIP events around palq_conv_run, separate run):", "",
            "| workload | kernel | us per launch | TOPS | roofline frac | peak |", "|---|---|---|---|---|---|"]
    for b in lines:
        rf = b["roofline"]
        out.append(f"| {b['config']['workload']} | {b['kernel']} | {b['us_per_launch']:.1f} | {b['value']:.0f} | "
                   f"{rf['frac']:.3f} | {rf['peak']:.0f} {rf['unit']} |")
    out += ["", "kernel_source_sha256: " + hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()]
    open(kernel_stats_file(workload), "w").write("\n".join(out) + "\n")
    print("wrote", kernel_stats_file(workload))


def summarize_profile(d, workload):
    """Writes the kernel-time summary of one profiling session (rocprofv3
    csv output under DIR: kt/ and bench.json) and, when DIR also holds the
    counter passes (fetch/, write/, cfetch/, cwrite/; ResNet-18 workload),
    the HBM-traffic summary under profiles/."""
    import csv
    import hashlib
    bench = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
    head = ["# commands (run from the repository root, on one MI355X, `cd /tmp && export TMPDIR=/tmp` first;",
            "# DIR is any output folder, W = " + workload + ")"]
    # ---- kernel time
    rows = list(csv.DictReader(open(os.path.join(d, "kt", "run_kernel_stats.csv"))))
    out = head + ["#   " + PROFILE_CMDS["kt"], "#   " + PROFILE_CMDS["bench"],
                  "#   python3 bench.py --workload W --summarize-profile DIR", "",
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
    src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    out += ["", "kernel_source_sha256: " + src]
    open(kernel_stats_file(workload), "w").write("\n".join(out) + "\n")
    print("wrote", kernel_stats_file(workload))
    if not os.path.isdir(os.path.join(d, "fetch")):
        return

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


COUNTER_PASSES = [
    "SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS SQ_INSTS_SALU "
    "SQ_VALU_MFMA_BUSY_CYCLES",
    "SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_VMEM SQ_INST_CYCLES_VMEM_RD SQ_LDS_BANK_CONFLICT "
    "SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_WAIT_INST_LDS",
    "GRBM_GUI_ACTIVE SQ_CYCLES SQ_ACTIVE_INST_ANY SQ_INSTS_VMEM_RD SQ_ACTIVE_INST_SCA SQ_INST_LEVEL_VMEM",
    # the memory path: address (TA) and data (TD) units, vector L1 (TCP)
    "TA_BUSY_avr TA_BUFFER_TOTAL_CYCLES_sum GRBM_GUI_ACTIVE TD_TD_BUSY_sum TD_TC_STALL_sum "
    "TCP_PENDING_STALL_CYCLES_sum TCP_TCP_TA_DATA_STALL_CYCLES_sum TCP_TCR_TCP_STALL_CYCLES_sum "
    "TCP_READ_TAGCONFLICT_STALL_CYCLES_sum",
    "TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCP_TOTAL_CACHE_ACCESSES_sum TCP_TCP_LATENCY_sum "
    "TA_ADDR_STALLED_BY_TC_CYCLES_sum TA_DATA_STALLED_BY_TC_CYCLES_sum GRBM_GUI_ACTIVE",
]
COUNTER_CMD = ("timeout -s KILL 120 rocprofv3 --pmc COUNTERS --output-format csv -d DIR/pPASS -o run -- "
               "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-histograms")


def summarize_counters(d, workload):
    """Per-layer counter summary of the network's conv launches (the
    rocprofv3 --pmc passes of COUNTER_PASSES under DIR/p1, p2, ... and the
    bench JSON DIR/bench.json): SQ instruction mix and busy fractions, then
    the memory path (TA, TD, vector L1 and its L2 requests)
    written to profiles/<workload>_sq_counters.md.  Counters are summed over
    the chip per dispatch; per-SIMD figures divide by 4 x CUs (256 CUs)."""
    import csv
    import hashlib
    bench = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
    convs = [L for L in bench["layers"] if L["op"] == "conv"]
    fams = {"stem_pool_kernel": [], DOMINANT: []}
    for L in convs:
        k = L["kernel"].split(" + ")[-1]
        if k in fams:
            fams[k].append(L)
    vals = {}  # (family, layer index within family) -> counter -> [values]
    for p in range(1, len(COUNTER_PASSES) + 1):
        rows = list(csv.DictReader(open(os.path.join(d, f"p{p}", "run_counter_collection.csv"))))
        seen = {}
        for r in rows:
            f = family(_short(r["Kernel_Name"]))
            if f not in fams or not fams[f]:
                continue
            key = (f, int(r["Dispatch_Id"]))
            seen.setdefault(f, {})
            if key not in seen[f]:
                seen[f][key] = len(seen[f])
            idx = seen[f][key] % len(fams[f])
            vals.setdefault((f, idx), {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    simds = 4 * 256
    out = ["# commands (from the repository root, on one MI355X, `cd /tmp && export TMPDIR=/tmp` first; DIR any folder)"]
    for i, c in enumerate(COUNTER_PASSES):
        out.append("#   " + COUNTER_CMD.replace("COUNTERS", c).replace("PASS", str(i + 1)))
    out += ["#   python3 bench.py --steps 50 --warmup 5 --no-cpu-baseline > DIR/bench.json",
            "#   python3 bench.py --summarize-counters DIR", "",
            "SQ counters per dispatch of the %s network's conv kernels (mean over the profiled forwards)." % workload,
            "Per SIMD = chip total / 1024.  mfma_busy = SQ_VALU_MFMA_BUSY_CYCLES per SIMD / (layer time x clock);",
            "valu_busy = 4 x SQ_INSTS_VALU per SIMD / the same cycles (a wave64 VALU instruction occupies a SIMD 4 cycles);",
            "lds_conflict = SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS; clock from GRBM_GUI_ACTIVE / 8 XCDs over the",
            "layer's HIP-event time.", "",
            "| layer | kernel | us | MFMA instr | VALU/MFMA | SALU/MFMA | LDS/MFMA | mfma_busy | valu_busy | "
            "lds_conflict | wait_inst_lds/wave | clock GHz |",
            "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for f, Ls in fams.items():
        for i, L in enumerate(Ls):
            v = {k: sum(x) / len(x) for k, x in vals.get((f, i), {}).items()}
            if not v:
                continue
            us = L["ms"] * 1e3
            cyc = v.get("GRBM_GUI_ACTIVE", 0) / 8
            clock = cyc / (us * 1e3) if us else 0
            mf = max(v.get("SQ_INSTS_MFMA", 1), 1)
            out.append("| %d | %s | %.1f | %d | %.1f | %.1f | %.2f | %.3f | %.3f | %.3f | %.0f | %.2f |" % (
                L["layer"], f, us, v.get("SQ_INSTS_MFMA", 0), v.get("SQ_INSTS_VALU", 0) / mf,
                v.get("SQ_INSTS_SALU", 0) / mf, v.get("SQ_INSTS_LDS", 0) / mf,
                v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / simds / max(cyc, 1),
                4 * v.get("SQ_INSTS_VALU", 0) / simds / max(cyc, 1),
                v.get("SQ_LDS_BANK_CONFLICT", 0) / max(v.get("SQ_ACTIVE_INST_LDS", 1), 1),
                v.get("SQ_WAIT_INST_LDS", 0) / max(v.get("SQ_WAVES", 1), 1), clock))
    cus = 256
    out += ["", "Memory path per dispatch (passes 4 and 5): busy and stall cycles per CU / (GRBM_GUI_ACTIVE / 8 XCDs);",
            "L2 requests = TCP_TCC_READ_REQ_sum (vector L1 misses sent to the L2), their mean latency in cycles.", "",
            "| layer | kernel | TA busy | TA buffer cycles/CU | TD busy/CU | TD stalled on TC | TCP pending stall | "
            "L2 read requests | L2 latency | L1 accesses | L1 latency |",
            "|---|---|---|---|---|---|---|---|---|---|---|"]
    for f, Ls in fams.items():
        for i, L in enumerate(Ls):
            v = {k: sum(x) / len(x) for k, x in vals.get((f, i), {}).items()}
            if "TA_BUSY_avr" not in v:
                continue
            cyc = max(v.get("GRBM_GUI_ACTIVE", 0) / 8, 1)
            req = max(v.get("TCP_TCC_READ_REQ_sum", 0), 1)
            acc = max(v.get("TCP_TOTAL_CACHE_ACCESSES_sum", 0), 1)
            out.append("| %d | %s | %.2f | %.2f | %.2f | %.2f | %.2f | %.0f | %.0f | %.0f | %.0f |" % (
                L["layer"], f, v["TA_BUSY_avr"] / cyc, v.get("TA_BUFFER_TOTAL_CYCLES_sum", 0) / cus / cyc,
                v.get("TD_TD_BUSY_sum", 0) / cus / cyc, v.get("TD_TC_STALL_sum", 0) / cus / cyc,
                v.get("TCP_PENDING_STALL_CYCLES_sum", 0) / cus / cyc, req,
                v.get("TCP_TCC_READ_REQ_LATENCY_sum", 0) / req, acc, v.get("TCP_TCP_LATENCY_sum", 0) / acc))
    out += ["", "raw means per dispatch (chip totals):", ""]
    for (f, i), cv in sorted(vals.items()):
        out.append("%s #%d: " % (f, i) + ", ".join("%s=%.0f" % (k, sum(x) / len(x)) for k, x in sorted(cv.items())))
    src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    out += ["", "kernel_source_sha256: " + src]
    path = os.path.join(ROOT, "profiles", f"{workload}_sq_counters.md")
    open(path, "w").write("\n".join(out) + "\n")
    print("wrote", path)


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


# the paper's ResNet-18 speed-ups over the M-bit baseline (Table 2, B = 2): context only
TABLE2_PAPER = {2: {"bit_fusion": 1.78, "bpvec": 1.77}, 3: {"bit_fusion": 2.52, "bpvec": 2.56},
                4: {"bit_fusion": 3.21, "bpvec": 3.12}}


def table2(args):
    """On-GPU analogue of the paper's Table 2 (Section 5.2) for M = 2G bits at
    B = 2, batch --batch, forward only, ResNet-18: PalQuant (G groups of
    2-bit convs on the FP4 matrix cores) against the M-bit network of the
    original width (G = 1) run two ways: directly on int8 matrix cores, and
    as the Eq. 4 bit decomposition the paper's accelerators perform (G^2
    2-bit chunk products per MAC, shifted and summed exactly, on the same FP4
    matrix cores as PalQuant; palq_set_conv_bitdecomp).  The two runs of the
    M-bit network must give identical logits.  One JSON line per G."""
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq

    ctx = palq.Context(0)
    n = args.batch

    def timed(spec, bitdecomp=False):
        ctx.set_conv_bitdecomp(bitdecomp)
        try:
            net = palq.Net(ctx, spec)
        finally:
            ctx.set_conv_bitdecomp(False)
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
        kern = net.layer_kernels()
        convs = [k for k, L in zip(kern, spec["layers"]) if L["op"] == "conv" and not L["in_signed"]]
        res = {"images_per_s": n / dt, "ms_per_forward": dt * 1e3, "int_ops": net.ops,
               "grouped_layer_kernels": sorted(set(convs))}
        del net
        return res, logits.cpu().numpy()

    for G in (2, 3, 4):
        M = 2 * G
        row = {"table2": f"ResNet-18, M = {M} bits vs G = {G} x B = 2", "batch": n,
               "data": "synthetic (seeded uniform codes and weights, stated parameters)"}
        row["palquant"], _ = timed(I.resnet18(n=n, groups=G, bits=2))
        dense = I.resnet18(n=n, groups=1, bits=M)
        row["dense_m_bit_int8"], l_direct = timed(dense)
        row["dense_m_bit_eq4_fp4"], l_eq4 = timed(dense, bitdecomp=True)
        row["eq4_logits_equal_direct"] = bool(np.array_equal(l_direct, l_eq4))
        for k in ("dense_m_bit_int8", "dense_m_bit_eq4_fp4"):
            row[f"palquant_speedup_vs_{k}"] = row["palquant"]["images_per_s"] / row[k]["images_per_s"]
        row["paper_speedup_vs_m_bit"] = TABLE2_PAPER[G]
        print(json.dumps(row), flush=True)


def host_cpu():
    """nproc and the CPU model name of this host (lscpu, else /proc/cpuinfo)."""
    import subprocess
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    if model is None and os.path.exists("/proc/cpuinfo"):
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    return os.cpu_count(), model


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
    nproc, model = host_cpu()
    return {"value": done / dt, "unit": "images/s", "cores": O.threads(), "kind": "oracle",
            "threads_used": O.threads(), "nproc": nproc, "cpu_model": model,
            "sample": f"{done} of {spec['n']} images of the same batch, quantise + full forward, "
                      f"{dt:.1f} s wall (the oracle's C convolution loop on an OpenMP team of "
                      f"{O.threads()} threads; its numpy requant and glue single-threaded)"}


NETWORKS = {
    # workload name -> (config name in the JSON line, metric)
    "resnet18_g4_b2": ("resnet18_palq_G4_b2_224_fwd_centred", METRIC),
    "resnet18_g4_b2_shuffles": ("resnet18_palq_G4_b2_224_fwd_centred_with_shuffle_modules_and_channel_shuffles",
                                "effective int TOPS + images/s, ResNet-18-shaped G=4 2-bit fwd with cyclic "
                                "shuffle modules and channel shuffles, batch 64"),
    "resnet50_g2_b2": ("resnet50_palq_G2_b2_224_fwd_centred",
                       "effective int TOPS + images/s, ResNet-50-shaped G=2 2-bit fwd, batch 128"),
}


def kernel_stats_file(workload):
    return os.path.join(ROOT, "profiles", f"{workload}_kernel_stats.md")


def rocprof_avg_us(workload, kernel):
    """Average launch duration of `kernel` in the committed rocprofv3
    summary of this workload, or None when the summary is missing or the
    kernel source changed since it was taken."""
    import hashlib
    path = kernel_stats_file(workload)
    if not os.path.exists(path):
        return None
    src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    avg, sha = None, None
    for line in open(path):
        if line.startswith("kernel_source_sha256:"):
            sha = line.split(":", 1)[1].strip()
        if line.startswith(kernel + ", all instantiations:"):
            avg = float(line.split("average", 1)[1].split("us")[0])
    return avg if sha == src else None


def network_algorithmic(spec, n):
    """Per layer: 2 x MACs and the bytes a launch must move at least once
    (packed input codes, packed weights, packed output codes, the residual /
    projection input and the per-channel requant arrays)."""
    def act_bytes(h, w, c, bits):
        return n * h * w * c * bits / 8

    shapes = {0: (spec["hw"], spec["hw"], 3, 8)}
    out = []
    for L in spec["layers"]:
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
            out.append(dict(ops=ops, bytes=nbytes))
        elif L["op"] == "shuffle_module":
            # 1x1 group conv on the cyclically permuted input plus the
            # unpermuted shortcut (Eq. 9-10): the input is read once
            g, co, _, _, ci = L["w"].shape
            ops = 2 * n * s[0] * s[1] * g * co * ci
            shapes[L["dst"]] = (s[0], s[1], g * co, L["out_bits"])
            nbytes = act_bytes(s[0], s[1], s[2], s[3]) + g * co * ci * L["w_bits"] / 8 \
                + act_bytes(s[0], s[1], g * co, L["out_bits"]) + 4 * 4 * g * co
            out.append(dict(ops=ops, bytes=nbytes))
        elif L["op"] == "channel_shuffle":
            shapes[L["dst"]] = s
            out.append(dict(bytes=2 * act_bytes(s[0], s[1], s[2], s[3])))
        else:
            if L["op"] == "maxpool":
                ho = (s[0] + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                shapes[L["dst"]] = (ho, ho, s[2], s[3])
            else:
                shapes[L["dst"]] = (1, 1, s[2], 32)
            out.append({})
    return out


def code_histograms(ctx, spec, xd, l, u):
    """Per conv layer of the network: how often each output code occurs on
    this batch (a KEEP_ALL build of the same network, untimed)."""
    import torch
    from paper_2208_01944_amd import palq
    net = palq.Net(ctx, spec, flags=palq.NET_KEEP_ALL)
    logits = torch.empty(spec["n"] * net.classes, dtype=torch.int32, device=ctx.dev)
    net.forward_image(xd, l, u, logits)
    ctx.sync()
    hist = {}
    for i, L in enumerate(spec["layers"]):
        if L["op"] == "conv":
            t = net.tensor(L["dst"])
            a = t.act
            nb = a.n * a.h * a.w * a.groups * a.ch_per_group
            codes = torch.empty(nb, dtype=torch.uint8, device=ctx.dev)
            ctx._check(palq._unpack(ctx.h, palq.ctypes.byref(a), codes.data_ptr()))
            hist[str(i)] = torch.bincount(codes, minlength=1 << L["out_bits"]).cpu().tolist()
    del net
    return hist


def run_network(args, workload):
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq

    cfg_name, metric = NETWORKS[workload]
    spec, x_f32, calib = I.workload(workload)
    spec = I.with_stored_biases(spec, workload)  # the centred variant (oracle-calibrated biases)
    n = spec["n"]
    l, u = I.IMAGE_RANGE

    ctx = palq.Context(0)
    # eager launches (--graph: replay from a captured HIP graph, which
    # measured about 1.5 % slower for the ResNet-18 network)
    lay = palq.NET_PIXEL_LAYOUT if args.pixel_layout else 0
    net = palq.Net(ctx, spec, flags=(palq.NET_GRAPH if args.graph else 0) | lay)
    net_t = palq.Net(ctx, spec, flags=palq.NET_TIMING | lay)
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
    distinct = int(torch.unique(logits).numel())
    if distinct < 100:
        raise SystemExit(f"the network's logits are degenerate ({distinct} distinct values)")

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
    labels = net_t.layer_kernels(image=True)
    alg = network_algorithmic(spec, n)

    kern = {}
    per_layer = []
    for i, L in enumerate(spec["layers"]):
        kname = labels[i] or "(covered by layer %d's launch)" % (i - 1)
        row = dict(layer=i, op=L["op"], kernel=kname, ms=float(layer_ms[i]), **alg[i])
        per_layer.append(row)
        K = kern.setdefault(kname, dict(launches=0, ops=0, bytes=0.0, ms=0.0))
        K["launches"] += 1
        K["ms"] += row["ms"]
        K["ops"] += row.get("ops", 0)
        K["bytes"] += row.get("bytes", 0.0)

    total_ops = net.ops
    img_s = n / (ms_per_step / 1e3)
    tops = total_ops / (ms_per_step / 1e3) / 1e12
    # the dominant kernel: the grouped 2-bit conv on FP4 matrix cores (int8
    # with PALQ_CONV_FP4=0); its peak is that of the format it runs on
    dom = DOMINANT if DOMINANT in kern else "conv_tile_kernel[int8]"
    D = kern[dom]
    peak = FP4_MFMA_PEAK_TFLOPS if dom == DOMINANT else INT8_MFMA_PEAK_TOPS
    launch_ms = D["ms"] / D["launches"]
    ops_per_launch = D["ops"] / D["launches"]
    achieved = ops_per_launch / (launch_ms / 1e3) / 1e12
    traffic = measured_traffic() if (dom == DOMINANT and workload == "resnet18_g4_b2") else None
    rp = rocprof_avg_us(workload, dom)
    res = {
        "metric": metric,
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
        "data": "synthetic (seeded random weights and codes, standard-normal fp32 images; "
                "centred conv biases calibrated by the oracle on images %s)" % calib,
        "config": {"workload": cfg_name, "global_batch": n, "image": [spec["hw"], spec["hw"], 3],
                   "groups": spec["groups"], "bits": spec["bits"], "variant": "centred",
                   "tensor_layout": "pixel" if args.pixel_layout else "group (conv outputs)",
                   "step": "palq_forward_image (quantize fp32 input + forward)"},
        "effective_tops": tops,
        "int_ops_per_step": total_ops,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak, "traffic": traffic,
                     "kernel": dom, "launches_per_step": D["launches"],
                     "avg_launch_us": launch_ms * 1e3, "int_ops_per_launch": ops_per_launch,
                     "algorithmic_bytes_per_launch": D["bytes"] / D["launches"],
                     "avg_launch_us_rocprof": rp,
                     "frac_rocprof": (ops_per_launch / (rp * 1e-6) / 1e12 / peak) if rp else None,
                     "timing": "avg_launch_us: HIP events on the library stream in this run; "
                               "avg_launch_us_rocprof: the committed rocprofv3 kernel trace of this "
                               "workload (null once the kernel source has changed)",
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"},
        "kernels": {k: dict(v, avg_launch_us=v["ms"] * 1e3 / v["launches"]) for k, v in kern.items()},
        "timing_pass_ms_per_step": wall_t * 1e3 / args.steps,
        "layers": per_layer,
        "distinct_logits": distinct,
    }
    if not args.no_histograms:
        res["code_histograms"] = code_histograms(ctx, spec, xd, l, u)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(spec, x_f32, l, u, args.cpu_seconds)
    print(json.dumps(res), flush=True)


SINGLE_DESC = {
    "c1": "single PalQuant 3x3 conv, batch 1, 56x56, G=2 x 64->64, 2-bit",
    "c2_l0": "ResNet-18 stage-1 3x3 conv, batch 32, 56x56, G=4 x 64->64, 2-bit",
    "c2_l1": "ResNet-18 stage-2 3x3 conv, batch 32, 28x28, G=4 x 128->128, 2-bit",
    "c2_l2": "ResNet-18 stage-3 3x3 conv, batch 32, 14x14, G=4 x 256->256, 2-bit",
    "c2_l3": "ResNet-18 stage-4 3x3 conv, batch 32, 7x7, G=4 x 512->512, 2-bit",
}


def oracle_layer_time(case, budget_s, single_thread):
    """Wall time per image of the oracle on one layer (C convolution loop +
    numpy epilogue), on whole images of the case's batch until the budget is
    spent.  single_thread: in a child process with OMP_NUM_THREADS=1."""
    import subprocess
    code = (
        "import sys, time, json; sys.path.insert(0, %r)\n"
        "from oracle import oracle as O\n"
        "from paper_2208_01944_amd import inputs as I\n"
        "case = I.single_workload(%r); L = case['layer']; x = case['x']; G = L['w'].shape[0]\n"
        "t0 = time.perf_counter(); done = 0\n"
        "while done < x.shape[0]:\n"
        "    acc = O.group_conv(x[done:done + 1], L['w'], L['stride'], L['pad'])\n"
        "    O.layer_epilogue(acc, G, L['mult'], L['shift'], L['bias'], L['out_bits'], L['shuffle'])\n"
        "    done += 1\n"
        "    if time.perf_counter() - t0 >= %r: break\n"
        "print(json.dumps(dict(images=done, seconds=time.perf_counter() - t0, threads=O.threads())))\n"
    ) % (ROOT, case, budget_s)
    env = dict(os.environ)
    if single_thread:
        env["OMP_NUM_THREADS"] = "1"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    if r.returncode != 0:
        raise RuntimeError(r.stderr[-2000:])
    return json.loads(r.stdout.strip().splitlines()[-1])


def run_single_layers(args, names):
    """One JSON line per single-layer case: the planned layer (palq_conv_run)
    timed over K runs with HIP events on the library's stream, its roofline
    fractions and the oracle's time on the same layer."""
    import torch
    from paper_2208_01944_amd import inputs as I
    from paper_2208_01944_amd import palq
    ctx = palq.Context(0)
    for name in names:
        case = I.single_workload(name)
        L = case["layer"]
        G, co, kh, kw, ci = L["w"].shape
        n, h, w, _ = case["x"].shape
        ho = (h + 2 * L["pad"] - kh) // L["stride"] + 1
        wo = (w + 2 * L["pad"] - kw) // L["stride"] + 1
        bias = I.single_stored_bias(name)
        i32 = lambda a: ctx.upload(np.asarray(a, np.int32))
        x = ctx.pack(case["x"], G, L["in_bits"])
        wt, wf = ctx.pack_filter(L["w"], L["w_bits"])
        out = ctx.empty_act(n, ho, wo, G, co, L["out_bits"])
        plan = palq.ConvPlan(ctx, x, wf, L["stride"], L["pad"], i32(L["mult"]), i32(L["shift"]), i32(bias), out,
                             shuffle=L["shuffle"])
        for _ in range(max(args.warmup, 1)):
            plan.run(x, out)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        ev0.record()
        for _ in range(args.steps):
            plan.run(x, out)
        ev1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        us = ev0.elapsed_time(ev1) * 1e3 / args.steps
        codes = ctx.unpack(out)
        hist = np.bincount(codes.reshape(-1), minlength=1 << L["out_bits"]).tolist()
        macs = n * ho * wo * G * co * kh * kw * ci
        ops = 2 * macs
        nbytes = (n * h * w * G * ci * L["in_bits"] + G * co * kh * kw * ci * L["w_bits"] +
                  n * ho * wo * G * co * L["out_bits"]) / 8 + 12 * G * co
        kern = plan.kernels
        fmt = {DOMINANT: "fp4", "conv_fp6_kernel": "fp6"}.get(kern, "int8")
        fp4 = fmt != "int8"  # FP4 and FP6 share the 10.1 PFLOP/s dense peak
        peak = FP4_MFMA_PEAK_TFLOPS if fp4 else INT8_MFMA_PEAK_TOPS
        tops = ops / (us * 1e-6) / 1e12
        gbs = nbytes / (us * 1e-6) / 1e9
        res = {
            "metric": "effective int TOPS of one PalQuant layer (palq_conv_run)",
            "value": tops, "unit": "TOPS", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": us / 1e3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": fmt,
            "data": "synthetic (seeded uniform codes and weights; centred bias over the batch's interior positions)",
            "config": {"workload": name, "description": SINGLE_DESC.get(name, f"ResNet-18 stage-3 3x3 conv, batch 128, "
                                                                             f"14x14, G={G} x 256->256, {L['in_bits']}-bit"),
                       "batch": n, "groups": G, "bits": L["in_bits"], "ci": ci, "co": co, "hw": h},
            "us_per_launch": us, "wall_us_per_launch": wall * 1e6 / args.steps, "kernel": kern,
            "int_ops": ops, "algorithmic_bytes": nbytes,
            "roofline": {"bound": "mfma", "achieved": tops, "peak": peak, "unit": "TFLOP/s" if fp4 else "TOP/s",
                         "frac": tops / peak, "traffic": None,
                         "hbm_gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS,
                         "arithmetic_intensity": ops / nbytes},
            "code_histogram": hist,
        }
        if not args.no_cpu_baseline:
            nproc, model = host_cpu()
            cb = {}
            for st in (False, True):
                if st and name.startswith("c4_g") and not name.startswith("c4_g1_b2"):
                    continue  # single-thread figures for C1, C2 and the G=1, b=2 sweep cell
                r = oracle_layer_time(name, args.cpu_seconds / 2, st)
                per = r["seconds"] / r["images"]
                cb["single_thread" if st else "all_threads"] = {
                    "value": macs * 2 / n / per / 1e9, "unit": "G int ops/s", "cores": r["threads"],
                    "us_per_batch": per * n * 1e6, "sample": f"{r['images']} of {n} images, {r['seconds']:.1f} s"}
            res["cpu_baseline"] = dict(cb["all_threads"], kind="oracle", nproc=nproc, cpu_model=model,
                                       single_thread=cb.get("single_thread"))
        print(json.dumps(res), flush=True)
        del plan


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1 "
                                   "(a batch-parallel split over GPUs is described in the design notes)"}))
        sys.exit(2)
    if args.summarize_profile:
        if args.workload in NETWORKS:
            summarize_profile(args.summarize_profile, args.workload)
        else:
            summarize_single_profile(args.summarize_profile, args.workload)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.workload)
        return
    if args.hbm_copy_probe:
        copy_probe(args.hbm_copy_probe)
        return
    if args.table2:
        table2(args)
        return
    if args.workload in NETWORKS:
        run_network(args, args.workload)
        return
    from paper_2208_01944_amd import inputs as I
    if args.workload == "layers":
        run_single_layers(args, I.SINGLE_WORKLOADS)
        return
    if args.workload in I.SINGLE_WORKLOADS or args.workload in ("c2", "c4"):
        names = [w for w in I.SINGLE_WORKLOADS if w == args.workload or w.startswith(args.workload + "_")]
        run_single_layers(args, names)
        return
    raise SystemExit(f"unknown workload {args.workload}")


if __name__ == "__main__":
    main()
