"""Writes tests/golden/centred_bias_<workload>.npz: the centred variant's
conv biases of each benchmark network (reading A14 of the design notes:
bias = -round_half_up(mean of the layer's pre-requant value), layer by
layer), calibrated by the CPU oracle on the workload's calibration images;
and tests/golden/centred_bias_single.npz: the centred bias of each
single-layer case, over the whole batch's interior positions (whose window
lies inside the image), as the full-size single-layer tests compute it.

Calls only the oracle and the seeded input generators:

    python tests/golden/make_centred_bias.py [workload ...]

Array "layer<i>" holds layer i's int32 bias (source channel order, as the
layer's requant arrays); "calib_images" the image indices used.
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2208_01944_amd import inputs as I  # noqa: E402

WORKLOADS = ["resnet18_g4_b2", "resnet18_g4_b2_shuffles", "resnet50_g2_b2", "single"]


def single_bias(name):
    case = I.single_workload(name)
    L = case["layer"]
    G = L["w"].shape[0]
    acc = O.group_conv(case["x"], L["w"], L["stride"], L["pad"])
    _, acc_d = O.layer_epilogue(acc, G, L["mult"], L["shift"], None, L["out_bits"], L["shuffle"])
    p = L["pad"] if L["stride"] == 1 else 0
    return O.centring_bias(acc_d[:, p:acc_d.shape[1] - p, p:acc_d.shape[2] - p], G, L["shuffle"])


def calibrate(name):
    spec, x, calib = I.workload(name)
    l, u = I.IMAGE_RANGE
    codes = O.quantize(x[calib], l, u, 8, signed=True)
    return O.calibrate_centring(spec, codes), calib


def main(names):
    for name in names:
        if name == "single":
            path = os.path.join(I.GOLDEN_DIR, "centred_bias_single.npz")
            np.savez_compressed(path, **{n: single_bias(n) for n in I.SINGLE_WORKLOADS})
            print("wrote", path)
            continue
        cen, calib = calibrate(name)
        arrays = {f"layer{i}": np.asarray(L["bias"], np.int32)
                  for i, L in enumerate(cen["layers"]) if L["op"] in ("conv", "shuffle_module")}
        arrays["calib_images"] = np.asarray(calib, np.int32)
        np.savez_compressed(I.centred_path(name), **arrays)
        print("wrote", I.centred_path(name))


if __name__ == "__main__":
    main(sys.argv[1:] or WORKLOADS)
