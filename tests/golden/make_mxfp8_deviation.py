"""Writes mxfp8_deviation.json: how far the emulated MXFP8 decoder (oracle/fp8.py) lies from the
fp64 oracle on the d7, d11, d17 and d25 networks, per distance the largest and the root-mean-square
logit difference over a seeded sample of windows. The MXFP8 GPU tests derive their tolerances
from these figures. Calls only the oracle (and the seeded input generators).

    python tests/golden/make_mxfp8_deviation.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import decoder as O          # noqa: E402
from oracle import fp8 as MX             # noqa: E402
from paper_2601_09921_amd import synth   # noqa: E402

SAMPLE = {"d7": 96, "d11": 24, "d17": 8, "d25": 6}
SEED = 20260


def main():
    out = {}
    for name, n in SAMPLE.items():
        wl = synth.WORKLOADS[name]
        w = synth.make_weights(wl)
        meas, types = synth.make_windows(wl, seed=SEED, B=n)
        o, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
        e, _ = MX.forward_windows_mx(meas, types, w, wl.d, wl.H)
        dev = np.abs(e - o)
        out[name] = {"windows": n, "seed": SEED, "max": float(dev.max()), "rms": float(np.sqrt(np.mean(dev ** 2))),
                     "mean_abs_logit": float(np.abs(o).mean())}
        print(name, out[name], flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "mxfp8_deviation.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
