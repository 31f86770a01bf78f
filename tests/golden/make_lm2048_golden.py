"""Write sampled expected values of the full-size regression workload
(2 layers, I = H = 2048, B = 256, T = 256, projection 2048 + MSE, bf16
inputs) computed by the float64 oracle.

    python tests/golden/make_lm2048_golden.py      # about 10-20 minutes, ~25 GiB RAM

Only oracle/ and the seeded input generator are called.  The sample
indices come from a fixed seed and are stored with the values.
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import steps  # noqa: E402
from paper_1812_01329_amd import workloads as wl  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lm2048_golden.json")
N_SAMPLES = 400


def sample(rng, arr, n=N_SAMPLES):
    arr = np.asarray(arr)
    flat = rng.choice(arr.size, size=min(n, arr.size), replace=False)
    idx = np.stack(np.unravel_index(flat, arr.shape), axis=1)
    return {"shape": list(arr.shape), "index": idx.tolist(), "value": arr.reshape(-1)[flat].tolist(),
            "absmax": float(np.abs(arr).max())}


def main():
    t0 = time.time()
    w = wl.lm2048_lstm()
    r = steps.lstm_step(w)
    rng = np.random.default_rng(20481)
    g = {"workload": "lm2048", "loss": r["loss"], "seconds": time.time() - t0}
    for k in ("y", "hT", "cT", "dh0", "dc0", "dWout", "dbout"):
        g[k] = sample(rng, r[k])
    for k in ("dWx", "dWh", "db"):
        for l in range(w.L):
            g[f"{k}[{l}]"] = sample(rng, r[k][l])
    with open(OUT, "w") as f:
        json.dump(g, f)
    print(f"wrote {OUT} in {time.time() - t0:.0f} s; loss {r['loss']:.9g}")


if __name__ == "__main__":
    main()
