"""Write expected values of the full-size regression workload (2 layers,
I = H = 2048, B = 256, T = 256, projection 2048 + MSE, bf16 inputs)
computed by the float64 oracle:

* lm2048_golden.json: 400 sampled entries of every output and gradient;
* lm2048_slices.npz: whole rows and whole columns of dWx[l] and dWh[l]
  (one row from each gate block i, f, g, o and four columns) and all of
  db[l], so an error confined to a few rows or columns of the weight
  gradients after 256 accumulated steps shows up.

    python tests/golden/make_lm2048_golden.py      # about 6-20 minutes, ~25 GiB RAM

Only oracle/ and the seeded input generator are called.  The sample,
row and column indices come from fixed seeds and are stored with the
values (the slices as float32, far below the 2e-2 tolerance they are
checked to).
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
OUT_SLICES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lm2048_slices.npz")
N_SAMPLES = 400
N_COLS = 4


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
    # whole rows (one unit per gate block) and columns of the weight
    # gradients, all of db
    rs = np.random.default_rng(20482)
    H = w.H
    sl = {}
    for k in ("dWx", "dWh"):
        for l in range(w.L):
            a = np.asarray(r[k][l])
            rows = np.array([gate * H + int(rs.integers(0, H)) for gate in range(4)])
            cols = np.sort(rs.choice(a.shape[1], size=N_COLS, replace=False))
            sl[f"{k}{l}_rows"] = rows
            sl[f"{k}{l}_rowvals"] = a[rows].astype(np.float32)
            sl[f"{k}{l}_cols"] = cols
            sl[f"{k}{l}_colvals"] = a[:, cols].astype(np.float32)
            sl[f"{k}{l}_absmax"] = np.array(np.abs(a).max())
    for l in range(w.L):
        sl[f"db{l}"] = np.asarray(r["db"][l]).astype(np.float32)
        sl[f"db{l}_absmax"] = np.array(np.abs(r["db"][l]).max())
    np.savez_compressed(OUT_SLICES, **sl)
    print(f"wrote {OUT} and {OUT_SLICES} in {time.time() - t0:.0f} s; loss {r['loss']:.9g}")


if __name__ == "__main__":
    main()
