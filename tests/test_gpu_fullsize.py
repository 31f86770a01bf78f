"""GPU parity at the full regression size (2 layers, input = hidden = 2048,
batch 256, length 256, projection 2048 + MSE, bf16 storage with float32
accumulation), in the launch configuration the benchmark times.

Three independent checks:
  * sampled elements of every output and gradient against values the
    float64 oracle wrote for the whole batch (tests/golden/lm2048_golden.json,
    written by tests/golden/make_lm2048_golden.py);
  * whole rows (one per gate block) and whole columns of the weight
    gradients dWx[l], dWh[l], and all of db[l], element by element, against
    the same oracle run (tests/golden/lm2048_slices.npz, same script): an
    error confined to a few rows or columns after 256 accumulated steps
    would slip past the samples;
  * whole rows of the per-sequence outputs (y, hT, cT, dh0, dc0) for a few
    sequences against the oracle run on just those sequences, which gives
    the same values because every per-sequence output depends only on its
    own sequence.
Errors are relative to the largest magnitude of the whole tensor, as in the
smaller parity tests."""
import json
import os

import numpy as np
import pytest

from oracle import steps as oracle_steps
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "lm2048_golden.json")
SLICES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "lm2048_slices.npz")


@pytest.fixture(scope="module")
def full_step():
    import torch
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    os.environ.pop("JANUS_PERSIST", None)
    print("[fullsize] lm2048 T=256 B=256 H=2048 I=2048 P=2048 bf16", flush=True)
    w = wl.lm2048_lstm()
    step = make_step(w)
    step.run()
    g = step.results()
    from paper_1812_01329_amd import janus as J
    rep = J.janus_lstm_device_report(step.desc, step.ws)   # raises if a barrier wait ran out
    print(f"[fullsize] device report {rep}", flush=True)
    return w, g


def _gpu_tensor(g, key):
    if "[" in key:
        name, l = key[:-1].split("[")
        return g[name][int(l)]
    return g[key]


def test_sampled_against_full_batch_oracle(full_step):
    w, g = full_step
    gold = json.load(open(GOLDEN))
    t = TOL["bf16"]
    check("loss", np.array([g["loss"]]), np.array([gold["loss"]]), t["out"])
    for key, rec in gold.items():
        if not isinstance(rec, dict):
            continue
        arr = _gpu_tensor(g, key)
        assert list(arr.shape) == rec["shape"], key
        idx = tuple(np.asarray(rec["index"]).T)
        got = arr[idx]
        ref = np.asarray(rec["value"])
        err = np.abs(got - ref).max() / max(rec["absmax"], 1e-30)
        tol = t["out"] if key in ("y", "hT", "cT") else t["grad"]
        assert err <= tol, f"{key}: sampled relative error {err:.3e} > {tol:.1e}"
        # the tensor's own scale agrees with the oracle's
        amax = float(np.abs(arr).max())
        assert abs(amax - rec["absmax"]) <= tol * rec["absmax"] + 1e-30, (key, amax, rec["absmax"])


def test_weight_gradient_rows_and_columns(full_step):
    w, g = full_step
    gold = np.load(SLICES, allow_pickle=False)
    t = TOL["bf16"]["grad"]
    for k in ("dWx", "dWh"):
        for l in range(w.L):
            got = g[k][l]
            scale = float(gold[f"{k}{l}_absmax"])
            rows, cols = gold[f"{k}{l}_rows"], gold[f"{k}{l}_cols"]
            for name, a, ref in ((f"{k}[{l}] rows {rows.tolist()}", got[rows], gold[f"{k}{l}_rowvals"]),
                                 (f"{k}[{l}] cols {cols.tolist()}", got[:, cols], gold[f"{k}{l}_colvals"])):
                assert a.shape == ref.shape, name
                err = np.abs(a - ref.astype(np.float64)).max() / max(scale, 1e-30)
                print(f"[fullsize] {name}: relative error {err:.3e}", flush=True)
                assert err <= t, f"{name}: relative error {err:.3e} > {t:.1e}"
    for l in range(w.L):
        check(f"db[{l}] (all)", g["db"][l], gold[f"db{l}"].astype(np.float64), t)


def test_whole_sequences_against_oracle(full_step):
    w, g = full_step
    rows = np.array([0, 97, 255])
    r = oracle_steps.lstm_step(w, batch_rows=rows)
    t = TOL["bf16"]
    check("y", g["y"][:, rows], r["y"], t["out"])
    check("hT", g["hT"][:, rows], r["hT"], t["out"])
    check("cT", g["cT"][:, rows], r["cT"], t["out"])
    check("dh0", g["dh0"][:, rows], r["dh0"], t["grad"])
    check("dc0", g["dc0"][:, rows], r["dc0"], t["grad"])
