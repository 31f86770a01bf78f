"""Helpers shared by the parity tests: per-tensor relative error and the
tolerances of the path (float32: 1e-4 on outputs, 1e-3 on gradients;
bf16 storage with float32 accumulation: 2e-2)."""
import numpy as np

TOL = {"f32": {"out": 1e-4, "grad": 1e-3}, "bf16": {"out": 2e-2, "grad": 2e-2}}


def rel_err(gpu, ref) -> float:
    """max |gpu - ref| / max(max |ref|, 1e-30) over the whole tensor."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    return float(np.abs(gpu - ref).max() / max(np.abs(ref).max(), 1e-30))


def check(name, gpu, ref, tol, report=None):
    e = rel_err(gpu, ref)
    if report is not None:
        report[name] = e
    assert e <= tol, f"{name}: relative error {e:.3e} > {tol:.1e}"
    return e


def compare_lstm(gpu, ref, dtype, with_dx=True, report=None):
    t = TOL[dtype]
    check("loss", np.array([gpu["loss"]]), np.array([ref["loss"]]), t["out"], report)
    for k in ("y", "hT", "cT"):
        check(k, gpu[k], ref[k], t["out"], report)
    for k in ("dh0", "dc0"):
        check(k, gpu[k], ref[k], t["grad"], report)
    for k in ("dWx", "dWh", "db"):
        for l, (g, r) in enumerate(zip(gpu[k], ref[k])):
            check(f"{k}[{l}]", g, r, t["grad"], report)
    if with_dx and "dx" in gpu:
        check("dx", gpu["dx"], ref["dx"], t["grad"], report)
    for k in ("dWout", "dbout", "dE"):
        if k in gpu:
            check(k, gpu[k], ref[k], t["grad"], report)
