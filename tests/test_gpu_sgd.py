"""GPU parity of the parameter update (janus_sgd_clip_update) against the
float64 oracle (oracle/sgd.py) on seeded parameters and gradients.

Tolerances: the norm is summed in float64 on the device and returned as
float32, so it matches to float32 precision.  The update is computed in
float32: a parameter is within 2^-22 (|p| + |lr s g|) of the float64 value
from the float32 operations (the product, lr s rounded to float32), plus
the rounding of the result: 2 float32 ulp, or one bf16 ulp for a bf16
parameter (the float32 result rounded to nearest even)."""
import math

import numpy as np
import pytest

from oracle import sgd as osgd
from paper_1812_01329_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _dev(a, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.cuda()


def _host(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def _run(params, grads, dtype, lr, max_norm, views=None):
    """Runs the update on device copies; returns (new params, stats)."""
    import torch
    from paper_1812_01329_amd import janus as J
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dt = J.BF16 if dtype == "bf16" else J.F32
    P = [_dev(p.ravel(), dtype) for p in params]
    G = [_dev(g.ravel(), "f32") for g in grads]
    if views:   # unaligned starts: the same data one element into a larger buffer
        for i in views:
            bp = torch.zeros(P[i].numel() + 1, dtype=P[i].dtype, device="cuda")
            bg = torch.zeros(G[i].numel() + 3, dtype=torch.float32, device="cuda")
            bp[1:].copy_(P[i])
            bg[3:].copy_(G[i])
            P[i], G[i] = bp[1:], bg[3:]
    d = J.SgdDesc(len(P), dt, lr, max_norm)
    ws = torch.empty(J.sgd_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    stats = torch.full((2,), -1.0, dtype=torch.float32, device="cuda")
    print(f"[sgd] n={len(P)} dtype={dtype} lr={lr} max_norm={max_norm} sizes={[p.numel() for p in P][:6]}",
          flush=True)
    J.janus_sgd_clip_update(d, P, G, stats=stats, ws=ws)
    torch.cuda.synchronize()
    return [_host(p) for p in P], _host(stats)


def _inputs(seed, shapes, dtype, gscale=1.0):
    rng = np.random.default_rng(seed)
    P = [rng.uniform(-1, 1, s).astype(np.float32) for s in shapes]
    if dtype == "bf16":
        P = [wl.bf16_round(p) for p in P]
    G = [(gscale * rng.normal(0, 1, s)).astype(np.float32) for s in shapes]
    return P, G


def _check(new, ref, P, G, dtype, lr, s):
    for k, o, p, g in zip(new, ref, P, G):
        k = k.reshape(o.shape)
        err = np.abs(k - o)
        mag = np.maximum(np.abs(k), np.abs(o))
        step = np.abs(lr * s * g.astype(np.float64)).reshape(o.shape)
        pin = np.abs(p.astype(np.float64)).reshape(o.shape)
        # float32 arithmetic on the operands (products, lr s rounded to float32)
        f32 = 2.0 ** -22 * (pin + step)
        if dtype == "bf16":
            bound = np.exp2(np.floor(np.log2(np.maximum(mag, 1e-30))) - 7) + f32
        else:
            bound = 2.0 * np.spacing(mag.astype(np.float32)).astype(np.float64) + f32
        assert np.all(err <= bound + 1e-30), (float(err.max()), float((err - bound).max()))


SHAPES = [(512, 64), (33,), (0,), (7, 5, 3), (1,), (4096,), (1000, 3)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("gscale,max_norm", [(1.0, 1.0), (0.001, 5.0), (1.0, 0.0), (1.0, math.inf)])
def test_update_matches_oracle(dtype, gscale, max_norm):
    P, G = _inputs(41, SHAPES, dtype, gscale)
    lr = 0.125
    new, stats = _run(P, G, dtype, lr, max_norm)
    ref, norm, s, applied = osgd.sgd_clip_update(P, G, lr, max_norm)
    assert applied
    assert stats[0] == pytest.approx(norm, rel=2e-7)
    assert stats[1] == pytest.approx(s, rel=2e-7)
    _check(new, ref, P, G, dtype, lr, s)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_views_and_many_tensors(dtype):
    """Starts not on a 16-byte boundary (scalar path for the parameters,
    vector path for the gradients after a head), and 130 tensors: three
    tables, whose block sums are added in order."""
    rng = np.random.default_rng(43)
    shapes = [(int(n),) for n in rng.integers(0, 3000, 130)]
    P, G = _inputs(44, shapes, dtype, 0.05)
    lr, max_norm = 0.5, 2.0
    new, stats = _run(P, G, dtype, lr, max_norm, views=[0, 5, 64, 129])
    ref, norm, s, _ = osgd.sgd_clip_update(P, G, lr, max_norm)
    assert stats[0] == pytest.approx(norm, rel=2e-7)
    _check(new, ref, P, G, dtype, lr, s)


@pytest.mark.parametrize("bad", [math.nan, math.inf])
def test_non_finite_gradient_leaves_parameters(bad):
    P, G = _inputs(45, SHAPES, "bf16")
    G[5] = G[5].copy()
    G[5][1234] = bad
    new, stats = _run(P, G, "bf16", 0.1, 1.0)
    assert not math.isfinite(stats[0]) and stats[1] == 0.0
    for k, p in zip(new, P):
        assert np.array_equal(k.reshape(p.shape), p.astype(np.float64))


def test_repeated_calls_identical():
    P, G = _inputs(46, SHAPES, "f32", 3.0)
    a, sa = _run(P, G, "f32", 0.01, 1.0)
    b, sb = _run(P, G, "f32", 0.01, 1.0)
    assert np.array_equal(sa, sb)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_full_size_parameter_set():
    """The parameters of the 2-layer, H = I = 2048 language model with its
    2048-wide projection (71.3 M entries, bf16) in one call, against the
    oracle on every entry."""
    H = I = P_ = 2048
    shapes = [(4 * H, I), (4 * H, H), (4 * H,), (4 * H, H), (4 * H, H), (4 * H,), (P_, H), (P_,)]
    P, G = _inputs(47, shapes, "bf16", 1e-3)
    lr, max_norm = 0.1, 5.0
    new, stats = _run(P, G, "bf16", lr, max_norm)
    ref, norm, s, _ = osgd.sgd_clip_update(P, G, lr, max_norm)
    assert s < 1.0   # the clipping is active at this scale
    assert stats[0] == pytest.approx(norm, rel=2e-7)
    _check(new, ref, P, G, "bf16", lr, s)


@pytest.mark.parametrize("max_norm", [1e-3, 0.0])
def test_training_step_with_update(max_norm):
    """One float32 LSTM language-model step (embedding, 2 layers, softmax
    cross-entropy) followed by the update, against the oracle's gradients and
    the oracle's update of the same initial parameters.  The device step's
    gradients match the oracle's to the step tolerance, so the parameter
    change is compared relative to its own size."""
    import torch
    from oracle import steps as osteps
    from paper_1812_01329_amd.train_step import make_step
    from tests.test_gpu_parity import _lstm
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w = _lstm("xent", "f32", L=2, I=16, H=32, B=8, T=6, seed=48, V=50)
    lr = 0.5
    print(f"[sgd-step] {w.name} max_norm={max_norm}", flush=True)
    step = make_step(w, update=(lr, max_norm))
    P0 = [_host(p) for p in step.parameters()[0]]
    step.run()
    torch.cuda.synchronize()
    P1 = [_host(p) for p in step.parameters()[0]]
    r = osteps.lstm_step(w)
    G = []
    for l in range(w.L):
        G += [r["dWx"][l], r["dWh"][l], r["db"][l]]
    G += [r["dWout"], r["dbout"], r["dE"]]
    ref, norm, s, applied = osgd.sgd_clip_update(P0, G, lr, max_norm)
    stats = _host(step.update.stats)
    assert applied
    assert stats[0] == pytest.approx(norm, rel=1e-3)
    if max_norm > 0:
        assert s < 1.0
    d_gpu = np.concatenate([(b - a).ravel() for a, b in zip(P0, P1)])
    d_ref = np.concatenate([(b - a).ravel() for a, b in zip(P0, ref)])
    assert np.linalg.norm(d_gpu - d_ref) <= 1e-3 * np.linalg.norm(d_ref)


def test_step_with_timed_out_recurrence_leaves_parameters(monkeypatch):
    """All-or-nothing state change (Section 4.2.3): when a bounded wait of
    the step's recurrences runs out, the update writes no parameter and the
    report says so after the backward.  The timeout is forced from the host
    by setting the workspace's timeout word between the forward and the
    backward call (every wait of the backward's persistent kernels then
    returns at once, so they drain normally).  A clean step before and after
    shows that the report covers the forward on its own too, and that the
    next forward clears the word."""
    import torch
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd.train_step import make_step
    from tests.test_gpu_parity import _lstm
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    # bf16, H = 1024, B = 64: the persistent forward (asked for in two
    # slices, so that it reports its unit groups) and backward kernels
    monkeypatch.setenv("JANUS_FWD_SLICES", "2")
    w = _lstm("mse", "bf16", L=2, I=64, H=1024, B=64, T=5, seed=52, P=16)
    print(f"[sgd-hold] {w.name}", flush=True)
    step = make_step(w, update=(0.5, 0.0))
    fwd_reports = []
    orig_bwd = J.janus_lstm_seq_bwd
    force = {"on": False}

    def bwd(*args, **kw):
        fwd_reports.append(J.janus_lstm_device_report(step.desc, step.ws))   # the forward's report
        if force["on"]:
            off = step.fault - step.ws.data_ptr()
            assert 0 <= off <= step.ws.numel() - 4
            step.ws[off:off + 4].copy_(torch.tensor([1, 0, 0, 0], dtype=torch.uint8))
        return orig_bwd(*args, **kw)

    monkeypatch.setattr(J, "janus_lstm_seq_bwd", bwd)
    # a clean step: the forward and the whole step report no timeout, and the update applies
    P0 = [_host(p) for p in step.parameters()[0]]
    step.run()
    rep = J.janus_lstm_device_report(step.desc, step.ws)
    assert fwd_reports[-1]["timed_out"] == 0 and fwd_reports[-1]["fwd_groups"] > 0
    assert rep["timed_out"] == 0 and rep["bwd_groups"] > 0
    P1 = [_host(p) for p in step.parameters()[0]]
    assert any(not np.array_equal(a, b) for a, b in zip(P0, P1))
    # the forced timeout: no parameter changes, the scale reads 0, the report raises
    force["on"] = True
    step.run()
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_device_report(step.desc, step.ws)
    assert e.value.status == J.ERR_DEVICE
    P2 = [_host(p) for p in step.parameters()[0]]
    for a, b in zip(P1, P2):
        assert np.array_equal(a, b)
    assert _host(step.update.stats)[1] == 0.0
    # the next step's forward clears the word: clean again, and it updates
    force["on"] = False
    step.run()
    assert J.janus_lstm_device_report(step.desc, step.ws)["timed_out"] == 0
    P3 = [_host(p) for p in step.parameters()[0]]
    assert any(not np.array_equal(a, b) for a, b in zip(P2, P3))


def test_held_update_writes_nothing():
    """janus_sgd_clip_update with a non-zero hold word writes no parameter
    and reports scale 0; with a zero word it matches the oracle."""
    import torch
    from paper_1812_01329_amd import janus as J
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    params, grads = _inputs(71, [(33,), (5, 7)], "f32")
    P = [_dev(p.ravel(), "f32") for p in params]
    G = [_dev(g.ravel(), "f32") for g in grads]
    d = J.SgdDesc(len(P), J.F32, 0.3, 0.0)
    ws = torch.empty(J.sgd_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    stats = torch.full((2,), -1.0, dtype=torch.float32, device="cuda")
    hold = torch.ones(1, dtype=torch.int32, device="cuda")
    print("[sgd-held] hold=1 then hold=0", flush=True)
    J.janus_sgd_clip_update(d, P, G, stats=stats, ws=ws, hold=hold.data_ptr())
    torch.cuda.synchronize()
    for p, ref in zip(P, params):
        assert np.array_equal(_host(p), np.asarray(ref, np.float32).ravel())
    assert _host(stats)[1] == 0.0
    hold.zero_()
    J.janus_sgd_clip_update(d, P, G, stats=stats, ws=ws, hold=hold.data_ptr())
    torch.cuda.synchronize()
    ref, norm, s, applied = osgd.sgd_clip_update(params, grads, 0.3, 0.0)
    assert applied and _host(stats)[1] == 1.0
    _check([_host(p) for p in P], ref, params, grads, "f32", 0.3, s)
