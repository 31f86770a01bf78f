"""GPU parity of a stream of batches whose recurrent state carries over
(janus_lstm_state_carry, Figure 1's self.state), with a smaller last batch,
against the oracle running the same batches with its own carried state; and
the device's split-call identity (T1 steps, carry, T2 steps = one call of
T1 + T2 steps)."""
import numpy as np
import pytest

from oracle import lstm as olstm
from oracle import steps as osteps
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check, compare_lstm

pytestmark = pytest.mark.gpu


def _batches(dtype, L, I, H, T, Bs, P, seed, lengths=False):
    """Workloads sharing one set of parameters, with their own data."""
    rng = np.random.default_rng(seed)
    a = 1.0 / np.sqrt(H)
    r = (lambda v: wl.bf16_round(v.astype(np.float32))) if dtype == "bf16" else (lambda v: v.astype(np.float32))
    Wx = [r(rng.uniform(-a, a, (4 * H, I if l == 0 else H))) for l in range(L)]
    Wh = [r(rng.uniform(-a, a, (4 * H, H))) for l in range(L)]
    b = [r(rng.uniform(-a, a, (4 * H,))) for l in range(L)]
    Wout, bout = r(rng.uniform(-a, a, (P, H))), r(rng.uniform(-a, a, (P,)))
    out = []
    for k, B in enumerate(Bs):
        x = r(rng.normal(0, 1, (T, B, I)))
        lens = rng.integers(0, T + 1, B).astype(np.int32) if lengths else None
        w = wl.LSTMWorkload(f"stream{k}-{dtype}-B{B}", dtype, L, I, H, B, T, x, lens, Wx, Wh, b, "mse")
        w.Wout, w.bout, w.target = Wout, bout, r(rng.normal(0, 1, (T, B, P)))
        out.append(w)
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("lengths", [False, True])
def test_stream_with_ragged_last_batch(dtype, lengths):
    import torch
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ws = _batches(dtype, L=2, I=32, H=64, T=8, Bs=[64, 64, 40], P=24, seed=61, lengths=lengths)
    prev, hT, cT = None, None, None
    for k, w in enumerate(ws):
        print(f"[state] batch {k} B={w.B} dtype={dtype} lengths={lengths}", flush=True)
        step = make_step(w)
        if prev is not None:
            step.carry_from(prev)
        step.run()
        g = step.results()
        wo = _batches(dtype, L=2, I=32, H=64, T=8, Bs=[64, 64, 40], P=24, seed=61, lengths=lengths)[k]
        wo.h0, wo.c0 = olstm.carry_state(hT, cT, w.B)
        r = osteps.lstm_step(wo)
        compare_lstm(g, r, dtype, with_dx=False)
        hT, cT = r["hT"], r["cT"]
        prev = step


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_split_call_equals_one_call(dtype):
    """On the device alone: the state carry loses nothing.  Rounding may
    differ only where the input projection of the shorter call is
    partitioned differently, far inside the output tolerance."""
    import torch
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    T1, T2 = 6, 5
    (w,) = _batches(dtype, L=2, I=32, H=64, T=T1 + T2, Bs=[48], P=24, seed=62)
    parts = []
    for lo, hi in ((0, T1), (T1, T1 + T2)):
        v = wl.LSTMWorkload(f"part{lo}", dtype, w.L, w.I, w.H, w.B, hi - lo, w.x[lo:hi], None, w.Wx, w.Wh, w.b,
                            "mse")
        v.Wout, v.bout, v.target = w.Wout, w.bout, w.target[lo:hi]
        parts.append(v)
    print(f"[state] split {T1}+{T2} dtype={dtype}", flush=True)
    whole = make_step(w)
    whole.run()
    g = whole.results()
    s1 = make_step(parts[0])
    s1.run()
    s2 = make_step(parts[1])
    s2.carry_from(s1)
    s2.run()
    g1, g2 = s1.results(), s2.results()
    tol = 1e-6 if dtype == "f32" else 1e-2
    check("y", np.concatenate([g1["y"], g2["y"]]), g["y"], tol)
    check("hT", g2["hT"], g["hT"], tol)
    check("cT", g2["cT"], g["cT"], tol)
