"""Pins of the LSTM oracle against facts that do not come from the oracle:
finite differences, closed forms, torch.nn.LSTM in float64, and invariants."""
import copy

import numpy as np
import pytest
import torch

from oracle import heads, lstm, steps
from paper_1812_01329_amd import workloads as wl


def small_lstm(head, L=2, I=3, H=4, B=3, T=5, lengths=None, seed=0, V=7, P=3, h0=False):
    rng = np.random.default_rng(seed)
    Wx = [rng.uniform(-0.6, 0.6, (4 * H, I if l == 0 else H)) for l in range(L)]
    Wh = [rng.uniform(-0.6, 0.6, (4 * H, H)) for l in range(L)]
    b = [rng.uniform(-0.6, 0.6, 4 * H) for l in range(L)]
    w = wl.LSTMWorkload("t", wl.F32, L, I, H, B, T, rng.standard_normal((T, B, I)),
                        None if lengths is None else np.asarray(lengths, np.int32),
                        Wx, Wh, b, head)
    if head == "xent":
        w.V = V
        w.tokens = rng.integers(0, V, (B, T + 1)).astype(np.int32)
        w.E = rng.uniform(-1, 1, (V, I))
        w.Wout = rng.uniform(-1, 1, (V, H))
        w.bout = rng.uniform(-1, 1, V)
    if head == "mse":
        w.Wout = rng.uniform(-1, 1, (P, H))
        w.bout = rng.uniform(-1, 1, P)
        w.target = rng.standard_normal((T, B, P))
    if h0:
        w.h0 = rng.uniform(-0.5, 0.5, (L, B, H))
        w.c0 = rng.uniform(-0.5, 0.5, (L, B, H))
    return w


def fd_check(w, getter_names, grad_of, eps=1e-5, tol=1e-6):
    """Central differences of the loss wrt every element of the named
    workload arrays, compared with the oracle's analytic gradient."""
    base = steps.lstm_step(w)
    for name in getter_names:
        arr_list, idx = name
        arr = getattr(w, arr_list)
        target = arr[idx] if idx is not None else arr
        an = np.asarray(grad_of(base, arr_list, idx), dtype=np.float64)
        fd = np.zeros(target.shape)
        flat = target.reshape(-1)
        for k in range(flat.size):
            old = flat[k]
            flat[k] = old + eps
            lp = steps.lstm_step(w)["loss"]
            flat[k] = old - eps
            lm = steps.lstm_step(w)["loss"]
            flat[k] = old
            fd.reshape(-1)[k] = (lp - lm) / (2 * eps)
        err = np.abs(fd - an).max() / max(np.abs(an).max(), 1e-30)
        assert err < tol, (name, err)


def _grad(base, arr, idx):
    return {"Wx": lambda: base["dWx"][idx], "Wh": lambda: base["dWh"][idx],
            "b": lambda: base["db"][idx], "x": lambda: base["dx"],
            "h0": lambda: base["dh0"], "c0": lambda: base["dc0"],
            "Wout": lambda: base["dWout"], "bout": lambda: base["dbout"],
            "E": lambda: base["dE"]}[arr]()


@pytest.mark.parametrize("head", ["sumsq", "mean_final", "mse", "xent"])
@pytest.mark.parametrize("lengths", [None, [5, 2, 0], [3, 5, 1]])
def test_finite_differences(head, lengths):
    w = small_lstm(head, lengths=lengths, h0=(head != "xent"))
    names = [("Wx", 0), ("Wx", 1), ("Wh", 0), ("Wh", 1), ("b", 0), ("b", 1)]
    if head == "xent":
        names += [("E", None), ("Wout", None), ("bout", None)]
    else:
        names += [("x", None), ("h0", None), ("c0", None)]
    if head == "mse":
        names += [("Wout", None), ("bout", None)]
    fd_check(w, names, _grad)


def test_closed_form_constant_gates():
    """W = 0 and a bias per gate block: the gates are constants
    i = s(bi), f = s(bf), g = tanh(bg), o = s(bo), so
    c_t = i g (1 - f^t) / (1 - f) and h_t = o tanh(c_t)."""
    T, B, I, H = 7, 2, 3, 5
    bi, bf, bg, bo = 0.3, -0.7, 1.1, 0.4
    b = np.concatenate([np.full(H, v) for v in (bi, bf, bg, bo)])
    x = np.random.default_rng(1).standard_normal((T, B, I))
    y, hT, cT, _ = lstm.layer_forward(x, None, np.zeros((4 * H, I)), np.zeros((4 * H, H)), b)
    s = lambda z: 1 / (1 + np.exp(-z))
    i, f, g, o = s(bi), s(bf), np.tanh(bg), s(bo)
    for t in range(1, T + 1):
        c = i * g * (1 - f ** t) / (1 - f)
        np.testing.assert_allclose(y[t - 1], np.full((B, H), o * np.tanh(c)), rtol=0, atol=1e-14)
    np.testing.assert_allclose(cT, i * g * (1 - f ** T) / (1 - f), atol=1e-14)
    # closed form: only b_g nonzero -> c_t = tanh(b)(1 - 2^-t)
    b2 = np.zeros(4 * H); b2[2 * H:3 * H] = 0.9
    _, _, c2, _ = lstm.layer_forward(x, None, np.zeros((4 * H, I)), np.zeros((4 * H, H)), b2)
    np.testing.assert_allclose(c2, np.tanh(0.9) * (1 - 2.0 ** -T), atol=1e-14)


def _torch_lstm(w):
    """torch.nn.LSTM in float64 on the CPU with packed variable lengths."""
    lstm_t = torch.nn.LSTM(w.I, w.H, num_layers=w.L, dtype=torch.float64)
    with torch.no_grad():
        for l in range(w.L):
            getattr(lstm_t, f"weight_ih_l{l}").copy_(torch.tensor(w.Wx[l]))
            getattr(lstm_t, f"weight_hh_l{l}").copy_(torch.tensor(w.Wh[l]))
            getattr(lstm_t, f"bias_ih_l{l}").copy_(torch.tensor(w.b[l]))
            getattr(lstm_t, f"bias_hh_l{l}").zero_()
    x = torch.tensor(np.asarray(w.x, np.float64), requires_grad=True)
    lengths = np.full(w.B, w.T) if w.lengths is None else np.asarray(w.lengths)
    packed = torch.nn.utils.rnn.pack_padded_sequence(x, torch.tensor(lengths), enforce_sorted=False)
    h0 = torch.tensor(w.h0, requires_grad=True) if w.h0 is not None else None
    c0 = torch.tensor(w.c0, requires_grad=True) if w.c0 is not None else None
    out, (hn, cn) = lstm_t(packed, None if h0 is None else (h0, c0))
    y, _ = torch.nn.utils.rnn.pad_packed_sequence(out, total_length=w.T)
    return lstm_t, x, h0, c0, y, hn, cn


@pytest.mark.parametrize("lengths", [None, [6, 1, 4, 6], [2, 2, 5, 3]])
def test_against_torch_lstm(lengths):
    w = small_lstm("sumsq", L=2, I=5, H=6, B=4, T=6, lengths=lengths, seed=3, h0=True)
    ref = steps.lstm_step(w)
    lstm_t, x, h0, c0, y, hn, cn = _torch_lstm(w)
    np.testing.assert_allclose(ref["y"], y.detach().numpy(), atol=1e-13)
    np.testing.assert_allclose(ref["hT"], hn.detach().numpy(), atol=1e-13)
    np.testing.assert_allclose(ref["cT"], cn.detach().numpy(), atol=1e-13)
    loss = (hn[-1] ** 2).sum()
    loss.backward()
    np.testing.assert_allclose(ref["loss"], loss.item(), rtol=1e-13)
    np.testing.assert_allclose(ref["dx"], x.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(ref["dh0"], h0.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(ref["dc0"], c0.grad.numpy(), atol=1e-12)
    for l in range(w.L):
        np.testing.assert_allclose(ref["dWx"][l], getattr(lstm_t, f"weight_ih_l{l}").grad.numpy(), atol=1e-12)
        np.testing.assert_allclose(ref["dWh"][l], getattr(lstm_t, f"weight_hh_l{l}").grad.numpy(), atol=1e-12)
        np.testing.assert_allclose(ref["db"][l], getattr(lstm_t, f"bias_ih_l{l}").grad.numpy(), atol=1e-12)


def test_torch_mse_and_xent_heads():
    rng = np.random.default_rng(5)
    R, H, V = 9, 4, 6
    h = rng.standard_normal((R, H)); W = rng.standard_normal((V, H)); b = rng.standard_normal(V)
    tgt = rng.integers(0, V, R)
    loss, dh, dW, db, _ = heads.softmax_xent(h, W, b, tgt)
    ht, Wt, bt = (torch.tensor(a, requires_grad=True) for a in (h, W, b))
    lt = torch.nn.functional.cross_entropy(ht @ Wt.T + bt, torch.tensor(tgt))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13
    for a, t in ((dh, ht), (dW, Wt), (db, bt)):
        np.testing.assert_allclose(a, t.grad.numpy(), atol=1e-14)
    tg = rng.standard_normal((R, V))
    loss, dh, dW, db, _ = heads.linear_mse(h, W, b, tg)
    ht, Wt, bt = (torch.tensor(a, requires_grad=True) for a in (h, W, b))
    lt = torch.nn.functional.mse_loss(ht @ Wt.T + bt, torch.tensor(tg))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13
    for a, t in ((dh, ht), (dW, Wt), (db, bt)):
        np.testing.assert_allclose(a, t.grad.numpy(), atol=1e-14)


def test_head_closed_forms():
    """W = 0, b = 0: cross-entropy is ln V exactly with dlogits = (1/V - onehot)/R;
    MSE is mean(target^2)."""
    R, H, V = 5, 3, 11
    rng = np.random.default_rng(2)
    h = rng.standard_normal((R, H))
    tgt = rng.integers(0, V, R)
    loss, dh, dW, db, _ = heads.softmax_xent(h, np.zeros((V, H)), np.zeros(V), tgt)
    assert abs(loss - np.log(V)) < 1e-15
    onehot = np.eye(V)[tgt]
    np.testing.assert_allclose(db, ((1.0 / V) - onehot).sum(0) / R, atol=1e-16)
    np.testing.assert_allclose(dW, ((1.0 / V - onehot).T @ h) / R, atol=1e-15)
    assert np.all(dh == 0)
    tg = rng.standard_normal((R, 4))
    loss, *_ = heads.linear_mse(h, np.zeros((4, H)), np.zeros(4), tg)
    assert abs(loss - np.mean(tg ** 2)) < 1e-15


def test_embedding_backward_against_add_at():
    rng = np.random.default_rng(4)
    ids = rng.integers(0, 6, 40)
    dx = rng.standard_normal((40, 3))
    ref = np.zeros((6, 3))
    np.add.at(ref, ids, dx)
    np.testing.assert_allclose(heads.embed_backward(6, dx, ids), ref, atol=1e-14)


def test_length_zero_returns_initial_state():
    w = small_lstm("sumsq", lengths=[0, 0, 0], h0=True)
    ref = steps.lstm_step(w)
    assert np.array_equal(ref["hT"], w.h0) and np.array_equal(ref["cT"], w.c0)
    assert np.all(ref["y"] == 0)
    # mixed: the zero-length row keeps its initial state, the others move
    w = small_lstm("sumsq", lengths=[5, 0, 2], h0=True)
    ref = steps.lstm_step(w)
    assert np.array_equal(ref["hT"][:, 1], w.h0[:, 1])
    assert not np.allclose(ref["hT"][:, 0], w.h0[:, 0])


def test_all_lengths_T_equals_unmasked():
    w1 = small_lstm("mse", lengths=None, h0=True)
    w2 = copy.deepcopy(w1)
    w2.lengths = np.full(w2.B, w2.T, np.int32)
    r1, r2 = steps.lstm_step(w1), steps.lstm_step(w2)
    for k in ("y", "hT", "cT", "dx", "dh0"):
        assert np.array_equal(r1[k], r2[k]), k


def test_batch_permutation_invariance():
    w = small_lstm("mse", lengths=[5, 2, 4], h0=True)
    ref = steps.lstm_step(w)
    p = np.array([2, 0, 1])
    wp = copy.deepcopy(w)
    wp.x = w.x[:, p]; wp.lengths = w.lengths[p]; wp.target = w.target[:, p]
    wp.h0 = w.h0[:, p]; wp.c0 = w.c0[:, p]
    rp = steps.lstm_step(wp)
    np.testing.assert_allclose(rp["y"], ref["y"][:, p], atol=1e-15)
    np.testing.assert_allclose(rp["dx"], ref["dx"][:, p], atol=1e-15)
    assert abs(rp["loss"] - ref["loss"]) < 1e-14
    for l in range(w.L):
        np.testing.assert_allclose(rp["dWh"][l], ref["dWh"][l], atol=1e-13)


def test_T1_is_one_cell_step_elementwise():
    """T = 1: a plain elementwise evaluation of the cell equations."""
    w = small_lstm("sumsq", L=1, T=1, h0=True)
    ref = steps.lstm_step(w)
    H = w.H
    for bi in range(w.B):
        for j in range(H):
            a = [w.b[0][g * H + j] + sum(w.Wx[0][g * H + j, k] * w.x[0, bi, k] for k in range(w.I))
                 + sum(w.Wh[0][g * H + j, k] * w.h0[0, bi, k] for k in range(H)) for g in range(4)]
            s = [1 / (1 + np.exp(-a[0])), 1 / (1 + np.exp(-a[1])), np.tanh(a[2]), 1 / (1 + np.exp(-a[3]))]
            c = s[1] * w.c0[0, bi, j] + s[0] * s[2]
            assert abs(ref["cT"][0, bi, j] - c) < 1e-14
            assert abs(ref["hT"][0, bi, j] - s[3] * np.tanh(c)) < 1e-14


def test_subset_rows_reproduce_full_batch_values():
    w = small_lstm("mse", lengths=[5, 2, 4], h0=True)
    full = steps.lstm_step(w)
    sub = steps.lstm_step(w, batch_rows=[2])
    np.testing.assert_allclose(sub["y"][:, 0], full["y"][:, 2], atol=1e-15)
    np.testing.assert_allclose(sub["dx"][:, 0], full["dx"][:, 2], atol=1e-15)
    np.testing.assert_allclose(sub["dh0"][:, 0], full["dh0"][:, 2], atol=1e-15)


@pytest.mark.parametrize("lengths", [None, [6, 1, 4, 6], [3, 0, 5, 2]])
def test_mean_final_loss_against_torch_lstm(lengths):
    """The variable-length workload's loss is the mean of the final h over
    B * H entries: torch.nn.LSTM with packed lengths, hn[-1].mean(), and
    autograd fix both its value and every gradient, so a wrong normalisation
    (1/B instead of 1/(B H), say) shows up here even though finite
    differences of the oracle would follow it."""
    w = small_lstm("mean_final", L=1, I=5, H=6, B=4, T=6, lengths=lengths, seed=11, h0=True)
    if lengths is not None and 0 in lengths:
        # torch's packed sequences reject length 0: run torch on the other
        # rows and rescale; a length-0 row keeps h0 (tested elsewhere)
        keep = [b for b in range(w.B) if lengths[b] > 0]
        sub = copy.deepcopy(w)
        sub.B = len(keep)
        sub.x = np.asarray(w.x)[:, keep]
        sub.lengths = np.asarray(lengths, np.int32)[keep]
        sub.h0 = np.asarray(w.h0)[:, keep]
        sub.c0 = np.asarray(w.c0)[:, keep]
        lstm_t, x, h0, c0, y, hn, cn = _torch_lstm(sub)
        zero = [b for b in range(w.B) if lengths[b] == 0]
        loss = (hn[-1].sum() + torch.tensor(np.asarray(w.h0)[-1, zero]).sum()) / (w.B * w.H)
    else:
        keep = list(range(w.B))
        lstm_t, x, h0, c0, y, hn, cn = _torch_lstm(w)
        loss = hn[-1].mean()
    loss.backward()
    ref = steps.lstm_step(w)
    np.testing.assert_allclose(ref["loss"], loss.item(), rtol=1e-13)
    np.testing.assert_allclose(ref["dx"][:, keep], x.grad.numpy(), atol=1e-13)
    np.testing.assert_allclose(ref["dh0"][:, keep], h0.grad.numpy(), atol=1e-13)
    np.testing.assert_allclose(ref["dc0"][:, keep], c0.grad.numpy(), atol=1e-13)
    for l in range(w.L):
        np.testing.assert_allclose(ref["dWx"][l], getattr(lstm_t, f"weight_ih_l{l}").grad.numpy(), atol=1e-13)
        np.testing.assert_allclose(ref["dWh"][l], getattr(lstm_t, f"weight_hh_l{l}").grad.numpy(), atol=1e-13)
        np.testing.assert_allclose(ref["db"][l], getattr(lstm_t, f"bias_ih_l{l}").grad.numpy(), atol=1e-13)


@pytest.mark.parametrize("shape", [(1,), (7,), (3, 5), (2, 4, 6)])
def test_mean_all_against_torch_mean(shape):
    """heads.mean_all: value and gradient of torch.mean under autograd, and
    the closed form mean(0..n-1) = (n-1)/2 with gradient 1/n everywhere."""
    rng = np.random.default_rng(sum(shape))
    h = rng.standard_normal(shape)
    loss, dh = heads.mean_all(h)
    ht = torch.tensor(h, requires_grad=True)
    lt = ht.mean()
    lt.backward()
    assert abs(loss - lt.item()) < 1e-14
    np.testing.assert_allclose(dh, ht.grad.numpy(), rtol=0, atol=0)
    n = int(np.prod(shape))
    loss, dh = heads.mean_all(np.arange(n, dtype=np.float64).reshape(shape))
    assert loss == (n - 1) / 2
    assert dh.shape == shape and np.all(dh == 1.0 / n)
