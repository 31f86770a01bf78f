"""GPU parity of the heads and losses called on their own through the C ABI
(janus_embed_softmax_xent, janus_linear_mse, janus_loss_reduce) against the
float64 oracle (oracle/heads.py), on the edge cases the training-step tests
do not reach: every row with the same id, ids at both ends of the
vocabulary, vocabularies and widths that are not multiples of a tile or of
8, the 5-class root classifier, unaligned and odd-length loss inputs.
Embedding lookups are bit-exact; the rest meets the float32 (1e-4 / 1e-3)
or bf16 (2e-2) tolerances."""
import numpy as np
import pytest

from oracle import heads as H_
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check

pytestmark = pytest.mark.gpu


def _dev(a, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.to("cuda:0")


def _host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def _vals(rng, shape, scale, dtype):
    a = rng.uniform(-scale, scale, shape).astype(np.float32)
    return wl.bf16_round(a) if dtype == "bf16" else a


def _ids(kind, rng, V, rows):
    if kind == "same":
        return np.full(rows, V // 2, np.int32)
    if kind == "ends":
        return np.where(np.arange(rows) % 2 == 0, 0, V - 1).astype(np.int32)
    return rng.integers(0, V, rows).astype(np.int32)


@pytest.mark.parametrize("dtype,V,Hd,rows", [("f32", 97, 37, 130), ("bf16", 1001, 64, 300), ("bf16", 50, 40, 7)])
@pytest.mark.parametrize("kind", ["same", "ends", "random"])
def test_embedding_gather_and_scatter(dtype, V, Hd, rows, kind):
    """EMBED_FWD copies rows exactly; EMBED_BWD sums the rows of each id
    (all rows on one id, or on ids 0 and V - 1 only) and leaves the other
    rows of dE at zero, identically on a second call."""
    import torch
    from paper_1812_01329_amd import janus as J
    rng = np.random.default_rng(V + rows)
    ids = _ids(kind, rng, V, rows)
    print(f"[embed] {dtype} V={V} H={Hd} rows={rows} ids={kind}", flush=True)
    E = _vals(rng, (V, Hd), 0.5, dtype)
    dx = _vals(rng, (rows, Hd), 1.0, dtype)
    dt = J.BF16 if dtype == "bf16" else J.F32
    desc = J.XentDesc(V, Hd, rows, dt)
    ids_dev = torch.from_numpy(ids).to("cuda:0")
    x = _dev(np.zeros((rows, Hd)), dtype)
    J.janus_embed_softmax_xent(desc, J.EMBED_FWD, ids, ids_dev, table=_dev(E, dtype), out=x)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(x), H_.embed_forward(E, ids))
    dE = torch.full((V, Hd), 7.0, dtype=torch.float32, device="cuda:0")   # overwritten, not accumulated
    ews = torch.empty(J.janus_xent_workspace_bytes(V, Hd, rows, dt, J.EMBED_BWD), dtype=torch.uint8, device="cuda:0")
    J.janus_embed_softmax_xent(desc, J.EMBED_BWD, ids, ids_dev, inp=_dev(dx, dtype), dtable=dE, ws=ews)
    torch.cuda.synchronize()
    first = dE.cpu().numpy().copy()
    ref = H_.embed_backward(V, dx, ids)
    check("dE", first, ref, TOL["f32"]["grad"])
    untouched = np.setdiff1d(np.arange(V), ids)
    assert np.all(first[untouched] == 0.0)
    J.janus_embed_softmax_xent(desc, J.EMBED_BWD, ids, ids_dev, inp=_dev(dx, dtype), dtable=dE, ws=ews)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dE.cpu().numpy(), first)


@pytest.mark.parametrize("dtype,V,Hd,rows", [("bf16", 10000, 650, 20000), ("f32", 20000, 300, 24000),
                                             ("bf16", 10000, 64, 1)])
def test_embedding_backward_many_zipf_rows(dtype, V, Hd, rows):
    """EMBED_BWD past the old 16384-row limit, with Zipf(1.1) ids (the most
    frequent id holds about 15 % of the rows): the sums in ascending row
    order of each id, against the oracle, and identical bits on a repeat."""
    import torch
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd import workloads as wl
    rng = np.random.default_rng(rows + V)
    ids = wl.zipf_truncated(rng, 1.1, V, rows).astype(np.int32)
    print(f"[embed-zipf] {dtype} V={V} H={Hd} rows={rows} distinct={len(np.unique(ids))}", flush=True)
    dx = _vals(rng, (rows, Hd), 1.0, dtype)
    dt = J.BF16 if dtype == "bf16" else J.F32
    desc = J.XentDesc(V, Hd, rows, dt)
    ids_dev = torch.from_numpy(ids).to("cuda:0")
    dE = torch.full((V, Hd), 7.0, dtype=torch.float32, device="cuda:0")
    ews = torch.empty(J.janus_xent_workspace_bytes(V, Hd, rows, dt, J.EMBED_BWD), dtype=torch.uint8, device="cuda:0")
    dxd = _dev(dx, dtype)
    J.janus_embed_softmax_xent(desc, J.EMBED_BWD, ids, ids_dev, inp=dxd, dtable=dE, ws=ews)
    torch.cuda.synchronize()
    first = dE.cpu().numpy().copy()
    check("dE", first, H_.embed_backward(V, dx, ids), TOL["f32"]["grad"])
    assert np.all(first[np.setdiff1d(np.arange(V), ids)] == 0.0)
    J.janus_embed_softmax_xent(desc, J.EMBED_BWD, ids, ids_dev, inp=dxd, dtable=dE, ws=ews)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dE.cpu().numpy(), first)


@pytest.mark.parametrize("dtype,V,Hd,rows,small", [("f32", 5, 150, 25, "1"), ("f32", 5, 150, 25, "0"),
                                                   ("f32", 1001, 36, 77, "1"), ("bf16", 1001, 64, 300, "1"),
                                                   ("bf16", 5, 64, 33, "1"), ("bf16", 5, 64, 33, "0"),
                                                   ("f32", 64, 96, 40, "1"), ("f32", 13001, 36, 9, "1")])
@pytest.mark.parametrize("kind", ["same", "ends", "random"])
def test_softmax_cross_entropy(dtype, V, Hd, rows, small, kind, monkeypatch):
    """XENT_FWD_BWD: mean loss, dh, dWout and dbout of one call, with the
    targets all on one class, on the two end classes, or random.  Heads of
    at most 64 classes whose operands fit 64 KB of LDS run in one workgroup
    (JANUS_XENT_SMALL=0 takes the contractions instead, as for the larger
    heads); a row of up to 12288 logits stays in LDS across the softmax
    passes; the 13001 class case takes the path that reads the row again."""
    import torch
    from paper_1812_01329_amd import janus as J
    monkeypatch.setenv("JANUS_XENT_SMALL", small)
    rng = np.random.default_rng(3 * V + rows)
    tgt = _ids(kind, rng, V, rows)
    print(f"[xent] {dtype} V={V} H={Hd} rows={rows} targets={kind}", flush=True)
    W = _vals(rng, (V, Hd), 0.5, dtype)
    b = _vals(rng, (V,), 0.5, dtype)
    h = _vals(rng, (rows, Hd), 1.0, dtype)
    dt = J.BF16 if dtype == "bf16" else J.F32
    desc = J.XentDesc(V, Hd, rows, dt)
    ws = torch.empty(J.janus_xent_workspace_bytes(V, Hd, rows, dt, J.XENT_FWD_BWD), dtype=torch.uint8,
                     device="cuda:0")
    dh = _dev(np.zeros((rows, Hd)), dtype)
    dW = torch.empty((V, Hd), dtype=torch.float32, device="cuda:0")
    db = torch.empty((V,), dtype=torch.float32, device="cuda:0")
    loss = torch.empty((1,), dtype=torch.float32, device="cuda:0")
    J.janus_trace_begin()
    J.janus_embed_softmax_xent(desc, J.XENT_FWD_BWD, tgt, torch.from_numpy(tgt).to("cuda:0"), table=_dev(W, dtype),
                               bias=_dev(b, dtype), inp=_dev(h, dtype), out=dh, dtable=dW, dbias=db, loss=loss,
                               ws=ws)
    labels = {r["label"] for r in J.janus_trace_end()}
    assert ("xent_small" in labels) == (small == "1" and V <= 64), labels
    torch.cuda.synchronize()
    rl, rdh, rdW, rdb, _ = H_.softmax_xent(h, W, b, tgt)
    t = TOL[dtype]
    check("loss", np.array([loss.item()]), np.array([rl]), t["out"])
    check("dh", _host(dh), rdh, t["grad"])
    check("dWout", dW.cpu().numpy(), rdW, t["grad"])
    check("dbout", db.cpu().numpy(), rdb, t["grad"])


@pytest.mark.parametrize("dtype,rows,Hd,P", [("f32", 77, 36, 20), ("bf16", 300, 128, 72), ("bf16", 520, 256, 256)])
def test_linear_mse(dtype, rows, Hd, P):
    """Projection + MSE on ragged float32 shapes and on bf16 shapes that take
    the fused epilogue (several 256-row tiles and a ragged last one)."""
    import torch
    from paper_1812_01329_amd import janus as J
    rng = np.random.default_rng(rows + P)
    print(f"[mse] {dtype} rows={rows} H={Hd} P={P}", flush=True)
    h = _vals(rng, (rows, Hd), 1.0, dtype)
    W = _vals(rng, (P, Hd), 1.0 / np.sqrt(Hd), dtype)
    b = _vals(rng, (P,), 0.5, dtype)
    tg = _vals(rng, (rows, P), 1.0, dtype)
    dt = J.BF16 if dtype == "bf16" else J.F32
    desc = J.MseDesc(rows, Hd, P, dt)
    ws = torch.empty(J.janus_mse_workspace_bytes(rows, Hd, P, dt), dtype=torch.uint8, device="cuda:0")
    dh = _dev(np.zeros((rows, Hd)), dtype)
    dW = torch.empty((P, Hd), dtype=torch.float32, device="cuda:0")
    db = torch.empty((P,), dtype=torch.float32, device="cuda:0")
    loss = torch.empty((1,), dtype=torch.float32, device="cuda:0")
    J.janus_linear_mse(desc, _dev(h, dtype), _dev(W, dtype), _dev(b, dtype), _dev(tg, dtype), dh, dW, db, loss, ws)
    torch.cuda.synchronize()
    rl, rdh, rdW, rdb, _ = H_.linear_mse(h, W, b, tg)
    t = TOL[dtype]
    check("loss", np.array([loss.item()]), np.array([rl]), t["out"])
    check("dh", _host(dh), rdh, t["grad"])
    check("dW", dW.cpu().numpy(), rdW, t["grad"])
    check("db", db.cpu().numpy(), rdb, t["grad"])


@pytest.mark.parametrize("kind", ["sumsq", "mean"])
@pytest.mark.parametrize("n,offset", [(1, 0), (4099, 0), (4099, 1), (1 << 20, 0), (1 << 20, 3)])
def test_loss_reduce(kind, n, offset):
    """Sum of squares and mean of n values (n not a multiple of 4, and the
    input starting off a 16-byte boundary), with the gradient; the same
    value on a second call."""
    import torch
    from paper_1812_01329_amd import janus as J
    rng = np.random.default_rng(n + offset)
    print(f"[loss_reduce] {kind} n={n} offset={offset}", flush=True)
    hv = rng.normal(0, 1, n + offset).astype(np.float32)
    h = torch.from_numpy(hv).to("cuda:0")[offset:]
    loss = torch.empty((1,), dtype=torch.float32, device="cuda:0")
    dh = torch.empty((n,), dtype=torch.float32, device="cuda:0")
    k = J.LOSS_SUMSQ if kind == "sumsq" else J.LOSS_MEAN
    J.janus_loss_reduce(k, h, n, loss, dh)
    torch.cuda.synchronize()
    first = loss.item()
    rl, rdh = (H_.sumsq if kind == "sumsq" else H_.mean_all)(hv[offset:])
    if kind == "sumsq":
        check("loss", np.array([first]), np.array([rl]), TOL["f32"]["out"])
    else:   # the mean is near 0: error of the sum against the sum of |h|
        err = abs(first - rl) * n / np.abs(hv[offset:].astype(np.float64)).sum()
        assert err <= 1e-6, f"mean: error {err:.3e} of the sum of |h|"
    check("dh", dh.cpu().numpy(), rdh, TOL["f32"]["grad"])
    J.janus_loss_reduce(k, h, n, loss, None)
    torch.cuda.synchronize()
    assert loss.item() == first
