"""The allocation-free parameter update (janus_sgd_clip_update_noalloc)
against the entry point that takes a caller workspace, through the C ABI.

Both run the same kernels, so the parameters and the statistics must agree
bit for bit.  The calls come in a row on one device, each input smaller than
the one before, so leftovers of a larger call in the library's fixed array
would show; a held call must leave everything unchanged."""
import numpy as np
import pytest

from oracle import sgd as osgd

pytestmark = pytest.mark.gpu


def _case(seed, shapes, dtype):
    rng = np.random.default_rng(seed)
    P = [rng.uniform(-1, 1, s).astype(np.float32) for s in shapes]
    G = [rng.normal(0, 1, s).astype(np.float32) for s in shapes]
    if dtype == "bf16":
        from paper_1812_01329_amd import workloads as wl
        P = [wl.bf16_round(p) for p in P]
    return P, G


def _both(P, G, dtype, lr, max_norm, hold_value=None):
    import torch
    from paper_1812_01329_amd import janus as J
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    pa = [torch.from_numpy(p.ravel()).to(tdt).cuda() for p in P]
    pb = [t.clone() for t in pa]
    g = [torch.from_numpy(x.ravel()).cuda() for x in G]
    d = J.SgdDesc(len(pa), J.BF16 if dtype == "bf16" else J.F32, lr, max_norm)
    ws = torch.empty(J.sgd_workspace_bytes(d), dtype=torch.uint8, device="cuda")
    sa = torch.full((2,), -1.0, dtype=torch.float32, device="cuda")
    sb = torch.full((2,), -1.0, dtype=torch.float32, device="cuda")
    hold = None
    if hold_value is not None:
        hold = torch.full((1,), hold_value, dtype=torch.int32, device="cuda")
    hp = None if hold is None else hold.data_ptr()
    print(f"[noalloc] n={len(pa)} dtype={dtype} lr={lr} max_norm={max_norm} hold={hold_value}", flush=True)
    J.janus_sgd_clip_update(d, pa, g, stats=sa, ws=ws, hold=hp)
    J.janus_sgd_clip_update_noalloc(d, pb, g, stats=sb, hold=hp)
    torch.cuda.synchronize()
    for a, b in zip(pa, pb):
        assert torch.equal(a, b)
    assert torch.equal(sa, sb)
    return [a.double().cpu().numpy() for a in pb], sa.double().cpu().numpy()


def test_noalloc_update_matches_workspace_update():
    # 1: 70 tensors (two tables of tensors, two chunks of block sums), bf16,
    #    clipping active; also against the oracle
    shapes = [(int(n),) for n in np.random.default_rng(3).integers(0, 5000, 70)]
    shapes[5] = (0,)
    P, G = _case(21, shapes, "bf16")
    new, st = _both(P, G, "bf16", 0.1, 1.0)
    ref, norm, s, applied = osgd.sgd_clip_update(P, G, 0.1, 1.0)
    assert applied and s < 1.0
    assert st[0] == pytest.approx(norm, rel=1e-5)
    for k, r in zip(new, ref):
        np.testing.assert_allclose(k, np.asarray(r).ravel(), rtol=2 ** -7, atol=1e-6)
    # 2: fewer, smaller float32 tensors, clipping off
    P, G = _case(22, [(1000,), (33,), (7, 9)], "f32")
    new, st = _both(P, G, "f32", 0.05, 0.0)
    assert st[1] == 1.0
    # 3: one tensor, held: nothing changes
    P, G = _case(23, [(17,)], "f32")
    new, st = _both(P, G, "f32", 0.5, 0.0, hold_value=1)
    assert np.array_equal(new[0], P[0].astype(np.float64))
    assert st[1] == 0.0


def test_noalloc_update_rejects_too_many_tensors():
    """Beyond the array's room the call fails before it touches the device."""
    import ctypes as C
    import torch
    from paper_1812_01329_amd import janus as J
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    n = J.SGD_NOALLOC_MAX_TENSORS + 1
    p = torch.zeros(n, dtype=torch.float32, device="cuda")
    g = torch.ones(n, dtype=torch.float32, device="cuda")
    P = [p[i:i + 1] for i in range(n)]
    G = [g[i:i + 1] for i in range(n)]
    d = J.SgdDesc(n, J.F32, 0.1, 0.0)
    with pytest.raises(J.JanusError) as e:
        J.janus_sgd_clip_update_noalloc(d, P, G)
    assert e.value.status == J.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.count_nonzero(p).item() == 0
