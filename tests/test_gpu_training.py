"""GPU parity of the readout, loss and Momentum update (called through the C
ABI) and of one whole training step against the oracle."""
import numpy as np
import pytest

import oracle as O
from gpu_helpers import TOL, relerr, say, dev, host, round_to

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
capi = pytest.importorskip("paper_1906_11786_amd.capi")


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    yield
    torch.cuda.synchronize()


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def _cands(rng, n, G, kmax=7):
    """Graph sizes 0..kmax candidates (an empty graph and a single-candidate
    graph included), distinct nodes, a target per graph."""
    ks = rng.integers(0, kmax + 1, G)
    ks[0], ks[1 % G] = 0, 1
    ptr = np.concatenate([[0], np.cumsum(ks)])
    node = rng.permutation(n)[:ptr[-1]]
    tgt = np.array([rng.integers(0, max(k, 1)) for k in ks])
    return node, ptr, tgt


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H", [32, 64, 128, 256])
def test_readout_loss_and_reverse(dt, H):
    say(f"readout_loss dt={dt} H={H}")
    rng = np.random.default_rng(H + (dt == "bf16"))
    n, G = 320, 37
    X = round_to(dt, rng.standard_normal((n, H)))
    w = rng.standard_normal(H).astype(np.float32).astype(np.float64)
    bo = 0.25
    node, ptr, tgt = _cands(rng, n, G)
    nc = int(ptr[-1])
    Xd = dev(X, dt)
    logits = torch.full((nc,), float("nan"), device="cuda")
    dlog = torch.full((nc,), float("nan"), device="cuda")
    loss = torch.full((G,), float("nan"), device="cuda")
    capi.ggnn_readout_loss(dt, n, H, G, nc, Xd, dev(w), dev(np.array([bo])), _i32(node), _i32(ptr), _i32(tgt),
                           logits, loss, dlog)
    wl = O.readout_logits(X, w, bo, node)
    wloss, _, wd = O.readout_loss(wl, ptr, tgt)
    assert relerr(host(logits), wl) <= 1e-5
    assert relerr(host(loss), wloss) <= 1e-5 and host(loss)[0] == 0.0
    assert relerr(host(dlog), wd) <= 1e-5
    # reverse: dX written whole, dw_out / db_out accumulated onto what is there
    dX = torch.full((n, H), float("nan"), device="cuda")
    dw = torch.ones((H,), device="cuda")
    db = torch.ones((1,), device="cuda")
    ws_n = capi.ggnn_readout_loss_bwd_workspace_bytes(H, nc)
    ws = torch.empty((ws_n,), dtype=torch.uint8, device="cuda")
    dl = rng.standard_normal(nc).astype(np.float32).astype(np.float64)
    capi.ggnn_readout_loss_bwd(dt, n, H, nc, Xd, dev(w), _i32(node), dev(dl), dX, dw, db, ws, ws_n)
    wdX, wdw, wdb = O.readout_backward(X, w, node, dl)
    np.testing.assert_allclose(host(dX), wdX, rtol=1e-6, atol=1e-30)
    assert relerr(host(dw) - 1.0, wdw) <= 1e-5
    assert abs(host(db)[0] - 1.0 - wdb) <= 1e-5 * max(1.0, np.abs(dl).sum())


@pytest.mark.parametrize("nesterov", [False, True])
@pytest.mark.parametrize("copy_dt", [None, "bf16", "f32"])
def test_sgd_momentum(nesterov, copy_dt):
    say(f"sgd_momentum nesterov={nesterov} copy={copy_dt}")
    rng = np.random.default_rng(7 + nesterov)
    count = 100_003
    th = rng.standard_normal(count).astype(np.float32).astype(np.float64)
    v = np.zeros(count)
    p, vel = dev(th), torch.zeros((count,), device="cuda")
    copy = None if copy_dt is None else torch.empty((count,), device="cuda",
                                                     dtype=torch.bfloat16 if copy_dt == "bf16" else torch.float32)
    for step in range(3):
        g = rng.standard_normal(count).astype(np.float32).astype(np.float64)
        capi.ggnn_sgd_momentum(count, p, vel, dev(g), 0.05, 0.9, 1e-3, nesterov, copy_dt or "f32", copy)
        th, v = O.momentum_update(th, v, g, 0.05, 0.9, 1e-3, nesterov)
        assert relerr(host(p), th) <= 1e-6 and relerr(host(vel), v) <= 1e-6
    if copy_dt == "bf16":
        np.testing.assert_array_equal(host(copy), round_to("bf16", host(p)))
    elif copy_dt == "f32":
        assert torch.equal(copy, p)


@pytest.mark.parametrize("dt,n,B,E,H,T", [("f32", 700, 64, 3, 32, 2), ("bf16", 1500, 128, 4, 64, 3),
                                          ("bf16", 900, 128, 2, 128, 2), ("bf16", 700, 64, 2, 256, 2)])
@pytest.mark.parametrize("band_format", ["bits", "dense"])
def test_train_step_matches_oracle(dt, n, B, E, H, T, band_format):
    """Two training steps (propagation, readout, loss, reverse pass, Momentum
    update of every parameter, with a per-type bias): the parameter updates
    and the loss against the oracle's training step."""
    from ggnn_synth import backbone_graph, scramble_graph, draw_params, draw_candidates, draw_readout
    from paper_1906_11786_amd.driver import compile_graphs, BandedGGNN
    say(f"train_step dt={dt} n={n} B={B} E={E} H={H} T={T} band={band_format}")
    graphs = [scramble_graph(50, gi, backbone_graph(50, gi, sz, E))[0] for gi, sz in enumerate([n // 2, n - n // 2])]
    comp = compile_graphs(graphs, B, E)
    # the oracle's own reordering and layout (the product's must agree)
    parts = []
    for g in graphs:
        _, rank = O.rcm_order(g.n, g.src, g.dst)
        parts.append((g.n, *O.relabel(rank, g.src, g.dst), g.etype))
    n_real, n_pad, src, dst, et, offs = O.batch_layout(parts, B)
    assert (n_real, n_pad) == (comp.n_real, comp.n_pad)
    np.testing.assert_array_equal(comp.src, src)
    np.testing.assert_array_equal(comp.dst, dst)
    prm = draw_params(50, n_real, n_pad, H, E, dt, with_bias=True)
    cands = draw_candidates(50, offs)
    w_out, b_out = draw_readout(50, H)
    m = BandedGGNN(comp, H, T, dt, prm, band_format=band_format)
    lr, mu = 0.05, 0.9
    m.setup_training(cands, w_out, b_out, lr=lr, momentum=mu)
    p_or = {"W": prm.W, "bias": prm.bias, "Wi": prm.Wi, "U": prm.U, "b": prm.b, "w_out": w_out, "b_out": b_out}
    vel = {k: np.zeros_like(np.asarray(x, np.float64)) for k, x in p_or.items()}
    prev = {k: np.asarray(x, np.float64) for k, x in p_or.items()}   # the GPU's parameters before the step
    for step in range(2):
        m.train_step()
        torch.cuda.synchronize()
        loss = host(m.loss)
        # the oracle's own chain: it propagates the compute copies of its
        # parameters (bf16-rounded in bf16 mode) and applies the update to
        # its float32-master stand-ins
        rp = dict(p_or)
        if dt == "bf16":
            for k in ("W", "Wi", "U"):
                rp[k] = round_to("bf16", p_or[k])
        newp, vel, mean, _ = O.train_step(n_pad, B, src, dst, et, prm.X, rp, vel, T,
                                          cands.node, cands.ptr, cands.target, lr, mu)
        nxt = {k: p_or[k] + (newp[k] - rp[k]) for k in p_or}
        assert abs(loss.mean() - mean) <= TOL[dt] * max(1.0, abs(mean)), (step, loss.mean(), mean)
        got = m.parameters()
        for k in p_or:
            d_got = got[k] - prev[k]
            d_want = np.asarray(nxt[k], np.float64) - np.asarray(p_or[k], np.float64)
            if k == "b_out":
                # each graph's dlogits sum to zero: only rounding moves b_out
                assert np.all(np.abs(d_got) <= 1e-5), (step, k, d_got)
                continue
            err = relerr(d_got, d_want)
            say(f"  step {step} {k}: {err:.2e}")
            assert err <= TOL[dt], (step, k, err)
        p_or, prev = nxt, got
