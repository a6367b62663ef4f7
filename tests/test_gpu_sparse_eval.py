"""GPU parity of the sparse evaluation path (ggnn_sparse_step over every
edge) and of the lossy regime: train on a block band narrower than the
graphs' bandwidth, evaluate the same weights with messages on all edges."""
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


def _csr(n, E, src, dst, et):
    row_ptr, col, _ = capi.ggnn_sparse_csr(n, E, src, dst, et)
    c = col if len(col) else np.zeros(1, np.int32)
    return torch.from_numpy(row_ptr).cuda(), torch.from_numpy(c).cuda(), len(col)


def _wt(W, dt):
    Wd = dev(W, dt)
    Wt = torch.empty_like(Wd)
    capi.ggnn_transpose_weights(dt, W.shape[1], W.shape[0], Wd, Wt)
    return Wt


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H,E,n", [(32, 3, 160), (64, 10, 512), (128, 2, 96), (256, 4, 224), (64, 1, 64), (128, 7, 128),
                                   (64, 10, 33280), (128, 3, 33280)])
def test_sparse_step_integer_exact(dt, H, E, n):
    """Random edges anywhere in the graph (no band), repeated edges, nodes
    without incoming edges, a bias: small integers, exact."""
    say(f"sparse_step int dt={dt} H={H} E={E} n={n}")
    rng = np.random.default_rng(H + E + n)
    m = 5 * n
    src, dst, et = rng.integers(0, n, m), rng.integers(0, n, m), rng.integers(0, E, m)
    dst[dst % 7 == 3] = 0            # several receivers get nothing, node 0 gets many
    src[:20], dst[:20], et[:20] = src[20:40], dst[20:40], et[20:40]
    X = rng.integers(-2, 3, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    bias = rng.integers(-2, 3, (E, H)).astype(np.float64)
    rp, col, nnz = _csr(n, E, src, dst, et)
    a = torch.full((n, H), float("nan"), device="cuda")
    capi.ggnn_sparse_step(dt, n, H, E, rp, col, nnz, dev(X, dt), _wt(W, dt), dev(bias), a)
    s, d, e, _ = O.dedupe_edges(src, dst, et)
    np.testing.assert_array_equal(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W, bias)))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H", [64, 256])
def test_sparse_step_real_values(dt, H):
    say(f"sparse_step real dt={dt} H={H}")
    rng = np.random.default_rng(3 * H)
    n, E, m = 640, 6, 6000
    src, dst, et = rng.integers(0, n, m), rng.integers(0, n, m), rng.integers(0, E, m)
    X = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    rp, col, nnz = _csr(n, E, src, dst, et)
    a = torch.empty((n, H), device="cuda")
    capi.ggnn_sparse_step(dt, n, H, E, rp, col, nnz, dev(X, dt), _wt(W, dt), None, a)
    s, d, e, _ = O.dedupe_edges(src, dst, et)
    assert relerr(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W))) <= 1e-4


@pytest.mark.parametrize("dt,B,H", [("f32", 32, 32), ("bf16", 32, 64), ("bf16", 64, 128), ("bf16", 64, 256)])
def test_lossy_training_then_sparse_evaluation(dt, B, H):
    """A batch whose bandwidth after reordering exceeds B: one banded training
    step drops the out-of-band edges; the updated weights are then evaluated
    along every edge.  Both losses against the oracle's own chain."""
    from ggnn_synth import backbone_graph, scramble_graph, draw_params, draw_candidates, draw_readout
    from paper_1906_11786_amd.driver import compile_graphs, BandedGGNN
    E, T = 3, 2
    say(f"lossy dt={dt} B={B} H={H}")
    # spans up to 120 > B: some edges fall outside the three block diagonals
    graphs = [scramble_graph(60, gi, backbone_graph(60, gi, sz, E, span_mean=30.0, max_span=120))[0]
              for gi, sz in enumerate([700, 500, 300])]
    comp = compile_graphs(graphs, B, E)
    parts = []
    for g in graphs:
        _, rank = O.rcm_order(g.n, g.src, g.dst)
        parts.append((g.n, *O.relabel(rank, g.src, g.dst), g.etype))
    n_real, n_pad, src, dst, et, offs = O.batch_layout(parts, B)
    np.testing.assert_array_equal(comp.src, src)
    np.testing.assert_array_equal(comp.dst, dst)
    prm = draw_params(60, n_real, n_pad, H, E, dt, with_bias=True)
    cands = draw_candidates(60, offs)
    w_out, b_out = draw_readout(60, H)
    m = BandedGGNN(comp, H, T, dt, prm, strict=False)
    assert comp.stats["n_dropped"] > 0
    m.setup_training(cands, w_out, b_out, lr=0.05, momentum=0.9)
    m.setup_sparse(comp.src, comp.dst, comp.etype)
    m.train_step()
    torch.cuda.synchronize()
    train_loss = host(m.loss).mean()
    m.evaluate_sparse()
    torch.cuda.synchronize()
    eval_loss = host(m.loss)
    p = {"W": prm.W, "bias": prm.bias, "Wi": prm.Wi, "U": prm.U, "b": prm.b, "w_out": w_out, "b_out": b_out}
    vel = {k: np.zeros_like(np.asarray(x, np.float64)) for k, x in p.items()}
    newp, _, mean, _ = O.train_step(n_pad, B, src, dst, et, prm.X, p, vel, T, cands.node, cands.ptr, cands.target,
                                    0.05, 0.9)
    assert abs(train_loss - mean) <= TOL[dt] * max(1.0, abs(mean))
    if dt == "bf16":    # the GPU propagates the bf16 copies of the updated weights
        for k in ("W", "Wi", "U"):
            newp[k] = round_to("bf16", newp[k])
    wl, wmean = O.evaluate(n_pad, None, src, dst, et, prm.X, newp, T, cands.node, cands.ptr, cands.target)
    _, banded_mean = O.evaluate(n_pad, B, src, dst, et, prm.X, newp, T, cands.node, cands.ptr, cands.target)
    say(f"  train {train_loss:.5f}/{mean:.5f}  eval all edges {eval_loss.mean():.5f}/{wmean:.5f}  "
        f"eval band only {banded_mean:.5f}  dropped {comp.stats['n_dropped']}")
    assert relerr(eval_loss, wl) <= TOL[dt]
    assert abs(wmean - banded_mean) > 1e-6     # the dropped edges matter for this loss
