"""T-step forward + reverse parity of the whole hot path (ggnn_forward /
ggnn_backward through the C ABI) against the CPU oracle, on the synthetic
workloads at their full sizes and on small cases spanning tiles and ragged
tails.  Large batches are checked on sampled graphs: graphs in a supergraph
do not interact, so the oracle runs on a few of them alone, and a second
reverse pass with the upstream gradient restricted to those graphs gives
weight gradients comparable with the oracle's."""
import os

import numpy as np
import pytest

import oracle as O
from ggnn_synth import BATCH_100K, PROGRAM_GRAPH, STRESS_1M, TINY, make_graphs, sweep_blocks, draw_params, backbone_graph, scramble_graph, Graph
from gpu_helpers import TOL, relerr, elemerr, record, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
drv = pytest.importorskip("paper_1906_11786_amd.driver")


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _oracle_edges(graphs, B, reorder):
    """Final labelling computed by the oracle's own reordering."""
    parts = []
    for g in graphs:
        if reorder:
            _, rank = O.rcm_order(g.n, g.src, g.dst)
            s, d = O.relabel(rank, g.src, g.dst)
        else:
            s, d = g.src, g.dst
        parts.append((g.n, s, d, g.etype))
    return O.batch_layout(parts, B)


def _compare(res, out, dt, keys=("XT", "dX0", "dW", "dWi", "dU", "db"), rows=None):
    want = dict(XT=out["X"][-1], dX0=out["dX0"], dW=out["dW"], dWi=out["dWi"], dU=out["dU"], db=out["db"])
    if "dbias" in res:
        want["dbias"] = out["dbias"]
        keys = tuple(keys) + ("dbias",)
    errs, elem = {}, {}
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    for k in keys:
        g = res[k] if rows is None or k not in ("XT", "dX0") else res[k][rows]
        w = want[k]
        errs[k] = relerr(g, w)
        elem[k] = elemerr(g, w)
        record(test, k, errs[k], elem[k])
    say("  errors (normwise / elementwise):", {k: f"{errs[k]:.2e} / {elem[k]:.2e}" for k in errs})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)
    return errs


def _run_full(graphs, spec_B, E, H, T, dt, cfg, reorder, with_bias=False, band_format="bits"):
    comp = drv.compile_graphs(graphs, spec_B, E, reorder=reorder)
    n_real, n_pad, s, d, e, offs = _oracle_edges(graphs, spec_B, reorder)
    assert (n_real, n_pad) == (comp.n_real, comp.n_pad)
    np.testing.assert_array_equal(comp.src, s)         # the product's reordering equals the oracle's
    np.testing.assert_array_equal(comp.dst, d)
    params = draw_params(cfg, n_real, n_pad, H, E, dt, with_bias=with_bias)
    m = drv.BandedGGNN(comp, H, T, dt, params, band_format=band_format)
    m.step()
    torch.cuda.synchronize()
    res = m.results()
    out = O.propagate(n_pad, spec_B, s, d, e, params.X, params.W, params.Wi, params.U, params.b, T, G=params.G,
                      bias=params.bias)
    assert comp.stats["n_dropped"] == out["n_dropped"]
    return m, res, out


@pytest.mark.parametrize("band_format", ["bits", "dense"])
def test_tiny_fp32_workload(band_format):
    spec = TINY
    say(f"workload {spec.name} band={band_format}")
    g = make_graphs(spec)
    _, res, out = _run_full(g, spec.B, spec.E, spec.H, spec.T, spec.dtype, spec.cfg, reorder=False,
                            band_format=band_format)
    assert out["n_dropped"] == 0
    _compare(res, out, "f32")


SMALL = [  # (dt, n_nodes, B, E, H, T, bias)
    ("f32", 700, 64, 2, 64, 2, True),
    ("f32", 1000, 128, 3, 128, 2, False),
    ("f32", 300, 32, 2, 32, 3, True),
    ("bf16", 1500, 128, 4, 64, 3, True),
    ("bf16", 900, 32, 3, 32, 4, False),
    ("bf16", 1300, 256, 2, 256, 2, True),
    ("bf16", 2000, 512, 2, 128, 2, False),
    ("bf16", 1100, 64, 5, 128, 3, True),
    ("f32", 600, 64, 2, 256, 2, True),
]


@pytest.mark.parametrize("band_format", ["bits", "dense"])
@pytest.mark.parametrize("dt,n,B,E,H,T,bias", SMALL)
def test_small_cases(dt, n, B, E, H, T, bias, band_format):
    say(f"small dt={dt} n={n} B={B} E={E} H={H} T={T} bias={bias} band={band_format}")
    g = scramble_graph(50 + n, 0, backbone_graph(50 + n, 0, n, E, span_mean=6.0, max_span=B))[0]
    _, res, out = _run_full([g], B, E, H, T, dt, 50 + n, reorder=True, with_bias=bias, band_format=band_format)
    _compare(res, out, dt)


@pytest.mark.parametrize("band_format", ["bits", "dense"])
def test_small_lossy_band(band_format):
    """Bandwidth above the block size: edges outside the three block
    diagonals are dropped identically by both sides."""
    dt, n, B, E, H, T = "bf16", 1200, 32, 3, 64, 2
    g = backbone_graph(77, 0, n, E, span_mean=20.0, max_span=90)
    comp = drv.compile_graphs([g], B, E, reorder=False)
    params = draw_params(77, comp.n_real, comp.n_pad, H, E, dt)
    m = drv.BandedGGNN(comp, H, T, dt, params, strict=False, band_format=band_format)
    assert comp.stats["n_dropped"] > 0
    m.step()
    out = O.propagate(comp.n_pad, B, g.src, g.dst, g.etype, params.X, params.W, params.Wi, params.U, params.b, T,
                      G=params.G)
    assert out["n_dropped"] == comp.stats["n_dropped"]
    _compare(m.results(), out, dt)


@pytest.mark.parametrize("band_format", ["bits", "dense"])
def test_program_graph_workload(band_format):
    spec = PROGRAM_GRAPH
    say(f"workload {spec.name} band={band_format}")
    g = make_graphs(spec)
    m, res, out = _run_full(g, spec.B, spec.E, spec.H, spec.T, spec.dtype, spec.cfg, reorder=True,
                            band_format=band_format)
    assert out["n_dropped"] == 0 and m.comp.bandwidth <= spec.B - 1
    _compare(res, out, spec.dtype)
    # determinism: a second pass gives identical bits
    m.step()
    torch.cuda.synchronize()
    res2 = m.results()
    for k in res:
        assert np.array_equal(res[k], res2[k]), k


@pytest.mark.parametrize("band_format", ["bits", "dense"])
@pytest.mark.parametrize("spec", sweep_blocks(), ids=lambda s: f"B{s.B}")
def test_sweep_workloads(spec, band_format):
    say(f"workload {spec.name} band={band_format}")
    g = make_graphs(spec)
    _, res, out = _run_full(g, spec.B, spec.E, spec.H, spec.T, spec.dtype, spec.cfg, reorder=False,
                            band_format=band_format)
    assert out["n_dropped"] == 0
    _compare(res, out, spec.dtype)


def _sampled_batch(spec, picks):
    graphs = make_graphs(spec)
    say(f"workload {spec.name}: {len(graphs)} graphs, {sum(g.n for g in graphs)} nodes; sampling {picks}")
    comp = drv.compile_graphs(graphs, spec.B, spec.E, reorder=True)
    params = draw_params(spec.cfg, comp.n_real, comp.n_pad, spec.H, spec.E, spec.dtype)
    m = drv.BandedGGNN(comp, spec.H, spec.T, spec.dtype, params)
    assert comp.stats["n_dropped"] == 0
    m.forward()
    m.backward()
    torch.cuda.synchronize()
    full = m.results()
    # restrict the upstream gradient to the sampled graphs and run the reverse pass again
    mask = np.zeros(comp.n_pad, bool)
    for gi in picks:
        mask[comp.offsets[gi]:comp.offsets[gi + 1]] = True
    m.G.mul_(torch.from_numpy(mask.astype(np.float32)).to(m.G.device)[:, None])
    m.backward()
    torch.cuda.synchronize()
    masked = m.results()
    acc = {}
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    for gi in picks:
        g = graphs[gi]
        o = slice(int(comp.offsets[gi]), int(comp.offsets[gi + 1]))
        _, rank = O.rcm_order(g.n, g.src, g.dst)
        s, d = O.relabel(rank, g.src, g.dst)
        np.testing.assert_array_equal(comp.src[(comp.src >= o.start) & (comp.src < o.stop)].size,
                                      s.size)
        out = O.propagate(g.n, g.n, s, d, g.etype, params.X[o], params.W, params.Wi, params.U, params.b, spec.T,
                          G=params.G[o])
        # rows of this graph, from the full run (graphs do not interact)
        rows = slice(o.start, o.stop)
        e1 = relerr(full["XT"][rows], out["X"][-1])
        e2 = relerr(full["dX0"][rows], out["dX0"])
        x1, x2 = elemerr(full["XT"][rows], out["X"][-1]), elemerr(full["dX0"][rows], out["dX0"])
        record(test, f"XT[graph {gi}]", e1, x1)
        record(test, f"dX0[graph {gi}]", e2, x2)
        say(f"  graph {gi} n={g.n}: XT {e1:.2e} / {x1:.2e}, dX0 {e2:.2e} / {x2:.2e} (normwise / elementwise)")
        assert e1 <= TOL[spec.dtype] and e2 <= TOL[spec.dtype]
        for k in ("dW", "dWi", "dU", "db"):
            acc[k] = acc.get(k, 0) + out[k]
    for k in ("dW", "dWi", "dU", "db"):
        e, x = relerr(masked[k], acc[k]), elemerr(masked[k], acc[k])
        record(test, f"{k} (sampled graphs)", e, x)
        say(f"  {k} (sampled graphs) {e:.2e} / {x:.2e}")
        assert e <= TOL[spec.dtype], k


def test_batch_100k_workload_every_graph():
    """All 34 graphs of the 100k-node batch, each against the oracle run on
    it alone, and the weight gradients against the sum over all of them."""
    _sampled_batch(BATCH_100K, picks=list(range(34)))


def test_stress_1m_workload_sampled():
    """Eight of the 141 graphs of the 1M-node batch: the first two, the last
    two (148 and 372 nodes), and four between them, one of the largest size
    (20,000 nodes)."""
    _sampled_batch(STRESS_1M, picks=[0, 1, 20, 50, 70, 100, 139, 140])


def _no_edges(n):
    z = np.zeros(0, np.int32)
    return Graph(n=n, src=z, dst=z, etype=z)


def _one_type(seed, n, E, keep):
    g = scramble_graph(seed, 0, backbone_graph(seed, 0, n, E, span_mean=5.0, max_span=32))[0]
    m = g.etype == keep
    return Graph(n=g.n, src=g.src[m], dst=g.dst[m], etype=g.etype[m])


DEGENERATE = {  # name: (graphs, B, E, H, T, dt, bias)
    "no_edges": (lambda: [_no_edges(200)], 64, 3, 64, 2, "bf16", True),
    "one_node": (lambda: [_no_edges(1)], 32, 2, 32, 3, "f32", True),
    "batch_of_edgeless_graphs": (lambda: [_no_edges(1), _no_edges(150), _no_edges(1)], 64, 2, 128, 2, "bf16", False),
    "one_edge_type_of_four": (lambda: [_one_type(83, 700, 4, 2)], 64, 4, 64, 2, "bf16", True),
    "mixed_with_empty": (lambda: [_no_edges(40), _one_type(84, 500, 3, 0), _no_edges(1)], 128, 3, 256, 2, "bf16",
                         True),
}


@pytest.mark.parametrize("band_format", ["bits", "dense"])
@pytest.mark.parametrize("case", list(DEGENERATE))
def test_degenerate_graphs(case, band_format):
    """Edgeless graphs (the aggregate is zero, only the GRU acts), a single
    node, a batch mixing edgeless graphs with one that has edges of a single
    type: the whole forward and reverse pass against the oracle."""
    make, B, E, H, T, dt, bias = DEGENERATE[case]
    say(f"degenerate {case} B={B} E={E} H={H} T={T} dt={dt} band={band_format}")
    _, res, out = _run_full(make(), B, E, H, T, dt, 90, reorder=True, with_bias=bias, band_format=band_format)
    assert out["n_dropped"] == 0
    _compare(res, out, dt)
    if case.startswith("no_edges") or case.startswith("one_node") or case.startswith("batch_of"):
        # no messages: the weight gradients of the transform are exactly zero
        assert not np.any(res["dW"]), case
        if "dbias" in res:
            assert not np.any(res["dbias"]), case


@pytest.mark.parametrize("band_format", ["bits", "dense"])
@pytest.mark.parametrize("n,B,E,H,T", [(1500, 128, 3, 128, 3), (1300, 256, 2, 256, 2)])
def test_gru_packed_weights_equal_gathered(n, B, E, H, T, band_format):
    """The large-width GRU kernels staging Wi, U from the packed copy give the
    same forward and reverse results, bit for bit, as staging them straight
    from the row-major weights; the packed copy holds every element of Wi
    and U once in each of its two regions."""
    dt = "bf16"
    say(f"gru packed vs gathered n={n} B={B} E={E} H={H} T={T} band={band_format}")
    g = scramble_graph(70 + H, 0, backbone_graph(70 + H, 0, n, E, span_mean=6.0, max_span=B))[0]
    comp = drv.compile_graphs([g], B, E, reorder=True)
    params = draw_params(70 + H, comp.n_real, comp.n_pad, H, E, dt, with_bias=True)
    res = {}
    for pack in (True, False):
        m = drv.BandedGGNN(comp, H, T, dt, params, band_format=band_format, gru_pack=pack)
        assert (m.gru_packed is not None) == pack
        m.step()
        torch.cuda.synchronize()
        res[pack] = m.results()
        if pack:
            pk = m.gru_packed.view(torch.int16).cpu().numpy().reshape(2, -1)
            w = np.concatenate([m.Wi.view(torch.int16).cpu().numpy().ravel(),
                                m.U.view(torch.int16).cpu().numpy().ravel()])
            for region in pk:
                np.testing.assert_array_equal(np.sort(region), np.sort(w))
        del m
    assert res[True].keys() == res[False].keys()
    for k in res[True]:
        assert np.array_equal(res[True][k], res[False][k]), k


@pytest.mark.parametrize("band_format", ["bits", "dense"])
@pytest.mark.parametrize("B,H", [(128, 64), (128, 128), (64, 256)])
def test_graph_replay_equals_eager(band_format, B, H):
    """The step captured as a HIP graph: every replay (with eager work and
    synchronizations between replays) gives the eager step's results bit for
    bit, and they match the oracle.  H = 64 runs the fused step kernels,
    H >= 128 the wide step kernels and the large-width GRU kernels (weights
    from their packed copy)."""
    dt, n, E, T = "bf16", 1500, 4, 3
    say(f"graph replay band={band_format} B={B} H={H}")
    g = scramble_graph(61, 0, backbone_graph(61, 0, n, E, span_mean=6.0, max_span=B))[0]
    m, res, out = _run_full([g], B, E, H, T, dt, 61, reorder=True, with_bias=True, band_format=band_format)
    _compare(res, out, dt)
    m.capture()
    for rep in range(3):
        m.replay()
        torch.cuda.synchronize()
        got = m.results()
        for k in res:
            assert np.array_equal(got[k], res[k]), (rep, k)
        # eager work between the replays: an eager step on the same buffers
        m.step()
        torch.cuda.synchronize()
        again = m.results()
        for k in res:
            assert np.array_equal(again[k], res[k]), (rep, k)
