"""Seeded input generators: reproducibility and the statistics the workloads promise."""
import numpy as np
import pytest

from ggnn_synth import (PROGRAM_GRAPH, TINY, make_graphs, sweep_blocks, draw_params, round_bf16, lognormal_batch_sizes,
                        backbone_graph, local_window_graph)


def test_generators_are_reproducible():
    a = make_graphs(PROGRAM_GRAPH)[0]
    b = make_graphs(PROGRAM_GRAPH)[0]
    assert np.array_equal(a.src, b.src) and np.array_equal(a.dst, b.dst) and np.array_equal(a.etype, b.etype)
    p1 = draw_params(1, 100, 128, 64, 10, "bf16")
    p2 = draw_params(1, 100, 128, 64, 10, "bf16")
    assert np.array_equal(p1.X, p2.X) and np.array_equal(p1.Wi, p2.Wi)


def test_tiny_config_edges():
    spec = TINY
    g = make_graphs(spec)[0]
    assert g.n == 512 and set(np.unique(g.etype)) == {0, 1}
    span = np.abs(g.src - g.dst)
    assert span.min() >= 1 and span.max() < 64
    # about 0.05 of the 60,480 ordered pairs per type
    for e in range(2):
        assert abs((g.etype == e).sum() - 0.05 * 60480) < 5 * np.sqrt(60480 * 0.05)


def test_program_graph_config_edges():
    g = make_graphs(PROGRAM_GRAPH)[0]
    assert g.n == 20000 and g.m == 2 * 19999 * 10


def test_batch_sizes_first_fit():
    s = lognormal_batch_sizes(2, 100000, 2000, 1.2, 100, 20000)
    assert sum(s) <= 100000 and min(s) >= 100 and max(s) <= 20000
    assert sum(s) > 99000
    s4 = lognormal_batch_sizes(4, 1048576, 5000, 1.2, 100, 20000)
    assert sum(s4) <= 1048576 and len(s4) > 100


def test_sweep_graph_density():
    for spec in sweep_blocks()[:3]:
        g = make_graphs(spec)[0]
        assert np.abs(g.src - g.dst).max() < spec.B
        deg = g.m / (spec.E * spec.n)
        assert abs(deg - 3.0) < 0.05


def test_params_padding_and_rounding():
    p = draw_params(3, 1000, 1024, 32, 2, "bf16", with_bias=True)
    assert np.all(p.X[1000:] == 0) and np.all(p.G[1000:] == 0)
    assert np.array_equal(round_bf16(p.X), p.X) and np.array_equal(round_bf16(p.W), p.W)
    assert p.bias.shape == (2, 32)
    assert abs(p.W.std() - 1 / np.sqrt(32)) < 0.01
    assert np.abs(p.Wi).max() <= 1 / np.sqrt(32)


def test_round_bf16_matches_torch():
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(0).standard_normal(20000).astype(np.float32) * 100
    assert np.array_equal(round_bf16(x), torch.from_numpy(x).to(torch.bfloat16).double().numpy())
