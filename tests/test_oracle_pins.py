"""Pins of the CPU oracle against things other than itself.

Each test ties one oracle function to the mathematics the paper fixes: a
dense-matrix form of Eq. 1, a library routine (scipy.sparse, torch's GRUCell,
torch autograd), closed forms, a hand-worked fixture, central finite
differences, or an invariance (relabelling, supergraph independence).
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp
from scipy.sparse.csgraph import reverse_cuthill_mckee, connected_components, breadth_first_order

import oracle as O
from ggnn_synth import BATCH_100K, TINY, make_graphs, backbone_graph, scramble_graph, local_window_graph

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_edges(rng, n, m, E, span=None):
    src = rng.integers(0, n, m)
    if span is None:
        dst = rng.integers(0, n, m)
    else:
        dst = np.clip(src + rng.integers(-span, span + 1, m), 0, n - 1)
    return src, dst, rng.integers(0, E, m)


def _rand_params(rng, n, H, E):
    X = rng.standard_normal((n, H))
    W = rng.standard_normal((E, H, H)) / np.sqrt(H)
    k = 1 / np.sqrt(H)
    Wi = rng.uniform(-k, k, (H, 3 * H))
    U = rng.uniform(-k, k, (H, 3 * H))
    b = rng.uniform(-k, k, 3 * H)
    bias = rng.uniform(-k, k, (E, H))
    G = rng.standard_normal((n, H))
    return X, W, Wi, U, b, bias, G


# --------------------------------------------------------------------------
# aggregation: dense adjacency, scipy.sparse, Eq. 3 band, Eq. 2, closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_aggregate_equals_dense_adjacency_matmul(seed):
    rng = np.random.default_rng(seed)
    n, E, H = 40, 3, 5
    src, dst, et = _rand_edges(rng, n, 300, E)
    M = rng.standard_normal((E, n, H))
    # Eq. 1 with dense 0/1 matrices A_e, a_ij = 1 iff an edge j -> i of type e
    A = np.zeros((E, n, n))
    for s_, d_, e_ in zip(src, dst, et):
        A[e_, d_, s_] = 1.0
    want = sum(A[e] @ M[e] for e in range(E))
    s, d, e, _ = O.dedupe_edges(src, dst, et)
    got = O.aggregate(n, s, d, e, M)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    # the transpose: dM_e = A_e^T da
    da = rng.standard_normal((n, H))
    got_t = O.aggregate_transpose(n, s, d, e, da, E)
    np.testing.assert_allclose(got_t, np.stack([A[k].T @ da for k in range(E)]), rtol=0, atol=1e-12)


def test_aggregate_equals_scipy_sparse():
    rng = np.random.default_rng(7)
    n, E, H = 500, 4, 8
    src, dst, et = _rand_edges(rng, n, 6000, E, span=30)
    M = rng.standard_normal((E, n, H))
    want = np.zeros((n, H))
    for k in range(E):
        sel = et == k
        A = sp.coo_matrix((np.ones(sel.sum()), (dst[sel], src[sel])), shape=(n, n)).tocsr()
        A.data[:] = 1.0          # repeated entries are one edge
        want += A @ M[k]
    s, d, e, _ = O.dedupe_edges(src, dst, et)
    np.testing.assert_allclose(O.aggregate(n, s, d, e, M), want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("B", [4, 8, 16])
def test_band_three_products_equal_scatter_on_kept_edges(B):
    rng = np.random.default_rng(B)
    nb, E, H = 6, 3, 4
    n = nb * B
    src, dst, et = _rand_edges(rng, n, 400, E, span=2 * B + 3)
    M = rng.integers(-4, 5, (E, n, H)).astype(np.float64)
    band = O.pack_band(n, E, B, src, dst, et)
    s, d, e, ndrop, ndup = O.kept_edges(src, dst, et, B)
    assert ndrop > 0, "the case should exercise the drop rule"
    np.testing.assert_array_equal(O.banded_apply(band, M), O.aggregate(n, s, d, e, M))


def test_block_diagonal_case_is_one_batched_matmul():
    """Eq. 2: with edges only inside diagonal blocks, A M = BMM(C, M_k)."""
    rng = np.random.default_rng(3)
    nb, B, H = 5, 8, 3
    n = nb * B
    C = (rng.random((nb, B, B)) < 0.3).astype(np.float64)
    k, r, c = np.nonzero(C)
    src, dst, et = k * B + c, k * B + r, np.zeros(len(k), np.int64)
    M = rng.integers(-3, 4, (1, n, H)).astype(np.float64)
    want = np.matmul(C, M[0].reshape(nb, B, H)).reshape(n, H)
    np.testing.assert_array_equal(O.aggregate(n, src, dst, et, M), want)
    band = O.pack_band(n, 1, B, src, dst, et)
    np.testing.assert_array_equal(band[0, :, 1], C)
    assert band[:, :, 0].sum() == 0 and band[:, :, 2].sum() == 0


def test_closed_forms_of_aggregation():
    B, nb, E, H = 4, 5, 2, 3
    n = nb * B
    rng = np.random.default_rng(11)
    M = rng.standard_normal((E, n, H))
    idx = np.arange(n)
    # self-loops of every type: a = sum_e M_e
    src = np.concatenate([idx, idx]); dst = src.copy(); et = np.repeat([0, 1], n)
    band = O.pack_band(n, E, B, src, dst, et)
    np.testing.assert_allclose(O.banded_apply(band, M), M.sum(0), atol=1e-13)
    np.testing.assert_allclose(O.aggregate(n, src, dst, et, M), M.sum(0), atol=1e-13)
    # chain i-1 -> i: a[i] = M[i-1], a[0] = 0; crosses into the L block at i = kB
    src, dst, et = idx[:-1], idx[1:], np.zeros(n - 1, np.int64)
    want = np.zeros((n, H)); want[1:] = M[0, :-1]
    band = O.pack_band(n, E, B, src, dst, et)
    assert band[0, 1:, 0].sum() == nb - 1          # one L entry per block boundary
    np.testing.assert_allclose(O.banded_apply(band, M), want, atol=1e-13)
    # chain i+1 -> i: a[i] = M[i+1]; U slot at the boundary
    src, dst = idx[1:], idx[:-1]
    want = np.zeros((n, H)); want[:-1] = M[0, 1:]
    band = O.pack_band(n, E, B, src, dst, et)
    assert band[0, :-1, 2].sum() == nb - 1
    np.testing.assert_allclose(O.banded_apply(band, M), want, atol=1e-13)
    # |i-j| < B always kept; |i-j| = B always kept; |i-j| = 2B never kept
    for span, kept in [(B - 1, True), (B, True), (2 * B, False)]:
        s_ = idx[: n - span]; d_ = s_ + span
        _, _, _, ndrop, _ = O.kept_edges(s_, d_, np.zeros_like(s_), B)
        assert (ndrop == 0) == kept
        _, _, _, ndrop, _ = O.kept_edges(d_, s_, np.zeros_like(s_), B)
        assert (ndrop == 0) == kept


def test_hand_worked_fixture():
    with open(os.path.join(GOLDEN, "hand_band_example.json")) as f:
        g = json.load(f)
    n, B, E = g["n"], g["B"], g["E"]
    j = np.arange(n, dtype=np.float64)
    M = np.stack([np.stack([j, np.ones(n)], 1), np.stack([10 * j, -np.ones(n)], 1)])
    ed = np.asarray(g["edges_src_dst_type"])
    s, d, e, ndrop, ndup = O.kept_edges(ed[:, 0], ed[:, 1], ed[:, 2], B)
    assert (ndrop, ndup) == (g["expected_n_dropped"], g["expected_n_duplicate"])
    np.testing.assert_array_equal(O.aggregate(n, s, d, e, M), np.asarray(g["expected_a"], float))
    band = O.pack_band(n, E, B, ed[:, 0], ed[:, 1], ed[:, 2])
    assert sorted(map(tuple, np.argwhere(band).tolist())) == sorted(map(tuple, g["expected_slots_e_k_s_r_c"]))
    np.testing.assert_array_equal(O.banded_apply(band, M), np.asarray(g["expected_a"], float))
    da = np.stack([j, np.ones(n)], 1)
    dM = O.aggregate_transpose(n, s, d, e, da, E)
    want = np.zeros_like(dM)
    for ee, jj, v in g["expected_dM_nonzero_e_j_value"]:
        want[ee, jj] = v
    np.testing.assert_array_equal(dM, want)


# --------------------------------------------------------------------------
# packing
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(3))
def test_pack_unpack_roundtrip_and_slots(seed):
    rng = np.random.default_rng(100 + seed)
    B, nb, E = 8, 7, 3
    n = B * nb
    src, dst, et = _rand_edges(rng, n, 700, E, span=3 * B)
    band = O.pack_band(n, E, B, src, dst, et)
    s, d, e, ndrop, _ = O.kept_edges(src, dst, et, B)
    us, ud, ue = O.unpack_band(band)
    assert set(zip(us.tolist(), ud.tolist(), ue.tolist())) == set(zip(s.tolist(), d.tolist(), e.tolist()))
    assert band.sum() == len(s)
    assert set(np.unique(band).tolist()) <= {0.0, 1.0}
    assert band[:, 0, 0].sum() == 0 and band[:, nb - 1, 2].sum() == 0


def test_triangularity_when_bandwidth_below_block():
    """Eq. 3 remark: with bandwidth <= B-1 the U blocks are strictly lower and
    the L blocks strictly upper triangular."""
    rng = np.random.default_rng(5)
    B, nb, E = 8, 6, 2
    n = B * nb
    src, dst, et = _rand_edges(rng, n, 500, E, span=B - 1)
    assert O.bandwidth(src, dst) <= B - 1
    band = O.pack_band(n, E, B, src, dst, et)
    U, L = band[:, :, 2], band[:, :, 0]
    assert np.all(np.triu(U) == 0)
    assert np.all(np.tril(L) == 0)


# --------------------------------------------------------------------------
# RCM
# --------------------------------------------------------------------------

def _is_perm(order, n):
    return sorted(order.tolist()) == list(range(n))


def test_rcm_path_graph_recovers_bandwidth_one():
    n = 300
    rng = np.random.default_rng(0)
    perm = rng.permutation(n)
    src, dst = perm[:-1], perm[1:]
    order, rank = O.rcm_order(n, src, dst)
    assert _is_perm(order, n)
    ns, nd = O.relabel(rank, src, dst)
    assert O.bandwidth(ns, nd) == 1
    # start is an endpoint of the path (pseudo-peripheral), the order is the path
    path = perm.tolist()
    assert order.tolist() in (path, path[::-1])


def test_rcm_star_closed_form():
    """Star with hub 0 and leaves 1..k: the start is leaf 1 (smallest degree,
    then label); the search visits hub 0 then leaves 2..k; reversed."""
    k = 9
    src = np.zeros(k, np.int64); dst = np.arange(1, k + 1)
    order, _ = O.rcm_order(k + 1, src, dst)
    assert order.tolist() == ([1, 0] + list(range(2, k + 1)))[::-1]


def test_rcm_components_contiguous_and_levels_monotone():
    rng = np.random.default_rng(9)
    parts, off = [], 0
    for sz in [50, 1, 80, 2, 30]:
        g = backbone_graph(99, len(parts), sz, 2, span_mean=3.0, max_span=10)
        parts.append((g.src + off, g.dst + off)); off += sz
    n = off
    perm = rng.permutation(n)
    src = perm[np.concatenate([p[0] for p in parts])]
    dst = perm[np.concatenate([p[1] for p in parts])]
    order, rank = O.rcm_order(n, src, dst)
    assert _is_perm(order, n)
    A = sp.coo_matrix((np.ones(len(src)), (src, dst)), shape=(n, n)).tocsr()
    A = ((A + A.T) > 0).astype(np.float64)
    ncomp, lab = connected_components(A, directed=False)
    assert ncomp == 5
    cm = order[::-1]                                # Cuthill-McKee order
    pos_lab = lab[cm]
    # every component occupies one contiguous range
    changes = np.count_nonzero(pos_lab[1:] != pos_lab[:-1])
    assert changes == ncomp - 1
    # components are taken in order of their smallest label
    firsts = [lab[v] for v in range(n)]
    comp_order = list(dict.fromkeys(firsts))
    assert list(dict.fromkeys(pos_lab.tolist())) == comp_order
    # inside a component the search order never goes back a level
    for c in range(ncomp):
        seq = cm[pos_lab == c]
        dist = sp.csgraph.shortest_path(A, indices=int(seq[0]), unweighted=True)
        lv = dist[seq]
        assert np.all(np.diff(lv) >= 0)
        bfs = breadth_first_order(A, int(seq[0]), directed=False, return_predecessors=False)
        assert set(bfs.tolist()) == set(seq.tolist())


def test_rcm_quality_on_program_graph_shape():
    """Within 25% of scipy's reverse Cuthill-McKee on a scrambled backbone
    graph, and inside the 128 band that the bf16 workloads use."""
    g = backbone_graph(1, 0, 4000, 10)
    g, _ = scramble_graph(1, 0, g)
    order, rank = O.rcm_order(g.n, g.src, g.dst)
    assert _is_perm(order, g.n)
    beta = O.bandwidth(*O.relabel(rank, g.src, g.dst))
    A = sp.coo_matrix((np.ones(g.m), (g.src, g.dst)), shape=(g.n, g.n)).tocsr()
    A = ((A + A.T) > 0).astype(np.float64)
    p = reverse_cuthill_mckee(A.tocsr(), symmetric_mode=True)
    rk = np.empty(g.n, np.int64); rk[p] = np.arange(g.n)
    beta_sp = O.bandwidth(rk[g.src], rk[g.dst])
    assert beta <= 1.25 * beta_sp
    assert beta <= 128
    assert O.bandwidth(g.src, g.dst) > 1000   # the scramble really destroyed the band


# --------------------------------------------------------------------------
# message transform and GRU
# --------------------------------------------------------------------------

def test_msg_transform_against_per_type_matmul():
    rng = np.random.default_rng(1)
    X, W, *_ , bias, _ = _rand_params(rng, 30, 6, 4)
    M = O.msg_transform(X, W, bias)
    for e in range(4):
        np.testing.assert_allclose(M[e], X @ W[e] + bias[e], atol=1e-13)


def test_gru_matches_torch_grucell_when_reset_is_open():
    """With r == 1 (b_r = +40) the Cho form and torch's GRUCell coincide."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    n, H = 17, 6
    a = rng.standard_normal((n, H)); h = rng.standard_normal((n, H))
    Wi = rng.uniform(-.3, .3, (H, 3 * H)); U = rng.uniform(-.3, .3, (H, 3 * H))
    b = rng.uniform(-.3, .3, 3 * H); b[:H] = 40.0
    cell = torch.nn.GRUCell(H, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(Wi.T.copy()))
        cell.weight_hh.copy_(torch.from_numpy(U.T.copy()))
        cell.bias_ih.copy_(torch.from_numpy(b))
        cell.bias_hh.zero_()
        want = cell(torch.from_numpy(a), torch.from_numpy(h)).numpy()
    got, r, z, nn = O.gru_forward(a, h, Wi, U, b)
    np.testing.assert_allclose(r, 1.0, atol=1e-14)
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_gru_closed_forms():
    rng = np.random.default_rng(4)
    n, H = 5, 4
    a = rng.standard_normal((n, H)); h = rng.standard_normal((n, H))
    Wi = rng.standard_normal((H, 3 * H)); U = rng.standard_normal((H, 3 * H))
    b = np.zeros(3 * H); b[H:2 * H] = 40.0                 # z == 1: state kept
    np.testing.assert_allclose(O.gru_forward(a, h, Wi, U, b)[0], h, atol=1e-14)
    b = rng.standard_normal(3 * H); b[H:2 * H] = -40.0     # z == 0, no inputs: tanh(b_n)
    hn = O.gru_forward(a, h, 0 * Wi, 0 * U, b)[0]
    np.testing.assert_allclose(hn, np.tile(np.tanh(b[2 * H:]), (n, 1)), atol=1e-14)


def test_gru_reset_gate_acts_before_state_weights():
    """H = 2, z = 1/2, r = (1, 0), U_n swaps the two features: the Cho form
    gives n = tanh((r*h) U_n) = (0, tanh(h1)), hence h' = (h1/2, (h2 + tanh(h1))/2).
    (Applying r after U_n would give (h1/2 + tanh(h2)/2, h2/2) instead.)"""
    H = 2
    h = np.array([[0.7, -1.3]])
    a = np.zeros((1, H))
    Wi = np.zeros((H, 3 * H)); U = np.zeros((H, 3 * H))
    U[:, 2 * H:] = [[0.0, 1.0], [1.0, 0.0]]
    b = np.zeros(3 * H); b[0], b[1] = 40.0, -40.0
    hn = O.gru_forward(a, h, Wi, U, b)[0]
    h1, h2 = h[0]
    np.testing.assert_allclose(hn[0], [h1 / 2, (h2 + np.tanh(h1)) / 2], atol=1e-14)


# --------------------------------------------------------------------------
# gradients: finite differences and torch autograd
# --------------------------------------------------------------------------

def _small_case(seed, n=24, B=8, E=2, H=4, m=120, T=2):
    rng = np.random.default_rng(seed)
    src, dst, et = _rand_edges(rng, n, m, E, span=2 * B)
    X, W, Wi, U, b, bias, G = _rand_params(rng, n, H, E)
    return dict(n=n, B=B, src=src, dst=dst, etype=et, X0=X, W=W, Wi=Wi, U=U, b=b, bias=bias, G=G, T=T)


def _loss(c, **over):
    d = dict(c); d.update(over)
    out = O.propagate(d["n"], d["B"], d["src"], d["dst"], d["etype"], d["X0"], d["W"], d["Wi"], d["U"], d["b"],
                      d["T"], bias=d["bias"])
    return float(np.sum(d["G"] * out["X"][-1]))


@pytest.mark.parametrize("seed", [0, 1])
def test_gradients_match_central_finite_differences(seed):
    c = _small_case(seed)
    out = O.propagate(c["n"], c["B"], c["src"], c["dst"], c["etype"], c["X0"], c["W"], c["Wi"], c["U"], c["b"],
                      c["T"], G=c["G"], bias=c["bias"])
    assert out["n_dropped"] > 0
    grads = {"X0": out["dX0"], "W": out["dW"], "bias": out["dbias"], "Wi": out["dWi"], "U": out["dU"], "b": out["db"]}
    rng = np.random.default_rng(1000 + seed)
    eps = 1e-5
    for name, gr in grads.items():
        base = c[name]
        for _ in range(4):                       # random directions
            v = rng.standard_normal(base.shape); v /= np.linalg.norm(v)
            fd = (_loss(c, **{name: base + eps * v}) - _loss(c, **{name: base - eps * v})) / (2 * eps)
            an = float(np.sum(gr * v))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)
        flat = rng.choice(base.size, size=min(8, base.size), replace=False)
        for f in flat:                           # coordinates
            v = np.zeros(base.size); v[f] = 1.0; v = v.reshape(base.shape)
            fd = (_loss(c, **{name: base + eps * v}) - _loss(c, **{name: base - eps * v})) / (2 * eps)
            assert abs(fd - gr.reshape(-1)[f]) <= 1e-6 * max(1.0, abs(fd)), (name, f)


def test_gru_gate_gradients_are_derivatives_in_the_gate_biases():
    """The gate gradients [r^, z^, n^] are dL/d(pre-activation): giving every
    node its own copy of the gate bias (b as an [n, 3H] matrix) makes row i
    of the bias gradient exactly row i of them; central differences of
    L = sum(g * h') in each such per-node bias entry must agree."""
    rng = np.random.default_rng(31)
    n, H = 6, 3
    a = rng.standard_normal((n, H)); h = rng.standard_normal((n, H))
    Wi = rng.standard_normal((H, 3 * H)) * 0.5; U = rng.standard_normal((H, 3 * H)) * 0.5
    b = rng.standard_normal((n, 3 * H)) * 0.3
    g = rng.standard_normal((n, H))
    _, r, z, nn = O.gru_forward(a, h, Wi, U, b)
    ghat = O.gru_gate_gradients(g, h, r, z, nn, U)
    assert ghat.shape == (n, 3 * H)
    eps = 1e-6
    for i in range(n):
        for c in range(3 * H):
            bp, bm = b.copy(), b.copy()
            bp[i, c] += eps
            bm[i, c] -= eps
            fd = (np.sum(g * O.gru_forward(a, h, Wi, U, bp)[0]) - np.sum(g * O.gru_forward(a, h, Wi, U, bm)[0])) / (2 * eps)
            assert abs(fd - ghat[i, c]) <= 1e-7 * max(1.0, abs(fd)), (i, c, fd, ghat[i, c])
    # and the reverse pass built on them: db is their column sum, dWi = a^T ghat
    _, _, dWi, _, db = O.gru_backward(g, a, h, r, z, nn, Wi, U)
    np.testing.assert_allclose(db, ghat.sum(axis=0), atol=1e-13)
    np.testing.assert_allclose(dWi, a.T @ ghat, atol=1e-13)


def test_gradients_match_torch_autograd():
    torch = pytest.importorskip("torch")
    c = _small_case(5, n=32, B=8, E=3, H=5, m=200, T=3)
    out = O.propagate(c["n"], c["B"], c["src"], c["dst"], c["etype"], c["X0"], c["W"], c["Wi"], c["U"], c["b"],
                      c["T"], G=c["G"], bias=c["bias"])
    s, d, e, _, _ = O.kept_edges(c["src"], c["dst"], c["etype"], c["B"])
    t = {k: torch.tensor(c[k], requires_grad=True) for k in ["X0", "W", "Wi", "U", "b", "bias"]}
    H = c["X0"].shape[1]
    h = t["X0"]
    si, di, ei = map(torch.from_numpy, (s, d, e))
    for _ in range(c["T"]):
        M = torch.einsum("nh,ehk->enk", h, t["W"]) + t["bias"][:, None, :]
        a = torch.zeros_like(h).index_add(0, di, M[ei, si])
        gi = a @ t["Wi"] + t["b"]
        r = torch.sigmoid(gi[:, :H] + h @ t["U"][:, :H])
        z = torch.sigmoid(gi[:, H:2 * H] + h @ t["U"][:, H:2 * H])
        nn_ = torch.tanh(gi[:, 2 * H:] + (r * h) @ t["U"][:, 2 * H:])
        h = z * h + (1 - z) * nn_
    (torch.from_numpy(c["G"]) * h).sum().backward()
    np.testing.assert_allclose(out["X"][-1], h.detach().numpy(), atol=1e-12)
    for k, ok in [("X0", "dX0"), ("W", "dW"), ("Wi", "dWi"), ("U", "dU"), ("b", "db"), ("bias", "dbias")]:
        np.testing.assert_allclose(out[ok], t[k].grad.numpy(), atol=1e-11, err_msg=k)


# --------------------------------------------------------------------------
# invariances
# --------------------------------------------------------------------------

def test_relabelling_equivariance():
    """Compilation section: outputs are equivariant to node permutation."""
    c = _small_case(8, n=24, B=24, T=2)      # one block: nothing is dropped
    rng = np.random.default_rng(8)
    pi = rng.permutation(c["n"])
    inv = np.argsort(pi)
    base = O.propagate(c["n"], c["B"], c["src"], c["dst"], c["etype"], c["X0"], c["W"], c["Wi"], c["U"], c["b"],
                       c["T"], G=c["G"], bias=c["bias"])
    per = O.propagate(c["n"], c["B"], pi[c["src"]], pi[c["dst"]], c["etype"], c["X0"][inv], c["W"], c["Wi"], c["U"],
                      c["b"], c["T"], G=c["G"][inv], bias=c["bias"])
    assert base["n_dropped"] == per["n_dropped"] == 0
    np.testing.assert_allclose(per["X"][-1], base["X"][-1][inv], atol=1e-12)
    np.testing.assert_allclose(per["dX0"], base["dX0"][inv], atol=1e-12)
    for k in ["dW", "dWi", "dU", "db", "dbias"]:
        np.testing.assert_allclose(per[k], base[k], atol=1e-11)


def test_supergraph_components_do_not_interact():
    """Background, sparse batching: graphs packed into one supergraph give the
    same rows as alone, and weight gradients add up."""
    B, E, H, T = 16, 2, 4, 2
    rng = np.random.default_rng(12)
    parts = []
    for gi, n in enumerate([40, 27, 33]):
        g = backbone_graph(77, gi, n, E, span_mean=2.0, max_span=6)
        parts.append((n, g.src, g.dst, g.etype))
    n_real, n_pad, src, dst, et, offs = O.batch_layout(parts, B)
    assert O.bandwidth(src, dst) <= B - 1
    X, W, Wi, U, b, bias, G = _rand_params(rng, n_pad, H, E)
    G[n_real:] = 0; X[n_real:] = 0
    full = O.propagate(n_pad, B, src, dst, et, X, W, Wi, U, b, T, G=G, bias=bias)
    acc = {k: 0 for k in ["dW", "dWi", "dU", "db", "dbias"]}
    for i, (n, s, d, e) in enumerate(parts):
        o = slice(offs[i], offs[i + 1])
        one = O.propagate(n, n, s, d, e, X[o], W, Wi, U, b, T, G=G[o], bias=bias)
        np.testing.assert_allclose(full["X"][-1][o], one["X"][-1], atol=1e-12)
        np.testing.assert_allclose(full["dX0"][o], one["dX0"], atol=1e-12)
        for k in acc:
            acc[k] = acc[k] + one[k]
    # padding rows have X = 0 and G = 0: they move only through the biases and
    # contribute nothing to the gradients
    for k in acc:
        np.testing.assert_allclose(full[k], acc[k], atol=1e-11)


def test_workload_graphs_fit_the_band_after_reordering():
    """The bf16 workloads are built so that reordering brings every edge into
    the 128 band (zero drops)."""
    for gi, g in enumerate(make_graphs(BATCH_100K, max_graphs=3)):
        order, rank = O.rcm_order(g.n, g.src, g.dst)
        s, d = O.relabel(rank, g.src, g.dst)
        assert O.bandwidth(s, d) <= BATCH_100K.B - 1, gi
    g = make_graphs(TINY)[0]
    assert O.bandwidth(g.src, g.dst) <= TINY.B - 1
