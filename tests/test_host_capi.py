"""Host side of the C-ABI, on the CPU: the library loads and exports every
declared symbol, reverse Cuthill-McKee and block packing are bit-exact
against the oracle, and argument validation reports errors."""
import os
import re

import numpy as np
import pytest

import oracle as O
from ggnn_synth import PROGRAM_GRAPH, make_graphs, backbone_graph, scramble_graph, local_window_graph

capi = pytest.importorskip("paper_1906_11786_amd.capi")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _need_lib():
    if not os.path.exists(capi.LIB_PATH):
        pytest.fail("libggnn.so is not built (python -m paper_1906_11786_amd.build)")


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "ggnn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ggnn_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    _need_lib()
    L = capi.lib()
    declared = _declared_functions()
    assert len(declared) >= 18
    for name in declared:
        assert hasattr(L, name), name
    assert set(declared) == set(capi.EXPORTS)
    header = open(os.path.join(ROOT, "include", "ggnn.h")).read()
    declared_abi = int(re.search(r"#define GGNN_ABI_VERSION (\d+)", header).group(1))
    assert capi.ggnn_abi_version() == capi.ABI_VERSION == declared_abi
    assert capi.ggnn_status_string(3) == "GGNN_ERR_OUT_OF_BAND"


def _graphs():
    out = []
    g = backbone_graph(11, 0, 3000, 4, span_mean=8.0)
    out.append(scramble_graph(11, 0, g)[0])
    out.append(local_window_graph(12, 0, 700, 3, 40, 0.02))     # several components, isolated nodes likely
    rng = np.random.default_rng(5)
    n = 400
    s = rng.integers(0, n, 600); d = rng.integers(0, n, 600)
    out.append(type(g)(n, s.astype(np.int32), d.astype(np.int32), np.zeros(600, np.int32)))
    # path, star, empty, single node, self-loops only
    p = rng.permutation(50)
    out.append(type(g)(50, p[:-1].astype(np.int32), p[1:].astype(np.int32), np.zeros(49, np.int32)))
    out.append(type(g)(9, np.zeros(8, np.int32), np.arange(1, 9, dtype=np.int32), np.zeros(8, np.int32)))
    out.append(type(g)(7, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)))
    out.append(type(g)(1, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)))
    out.append(type(g)(5, np.arange(5, dtype=np.int32), np.arange(5, dtype=np.int32), np.zeros(5, np.int32)))
    return out


def test_rcm_bit_exact_against_oracle():
    _need_lib()
    for g in _graphs():
        order, rank, bw = capi.ggnn_rcm_order(g.n, g.src, g.dst)
        o_order, o_rank = O.rcm_order(g.n, g.src, g.dst)
        np.testing.assert_array_equal(order, o_order)
        np.testing.assert_array_equal(rank, o_rank)
        s, d = O.relabel(o_rank, g.src, g.dst)
        assert bw == O.bandwidth(s, d)
        assert capi.ggnn_bandwidth(g.n, g.src, g.dst, rank) == bw
        assert capi.ggnn_bandwidth(g.n, g.src, g.dst) == O.bandwidth(g.src, g.dst)


def test_batch_graphs_against_oracle_rcm_per_graph():
    """Sparse batching in the host library: each graph reordered alone and
    offset by the nodes before it, edges in order (oracle RCM per graph)."""
    _need_lib()
    from host_sanitized_cases import check_batch
    check_batch()
    # the composition the driver builds on: the program-graph batch keeps every graph's bandwidth below B
    gs = make_graphs(PROGRAM_GRAPH)
    s, d, offs, bw = capi.ggnn_batch_graphs([g.n for g in gs], [len(g.src) for g in gs],
                                            np.concatenate([g.src for g in gs]), np.concatenate([g.dst for g in gs]))
    assert offs[-1] == sum(g.n for g in gs) and bw == int(np.abs(s.astype(np.int64) - d).max()) <= PROGRAM_GRAPH.B - 1


def test_rcm_bit_exact_on_program_graph_workload():
    _need_lib()
    g = make_graphs(PROGRAM_GRAPH)[0]
    order, rank, bw = capi.ggnn_rcm_order(g.n, g.src, g.dst)
    o_order, _ = O.rcm_order(g.n, g.src, g.dst)
    np.testing.assert_array_equal(order, o_order)
    assert bw <= PROGRAM_GRAPH.B - 1


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B", [4, 8, 32])
def test_pack_bit_exact_against_oracle(dt, B):
    _need_lib()
    rng = np.random.default_rng(B)
    nb, E = 9, 3
    n = nb * B
    src = rng.integers(0, n, 900)
    dst = np.clip(src + rng.integers(-3 * B, 3 * B + 1, 900), 0, n - 1)
    et = rng.integers(0, E, 900)
    src = np.concatenate([src, src[:50]]); dst = np.concatenate([dst, dst[:50]]); et = np.concatenate([et, et[:50]])
    band, packed, dropped, dup = capi.ggnn_banded_pack(n, E, B, src, dst, et, dt=dt)
    ob = O.pack_band(n, E, B, src, dst, et)
    s, d, e, odrop, odup = O.kept_edges(src, dst, et, B)
    bits = (band == (1.0 if dt == "f32" else 0x3F80))
    assert set(np.unique(band).tolist()) <= ({0.0, 1.0} if dt == "f32" else {0, 0x3F80})
    np.testing.assert_array_equal(bits, ob == 1.0)
    assert (packed, dropped, dup) == (len(s), odrop, odup)
    assert dropped > 0 and dup >= 50


def test_pack_with_rank_equals_pack_of_relabelled_edges():
    _need_lib()
    g = scramble_graph(13, 0, backbone_graph(13, 0, 1000, 2))[0]
    order, rank, bw = capi.ggnn_rcm_order(g.n, g.src, g.dst)
    n_pad = 1024
    rk = np.concatenate([rank, np.arange(g.n, n_pad, dtype=np.int32)])
    a, *ca = capi.ggnn_banded_pack(n_pad, 2, 32, g.src, g.dst, g.etype, rank=rk, dt="bf16")
    s, d = O.relabel(rank, g.src, g.dst)
    b, *cb = capi.ggnn_banded_pack(n_pad, 2, 32, s, d, g.etype, dt="bf16")
    np.testing.assert_array_equal(a, b)
    assert ca == cb


def test_pack_strict_and_validation_errors():
    _need_lib()
    src = np.array([0, 100]); dst = np.array([1, 0]); et = np.array([0, 0])
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_banded_pack(128, 1, 32, src, dst, et, strict=True)
    assert ei.value.status_name == "GGNN_ERR_OUT_OF_BAND"
    _, p, d, u = capi.ggnn_banded_pack(128, 1, 32, src, dst, et, strict=False)
    assert (p, d, u) == (1, 1, 0)
    bad = [
        dict(n_pad=100, E=1, B=32, src=src, dst=dst, et=et),            # n_pad not a multiple of B
        dict(n_pad=128, E=1, B=32, src=np.array([128]), dst=np.array([0]), et=np.array([0])),  # id out of range
        dict(n_pad=128, E=1, B=32, src=src, dst=dst, et=np.array([0, 1])),  # type out of range
        dict(n_pad=128, E=0, B=32, src=src, dst=dst, et=et),            # no edge types
    ]
    for kw in bad:
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_banded_pack(kw["n_pad"], kw["E"], kw["B"], kw["src"], kw["dst"], kw["et"])
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG"
        assert capi.ggnn_last_error().startswith("GGNN_ERR_INVALID_ARG")
    with pytest.raises(capi.GGNNError):
        capi.ggnn_rcm_order(3, [0, 5], [1, 2])
    assert capi.ggnn_band_bytes(512, 2, 64, "f32") == 2 * 8 * 3 * 64 * 64 * 4
    assert capi.ggnn_band_bytes(20096, 10, 128, "bf16") == 10 * 157 * 3 * 128 * 128 * 2
    assert capi.ggnn_band_bytes(100, 2, 64, "f32") == 0


def test_device_entry_points_validate_before_touching_the_gpu():
    """Invalid sizes are rejected on the host, so this runs without a GPU."""
    _need_lib()
    for H in [16, 48, 512]:
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_msg_transform("bf16", 128, H, 2, 16, 16, None, 16, stream=0)
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG"
    with pytest.raises(capi.GGNNError):
        capi.ggnn_banded_propagate("bf16", 96, 64, 64, 2, 16, 16, 16, stream=0)   # 96 % 64 != 0
    with pytest.raises(capi.GGNNError):
        capi.ggnn_banded_propagate("bf16", 128, 48, 64, 2, 16, 16, 16, stream=0)  # unsupported B
    with pytest.raises(capi.GGNNError):
        capi.ggnn_banded_propagate("bf16", 128, 64, 64, 2, None, 16, 16, stream=0)  # NULL band
    with pytest.raises(capi.GGNNError):
        capi.ggnn_banded_propagate("bf16", 128, 64, 64, 2, 8, 16, 16, stream=0)   # misaligned band
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_gru_update_bwd("bf16", 128, 64, 16, 16, 16, 16, 16, 16, 16, 32, 16, 16, 16, 16, 0, stream=0)
    assert ei.value.status_name == "GGNN_ERR_WORKSPACE"
    assert capi.ggnn_gru_update_bwd_workspace_bytes("bf16", 20096, 64) > 0
    assert capi.ggnn_msg_transform_bwd_workspace_bytes("bf16", 20096, 64, 10) > 0
    assert capi.ggnn_msg_transform_bwd_workspace_bytes("bf16", 20096, 48, 10) == 0


def test_training_entry_points_validate_before_touching_the_gpu():
    """Readout, loss and Momentum update reject bad arguments on the host."""
    _need_lib()
    P = 16   # a 16-byte aligned stand-in address; nothing is launched
    bad_readout = [
        dict(n_graphs=0), dict(n_cand=-1), dict(H=48), dict(X=None), dict(cand_ptr=None), dict(loss=8),
    ]
    for over in bad_readout:
        kw = dict(dt="bf16", n_pad=128, H=64, n_graphs=2, n_cand=4, X=P, w_out=P, b_out=P, cand_node=P, cand_ptr=P,
                  target=P, logits=P, loss=P, dlogit=P)
        kw.update(over)
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_readout_loss(**kw, stream=0)
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG", over
    need = capi.ggnn_readout_loss_bwd_workspace_bytes(64, 1000)
    assert need == 16 * 65 * 4   # one partial row of H + 1 floats per block of 64 candidates
    assert capi.ggnn_readout_loss_bwd_workspace_bytes(48, 10) == 0
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_readout_loss_bwd("bf16", 128, 64, 1000, P, P, P, P, P, P, P, P, need - 4, stream=0)
    assert ei.value.status_name == "GGNN_ERR_WORKSPACE"
    for args in [dict(count=-1), dict(momentum=-0.5), dict(weight_decay=-1.0), dict(lr=float("nan")),
                 dict(param=None), dict(velocity=P, param=P), dict(param_copy=P, param=P)]:
        kw = dict(count=10, param=P, velocity=32, grad=48, lr=0.1, momentum=0.9)
        kw.update(args)
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_sgd_momentum(**kw, stream=0)
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG", args
    capi.ggnn_sgd_momentum(0, None, None, None, 0.1, 0.9, stream=0)   # nothing to do: OK


def test_gru_pack_sizes_and_validation_before_touching_the_gpu():
    """Packed GRU weights: 12 H^2 bf16 elements where the large-width kernels
    read them, nothing elsewhere (the call is then a no-op); bad pointers and
    overlaps are rejected on the host."""
    _need_lib()
    assert capi.ggnn_gru_pack_bytes("bf16", 128) == 12 * 128 * 128 * 2
    assert capi.ggnn_gru_pack_bytes("bf16", 256) == 12 * 256 * 256 * 2
    for dt, H in [("bf16", 32), ("bf16", 64), ("f32", 128), ("f32", 256), ("bf16", 48)]:
        assert capi.ggnn_gru_pack_bytes(dt, H) == 0, (dt, H)
    capi.ggnn_gru_pack_weights("f32", 128, None, None, None, stream=0)   # nothing to pack: OK
    capi.ggnn_gru_pack_weights("bf16", 64, None, None, None, stream=0)
    H = 128
    wb = H * 3 * H * 2
    Wi, U, pk = 1 << 20, 2 << 20, 4 << 20   # 16-byte aligned stand-in addresses; nothing is launched
    for args in [(None, U, pk), (Wi, U, None), (Wi + 8, U, pk), (Wi, U, Wi + wb - 16), (Wi, U, U - 16),
                 (Wi, U, Wi - capi.ggnn_gru_pack_bytes("bf16", H) + 16)]:
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_gru_pack_weights("bf16", H, *args, stream=0)
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG", args
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_gru_pack_weights("bf16", 48, Wi, U, pk, stream=0)
    assert ei.value.status_name == "GGNN_ERR_INVALID_ARG"


def test_step_bits_gru_rejects_overlapping_state_buffers():
    """The fused forward step reads neighbour rows of X while writing h_out:
    any shared byte is rejected on the host (nothing is launched)."""
    _need_lib()
    n_pad, B, H, E = 256, 64, 64, 2
    xb = n_pad * H * 2
    X = 1 << 24
    P = 1 << 28   # 16-byte aligned stand-in addresses for the other operands
    for h_out in (X, X + xb - 16, X - xb + 16):
        with pytest.raises(capi.GGNNError) as ei:
            capi.ggnn_step_bits_gru("bf16", n_pad, B, H, E, P, X, P, None, None, P, P, P, P, h_out, P, stream=0)
        assert ei.value.status_name == "GGNN_ERR_INVALID_ARG", h_out
        assert "overlap" in capi.ggnn_last_error()


def test_candidate_lists_are_checked_on_the_host():
    """The readout's reverse writes each candidate's dX row once: repeated
    nodes, ids outside the supergraph, malformed offsets and targets outside
    a list are refused before anything reaches the device."""
    from ggnn_synth.readout import Candidates, draw_candidates
    from paper_1906_11786_amd.driver import check_candidates
    good = draw_candidates(1, np.array([0, 50, 120, 121, 400]))
    check_candidates(good, 512)
    i32 = lambda *v: np.array(v, np.int32)
    bad = [
        Candidates(i32(3, 7, 3), i32(0, 3), i32(0)),            # node 3 twice in one graph
        Candidates(i32(3, 7, 9, 7), i32(0, 2, 4), i32(0, 1)),   # node 7 in two graphs
        Candidates(i32(3, 600), i32(0, 2), i32(0)),             # id beyond n_pad
        Candidates(i32(3, 4), i32(0, 3), i32(0)),               # offsets do not end at the count
        Candidates(i32(3, 4), i32(0, 2), i32(2)),               # target outside the list
        Candidates(i32(3, 4), i32(0, 2), i32(0, 0)),            # one target per graph
    ]
    for c in bad:
        with pytest.raises(ValueError):
            check_candidates(c, 512)


def _unpack_bits(bits):
    return np.unpackbits(bits, axis=-1, bitorder="little").astype(np.float64)


@pytest.mark.parametrize("B", [8, 32, 64])
def test_pack_bits_bit_exact_against_oracle(B):
    _need_lib()
    rng = np.random.default_rng(300 + B)
    nb, E = 7, 3
    n = nb * B
    src = rng.integers(0, n, 1200)
    dst = np.clip(src + rng.integers(-3 * B, 3 * B + 1, 1200), 0, n - 1)
    et = rng.integers(0, E, 1200)
    src = np.concatenate([src, src[:40]]); dst = np.concatenate([dst, dst[:40]]); et = np.concatenate([et, et[:40]])
    bits, bits_t, packed, dropped, dup = capi.ggnn_banded_pack_bits(n, E, B, src, dst, et)
    assert bits.shape == (E, nb, 3, B, B // 8)
    assert capi.ggnn_band_bits_bytes(n, E, B) == bits.nbytes
    band = O.pack_band(n, E, B, src, dst, et)
    np.testing.assert_array_equal(_unpack_bits(bits), band)
    s, d, e, odrop, odup = O.kept_edges(src, dst, et, B)
    assert (packed, dropped, dup) == (len(s), odrop, odup)
    # transposed blocks with roles swapped: bits_t[e][j][s] = band[e][j-1+s][2-s]^T
    bt = _unpack_bits(bits_t)
    for j in range(nb):
        for sl in range(3):
            kr = j - 1 + sl
            want = band[:, kr, 2 - sl].transpose(0, 2, 1) if 0 <= kr < nb else np.zeros((E, B, B))
            np.testing.assert_array_equal(bt[:, j, sl], want)
    # and, semantically, the transposed band applied to da is the oracle's gather
    da = rng.integers(-3, 4, (n, 5)).astype(np.float64)
    dap = np.zeros((nb + 2, B, 5)); dap[1:nb + 1] = da.reshape(nb, B, 5)
    dM = np.zeros((E, nb, B, 5))
    for sl in range(3):
        dM += np.einsum("ejcr,jrh->ejch", bt[:, :, sl], dap[sl:sl + nb])
    np.testing.assert_array_equal(dM.reshape(E, n, 5), O.aggregate_transpose(n, s, d, e, da, E))


def test_pack_bits_strict_and_errors():
    _need_lib()
    src = np.array([0, 100]); dst = np.array([1, 0]); et = np.array([0, 0])
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_banded_pack_bits(128, 1, 32, src, dst, et, strict=True)
    assert ei.value.status_name == "GGNN_ERR_OUT_OF_BAND"
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_banded_pack_bits(120, 1, 12, src, dst, et)      # B not a multiple of 8
    assert ei.value.status_name == "GGNN_ERR_INVALID_ARG"
    bits, bits_t, *_ = capi.ggnn_banded_pack_bits(128, 1, 32, src, dst, et, with_transpose=False)
    assert bits_t is None and int(np.unpackbits(bits).sum()) == 1


def test_sparse_csr_bit_exact_against_oracle_dedupe():
    """Receiver-major lists of every edge: rows (receiver, type), senders
    ascending, duplicates merged -- the oracle's deduplicated edge set."""
    _need_lib()
    rng = np.random.default_rng(11)
    n, E, m = 300, 5, 4000
    src = rng.integers(0, n, m)
    dst = rng.integers(0, n, m)
    et = rng.integers(0, E, m)
    src[:50], dst[:50], et[:50] = src[50:100], dst[50:100], et[50:100]      # planted duplicates
    row_ptr, col, dup = capi.ggnn_sparse_csr(n, E, src, dst, et)
    s, d, e, ndup = O.dedupe_edges(src, dst, et)
    assert dup == ndup and len(col) == len(s)
    order = np.lexsort((s, e, d))
    np.testing.assert_array_equal(col, s[order])
    want_ptr = np.concatenate([[0], np.cumsum(np.bincount(d * E + e, minlength=n * E))])
    np.testing.assert_array_equal(row_ptr, want_ptr)
    # empty edge list, and errors
    rp, c, dup = capi.ggnn_sparse_csr(64, 2, [], [], [])
    assert (rp == 0).all() and len(c) == 0 and dup == 0
    with pytest.raises(capi.GGNNError):
        capi.ggnn_sparse_csr(64, 2, [0], [64], [0])      # node out of range
    with pytest.raises(capi.GGNNError):
        capi.ggnn_sparse_csr(64, 2, [0], [1], [2])       # type out of range


def test_dropped_edges_counts_against_oracle():
    """The host measurement of dropped edges equals the oracle's coverage
    rule on the same (oracle-reordered) labels; nothing drops when B exceeds
    the bandwidth."""
    _need_lib()
    from paper_1906_11786_amd.driver import dropped_edges
    graphs = [scramble_graph(9, gi, backbone_graph(9, gi, sz, 3, span_mean=20.0, max_span=200))[0]
              for gi, sz in enumerate([400, 250])]
    parts = []
    for g in graphs:
        _, rank = O.rcm_order(g.n, g.src, g.dst)
        parts.append((g.n, *O.relabel(rank, g.src, g.dst), g.etype))
    _, _, s, d, e, _ = O.batch_layout(parts, 32)
    for B in (32, 64, 128, 512):
        r = dropped_edges(graphs, B, 3)
        ks, kd, ke, ndrop, ndup = O.kept_edges(s, d, e, B)
        assert (r["dropped"], r["kept"], r["duplicates"]) == (ndrop, len(ks), ndup), B
        if r["bandwidth"] < B:
            assert r["dropped"] == 0


def _expected_slices(n, E, s, src, dst, et):
    s_, d_, e_, _ = O.dedupe_edges(src, dst, et)
    R = np.zeros((E, s, n), np.uint8)
    Cc = np.zeros((E, n, s), np.uint8)
    into = d_ < s
    R[e_[into], d_[into], s_[into]] = 1
    out = (~into) & (s_ < s)
    Cc[e_[out], d_[out], s_[out]] = 1
    return R, Cc, int(into.sum()), int(out.sum()), int((~into & ~out).sum())


@pytest.mark.parametrize("s", [32, 64, 128])
def test_super_pack_bit_exact_against_oracle(s):
    """Rows slice = edges into nodes < s, cols slice = edges out of them into
    the others, transposes consistent, counts = the oracle's deduplicated
    edge split."""
    _need_lib()
    rng = np.random.default_rng(s)
    n, E, m = 448, 3, 5000
    src, dst, et = rng.integers(0, n, m), rng.integers(0, n, m), rng.integers(0, E, m)
    src[:200] = rng.integers(0, s, 200)      # plenty of edges touching the supernodes
    dst[200:400] = rng.integers(0, s, 200)
    rows, cols, rows_t, cols_t, cnt = capi.ggnn_super_pack(n, E, s, src, dst, et)
    R, Cc, nr, nc, rest = _expected_slices(n, E, s, src, dst, et)
    unpack = lambda b: np.unpackbits(b, axis=-1, bitorder="little")
    np.testing.assert_array_equal(unpack(rows), R)
    np.testing.assert_array_equal(unpack(cols), Cc)
    np.testing.assert_array_equal(unpack(rows_t), R.transpose(0, 2, 1))
    np.testing.assert_array_equal(unpack(cols_t), Cc.transpose(0, 2, 1))
    _, _, _, ndup = O.dedupe_edges(src, dst, et)
    assert (cnt["rows"], cnt["cols"]) == (nr, nc)
    assert cnt["rest"] + cnt["rows"] + cnt["cols"] + cnt["duplicates"] == m
    assert cnt["rest"] >= rest and cnt["duplicates"] <= ndup
    with pytest.raises(capi.GGNNError):
        capi.ggnn_super_pack(448, 3, 48, src, dst, et)     # s not a multiple of 32
    with pytest.raises(capi.GGNNError):
        capi.ggnn_super_pack(480, 3, 32, src, dst, et)     # n_pad not a multiple of 64


@pytest.mark.parametrize("s", [32, 64, 128])
def test_super_active_is_the_highest_supernode_with_an_edge(s):
    """ggnn_super_active: the smallest multiple of 16 above every supernode
    index that has an edge into it (row slice) or out of it into another node
    (column slice); 0 for empty slices; edges among the other nodes do not
    count."""
    _need_lib()
    n, E = 448, 3
    rng = np.random.default_rng(s + 1)
    src = rng.integers(s, n, 300)
    dst = rng.integers(s, n, 300)
    et = rng.integers(0, E, 300)
    rows, cols, _, _, _ = capi.ggnn_super_pack(n, E, s, src, dst, et)
    assert capi.ggnn_super_active(n, E, s, rows, cols) == 0
    for top, into in [(0, True), (5, False), (15, True), (16, False), (31, True), (32, False), (s - 1, True),
                      (s - 1, False)]:
        if top >= s:
            continue
        a = np.append(src, s + 3 if into else top)
        b = np.append(dst, top if into else s + 7)
        c = np.append(et, E - 1)
        rows, cols, _, _, _ = capi.ggnn_super_pack(n, E, s, a, b, c)
        assert capi.ggnn_super_active(n, E, s, rows, cols) == (top // 16 + 1) * 16, (top, into)
    with pytest.raises(capi.GGNNError):
        capi.ggnn_super_active(n, E, 48, rows, cols)


def test_compile_with_supernodes_matches_oracle_reordering():
    """Hubs take the first labels; the other nodes of each graph follow in
    the oracle's reverse Cuthill-McKee order of the edges between them."""
    _need_lib()
    from ggnn_synth import add_hubs
    from paper_1906_11786_amd.driver import compile_with_supernodes
    graphs, hubs = [], []
    for gi, sz in enumerate([300, 200]):
        g, h = add_hubs(4, gi, scramble_graph(4, gi, backbone_graph(4, gi, sz, 3))[0], 3, 0.4, 3)
        graphs.append(g)
        hubs.append(h)
    comp = compile_with_supernodes(graphs, hubs, 64, 3, 32)
    assert comp.n_pad % 64 == 0 and comp.n_real == 32 + 500 - 6
    base, nh = 32, 0
    S, D = [], []
    for g, h in zip(graphs, hubs):
        label = np.full(g.n, -1, np.int64)
        label[h] = np.arange(nh, nh + len(h))
        nh += len(h)
        rest = np.flatnonzero(label < 0)
        local = np.full(g.n, -1, np.int64)
        local[rest] = np.arange(len(rest))
        inner = (label[g.src] < 0) & (label[g.dst] < 0)
        _, rank = O.rcm_order(len(rest), local[g.src[inner]], local[g.dst[inner]])
        label[rest] = base + np.asarray(rank)
        base += len(rest)
        S.append(label[g.src])
        D.append(label[g.dst])
    np.testing.assert_array_equal(comp.src, np.concatenate(S))
    np.testing.assert_array_equal(comp.dst, np.concatenate(D))
    from host_sanitized_cases import check_batch_super
    check_batch_super()
