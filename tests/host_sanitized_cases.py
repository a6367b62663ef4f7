"""Cases for the host compilation code built with the address and
undefined-behaviour sanitizers (tests/test_host_sanitized.py runs this file
in a child process with the sanitizer runtime preloaded).

Every host entry point of csrc/host.cpp is driven through the C ABI -- the
ctypes binding pointed at the sanitized build -- over graphs that reach the
edges of its index arithmetic: ids 0 and n_pad - 1, empty and one-node
graphs, self-loops and repeated edges, every supported block size, the
largest edge counts of a full band, the transposed bit band, the sparse
lists and the supernode slices, plus every validation error path.  Results
are checked against the oracle (the same checks as the unsanitized tests),
so a silent out-of-bounds write that happened to leave results intact is
still reported by the sanitizer.  Prints "ALL OK" at the end.
"""
import ctypes as C
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
from ggnn_synth import backbone_graph, scramble_graph, local_window_graph  # noqa: E402
from paper_1906_11786_amd import capi  # noqa: E402

HOST_FUNCS = ["ggnn_abi_version", "ggnn_last_error", "ggnn_status_string", "ggnn_rcm_order", "ggnn_bandwidth",
              "ggnn_band_bytes", "ggnn_banded_pack", "ggnn_band_bits_bytes", "ggnn_banded_pack_bits",
              "ggnn_sparse_csr", "ggnn_super_bytes", "ggnn_super_pack", "ggnn_batch_graphs",
              "ggnn_batch_graphs_super"]


def bind(path):
    L = C.CDLL(path)
    for name in HOST_FUNCS:
        res, args = capi._SIGS[name]
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    capi._lib = L


def expect_error(fn, *a, status="GGNN_ERR_INVALID_ARG", **kw):
    try:
        fn(*a, **kw)
    except capi.GGNNError as e:
        assert e.status_name == status, (e.status_name, status)
        return
    raise AssertionError(f"{fn.__name__} accepted invalid arguments")


def unpack(bits):
    return np.unpackbits(bits, axis=-1, bitorder="little").astype(np.float64)


def graphs():
    rng = np.random.default_rng(7)
    G = type(backbone_graph(1, 0, 10, 1))
    out = [scramble_graph(21, 0, backbone_graph(21, 0, 2500, 3, span_mean=8.0))[0],
           local_window_graph(22, 0, 600, 2, 40, 0.03),
           G(1, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)),
           G(6, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)),
           G(5, np.arange(5, dtype=np.int32), np.arange(5, dtype=np.int32), np.zeros(5, np.int32))]
    n = 333   # random multigraph with repeats and self-loops, ids at both ends
    s = rng.integers(0, n, 2000).astype(np.int32)
    d = rng.integers(0, n, 2000).astype(np.int32)
    s[:3], d[:3] = [0, n - 1, 0], [n - 1, 0, 0]
    s[3:40], d[3:40] = s[40:77], d[40:77]
    out.append(G(n, s, d, rng.integers(0, 1, 2000).astype(np.int32)))
    star = G(64, np.zeros(63, np.int32), np.arange(1, 64, dtype=np.int32), np.zeros(63, np.int32))
    out.append(star)
    return out


def check_rcm():
    for g in graphs():
        order, rank, bw = capi.ggnn_rcm_order(g.n, g.src, g.dst)
        o_order, o_rank = O.rcm_order(g.n, g.src, g.dst)
        assert np.array_equal(order, o_order) and np.array_equal(rank, o_rank)
        s, d = O.relabel(o_rank, g.src, g.dst)
        assert bw == O.bandwidth(s, d)
        assert capi.ggnn_bandwidth(g.n, g.src, g.dst, rank) == bw
        assert capi.ggnn_bandwidth(g.n, g.src, g.dst) == O.bandwidth(g.src, g.dst)
    expect_error(capi.ggnn_rcm_order, 3, [0, 5], [1, 2])
    expect_error(capi.ggnn_rcm_order, 3, [0, -1], [1, 2])
    expect_error(capi.ggnn_bandwidth, 4, [0, 1], [1, 4])
    expect_error(capi.ggnn_bandwidth, 4, [0, 1], [1, 2], rank=[0, 1, 2, 4])


def batch_expected(gs, reorder):
    """Supergraph edges, offsets and bandwidth from the oracle's RCM, one
    graph at a time."""
    S, D, offs, bw = [], [], [0], 0
    for g in gs:
        if reorder:
            s, d = O.relabel(O.rcm_order(g.n, g.src, g.dst)[1], g.src, g.dst)
        else:
            s, d = g.src, g.dst
        bw = max(bw, O.bandwidth(s, d) if len(s) else 0)
        S.append(np.asarray(s, np.int64) + offs[-1])
        D.append(np.asarray(d, np.int64) + offs[-1])
        offs.append(offs[-1] + g.n)
    cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int64))
    return cat(S), cat(D), np.asarray(offs, np.int64), bw


def check_batch():
    gs = graphs()
    for reorder in (True, False):
        for sel in (gs, gs[::-1], gs[2:4], []):
            cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int32))
            s, d, offs, bw = capi.ggnn_batch_graphs([g.n for g in sel], [len(g.src) for g in sel],
                                                    cat([g.src for g in sel]), cat([g.dst for g in sel]),
                                                    reorder=reorder)
            es, ed, eo, ebw = batch_expected(sel, reorder)
            assert np.array_equal(s, es) and np.array_equal(d, ed) and np.array_equal(offs, eo) and bw == ebw
    expect_error(capi.ggnn_batch_graphs, [3, 4], [1, 1], [0, 1], [2, 4])     # graph 1: id 4 of 4 nodes
    expect_error(capi.ggnn_batch_graphs, [3, -1], [1, 0], [0], [2])
    expect_error(capi.ggnn_batch_graphs, [3], [-1], [], [])
    expect_error(capi.ggnn_batch_graphs, [3, 4], [1, 1], [0, -1], [2, 1], reorder=False)


def check_batch_super():
    """Hubs first (list order, graph after graph), then each graph's other
    nodes in the oracle's RCM order of the edges between them, from s on."""
    gs = [g for g in graphs() if g.n >= 5]
    rng = np.random.default_rng(3)
    hubs = [np.sort(rng.choice(g.n, size=min(3, g.n - 2), replace=False)).astype(np.int32) for g in gs]
    hubs[0] = hubs[0][::-1].copy()      # list order, not id order, decides the labels
    hubs[1] = np.zeros(0, np.int32)     # a graph without hubs
    s = 32
    cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int32))
    out_s, out_d, nn, bw = capi.ggnn_batch_graphs_super([g.n for g in gs], [len(g.src) for g in gs],
                                                       cat([g.src for g in gs]), cat([g.dst for g in gs]),
                                                       [len(h) for h in hubs], cat(hubs), s)
    base, nh, ebw, S, D = s, 0, 0, [], []
    for g, h in zip(gs, hubs):
        label = np.full(g.n, -1, np.int64)
        label[h] = np.arange(nh, nh + len(h))
        nh += len(h)
        rest = np.flatnonzero(label < 0)
        local = np.full(g.n, -1, np.int64)
        local[rest] = np.arange(len(rest))
        inner = (label[g.src] < 0) & (label[g.dst] < 0)
        ls, ld = local[g.src[inner]], local[g.dst[inner]]
        rank = np.asarray(O.rcm_order(len(rest), ls, ld)[1])
        if inner.any():
            ebw = max(ebw, O.bandwidth(*O.relabel(rank, ls, ld)))
        label[rest] = base + rank
        base += len(rest)
        S.append(label[g.src])
        D.append(label[g.dst])
    assert np.array_equal(out_s, np.concatenate(S)) and np.array_equal(out_d, np.concatenate(D))
    assert nn == base and bw == ebw
    expect_error(capi.ggnn_batch_graphs_super, [4], [1], [0], [1], [3], [0, 1, 2], 2)     # 3 hubs, 2 slots
    expect_error(capi.ggnn_batch_graphs_super, [4], [1], [0], [1], [2], [1, 1], 4)        # repeated hub
    expect_error(capi.ggnn_batch_graphs_super, [4], [1], [0], [1], [1], [4], 4)           # hub out of range
    expect_error(capi.ggnn_batch_graphs_super, [4], [1], [0], [5], [1], [0], 4)           # edge out of range
    expect_error(capi.ggnn_batch_graphs_super, [2], [0], [], [], [3], [0, 1, 0], 4)       # more hubs than nodes


def full_band(n, E, B, rng):
    """Every in-band (receiver, sender, type) triple of an n-node graph, plus
    repeats and a few out-of-band edges: the largest edge lists a band of
    this size can hold."""
    i = np.arange(n)
    src, dst = np.meshgrid(i, i)
    keep = np.abs(src // B - dst // B) <= 1
    s, d = src[keep].ravel(), dst[keep].ravel()
    et = np.repeat(np.arange(E), len(s))
    s, d = np.tile(s, E), np.tile(d, E)
    extra = rng.integers(0, len(s), len(s) // 10)
    far_s = np.array([0, n - 1]); far_d = np.array([n - 1, 0])
    return (np.concatenate([s, s[extra], far_s]).astype(np.int32),
            np.concatenate([d, d[extra], far_d]).astype(np.int32),
            np.concatenate([et, et[extra], [0, E - 1]]).astype(np.int32))


def check_pack():
    rng = np.random.default_rng(11)
    for B in (8, 32, 64, 128, 256, 512):
        nb = 3 if B >= 256 else 5
        n, E = nb * B, 2
        if B <= 64:
            src, dst, et = full_band(n, E, B, rng)
        else:
            m = 20000
            src = rng.integers(0, n, m).astype(np.int32)
            dst = np.clip(src + rng.integers(-2 * B, 2 * B + 1, m), 0, n - 1).astype(np.int32)
            et = rng.integers(0, E, m).astype(np.int32)
            src[:2], dst[:2] = [0, n - 1], [n - 1, 0]
        band = O.pack_band(n, E, B, src, dst, et)
        ks, kd, ke, ndrop, ndup = O.kept_edges(src, dst, et, B)
        for dt in ("f32", "bf16"):
            b, p, dr, du = capi.ggnn_banded_pack(n, E, B, src, dst, et, dt=dt)
            one = 1.0 if dt == "f32" else 0x3F80
            assert np.array_equal(b == one, band == 1.0) and (p, dr, du) == (len(ks), ndrop, ndup), (B, dt)
            assert capi.ggnn_band_bytes(n, E, B, dt) == b.nbytes
        bits, bits_t, p, dr, du = capi.ggnn_banded_pack_bits(n, E, B, src, dst, et)
        assert np.array_equal(unpack(bits), band) and (p, dr, du) == (len(ks), ndrop, ndup), B
        bt = unpack(bits_t)
        for j in range(nb):
            for sl in range(3):
                kr = j - 1 + sl
                want = band[:, kr, 2 - sl].transpose(0, 2, 1) if 0 <= kr < nb else np.zeros((E, B, B))
                assert np.array_equal(bt[:, j, sl], want), (B, j, sl)
        # with a relabelling (rank) applied inside the packer
        rank = rng.permutation(n).astype(np.int32)
        b1, *c1 = capi.ggnn_banded_pack_bits(n, E, B, src, dst, et, rank=rank)
        b2, *c2 = capi.ggnn_banded_pack_bits(n, E, B, rank[src], rank[dst], et)
        assert np.array_equal(b1, b2) and c1[1:] == c2[1:]
    # empty edge list, one block, strict mode and every validation error
    bits, bits_t, p, dr, du = capi.ggnn_banded_pack_bits(64, 1, 64, [], [], [])
    assert not bits.any() and not bits_t.any() and (p, dr, du) == (0, 0, 0)
    src, dst, et = np.array([0, 100]), np.array([1, 0]), np.array([0, 0])
    expect_error(capi.ggnn_banded_pack, 128, 1, 32, src, dst, et, strict=True, status="GGNN_ERR_OUT_OF_BAND")
    expect_error(capi.ggnn_banded_pack_bits, 128, 1, 32, src, dst, et, strict=True, status="GGNN_ERR_OUT_OF_BAND")
    for args in [(100, 1, 32, src, dst, et), (128, 1, 32, [128], [0], [0]), (128, 1, 32, [-1], [0], [0]),
                 (128, 1, 32, src, dst, [0, 1]), (128, 0, 32, src, dst, et), (128, 1, 0, src, dst, et)]:
        expect_error(capi.ggnn_banded_pack_bits, *args)
        expect_error(capi.ggnn_banded_pack, *args)
    expect_error(capi.ggnn_banded_pack_bits, 120, 1, 12, src, dst, et)    # bit rows need B % 8 == 0
    b, p, dr, du = capi.ggnn_banded_pack(120, 1, 12, [0, 11, 119], [11, 12, 10], [0, 0, 0], dt="f32")
    assert (p, dr, du) == (2, 1, 0) and b.sum() == 2
    expect_error(capi.ggnn_banded_pack_bits, 128, 1, 32, src, dst, et, rank=[0] * 127 + [128])


def check_csr():
    rng = np.random.default_rng(12)
    n, E, m = 257, 4, 6000
    src, dst, et = rng.integers(0, n, m), rng.integers(0, n, m), rng.integers(0, E, m)
    src[:2], dst[:2], et[:2] = [0, n - 1], [n - 1, 0], [E - 1, 0]
    src[2:60], dst[2:60], et[2:60] = src[60:118], dst[60:118], et[60:118]
    row_ptr, col, dup = capi.ggnn_sparse_csr(n, E, src, dst, et)
    s, d, e, ndup = O.dedupe_edges(src, dst, et)
    assert dup == ndup and np.array_equal(col, s[np.lexsort((s, e, d))])
    want = np.concatenate([[0], np.cumsum(np.bincount(d * E + e, minlength=n * E))])
    assert np.array_equal(row_ptr, want)
    rp, c, dup = capi.ggnn_sparse_csr(1, 1, [], [], [])
    assert (rp == 0).all() and len(c) == 0
    expect_error(capi.ggnn_sparse_csr, 64, 2, [0], [64], [0])
    expect_error(capi.ggnn_sparse_csr, 64, 2, [0], [1], [2])
    expect_error(capi.ggnn_sparse_csr, 64, 0, [0], [1], [0])


def check_super():
    rng = np.random.default_rng(13)
    for s in (32, 64, 96, 128):
        n, E, m = 512, 3, 8000
        src, dst, et = rng.integers(0, n, m), rng.integers(0, n, m), rng.integers(0, E, m)
        src[:300] = rng.integers(0, s, 300)
        dst[300:600] = rng.integers(0, s, 300)
        src[600:602], dst[600:602] = [s - 1, n - 1], [n - 1, s - 1]
        rows, cols, rows_t, cols_t, cnt = capi.ggnn_super_pack(n, E, s, src, dst, et)
        s_, d_, e_, _ = O.dedupe_edges(src, dst, et)
        R = np.zeros((E, s, n), np.uint8)
        Cc = np.zeros((E, n, s), np.uint8)
        into = d_ < s
        R[e_[into], d_[into], s_[into]] = 1
        out = (~into) & (s_ < s)
        Cc[e_[out], d_[out], s_[out]] = 1
        u = lambda b: np.unpackbits(b, axis=-1, bitorder="little")
        assert np.array_equal(u(rows), R) and np.array_equal(u(cols), Cc)
        assert np.array_equal(u(rows_t), R.transpose(0, 2, 1)) and np.array_equal(u(cols_t), Cc.transpose(0, 2, 1))
        assert (cnt["rows"], cnt["cols"]) == (int(into.sum()), int(out.sum()))
        assert cnt["rest"] + cnt["rows"] + cnt["cols"] + cnt["duplicates"] == m
    expect_error(capi.ggnn_super_pack, 448, 3, 48, [0], [1], [0])
    expect_error(capi.ggnn_super_pack, 480, 3, 32, [0], [1], [0])
    expect_error(capi.ggnn_super_pack, 512, 3, 32, [0], [512], [0])
    expect_error(capi.ggnn_super_pack, 512, 3, 32, [0], [1], [3])


def sanitizer_loaded():
    with open("/proc/self/maps") as f:
        maps = f.read()
    return "libasan" in maps and "libubsan" in maps


if __name__ == "__main__":
    bind(sys.argv[1])
    assert sanitizer_loaded(), "the address / undefined-behaviour sanitizer runtimes are not loaded"
    assert capi.ggnn_abi_version() == capi.ABI_VERSION
    assert capi.ggnn_status_string(3) == "GGNN_ERR_OUT_OF_BAND"
    for step in (check_rcm, check_batch, check_batch_super, check_pack, check_csr, check_super):
        step()
        print(f"{step.__name__} ok", flush=True)
    print("ALL OK", flush=True)
