"""Per-entry-point parity of the HIP kernels against the CPU oracle, called
through the C ABI.  Integer-valued cases (every partial sum exact in fp32)
are compared bitwise, so any indexing slip shows; real-valued cases use the
fp32 / bf16 tolerances."""
import os

import numpy as np
import pytest

import oracle as O
from gpu_helpers import elemerr, record, TOL, relerr, say, dev, host, round_to, torch_dt

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
capi = pytest.importorskip("paper_1906_11786_amd.capi")


@pytest.fixture(autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    yield
    torch.cuda.synchronize()


def _edges(rng, n, m, E, span):
    src = rng.integers(0, n, m)
    dst = np.clip(src + rng.integers(-span, span + 1, m), 0, n - 1)
    return src, dst, rng.integers(0, E, m)


def _band(dt, n_pad, E, B, src, dst, et):
    band, packed, dropped, dup = capi.ggnn_banded_pack(n_pad, E, B, src, dst, et, dt=dt)
    if dt == "bf16":
        return torch.from_numpy(band.view(np.int16)).cuda().view(torch.bfloat16), dropped
    return torch.from_numpy(band).cuda(), dropped


# (B, H, E, nb): several block rows, each block size and feature width.
BANDED_CASES = [(32, 32, 2, 7), (64, 64, 3, 5), (128, 64, 2, 4), (128, 128, 2, 3), (256, 128, 1, 3),
                (512, 32, 2, 2), (128, 256, 2, 3), (256, 256, 1, 2), (64, 32, 1, 1)]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", BANDED_CASES)
def test_banded_propagate_integer_exact(dt, B, H, E, nb):
    say(f"banded_propagate int dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B * 131 + H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    band, dropped = _band(dt, n, E, B, src, dst, et)
    assert nb < 3 or dropped > 0      # with fewer than three blocks nothing can fall outside the band
    M = rng.integers(-4, 5, (E, n, H)).astype(np.float64)
    Mt = dev(M.transpose(0, 2, 1))                      # feature-major [E][H][n], float
    a = torch.full((n, H), float("nan"), device="cuda")
    capi.ggnn_banded_propagate(dt, n, B, H, E, band, Mt, a)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    np.testing.assert_array_equal(host(a), O.aggregate(n, s, d, e, M))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", BANDED_CASES)
def test_banded_propagate_bwd_integer_exact(dt, B, H, E, nb):
    say(f"banded_propagate_bwd int dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B * 17 + H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    band, _ = _band(dt, n, E, B, src, dst, et)
    da = rng.integers(-4, 5, (n, H)).astype(np.float64)
    dM = torch.full((E, H, n), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_banded_propagate_bwd(dt, n, B, H, E, band, dev(da.T, dt), dM)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    want = O.aggregate_transpose(n, s, d, e, da, E)
    np.testing.assert_array_equal(host(dM), want.transpose(0, 2, 1))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_banded_forward_backward_adjoint(dt):
    """<A M, D> = <M, A^T D> through the two kernels (real values)."""
    rng = np.random.default_rng(3)
    B, H, E, nb = 128, 64, 3, 4
    n = B * nb
    src, dst, et = _edges(rng, n, 8 * n, E, 2 * B)
    band, _ = _band(dt, n, E, B, src, dst, et)
    M = round_to("f32", rng.standard_normal((E, n, H)))
    D = round_to(dt, rng.standard_normal((n, H)))
    a = torch.empty((n, H), device="cuda")
    capi.ggnn_banded_propagate(dt, n, B, H, E, band, dev(M.transpose(0, 2, 1)), a)
    dM = torch.empty((E, H, n), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_banded_propagate_bwd(dt, n, B, H, E, band, dev(D.T, dt), dM)
    lhs = float(np.sum(host(a) * D))
    rhs = float(np.sum(M.transpose(0, 2, 1) * host(dM)))
    assert abs(lhs - rhs) <= TOL[dt] * np.sqrt(np.sum(host(a) ** 2) * np.sum(D ** 2))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H", [32, 64, 128, 256])
@pytest.mark.parametrize("n", [96, 1184])
def test_msg_transform(dt, H, n):
    say(f"msg_transform dt={dt} H={H} n={n}")
    rng = np.random.default_rng(H + n)
    E = 3
    # integer-valued: exact in every dtype
    X = rng.integers(-1, 2, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    M = torch.full((E, H, n), float("nan"), device="cuda")
    capi.ggnn_msg_transform(dt, n, H, E, dev(X, dt), dev(W, dt), None, M)
    np.testing.assert_array_equal(host(M), O.msg_transform(X, W).transpose(0, 2, 1))
    # real-valued with bias
    X = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    bias = rng.uniform(-0.2, 0.2, (E, H)).astype(np.float32).astype(np.float64)
    capi.ggnn_msg_transform(dt, n, H, E, dev(X, dt), dev(W, dt), dev(bias), M)
    assert relerr(host(M), O.msg_transform(X, W, bias).transpose(0, 2, 1)) <= TOL["f32"]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H", [32, 64, 128, 256])
@pytest.mark.parametrize("n", [96, 1184])
def test_msg_transform_bwd(dt, H, n):
    say(f"msg_transform_bwd dt={dt} H={H} n={n}")
    rng = np.random.default_rng(7 * H + n)
    E = 3
    X = rng.integers(-1, 2, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    dM = rng.integers(-2, 3, (E, n, H)).astype(np.float64)
    dX_in = rng.integers(-3, 4, (n, H)).astype(np.float64)
    ws_n = capi.ggnn_msg_transform_bwd_workspace_bytes(dt, n, H, E)
    ws = torch.empty(ws_n, dtype=torch.uint8, device="cuda")
    dX = torch.full((n, H), float("nan"), device="cuda")
    dW = dev(np.ones((E, H, H)))            # += semantics: start from ones
    dbias = dev(np.ones((E, H)))
    capi.ggnn_msg_transform_bwd(dt, n, H, E, dev(X, dt), dev(W, dt), dev(dM.transpose(0, 2, 1), dt), dev(dX_in),
                                dX, dW, dbias, ws, ws_n)
    wdX, wdW, wdb = O.msg_transform_backward(X, W, dM)
    np.testing.assert_array_equal(host(dX), dX_in + wdX)
    np.testing.assert_array_equal(host(dW), 1 + wdW)
    np.testing.assert_array_equal(host(dbias), 1 + wdb)
    # in place (dX_in == dX_out), no bias gradient
    dX2 = dev(dX_in)
    capi.ggnn_msg_transform_bwd(dt, n, H, E, dev(X, dt), dev(W, dt), dev(dM.transpose(0, 2, 1), dt), dX2, dX2,
                                dW, None, ws, ws_n)
    np.testing.assert_array_equal(host(dX2), dX_in + wdX)
    np.testing.assert_array_equal(host(dW), 1 + 2 * wdW)


def _gru_inputs(dt, rng, n, H):
    a = rng.standard_normal((n, H)).astype(np.float32).astype(np.float64)
    h = round_to(dt, rng.standard_normal((n, H)))
    k = 1 / np.sqrt(H)
    Wi = round_to(dt, rng.uniform(-k, k, (H, 3 * H)))
    U = round_to(dt, rng.uniform(-k, k, (H, 3 * H)))
    b = rng.uniform(-k, k, 3 * H).astype(np.float32).astype(np.float64)
    return a, h, Wi, U, b


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H", [32, 64, 128, 256])
@pytest.mark.parametrize("n", [96, 1184])
def test_gru_update(dt, H, n):
    say(f"gru_update dt={dt} H={H} n={n}")
    rng = np.random.default_rng(11 * H + n)
    a, h, Wi, U, b = _gru_inputs(dt, rng, n, H)
    h_out = torch.full((n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    saved = torch.full((n, 3 * H), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_gru_update(dt, n, H, dev(a), dev(h, dt), dev(Wi, dt), dev(U, dt), dev(b), h_out, saved)
    hn, r, z, nn = O.gru_forward(a, h, Wi, U, b)
    assert relerr(host(h_out), hn) <= TOL[dt]
    assert relerr(host(saved), np.concatenate([r, z, nn], axis=1)) <= TOL[dt]
    h_out2 = torch.full((n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_gru_update(dt, n, H, dev(a), dev(h, dt), dev(Wi, dt), dev(U, dt), dev(b), h_out2, None)
    assert torch.equal(h_out, h_out2)


# n = 9504 at H = 256: the bf16 weight-gradient contraction there splits the
# rows into 38 splits of 8 chunks of 32 rows (ring of three LDS slots wraps)
# and a last split of one chunk.
GRU_BWD_CASES = [(H, n) for H in (32, 64, 128, 256) for n in (96, 1184)] + [(256, 9504)]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("H,n", GRU_BWD_CASES)
def test_gru_update_bwd(dt, H, n):
    say(f"gru_update_bwd dt={dt} H={H} n={n}")
    rng = np.random.default_rng(13 * H + n)
    a, h, Wi, U, b = _gru_inputs(dt, rng, n, H)
    _, r, z, nn = O.gru_forward(a, h, Wi, U, b)
    saved = round_to(dt, np.concatenate([r, z, nn], axis=1))
    r, z, nn = saved[:, :H], saved[:, H:2 * H], saved[:, 2 * H:]
    g = rng.standard_normal((n, H)).astype(np.float32).astype(np.float64)
    ws_n = capi.ggnn_gru_update_bwd_workspace_bytes(dt, n, H)
    ws = torch.empty(ws_n, dtype=torch.uint8, device="cuda")
    da = torch.full((H, n), float("nan"), device="cuda", dtype=torch_dt(dt))
    dh = torch.full((n, H), float("nan"), device="cuda")
    dWi, dU, db = dev(np.ones((H, 3 * H))), dev(np.ones((H, 3 * H))), dev(np.ones(3 * H))
    capi.ggnn_gru_update_bwd(dt, n, H, dev(g), dev(a), dev(h, dt), dev(saved, dt), dev(Wi, dt), dev(U, dt), da, dh,
                             dWi, dU, db, ws, ws_n)
    wda, wdh, wdWi, wdU, wdb = O.gru_backward(g, a, h, r, z, nn, Wi, U)
    assert relerr(host(da).T, wda) <= TOL[dt]
    assert relerr(host(dh), wdh) <= TOL[dt]
    assert relerr(host(dWi) - 1, wdWi) <= TOL[dt]
    assert relerr(host(dU) - 1, wdU) <= TOL[dt]
    assert relerr(host(db) - 1, wdb) <= TOL[dt]


def _bits(n_pad, E, B, src, dst, et):
    bits, bits_t, packed, dropped, dup = capi.ggnn_banded_pack_bits(n_pad, E, B, src, dst, et)
    return torch.from_numpy(bits).cuda(), torch.from_numpy(bits_t).cuda(), dropped


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", BANDED_CASES)
def test_banded_step_bits_integer_exact(dt, B, H, E, nb):
    """a = sum_e (A_e X) W_e on the 1-bit band, small integers: exact."""
    say(f"banded_step_bits int dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B * 7 + H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    bits, _, dropped = _bits(n, E, B, src, dst, et)
    X = rng.integers(-2, 3, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    bias = rng.integers(-2, 3, (E, H)).astype(np.float64)
    a = torch.full((n, H), float("nan"), device="cuda")
    capi.ggnn_banded_step_bits(dt, n, B, H, E, bits, dev(X, dt), dev(W, dt), dev(bias), a)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    np.testing.assert_array_equal(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W, bias)))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", [(128, 64, 3, 5), (64, 128, 2, 6), (256, 256, 2, 3), (32, 32, 4, 9)])
def test_banded_step_bits_real_values(dt, B, H, E, nb):
    """bf16 inputs, fp32 results: the aggregate enters the transform as a hi +
    lo pair, so the result is close to fp32 accuracy."""
    say(f"banded_step_bits real dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B + 3 * H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 4 * n, E, B + 3)
    bits, _, _ = _bits(n, E, B, src, dst, et)
    X = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    a = torch.empty((n, H), device="cuda")
    capi.ggnn_banded_step_bits(dt, n, B, H, E, bits, dev(X, dt), dev(W, dt), None, a)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    assert relerr(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W))) <= 1e-4


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", BANDED_CASES)
def test_banded_propagate_bits_bwd_integer_exact(dt, B, H, E, nb):
    say(f"banded_propagate_bits_bwd int dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B * 19 + H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    _, bits_t, _ = _bits(n, E, B, src, dst, et)
    da = rng.integers(-4, 5, (n, H)).astype(np.float64)
    dM = torch.full((E, H, n), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_banded_propagate_bits_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), dM)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    np.testing.assert_array_equal(host(dM), O.aggregate_transpose(n, s, d, e, da, E).transpose(0, 2, 1))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", BANDED_CASES)
def test_banded_step_bits_bwd_integer_exact(dt, B, H, E, nb):
    """Fused reverse step, small integers: dM_e = A_e^T da (node-major rows,
    row stride ldm > n_pad: the rows past n_pad stay untouched) and
    dX = dX_in + sum_e dM_e W_e^T, exact."""
    say(f"banded_step_bits_bwd int dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B * 23 + H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    _, bits_t, _ = _bits(n, E, B, src, dst, et)
    da = rng.integers(-4, 5, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    dX_in = rng.integers(-3, 4, (n, H)).astype(np.float64)
    ldm = n + 32
    dM = torch.full((E, ldm, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    dX = torch.full((n, H), float("nan"), device="cuda")
    capi.ggnn_banded_step_bits_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), dev(W, dt), dev(dX_in), dX, dM, ldm)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    want_dM = O.aggregate_transpose(n, s, d, e, da, E)
    got = host(dM)
    np.testing.assert_array_equal(got[:, :n], want_dM)
    assert np.isnan(got[:, n:]).all()
    want_dX, _, _ = O.msg_transform_backward(np.zeros((n, H)), W, want_dM)
    np.testing.assert_array_equal(host(dX), dX_in + want_dX)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", [(128, 64, 10, 5), (64, 128, 2, 6), (256, 256, 2, 3), (32, 32, 4, 9)])
def test_banded_step_bits_bwd_real_values(dt, B, H, E, nb):
    """Real values, in place (dX_in is dX_out) and without dX_in: dX agrees
    with the oracle to the dtype's tolerance (dM enters the transform as its
    stored, rounded value)."""
    say(f"banded_step_bits_bwd real dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B + 5 * H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 4 * n, E, B + 3)
    _, bits_t, _ = _bits(n, E, B, src, dst, et)
    da = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    dX0 = rng.standard_normal((n, H))
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    want_dM = O.aggregate_transpose(n, s, d, e, da, E)
    want_dX, _, _ = O.msg_transform_backward(np.zeros((n, H)), W, want_dM)
    dM = torch.empty((E, n, H), device="cuda", dtype=torch_dt(dt))
    dX = dev(dX0)
    capi.ggnn_banded_step_bits_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), dev(W, dt), dX, dX, dM, n)
    assert relerr(host(dM), want_dM) <= TOL[dt]
    assert relerr(host(dX), dX0 + want_dX) <= TOL[dt]
    capi.ggnn_banded_step_bits_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), dev(W, dt), None, dX, dM, n)
    assert relerr(host(dX), want_dX) <= TOL[dt]


STEP_GRU_CASES = [(128, 64, 10, 5), (64, 128, 2, 6), (32, 32, 4, 9), (256, 256, 2, 3)]


def _wide(dt, B, H):
    """Shapes served by the sliced wide step kernel (bf16, H of 128 or 256,
    B of 32 to 512; the forward only when W_e^T is given)."""
    return dt == "bf16" and H in (128, 256) and B in (32, 64, 128, 256, 512)


# Wide-kernel shapes: E = 1 stages most of each next feature slice after the
# slice's last type, B = 512 keeps a single node-slice buffer, nb = 1 has no
# neighbouring blocks, nb >= 3 has interior block rows.
WIDE_CASES = [(128, 128, 2, 3), (256, 128, 1, 3), (512, 128, 2, 2), (128, 256, 3, 3), (256, 256, 1, 2),
              (256, 256, 4, 1), (256, 256, 3, 3), (512, 256, 2, 2), (64, 128, 3, 5), (32, 128, 2, 7),
              (64, 256, 1, 4), (32, 256, 3, 1)]


@pytest.mark.parametrize("B,H,E,nb", WIDE_CASES)
@pytest.mark.parametrize("with_bias", [False, True])
def test_step_wide_forward_integer_exact(B, H, E, nb, with_bias):
    """a = sum_e (A_e X) W_e (+ deg_e b_e) through the wide forward step
    (bf16, W_e^T given), small integers: every partial sum exact."""
    dt = "bf16"
    say(f"step_wide fwd int B={B} H={H} E={E} nb={nb} bias={with_bias}")
    rng = np.random.default_rng(B * 29 + H + E + nb)
    n = B * nb
    src, dst, et = _edges(rng, n, 6 * n, E, 2 * B + 5)
    bits, _, _ = _bits(n, E, B, src, dst, et)
    X = rng.integers(-2, 3, (n, H)).astype(np.float64)
    W = rng.integers(-1, 2, (E, H, H)).astype(np.float64)
    bias = rng.integers(-2, 3, (E, H)).astype(np.float64) if with_bias else None
    _, _, Wi, U, b = _gru_inputs(dt, rng, n, H)
    Wd = dev(W, dt)
    Wt = torch.empty_like(Wd)
    capi.ggnn_transpose_weights(dt, H, E, Wd, Wt)
    a = torch.full((n, H), float("nan"), device="cuda")
    h_out = torch.full((n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    saved = torch.full((n, 3 * H), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_step_bits_gru(dt, n, B, H, E, bits, dev(X, dt), Wd, Wt, None if bias is None else dev(bias),
                            dev(Wi, dt), dev(U, dt), dev(b), a, h_out, saved)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    np.testing.assert_array_equal(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W, bias)))


@pytest.mark.parametrize("B,H,E,nb", WIDE_CASES)
def test_step_wide_reverse_integer_exact(B, H, E, nb):
    """dM_e = A_e^T da and dX = dX_in + sum_e dM_e W_e^T through the wide
    reverse step, small integers: exact (rows past n_pad untouched)."""
    test_banded_step_bits_bwd_integer_exact("bf16", B, H, E, nb)


@pytest.mark.parametrize("B,H,nb", [(256, 256, 3), (128, 128, 4), (512, 128, 2)])
def test_step_wide_real_values(B, H, nb):
    """Ten edge types, real values, both directions of the wide step against
    the oracle at the bf16 tolerance (the forward aggregate as hi + lo)."""
    dt, E = "bf16", 10
    say(f"step_wide real B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B + 13 * H + nb)
    n = B * nb
    src, dst, et = _edges(rng, n, 20 * n, E, B + 3)
    bits, bits_t, _ = _bits(n, E, B, src, dst, et)
    X = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    _, _, Wi, U, b = _gru_inputs(dt, rng, n, H)
    Wd = dev(W, dt)
    Wt = torch.empty_like(Wd)
    capi.ggnn_transpose_weights(dt, H, E, Wd, Wt)
    a = torch.empty((n, H), device="cuda")
    h_out = torch.empty((n, H), device="cuda", dtype=torch_dt(dt))
    saved = torch.empty((n, 3 * H), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_step_bits_gru(dt, n, B, H, E, bits, dev(X, dt), Wd, Wt, None, dev(Wi, dt), dev(U, dt), dev(b), a,
                            h_out, saved)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    assert relerr(host(a), O.aggregate(n, s, d, e, O.msg_transform(X, W))) <= 1e-4
    da = X                                   # any bf16 values serve as the upstream gradient
    want_dM = O.aggregate_transpose(n, s, d, e, da, E)
    want_dX, _, _ = O.msg_transform_backward(np.zeros((n, H)), W, want_dM)
    dM = torch.empty((E, n, H), device="cuda", dtype=torch_dt(dt))
    dX = torch.empty((n, H), device="cuda")
    capi.ggnn_banded_step_bits_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), Wd, None, dX, dM, n)
    assert relerr(host(dM), want_dM) <= TOL[dt]
    assert relerr(host(dX), want_dX) <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", STEP_GRU_CASES)
def test_step_bits_gru(dt, B, H, E, nb):
    """One forward step (propagation + GRU, fused where the shape allows):
    the aggregate against the oracle's, the GRU outputs against the oracle's
    GRU of that aggregate."""
    say(f"step_bits_gru dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B + 7 * H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 4 * n, E, B + 3)
    bits, _, _ = _bits(n, E, B, src, dst, et)
    X = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    bias = rng.standard_normal((E, H)) * 0.1
    _, _, Wi, U, b = _gru_inputs(dt, rng, n, H)
    a = torch.full((n, H), float("nan"), device="cuda")
    h_out = torch.full((n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    saved = torch.full((n, 3 * H), float("nan"), device="cuda", dtype=torch_dt(dt))
    Wd = dev(W, dt)
    Wt = torch.empty_like(Wd)
    capi.ggnn_transpose_weights(dt, H, E, Wd, Wt)
    assert torch.equal(Wt.float().cpu(), Wd.float().cpu().transpose(1, 2))
    capi.ggnn_step_bits_gru(dt, n, B, H, E, bits, dev(X, dt), Wd, Wt, dev(bias), dev(Wi, dt), dev(U, dt),
                            dev(b), a, h_out, saved)
    # without the transposed weights (column gathers): the same bits
    a2 = torch.full((n, H), float("nan"), device="cuda")
    h2 = torch.full((n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    s2 = torch.full((n, 3 * H), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_step_bits_gru(dt, n, B, H, E, bits, dev(X, dt), Wd, None, dev(bias), dev(Wi, dt), dev(U, dt),
                            dev(b), a2, h2, s2)
    if _wide(dt, B, H):
        # with Wt the sliced wide kernel runs: another summation order
        assert relerr(host(a2), host(a)) <= 1e-5
    else:
        assert torch.equal(a, a2) and torch.equal(h_out, h2) and torch.equal(saved, s2)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    wa = O.aggregate(n, s, d, e, O.msg_transform(X, W, bias))
    assert relerr(host(a), wa) <= 1e-4
    # the GRU half consumes the aggregate the kernel produced (fp32)
    hn, r, z, nn = O.gru_forward(host(a), X, Wi, U, b)
    assert relerr(host(h_out), hn) <= TOL[dt]
    assert relerr(host(saved), np.concatenate([r, z, nn], axis=1)) <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,E,nb", STEP_GRU_CASES)
def test_step_bits_gru_bwd(dt, B, H, E, nb):
    """One reverse step (propagation reverse of step t + GRU reverse of step
    t-1, fused where the shape allows) against the oracle."""
    say(f"step_bits_gru_bwd dt={dt} B={B} H={H} E={E} nb={nb}")
    rng = np.random.default_rng(B + 11 * H + E)
    n = B * nb
    src, dst, et = _edges(rng, n, 4 * n, E, B + 3)
    _, bits_t, _ = _bits(n, E, B, src, dst, et)
    da = round_to(dt, rng.standard_normal((n, H)))
    W = round_to(dt, rng.standard_normal((E, H, H)) / np.sqrt(H))
    dX_in = rng.standard_normal((n, H))
    a_prev, h_prev, Wi, U, b = _gru_inputs(dt, rng, n, H)
    _, r, z, nn = O.gru_forward(a_prev, h_prev, Wi, U, b)
    saved = round_to(dt, np.concatenate([r, z, nn], axis=1))
    r, z, nn = saved[:, :H], saved[:, H:2 * H], saved[:, 2 * H:]
    dM = torch.full((E, n, H), float("nan"), device="cuda", dtype=torch_dt(dt))
    da_prev = torch.full((H, n), float("nan"), device="cuda", dtype=torch_dt(dt))
    dh_prev = torch.full((n, H), float("nan"), device="cuda")
    ghat = torch.full((n, 3 * H), float("nan"), device="cuda", dtype=torch_dt(dt))
    capi.ggnn_step_bits_gru_bwd(dt, n, B, H, E, bits_t, dev(da.T, dt), dev(W, dt), dev(dX_in), dM, n, dev(Wi, dt),
                                dev(U, dt), dev(h_prev, dt), dev(saved, dt), da_prev, dh_prev, ghat)
    s, d, e, _, _ = O.kept_edges(src, dst, et, B)
    want_dM = O.aggregate_transpose(n, s, d, e, da, E)
    g, _, _ = O.msg_transform_backward(np.zeros((n, H)), W, want_dM)
    wda, wdh, wdWi, _, wdb = O.gru_backward(dX_in + g, a_prev, h_prev, r, z, nn, Wi, U)
    assert relerr(host(dM), want_dM) <= TOL[dt]
    assert relerr(host(da_prev).T, wda) <= TOL[dt]
    assert relerr(host(dh_prev), wdh) <= TOL[dt]
    gh = host(ghat)
    assert relerr(gh.sum(axis=0), wdb) <= TOL[dt]
    assert relerr(a_prev.T @ gh, wdWi) <= TOL[dt]
    # the gate gradients themselves against the oracle's, every element (the
    # normwise bound; the elementwise figure is reported: in bf16 the stored
    # dM feeding dX carries 2^-9 relative rounding, which elements of dX that
    # nearly cancel turn into large relative errors of small G^ entries)
    want_gh = O.gru_gate_gradients(dX_in + g, h_prev, r, z, nn, U)
    nw, ew = relerr(gh, want_gh), elemerr(gh, want_gh)
    record(os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0], "G^", nw, ew)
    say(f"  G^ normwise {nw:.2e} elementwise {ew:.2e}")
    assert nw <= TOL[dt], nw


def test_device_errors_are_reported():
    n, H = 128, 64
    ws_n = capi.ggnn_gru_update_bwd_workspace_bytes("bf16", n, H)
    small = torch.empty(ws_n // 2, dtype=torch.uint8, device="cuda")
    x = [torch.zeros((n, 3 * H), device="cuda") for _ in range(11)]
    with pytest.raises(capi.GGNNError) as ei:
        capi.ggnn_gru_update_bwd("bf16", n, H, *x, small, ws_n // 2)
    assert ei.value.status_name == "GGNN_ERR_WORKSPACE"
