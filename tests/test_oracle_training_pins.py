"""Pins of the oracle's readout, loss and Momentum update (the step that
closes one training iteration) against library routines, closed forms and
finite differences."""
import numpy as np
import pytest

import oracle as O

torch = pytest.importorskip("torch")


def _cands(rng, n, G, kmax=6):
    """G graphs, each with 1..kmax distinct candidate nodes (distinct across
    graphs too), and a target index per graph."""
    nodes = rng.permutation(n)
    ks = rng.integers(1, kmax + 1, G)
    ptr = np.concatenate([[0], np.cumsum(ks)])
    return nodes[:ptr[-1]], ptr, np.array([rng.integers(0, k) for k in ks])


def test_loss_matches_torch_cross_entropy():
    rng = np.random.default_rng(0)
    n, H, G = 60, 5, 7
    XT = rng.standard_normal((n, H))
    w, b = rng.standard_normal(H), 0.3
    cand, ptr, tgt = _cands(rng, n, G)
    logits = O.readout_logits(XT, w, b, cand)
    np.testing.assert_allclose(logits, np.array([XT[c] @ w + b for c in cand]), rtol=1e-13)
    loss, mean, dlog = O.readout_loss(logits, ptr, tgt)
    lt = torch.tensor(logits, dtype=torch.float64, requires_grad=True)
    want = []
    for g in range(G):
        seg = lt[ptr[g]:ptr[g + 1]].unsqueeze(0)
        want.append(torch.nn.functional.cross_entropy(seg, torch.tensor([int(tgt[g])])))
    tot = torch.stack(want).mean()
    tot.backward()
    np.testing.assert_allclose(loss, torch.stack(want).detach().numpy(), rtol=1e-12)
    assert abs(mean - tot.item()) < 1e-12
    np.testing.assert_allclose(dlog, lt.grad.numpy(), atol=1e-14)


def test_loss_closed_forms():
    # two equal logits: loss log 2, gradient (1/2 - 1) / G on the target
    loss, mean, d = O.readout_loss(np.array([1.5, 1.5, 0.2]), np.array([0, 2, 3]), np.array([1, 0]))
    assert abs(loss[0] - np.log(2)) < 1e-15 and loss[1] == 0.0
    np.testing.assert_allclose(d, [0.25, -0.25, 0.0], atol=1e-15)
    # empty graph: no loss, no gradient; shifting a graph's logits changes nothing
    loss, _, d = O.readout_loss(np.array([0.1, -2.0]), np.array([0, 0, 2]), np.array([0, 1]))
    assert loss[0] == 0.0
    l2, _, d2 = O.readout_loss(np.array([7.1, 5.0]), np.array([0, 0, 2]), np.array([0, 1]))
    np.testing.assert_allclose(l2, loss, rtol=1e-12)
    np.testing.assert_allclose(d2, d, atol=1e-15)
    # each graph's gradient sums to zero, so the readout bias gets none
    rng = np.random.default_rng(1)
    cand, ptr, tgt = _cands(rng, 50, 9)
    _, _, d = O.readout_loss(rng.standard_normal(len(cand)), ptr, tgt)
    for g in range(9):
        assert abs(d[ptr[g]:ptr[g + 1]].sum()) < 1e-15


def test_readout_backward_matches_finite_differences():
    rng = np.random.default_rng(2)
    n, H, G = 40, 4, 5
    XT = rng.standard_normal((n, H))
    w, b = rng.standard_normal(H), -0.4
    cand, ptr, tgt = _cands(rng, n, G)

    def L(XT_, w_, b_):
        return O.readout_loss(O.readout_logits(XT_, w_, b_, cand), ptr, tgt)[1]

    _, _, dlog = O.readout_loss(O.readout_logits(XT, w, b, cand), ptr, tgt)
    dXT, dw, db = O.readout_backward(XT, w, cand, dlog)
    eps = 1e-6
    D = rng.standard_normal(XT.shape)
    fd = (L(XT + eps * D, w, b) - L(XT - eps * D, w, b)) / (2 * eps)
    assert abs(fd - np.sum(D * dXT)) < 1e-8
    dwv = rng.standard_normal(H)
    fd = (L(XT, w + eps * dwv, b) - L(XT, w - eps * dwv, b)) / (2 * eps)
    assert abs(fd - dwv @ dw) < 1e-8
    fd = (L(XT, w, b + eps) - L(XT, w, b - eps)) / (2 * eps)
    assert abs(fd - db) < 1e-8 and abs(db) < 1e-14
    # rows of non-candidates get nothing
    mask = np.ones(n, bool)
    mask[cand] = False
    assert np.all(dXT[mask] == 0)


@pytest.mark.parametrize("nesterov", [False, True])
@pytest.mark.parametrize("wd", [0.0, 1e-2])
def test_momentum_matches_torch_sgd(nesterov, wd):
    rng = np.random.default_rng(3)
    theta0 = rng.standard_normal(17)
    grads = [rng.standard_normal(17) for _ in range(4)]
    p = torch.tensor(theta0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=0.05, momentum=0.9, nesterov=nesterov, weight_decay=wd)
    th, v = theta0.copy(), np.zeros(17)
    for gr in grads:
        opt.zero_grad()
        p.grad = torch.tensor(gr, dtype=torch.float64)
        opt.step()
        th, v = O.momentum_update(th, v, gr, 0.05, 0.9, wd, nesterov)
        np.testing.assert_allclose(th, p.detach().numpy(), rtol=1e-13, atol=1e-14)


def test_momentum_closed_form_constant_gradient():
    g, mu, lr, k = np.array([0.5, -2.0]), 0.8, 0.1, 6
    th, v = np.zeros(2), np.zeros(2)
    for _ in range(k):
        th, v = O.momentum_update(th, v, g, lr, mu)
    np.testing.assert_allclose(v, g * (1 - mu ** k) / (1 - mu), rtol=1e-14)
    # theta = -lr * sum_{j=1..k} g (1 - mu^j) / (1 - mu)
    want = -lr * g * sum((1 - mu ** j) / (1 - mu) for j in range(1, k + 1))
    np.testing.assert_allclose(th, want, rtol=1e-14)


def _tiny_model(seed):
    rng = np.random.default_rng(seed)
    n, B, E, H, T = 16, 4, 2, 3, 2
    src = rng.integers(0, n, 50)
    dst = np.clip(src + rng.integers(-5, 6, 50), 0, n - 1)
    et = rng.integers(0, E, 50)
    k = 1 / np.sqrt(H)
    p = {"W": rng.standard_normal((E, H, H)) / np.sqrt(H), "bias": rng.uniform(-k, k, (E, H)),
         "Wi": rng.uniform(-k, k, (H, 3 * H)), "U": rng.uniform(-k, k, (H, 3 * H)), "b": rng.uniform(-k, k, 3 * H),
         "w_out": rng.standard_normal(H), "b_out": np.float64(0.1)}
    X0 = rng.standard_normal((n, H))
    cand, ptr, tgt = _cands(rng, n, 3, kmax=4)
    return n, B, src, dst, et, X0, T, p, cand, ptr, tgt


def _mean_loss(n, B, src, dst, et, X0, T, p, cand, ptr, tgt):
    out = O.propagate(n, B, src, dst, et, X0, p["W"], p["Wi"], p["U"], p["b"], T, bias=p["bias"])
    return O.readout_loss(O.readout_logits(out["X"][T], p["w_out"], p["b_out"], cand), ptr, tgt)[1]


@pytest.mark.parametrize("seed", [0, 1])
def test_train_step_gradients_match_finite_differences(seed):
    """Every gradient of the composed step (propagation, readout, softmax
    loss) against central differences of the mean loss along a random
    direction; then the update is lr * grad for zero momentum state."""
    n, B, src, dst, et, X0, T, p, cand, ptr, tgt = _tiny_model(seed)
    vel = {k: np.zeros_like(np.asarray(v, np.float64)) for k, v in p.items()}
    newp, newv, mean, grads = O.train_step(n, B, src, dst, et, X0, p, vel, T, cand, ptr, tgt, lr=0.1, momentum=0.9)
    assert abs(mean - _mean_loss(n, B, src, dst, et, X0, T, p, cand, ptr, tgt)) < 1e-14
    rng = np.random.default_rng(100 + seed)
    eps = 1e-6
    for key in ["W", "bias", "Wi", "U", "b", "w_out", "b_out"]:
        D = rng.standard_normal(np.shape(p[key]))
        pp, pm = dict(p), dict(p)
        pp[key] = p[key] + eps * D
        pm[key] = p[key] - eps * D
        fd = (_mean_loss(n, B, src, dst, et, X0, T, pp, cand, ptr, tgt) -
              _mean_loss(n, B, src, dst, et, X0, T, pm, cand, ptr, tgt)) / (2 * eps)
        an = float(np.sum(D * grads[key]))
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(fd)), key
        np.testing.assert_allclose(newp[key], p[key] - 0.1 * grads[key], rtol=1e-14, atol=1e-16)
        np.testing.assert_allclose(newv[key], grads[key], rtol=1e-14, atol=1e-16)


def test_all_edge_propagation_equals_a_band_wide_enough():
    """B = None (every edge) agrees with a band wide enough to drop nothing,
    and differs from a narrow band that drops edges."""
    rng = np.random.default_rng(5)
    n, E, H, T = 48, 2, 3, 2
    src = rng.integers(0, n, 150)
    dst = rng.integers(0, n, 150)            # spans up to n-1: outside any narrow band
    et = rng.integers(0, E, 150)
    k = 1 / np.sqrt(H)
    W = rng.standard_normal((E, H, H)) / np.sqrt(H)
    Wi, U, b = rng.uniform(-k, k, (H, 3 * H)), rng.uniform(-k, k, (H, 3 * H)), rng.uniform(-k, k, 3 * H)
    X0 = rng.standard_normal((n, H))
    full = O.propagate(n, None, src, dst, et, X0, W, Wi, U, b, T)
    wide = O.propagate(n, 64, src, dst, et, X0, W, Wi, U, b, T)      # one block: nothing dropped
    narrow = O.propagate(n, 4, src, dst, et, X0, W, Wi, U, b, T)
    assert wide["n_dropped"] == 0 and narrow["n_dropped"] > 0 and full["n_dropped"] == 0
    np.testing.assert_allclose(full["X"][T], wide["X"][T], rtol=1e-13, atol=1e-13)
    assert np.abs(full["X"][T] - narrow["X"][T]).max() > 1e-3


def test_supernode_edge_set():
    """With supernodes, every edge touching a node < n_super is propagated:
    equal to propagation on all edges when the other edges fit the band, and
    to the plain band when no edge touches a supernode."""
    rng = np.random.default_rng(8)
    n, B, E, H, T, ns = 64, 8, 2, 3, 2, 4
    far_s = rng.integers(0, ns, 40)                  # supernode edges spanning the whole graph
    far_d = rng.integers(0, n, 40)
    near_s = rng.integers(ns, n, 120)
    near_d = np.clip(near_s + rng.integers(-3, 4, 120), ns, n - 1)
    src = np.concatenate([far_s, far_d, near_s])
    dst = np.concatenate([far_d, far_s, near_d])
    et = rng.integers(0, E, len(src))
    k = 1 / np.sqrt(H)
    W = rng.standard_normal((E, H, H)) / np.sqrt(H)
    Wi, U, b = rng.uniform(-k, k, (H, 3 * H)), rng.uniform(-k, k, (H, 3 * H)), rng.uniform(-k, k, 3 * H)
    X0, G = rng.standard_normal((n, H)), rng.standard_normal((n, H))
    sup = O.propagate(n, B, src, dst, et, X0, W, Wi, U, b, T, G=G, n_super=ns)
    full = O.propagate(n, None, src, dst, et, X0, W, Wi, U, b, T, G=G)
    band = O.propagate(n, B, src, dst, et, X0, W, Wi, U, b, T, G=G)
    assert sup["n_dropped"] == 0 and band["n_dropped"] > 0
    for key in ("dX0", "dW", "dWi"):
        np.testing.assert_allclose(sup[key], full[key], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sup["X"][T], full["X"][T], rtol=1e-12, atol=1e-12)
    ns_ = O.propagate(n, B, near_s, near_d, et[:120], X0, W, Wi, U, b, T, n_super=ns)
    nb_ = O.propagate(n, B, near_s, near_d, et[:120], X0, W, Wi, U, b, T)
    np.testing.assert_array_equal(ns_["X"][T], nb_["X"][T])
