"""Plain fp64 reference of banded GGNN propagation -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
module.  Every function cites the passage of the paper (arXiv 1906.11786) it
follows.  Readings of passages that the paper leaves open are marked
"Reading:".

Conventions (Background, Eq. 1 and the typed form after it):
  * edges are (src j, dst i, type e): node i receives from node j, i.e.
    a_ij = 1 in the transposed adjacency matrix A_e;
  * node states X are [n, H]; messages M_e = X W_e (+ b_e) are [E, n, H];
  * the aggregated input is a = sum_e A_e M_e, messages summed, not averaged
    (Appendix, hyper-parameters: "Model").

Parity status: every function here is pinned by tests/test_oracle_pins.py
against closed forms, a library routine or finite differences; nothing is
"parity unpinned".
"""
from __future__ import annotations

from collections import deque

import numpy as np


# ----------------------------------------------------------------------------
# Graph structure: bandwidth, coverage of the three block diagonals, RCM
# ----------------------------------------------------------------------------

def bandwidth(src: np.ndarray, dst: np.ndarray) -> int:
    """Bandwidth of the adjacency matrix: the smallest b with a_ij = 0 whenever
    |i - j| > b (Background, "Sparse numerical linear algebra")."""
    if len(src) == 0:
        return 0
    return int(np.max(np.abs(np.asarray(src, np.int64) - np.asarray(dst, np.int64))))


def dedupe_edges(src, dst, etype):
    """A_e has entries in {0, 1} (Background, Eq. 1): repeated (j -> i, e)
    triples are one edge.  Reading: edges of different types between the same
    pair stay distinct.  Returns (src, dst, etype, n_duplicates), sorted by
    (type, dst, src)."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    etype = np.asarray(etype, np.int64)
    if src.size == 0:
        z = np.zeros(0, np.int64)
        return z, z.copy(), z.copy(), 0
    key = np.stack([etype, dst, src], axis=1)
    uniq = np.unique(key, axis=0)
    return uniq[:, 2], uniq[:, 1], uniq[:, 0], int(src.size - uniq.shape[0])


def covered_mask(src, dst, B: int) -> np.ndarray:
    """Which edges the three-block-diagonal product sees (Eq. 3, and the
    coverage remark after it).  Reading: an edge j -> i is covered iff its
    block row floor(i/B) and block column floor(j/B) differ by at most one;
    this keeps every |i-j| < B, some B <= |i-j| < 2B, and no |i-j| >= 2B."""
    bi = np.asarray(dst, np.int64) // B
    bj = np.asarray(src, np.int64) // B
    return np.abs(bi - bj) <= 1


def kept_edges(src, dst, etype, B: int):
    """The edge set the banded method propagates along: deduplicated, then
    restricted to the covered block diagonals.  Returns
    (src, dst, etype, n_dropped, n_duplicates)."""
    s, d, e, ndup = dedupe_edges(src, dst, etype)
    keep = covered_mask(s, d, B)
    return s[keep], d[keep], e[keep], int((~keep).sum()), ndup


def kept_edges_super(src, dst, etype, B: int, n_super: int):
    """The edge set propagated with n_super supernodes next to the band
    (Discussion section: dense slices of the first rows and columns of the
    adjacency matrix): every edge into or out of a node labelled < n_super,
    and the other edges when the three block diagonals cover them.  Returns
    (src, dst, etype, n_dropped, n_duplicates)."""
    s, d, e, ndup = dedupe_edges(src, dst, etype)
    keep = (d < n_super) | (s < n_super) | covered_mask(s, d, B)
    return s[keep], d[keep], e[keep], int((~keep).sum()), ndup


def _sym_neighbours(n: int, src, dst):
    """Neighbour lists of the undirected simple graph that is the union of all
    edge types, symmetrised, without self-loops or repeats."""
    s = np.asarray(src, np.int64)
    d = np.asarray(dst, np.int64)
    u = np.concatenate([s, d])
    v = np.concatenate([d, s])
    m = u != v
    pairs = np.unique(np.stack([u[m], v[m]], axis=1), axis=0) if m.any() else np.zeros((0, 2), np.int64)
    deg = np.bincount(pairs[:, 0], minlength=n) if len(pairs) else np.zeros(n, np.int64)
    nbrs = [[] for _ in range(n)]
    for a, b in pairs.tolist():
        nbrs[a].append(b)
    return nbrs, deg


def _levels(root: int, nbrs) -> list[list[int]]:
    """Rooted level structure (breadth-first levels) of root's component."""
    seen = {root}
    levels = [[root]]
    while True:
        nxt = []
        for v in levels[-1]:
            for w in nbrs[v]:
                if w not in seen:
                    seen.add(w)
                    nxt.append(w)
        if not nxt:
            return levels
        levels.append(nxt)


def rcm_order(n: int, src, dst):
    """Reverse Cuthill-McKee node order (Compilation section: permute the
    nodes with RCMK to expose low bandwidth; Cuthill & McKee 1969).

    Reading of the details the paper leaves open:
      * the graph is the union of all edge types, symmetrised, without
        self-loops and repeats;
      * components are taken in order of their smallest node label;
      * each component starts at a pseudo-peripheral node found by the
        George-Liu iteration started from the component's node of smallest
        (degree, label): build the level structure, move to the smallest
        (degree, label) node of the last level while that increases the
        number of levels;
      * breadth-first search from the start, appending each node's unvisited
        neighbours in increasing (degree, label) order;
      * the concatenated sequence is reversed.
    Returns (order, rank): order[p] is the old label placed at new position
    p, rank[v] is the new position of old node v.  Both int32.
    """
    nbrs, deg = _sym_neighbours(n, src, dst)
    for v in range(n):
        nbrs[v].sort(key=lambda w: (deg[w], w))
    visited = np.zeros(n, dtype=bool)
    seq: list[int] = []
    for v0 in range(n):
        if visited[v0]:
            continue
        comp = [x for lev in _levels(v0, nbrs) for x in lev]
        root = min(comp, key=lambda w: (deg[w], w))
        lev = _levels(root, nbrs)
        while True:
            cand = min(lev[-1], key=lambda w: (deg[w], w))
            lev_c = _levels(cand, nbrs)
            if len(lev_c) > len(lev):
                root, lev = cand, lev_c
            else:
                break
        visited[root] = True
        q = deque([root])
        while q:
            x = q.popleft()
            seq.append(x)
            for w in nbrs[x]:
                if not visited[w]:
                    visited[w] = True
                    q.append(w)
    order = np.asarray(seq[::-1], dtype=np.int32)
    rank = np.empty(n, dtype=np.int32)
    rank[order] = np.arange(n, dtype=np.int32)
    return order, rank


def relabel(rank, src, dst):
    """Apply a node relabelling old v -> rank[v] to an edge list (Compilation
    section: predictions are permuted along with the nodes)."""
    rank = np.asarray(rank, np.int64)
    return rank[np.asarray(src, np.int64)], rank[np.asarray(dst, np.int64)]


def batch_layout(graphs_edges, B: int):
    """Sparse batching (Background, "Sparse batching"): graphs become disjoint
    components of one supergraph by offsetting their labels.  Input: list of
    (n, src, dst, etype) already in their final per-graph labelling.  Returns
    (n_real, n_pad, src, dst, etype, offsets) with n_pad the next multiple of
    B."""
    offs = [0]
    S, D, T = [], [], []
    for n, s, d, e in graphs_edges:
        S.append(np.asarray(s, np.int64) + offs[-1])
        D.append(np.asarray(d, np.int64) + offs[-1])
        T.append(np.asarray(e, np.int64))
        offs.append(offs[-1] + n)
    n_real = offs[-1]
    n_pad = -(-n_real // B) * B
    cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int64))
    return n_real, n_pad, cat(S), cat(D), cat(T), np.asarray(offs, np.int64)


# ----------------------------------------------------------------------------
# Block-band packing (Eq. 3; Algorithm 1's Cks, Uks, Lks inputs)
# ----------------------------------------------------------------------------

def pack_band(n_pad: int, E: int, B: int, src, dst, etype) -> np.ndarray:
    """Dense block band band[e, k, s, r, c] (float64) of A_e, with k the block
    row, s = 0, 1, 2 the sub-diagonal, diagonal and super-diagonal block
    (block column k-1+s), r the receiver row and c the sender column inside
    the blocks (Eq. 3: L blocks, C blocks, U blocks).  Edges outside the
    three block diagonals are left out, repeats count once."""
    nb = n_pad // B
    band = np.zeros((E, nb, 3, B, B), dtype=np.float64)
    s, d, e, _, _ = kept_edges(src, dst, etype, B)
    k = d // B
    band[e, k, s // B - k + 1, d % B, s % B] = 1.0
    return band


def unpack_band(band: np.ndarray):
    """Inverse of pack_band: the (src, dst, etype) of every nonzero entry."""
    E, nb, _, B, _ = band.shape
    e, k, s, r, c = np.nonzero(band)
    dst = k * B + r
    src = (k - 1 + s) * B + c
    return src.astype(np.int64), dst.astype(np.int64), e.astype(np.int64)


def banded_apply(band: np.ndarray, M: np.ndarray) -> np.ndarray:
    """a = sum_e A_e M_e evaluated as the three batched block products of
    Eq. 3: a_k = sum_e C_k M_e[k] + U_k M_e[k+1] + L_k M_e[k-1].
    band [E, nb, 3, B, B], M [E, nb*B, H] -> a [nb*B, H]."""
    E, nb, _, B, _ = band.shape
    H = M.shape[2]
    Mb = M.reshape(E, nb, B, H)
    Mp = np.zeros((E, nb + 2, B, H))
    Mp[:, 1:nb + 1] = Mb
    a = np.zeros((nb, B, H))
    for s in range(3):
        a += np.einsum("ekrc,ekch->krh", band[:, :, s], Mp[:, s:s + nb])
    return a.reshape(nb * B, H)


# ----------------------------------------------------------------------------
# Model math (Eq. 1 with typed edges; GRU of Cho et al. 2014)
# ----------------------------------------------------------------------------

def msg_transform(X: np.ndarray, W: np.ndarray, bias=None) -> np.ndarray:
    """Messages M_e = X W_e (+ 1 b_e^T) for every edge type (typed form of
    Eq. 1; the per-type bias of the Appendix's "Model" paragraph)."""
    M = np.stack([X @ W[e] for e in range(W.shape[0])])
    if bias is not None:
        M = M + bias[:, None, :]
    return M


def _scatter_rows(n: int, rows: np.ndarray, vals: np.ndarray) -> np.ndarray:
    """out[i] = sum of vals[k] over all k with rows[k] == i (a weighted count
    per output row, one feature column at a time)."""
    out = np.zeros((n, vals.shape[1]))
    for h in range(vals.shape[1]):
        out[:, h] = np.bincount(rows, weights=vals[:, h], minlength=n)
    return out


def aggregate(n: int, src, dst, etype, M: np.ndarray) -> np.ndarray:
    """a[i] = sum over edges (j -> i, e) of M_e[j]: the sparse product
    sum_e A_e M_e by explicit scatter-add (Eq. 1; messages are summed)."""
    src, dst, etype = (np.asarray(x, np.int64) for x in (src, dst, etype))
    return _scatter_rows(n, dst, M[etype, src])


def aggregate_transpose(n: int, src, dst, etype, da: np.ndarray, E: int) -> np.ndarray:
    """Adjoint of `aggregate`: dM_e[j] = sum over edges (j -> i, e) of da[i]
    (a gather along reversed edges, i.e. A_e^T da)."""
    src, dst, etype = (np.asarray(x, np.int64) for x in (src, dst, etype))
    dM = np.zeros((E, n, da.shape[1]))
    for e in range(E):
        sel = etype == e
        dM[e] = _scatter_rows(n, src[sel], da[dst[sel]])
    return dM


def msg_transform_backward(X: np.ndarray, W: np.ndarray, dM: np.ndarray):
    """Reverse of msg_transform: dX = sum_e dM_e W_e^T, dW_e = X^T dM_e,
    db_e = column sums of dM_e."""
    dX = sum(dM[e] @ W[e].T for e in range(W.shape[0]))
    dW = np.stack([X.T @ dM[e] for e in range(W.shape[0])])
    dbias = dM.sum(axis=1)
    return dX, dW, dbias


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def gru_forward(a, h, Wi, U, b):
    """GRU node update (Eq. 1's GRU; Cho et al. 2014).  Reading: the reset gate
    multiplies the state before U_n, one bias per gate, gates ordered
    (r, z, n) along the 3H columns of Wi [H, 3H] and U [H, 3H]:
        r = sigmoid(a Wi_r + h U_r + b_r)
        z = sigmoid(a Wi_z + h U_z + b_z)
        n = tanh(a Wi_n + (r * h) U_n + b_n)
        h' = z * h + (1 - z) * n
    Returns (h', r, z, n)."""
    H = h.shape[1]
    gi = a @ Wi + b
    r = _sigmoid(gi[:, :H] + h @ U[:, :H])
    z = _sigmoid(gi[:, H:2 * H] + h @ U[:, H:2 * H])
    nn = np.tanh(gi[:, 2 * H:] + (r * h) @ U[:, 2 * H:])
    return z * h + (1.0 - z) * nn, r, z, nn


def gru_gate_gradients(g, h, r, z, nn, U):
    """Gradients of the three gate pre-activations of gru_forward (the sums
    inside sigma, sigma and tanh, bias included) for the upstream gradient g
    of h': the [n, 3H] matrix [r^, z^, n^] that the reverse pass multiplies
    by Wi^T and U^T and that the weight gradients contract with a and h."""
    H = h.shape[1]
    gn = g * (1.0 - z) * (1.0 - nn * nn)  # d/d(pre-activation of n)
    gz = g * (h - nn) * z * (1.0 - z)     # d/d(pre-activation of z)
    q = gn @ U[:, 2 * H:].T               # d/d(r * h)
    gr = q * h * r * (1.0 - r)            # d/d(pre-activation of r)
    return np.concatenate([gr, gz, gn], axis=1)


def gru_backward(g, a, h, r, z, nn, Wi, U):
    """Reverse-mode derivative of gru_forward for the upstream gradient g of
    h'.  Returns (da, dh, dWi, dU, db)."""
    H = h.shape[1]
    ghat = gru_gate_gradients(g, h, r, z, nn, U)
    gr, gz, gn = ghat[:, :H], ghat[:, H:2 * H], ghat[:, 2 * H:]
    q = gn @ U[:, 2 * H:].T               # d/d(r * h)
    dh = g * z + q * r
    da = ghat @ Wi.T
    dh = dh + gr @ U[:, :H].T + gz @ U[:, H:2 * H].T
    dWi = a.T @ ghat
    dU = np.concatenate([h.T @ gr, h.T @ gz, (r * h).T @ gn], axis=1)
    db = ghat.sum(axis=0)
    return da, dh, dWi, dU, db


def propagate(n: int, B, src, dst, etype, X0, W, Wi, U, b, T: int, G=None, bias=None, n_super: int = 0):
    """T steps of banded GGNN propagation (Eq. 1, Algorithm 1 semantics) on the
    edges the three block diagonals cover, and, when G is given, the reverse
    pass for the loss L = sum(G * X_T).  n_super > 0 adds every edge touching
    the supernodes 0 .. n_super-1 (kept_edges_super).  B = None propagates
    along every (deduplicated) edge: the sparse model that evaluates the weights of a
    banded one on all edges (Experiments, "Training time to validation
    accuracy").

    Returns a dict with 'X' (list of X_0..X_T), 'a', 'r', 'z', 'n' (per step),
    'n_dropped', 'n_duplicate', and with G: 'dX0', 'dW', 'dbias', 'dWi', 'dU',
    'db', 'dX' (list of dX_0..dX_T)."""
    E = W.shape[0]
    if B is None:
        s, d, e, ndup = dedupe_edges(src, dst, etype)
        ndrop = 0
    elif n_super > 0:
        s, d, e, ndrop, ndup = kept_edges_super(src, dst, etype, B, n_super)
    else:
        s, d, e, ndrop, ndup = kept_edges(src, dst, etype, B)
    out = {"X": [np.asarray(X0, np.float64)], "a": [], "r": [], "z": [], "n": [],
           "n_dropped": ndrop, "n_duplicate": ndup}
    for t in range(T):
        h = out["X"][t]
        M = msg_transform(h, W, bias)
        a = aggregate(n, s, d, e, M)
        hn, r, z, nn = gru_forward(a, h, Wi, U, b)
        out["X"].append(hn)
        out["a"].append(a)
        out["r"].append(r)
        out["z"].append(z)
        out["n"].append(nn)
    if G is None:
        return out
    H = X0.shape[1]
    dW = np.zeros_like(W, dtype=np.float64)
    dbias = np.zeros((E, H))
    dWi = np.zeros_like(Wi, dtype=np.float64)
    dU = np.zeros_like(U, dtype=np.float64)
    db = np.zeros_like(b, dtype=np.float64)
    g = np.asarray(G, np.float64)
    dXs = [None] * (T + 1)
    dXs[T] = g
    for t in range(T - 1, -1, -1):
        h = out["X"][t]
        da, dh, dWi_t, dU_t, db_t = gru_backward(g, out["a"][t], h, out["r"][t], out["z"][t], out["n"][t], Wi, U)
        dM = aggregate_transpose(n, s, d, e, da, E)
        dXm, dW_t, dbias_t = msg_transform_backward(h, W, dM)
        g = dh + dXm
        dXs[t] = g
        dW += dW_t
        dbias += dbias_t
        dWi += dWi_t
        dU += dU_t
        db += db_t
    out.update(dX0=g, dW=dW, dbias=dbias, dWi=dWi, dU=dU, db=db, dX=dXs)
    return out


# ----------------------------------------------------------------------------
# Readout, loss and the parameter update closing one training step
# ----------------------------------------------------------------------------

def readout_logits(XT, w_out, b_out, cand_node):
    """Per-candidate logits: a learned linear map R^H -> R applied to the
    final embeddings of the candidate nodes (Background, "Variable misuse").
    Returns logits[c] = XT[cand_node[c]] . w_out + b_out."""
    XT = np.asarray(XT, np.float64)
    return XT[np.asarray(cand_node, np.int64)] @ np.asarray(w_out, np.float64) + float(b_out)


def readout_loss(logits, cand_ptr, target):
    """Softmax over each graph's candidates (Background, "Variable misuse":
    the softmax gives the probability of each candidate filling the hole) and
    the cross-entropy of the correct one.  Graph g owns candidates
    cand_ptr[g] .. cand_ptr[g+1]-1, target[g] is the index of the correct one
    within them.  Reading: the training loss is the mean over graphs.
    Returns (loss per graph [G], mean loss, dlogits = d mean / d logits).
    A graph without candidates contributes loss 0 and no gradient."""
    logits = np.asarray(logits, np.float64)
    ptr = np.asarray(cand_ptr, np.int64)
    G = len(ptr) - 1
    loss = np.zeros(G)
    dlog = np.zeros_like(logits)
    for g in range(G):
        lo, hi = ptr[g], ptr[g + 1]
        if hi == lo:
            continue
        z = logits[lo:hi]
        p = np.exp(z - z.max())
        p /= p.sum()
        loss[g] = -np.log(p[target[g]])
        onehot = np.zeros(hi - lo)
        onehot[target[g]] = 1.0
        dlog[lo:hi] = (p - onehot) / G
    return loss, float(loss.mean()), dlog


def readout_backward(XT, w_out, cand_node, dlogits):
    """Reverse of readout_logits: dXT (zero except candidate rows),
    dw_out = sum_c dlogits[c] XT[cand_node[c]], db_out = sum_c dlogits[c]."""
    XT = np.asarray(XT, np.float64)
    cand = np.asarray(cand_node, np.int64)
    dl = np.asarray(dlogits, np.float64)
    dXT = np.zeros_like(XT)
    np.add.at(dXT, cand, dl[:, None] * np.asarray(w_out, np.float64)[None, :])
    return dXT, XT[cand].T @ dl, float(dl.sum())


def momentum_update(theta, velocity, grad, lr, momentum, weight_decay=0.0, nesterov=False):
    """One step of the Momentum optimizer (Appendix, "Optimization": momentum,
    optionally Nesterov, with L2 weight decay):
        g' = grad + weight_decay * theta
        v  = momentum * v + g'
        theta -= lr * (g' + momentum * v)   (Nesterov)   or   lr * v
    Returns (theta, v)."""
    theta = np.asarray(theta, np.float64)
    g = np.asarray(grad, np.float64) + weight_decay * theta
    v = momentum * np.asarray(velocity, np.float64) + g
    step = g + momentum * v if nesterov else v
    return theta - lr * step, v


def evaluate(n: int, B, src, dst, etype, X0, params: dict, T: int, cand_node, cand_ptr, target):
    """Mean readout loss of the parameters after T propagation steps (B = None:
    along every edge).  Returns (loss per graph, mean loss)."""
    out = propagate(n, B, src, dst, etype, X0, params["W"], params["Wi"], params["U"], params["b"], T,
                    bias=params.get("bias"))
    logits = readout_logits(out["X"][T], params["w_out"], params["b_out"], cand_node)
    loss, mean, _ = readout_loss(logits, cand_ptr, target)
    return loss, mean


def train_step(n: int, B: int, src, dst, etype, X0, params: dict, velocity: dict, T: int,
               cand_node, cand_ptr, target, lr, momentum, weight_decay=0.0, nesterov=False):
    """One training step (Background: propagation, then the readout and the
    softmax loss; Appendix, "Optimization": the Momentum update of every
    parameter).  params holds W, bias (or None), Wi, U, b, w_out, b_out;
    velocity the same keys.  Returns (new params, new velocity, mean loss,
    gradients)."""
    bias = params.get("bias")
    out = propagate(n, B, src, dst, etype, X0, params["W"], params["Wi"], params["U"], params["b"], T, bias=bias)
    XT = out["X"][T]
    logits = readout_logits(XT, params["w_out"], params["b_out"], cand_node)
    _, mean_loss, dlog = readout_loss(logits, cand_ptr, target)
    dXT, dw_out, db_out = readout_backward(XT, params["w_out"], cand_node, dlog)
    rev = propagate(n, B, src, dst, etype, X0, params["W"], params["Wi"], params["U"], params["b"], T, G=dXT,
                    bias=bias)
    grads = {"W": rev["dW"], "Wi": rev["dWi"], "U": rev["dU"], "b": rev["db"], "w_out": dw_out,
             "b_out": np.float64(db_out)}
    if bias is not None:
        grads["bias"] = rev["dbias"]
    new_p, new_v = dict(params), dict(velocity)
    for k, g in grads.items():
        new_p[k], new_v[k] = momentum_update(params[k], velocity[k], g, lr, momentum, weight_decay, nesterov)
    return new_p, new_v, mean_loss, grads
