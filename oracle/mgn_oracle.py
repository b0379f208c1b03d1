"""Plain fp64 CPU oracle of the scaled-MeshGraphNets message-passing path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module.  It shares no
code with the GPU library: it reads the same seeded inputs (from ``synth``)
and nothing else.

Everything here is written from the paper (Bartoldson, Hu et al.,
"Scientific Computing Algorithms to Learn Enhanced Scalable Surrogates for
Mesh Physics", ICLR 2023 workshop; arXiv 2304.00338):

* Sec. 2.1 -- one MGN message-passing step updates every edge from its two
  incident nodes, then every node from the aggregate of its incident edges;
  the next state is ``y + MGN(y)``.
* Sec. 2.2 -- subdomains from an equal split of every axis; a patch is a
  subdomain plus its k-hop ghost zone; with m <= k message-passing steps the
  subdomain nodes of a patch are updated exactly as on the whole mesh
  (condition 1), the loss covers subdomain nodes only (condition 2) and
  gradients are summed over all patches before an update (condition 3).
* Sec. 2.3 and App. A -- Heun's second-order update (equation FE_HUEN and the
  MGN-scaled form in equation heun) and Heun's third-order method; the
  outlook (App. D) names Ralston's methods and predict-evaluate-correct at
  inference.
* App. B -- mesh edges come from the simplices of the mesh; App. C -- the
  MGN edge features (relative displacement and its length), latent width 128.

Readings where the paper is silent (recorded in the design notes): MLPs are
two Linear layers with one ReLU; every encoder and processor MLP ends in a
LayerNorm (biased variance, eps 1e-5, affine); the decoder has none; the
aggregate is the sum over a node's in-edges of the new edge message (the
LayerNorm output, before the edge residual); residuals are added after both
updates, and the node update uses the node latents from before the step;
processor blocks do not share weights; the integrator replaces ``h f`` by
MGN, so a stage state is ``y + sum_j a_ij K_j`` with ``K_j = MGN(stage j)``;
Heun's third-order method uses the tableau c = (0, 1/3, 2/3),
a21 = 1/3, a32 = 2/3, b = (1/4, 0, 3/4).

Parity pins for every function live in ``tests/test_oracle_*.py``.  The whole
network's output values have no printed example in the paper: beyond the
structural pins (dense brute force, permutation equivariance, locality,
patch equivalence, finite differences, integrator closed forms) they are
"parity unpinned".
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

__all__ = [
    "Graph", "Patch", "build_graph", "partition", "extract_patch",
    "param_layout", "unpack_params", "n_params", "mlp", "layer_norm", "hop_distance", "edge_features", "pack_grads",
    "mgn_forward", "mgn_backward", "TABLEAUS", "integrate_step",
    "integrate_backward", "masked_mse_grad", "relu_kinks", "pec_step", "pec_rollout",
    "NOISE_STD_3D", "lr_schedule", "adam_update", "masked_mse", "train_step",
]

LN_EPS = 1e-5


# --------------------------------------------------------------------------
# a0: mesh graph (App. B: edges from the mesh simplices; App. C: MGN edge
# features = sender-minus-receiver displacement and its Euclidean length)
# --------------------------------------------------------------------------
class Graph:
    """Receiver-sorted directed mesh graph.

    rowptr[N+1]  in-edge segment of node v is rowptr[v]:rowptr[v+1]
    senders[E]   sender of edge e (receivers ascending, then senders)
    receivers[E] receiver of edge e
    rev[E]       index of the opposite edge (receiver->sender)
    efeat[E,4]   float32 [x_s - x_r, |x_s - x_r|] (2D: [dx, dy, |d|, 0])
    """

    def __init__(self, rowptr, senders, receivers, rev, efeat):
        self.rowptr = rowptr
        self.senders = senders
        self.receivers = receivers
        self.rev = rev
        self.efeat = efeat

    @property
    def n_nodes(self):
        return self.rowptr.shape[0] - 1

    @property
    def n_edges(self):
        return self.senders.shape[0]


def _csr_from_pairs(recv, send, n):
    """Sort directed pairs by (receiver, sender), drop duplicates, return
    rowptr, senders, receivers, rev."""
    key = np.unique(recv.astype(np.int64) * n + send.astype(np.int64))
    receivers = key // n
    senders = key % n
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(receivers, minlength=n), out=rowptr[1:])
    rev = np.searchsorted(key, senders * n + receivers)
    if rev.size and not np.all(key[np.minimum(rev, key.size - 1)]
                               == senders * n + receivers):
        raise ValueError("graph is not symmetric")
    return rowptr, senders, receivers, rev


def edge_features(pos, senders, receivers):
    """MGN edge features: displacement sender - receiver and its length,
    evaluated in fp64 from the float32 positions and rounded once to
    float32; 2D pads a zero so every edge has four features."""
    p = np.asarray(pos, dtype=np.float32).astype(np.float64)
    dim = p.shape[1]
    d = p[senders] - p[receivers]
    sq = d[:, 0] * d[:, 0]
    for c in range(1, dim):
        sq = sq + d[:, c] * d[:, c]
    nrm = np.sqrt(sq)
    f = np.zeros((senders.shape[0], 4), dtype=np.float64)
    f[:, :dim] = d
    f[:, dim] = nrm
    return f.astype(np.float32)


def build_graph(cells, pos) -> Graph:
    """Every unordered pair of distinct vertices sharing a cell becomes an
    undirected mesh edge, stored as two directed edges."""
    cells = np.asarray(cells, dtype=np.int64)
    pos = np.asarray(pos, dtype=np.float32)
    n = pos.shape[0]
    if cells.ndim != 2 or cells.shape[1] not in (2, 3, 4):
        raise ValueError("cells must be [n_cells, 2|3|4]")
    if pos.ndim != 2 or pos.shape[1] not in (2, 3):
        raise ValueError("pos must be [N, 2|3]")
    if cells.size and (cells.min() < 0 or cells.max() >= n):
        raise ValueError("cell vertex id out of range")
    recv, send = [], []
    k = cells.shape[1]
    for a in range(k):
        for b in range(k):
            if a == b:
                continue
            keep = cells[:, a] != cells[:, b]
            recv.append(cells[keep, b])
            send.append(cells[keep, a])
    recv = np.concatenate(recv) if recv else np.zeros(0, np.int64)
    send = np.concatenate(send) if send else np.zeros(0, np.int64)
    rowptr, senders, receivers, rev = _csr_from_pairs(recv, send, n)
    return Graph(rowptr, senders, receivers, rev,
                 edge_features(pos, senders, receivers))


# --------------------------------------------------------------------------
# a1: subdomains and ghost-zone patches (Sec. 2.2; App. C patch counts)
# --------------------------------------------------------------------------
def partition(pos, splits):
    """Equal split of the bounding box along every axis.  Per axis the index
    is floor(splits * (x - lo) / (hi - lo)) in fp64 (left to right), clamped
    to [0, splits-1]; a degenerate axis (hi == lo) gives 0.  The subdomain id
    runs x fastest."""
    p = np.asarray(pos, dtype=np.float32).astype(np.float64)
    splits = [int(s) for s in splits]
    if len(splits) != p.shape[1] or min(splits) < 1:
        raise ValueError("one positive split per axis")
    part = np.zeros(p.shape[0], dtype=np.int64)
    stride = 1
    for ax, s in enumerate(splits):
        x = p[:, ax]
        lo, hi = x.min(), x.max()
        if hi > lo:
            idx = np.floor((s * (x - lo)) / (hi - lo)).astype(np.int64)
            idx = np.clip(idx, 0, s - 1)
        else:
            idx = np.zeros_like(part)
        part += idx * stride
        stride *= s
    return part


class Patch(Graph):
    """A subdomain plus its k-hop ghost zone, as an induced subgraph with
    ascending global ids as local ids."""

    def __init__(self, rowptr, senders, receivers, rev, efeat, node_l2g, hop,
                 edge_l2g):
        super().__init__(rowptr, senders, receivers, rev, efeat)
        self.node_l2g = node_l2g
        self.hop = hop
        self.edge_l2g = edge_l2g

    @property
    def interior(self):
        return (self.hop == 0).astype(np.uint8)

    @property
    def n_interior(self):
        return int(np.count_nonzero(self.hop == 0))


def hop_distance(g: Graph, sources_mask, k):
    """Breadth-first hop count from the source set over the (symmetric) mesh
    graph, up to k hops; -1 for nodes farther than k."""
    hop = np.full(g.n_nodes, -1, dtype=np.int64)
    hop[sources_mask] = 0
    frontier = np.asarray(sources_mask, dtype=bool).copy()
    for d in range(1, k + 1):
        # neighbours of the frontier: senders of edges whose receiver is on it
        cand = g.senders[frontier[g.receivers]]
        new = np.zeros(g.n_nodes, dtype=bool)
        new[cand] = True
        new &= hop < 0
        if not new.any():
            break
        hop[new] = d
        frontier = new
    return hop


def extract_patch(g: Graph, part, p, k) -> Patch:
    """Patch p: all nodes within k hops of subdomain p, induced edges."""
    part = np.asarray(part)
    if k < 0:
        raise ValueError("k must be >= 0")
    if part.shape[0] != g.n_nodes:
        raise ValueError("part has wrong length")
    if p < 0 or (part.size and p > part.max()):
        raise ValueError("subdomain id out of range")
    hop = hop_distance(g, part == p, k)
    nodes = np.nonzero(hop >= 0)[0]
    g2l = np.full(g.n_nodes, -1, dtype=np.int64)
    g2l[nodes] = np.arange(nodes.size)
    keep = (g2l[g.receivers] >= 0) & (g2l[g.senders] >= 0)
    eids = np.nonzero(keep)[0]
    lr = g2l[g.receivers[eids]]
    ls = g2l[g.senders[eids]]
    order = np.lexsort((ls, lr))
    eids, lr, ls = eids[order], lr[order], ls[order]
    n = nodes.size
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(lr, minlength=n), out=rowptr[1:])
    key = lr * max(n, 1) + ls
    rev = np.searchsorted(key, ls * max(n, 1) + lr)
    return Patch(rowptr, ls, lr, rev, g.efeat[eids].copy(), nodes,
                 hop[nodes], eids)


# --------------------------------------------------------------------------
# parameters: flat float32 buffer, order documented in include/mgn.h
# --------------------------------------------------------------------------
def param_layout(mp_steps, latent=128, node_in=8, edge_in=4, out=4):
    """List of (mlp_name, [(field, shape), ...]) in buffer order.  Weights are
    [out_features, in_features] row-major."""
    D = latent

    def mlp_fields(din, dout, ln):
        f = [("W1", (D, din)), ("b1", (D,)), ("W2", (dout, D)),
             ("b2", (dout,))]
        if ln:
            f += [("gamma", (dout,)), ("beta", (dout,))]
        return f

    lay = [("enc_node", mlp_fields(node_in, D, True)),
           ("enc_edge", mlp_fields(edge_in, D, True))]
    for i in range(mp_steps):
        lay.append((f"block{i}.edge", mlp_fields(3 * D, D, True)))
        lay.append((f"block{i}.node", mlp_fields(2 * D, D, True)))
    lay.append(("dec", mlp_fields(D, out, False)))
    return lay


def n_params(mp_steps, latent=128):
    return sum(int(np.prod(s)) for _, fs in param_layout(mp_steps, latent)
               for _, s in fs)


def unpack_params(flat, mp_steps, latent=128):
    """Views of the flat buffer as fp64 arrays, keyed by MLP then field."""
    flat = np.asarray(flat, dtype=np.float64)
    if flat.shape != (n_params(mp_steps, latent),):
        raise ValueError("parameter buffer has wrong size")
    P, off = {}, 0
    for name, fields in param_layout(mp_steps, latent):
        d = {}
        for f, shape in fields:
            sz = int(np.prod(shape))
            d[f] = flat[off:off + sz].reshape(shape)
            off += sz
        P[name] = d
    return P


def pack_grads(G, mp_steps, latent=128):
    out = []
    for name, fields in param_layout(mp_steps, latent):
        for f, shape in fields:
            out.append(G[name][f].reshape(-1))
    return np.concatenate(out)


def zero_grads(P):
    return {n: {f: np.zeros_like(v) for f, v in d.items()} for n, d in P.items()}


# --------------------------------------------------------------------------
# MLP and LayerNorm (textbook definitions)
# --------------------------------------------------------------------------
def _rows_times(x, W):
    """x W^T computed one row at a time (a vector-matrix product per row), so
    every row's result depends only on that row and never on how many rows
    are multiplied together: a matrix-matrix BLAS call may block the
    products differently for different row counts.  With this, the
    subdomain rows of a patch get bitwise the whole mesh's values (Sec. 2.2,
    condition 1, with ascending local ids and in-segment sums in ascending
    order)."""
    return (x[:, None, :] @ W.T)[:, 0, :]


def mlp(x, p):
    """Two Linear layers with a ReLU between: W2 relu(W1 x + b1) + b2."""
    z1 = _rows_times(x, p["W1"]) + p["b1"]
    a1 = np.maximum(z1, 0.0)
    return _rows_times(a1, p["W2"]) + p["b2"], (x, z1, a1)


def layer_norm(z, gamma, beta, eps=LN_EPS):
    """gamma * (z - mean) / sqrt(var + eps) + beta over the last axis, with
    the biased variance."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mu) * rstd
    return gamma * xhat + beta, (xhat, rstd)


def _mlp_ln(x, p, eps):
    z2, t_mlp = mlp(x, p)
    if "gamma" in p:
        y, t_ln = layer_norm(z2, p["gamma"], p["beta"], eps)
    else:
        y, t_ln = z2, None
    return y, (t_mlp, t_ln)


def _mlp_ln_bwd(tape, ybar, p, g, flip=None):
    """Reverse mode of _mlp_ln; adds parameter gradients into g and returns
    the gradient with respect to the MLP input.  ``flip`` (rows, units)
    selects ReLU inputs at which the other one-sided derivative is taken
    (a different valid subgradient at a kink)."""
    (x, z1, a1), t_ln = tape
    if t_ln is not None:
        xhat, rstd = t_ln
        g["gamma"] += (ybar * xhat).sum(axis=0)
        g["beta"] += ybar.sum(axis=0)
        xhb = ybar * p["gamma"]
        z2bar = rstd * (xhb - xhb.mean(axis=-1, keepdims=True)
                        - xhat * (xhb * xhat).mean(axis=-1, keepdims=True))
    else:
        z2bar = ybar
    g["W2"] += z2bar.T @ a1
    g["b2"] += z2bar.sum(axis=0)
    a1bar = z2bar @ p["W2"]
    mask = z1 > 0.0
    if flip is not None:
        mask = mask.copy()
        mask[flip[0], flip[1]] ^= True
    z1bar = a1bar * mask
    g["W1"] += z1bar.T @ x
    g["b1"] += z1bar.sum(axis=0)
    return z1bar @ p["W1"]


def _incidence(index, n_nodes):
    """Sparse [N, E] matrix with a one at (index[e], e)."""
    E = index.shape[0]
    return sp.csr_matrix((np.ones(E), (index, np.arange(E))),
                         shape=(n_nodes, E))


# --------------------------------------------------------------------------
# a2-a7: one MGN call (Sec. 2.1)
# --------------------------------------------------------------------------
def mgn_forward(g: Graph, params, node_in, efeat, mp_steps, latent=128,
                eps=LN_EPS, keep=False):
    """Encode, ``mp_steps`` message-passing steps, decode.  Returns the
    decoder output [N, 4] (and the tape for mgn_backward when keep)."""
    P = unpack_params(params, mp_steps, latent)
    x_n = np.asarray(node_in, dtype=np.float64)
    x_e = np.asarray(efeat, dtype=np.float64)
    s, r = g.senders, g.receivers
    N = g.n_nodes
    R = _incidence(r, N)
    h, t_enc_n = _mlp_ln(x_n, P["enc_node"], eps)
    e, t_enc_e = _mlp_ln(x_e, P["enc_edge"], eps)
    blocks = []
    for i in range(mp_steps):
        # edge update from the edge and its two incident nodes
        xe = np.concatenate([e, h[s], h[r]], axis=1)
        m, t_e = _mlp_ln(xe, P[f"block{i}.edge"], eps)
        # node update from the sum of its incident (in-)edge messages
        agg = R @ m
        xn = np.concatenate([h, agg], axis=1)
        dh, t_n = _mlp_ln(xn, P[f"block{i}.node"], eps)
        e = e + m
        h = h + dh
        if keep:
            blocks.append((t_e, t_n))
    out, t_dec = mlp(h, P["dec"])
    if not keep:
        return out
    tape = {"P": P, "g": g, "R": R, "mp_steps": mp_steps, "latent": latent,
            "enc_n": t_enc_n, "enc_e": t_enc_e, "blocks": blocks,
            "dec": (t_dec, None)}
    return out, tape


def relu_kinks(tape, tau):
    """ReLU inputs of one saved MGN call with |z| < tau: where an evaluation
    in another precision may take the other branch.  Returns a list of
    (mlp_name, row, unit)."""
    out = []
    named = [("enc_node", tape["enc_n"]), ("enc_edge", tape["enc_e"]), ("dec", tape["dec"])]
    for i, (t_e, t_n) in enumerate(tape["blocks"]):
        named += [(f"block{i}.edge", t_e), (f"block{i}.node", t_n)]
    for name, t in named:
        z1 = t[0][1]
        rows, units = np.nonzero(np.abs(z1) < tau)
        out += [(name, int(r), int(u)) for r, u in zip(rows, units)]
    return out


def _flip_sets(kinks):
    fl = {}
    for name, r, u in kinks or ():
        fl.setdefault(name, ([], []))
        fl[name][0].append(r)
        fl[name][1].append(u)
    return {k: (np.array(v[0]), np.array(v[1])) for k, v in fl.items()}


def mgn_backward(tape, grad_out, flips=None):
    """Reverse mode of mgn_forward.  Returns (flat parameter gradient,
    gradient with respect to node_in).  ``flips``: optional list of
    (mlp_name, row, unit) ReLU inputs at which the other one-sided
    derivative is used (see relu_kinks)."""
    fl = _flip_sets(flips)
    P, g, R = tape["P"], tape["g"], tape["R"]
    m_steps, D = tape["mp_steps"], tape["latent"]
    S = _incidence(g.senders, g.n_nodes)
    G = zero_grads(P)
    ybar = np.asarray(grad_out, dtype=np.float64)
    hbar = _mlp_ln_bwd(tape["dec"], ybar, P["dec"], G["dec"], fl.get("dec"))
    ebar = np.zeros((g.n_edges, D))
    for i in reversed(range(m_steps)):
        t_e, t_n = tape["blocks"][i]
        xnbar = _mlp_ln_bwd(t_n, hbar, P[f"block{i}.node"], G[f"block{i}.node"],
                            fl.get(f"block{i}.node"))
        hbar = hbar + xnbar[:, :D]
        aggbar = xnbar[:, D:]
        mbar = ebar + aggbar[g.receivers]
        xebar = _mlp_ln_bwd(t_e, mbar, P[f"block{i}.edge"], G[f"block{i}.edge"],
                            fl.get(f"block{i}.edge"))
        ebar = ebar + xebar[:, :D]
        hbar = hbar + S @ xebar[:, D:2 * D] + R @ xebar[:, 2 * D:]
    _mlp_ln_bwd(tape["enc_e"], ebar, P["enc_edge"], G["enc_edge"], fl.get("enc_edge"))
    gin = _mlp_ln_bwd(tape["enc_n"], hbar, P["enc_node"], G["enc_node"], fl.get("enc_node"))
    return pack_grads(G, m_steps, D), gin


# --------------------------------------------------------------------------
# a8: explicit integrators, MGN in place of h*f (Sec. 2.3, App. A)
# --------------------------------------------------------------------------
TABLEAUS = {
    # name: (a [s x s] strictly lower, b [s])
    "euler": ([[0.0]], [1.0]),
    "heun2": ([[0.0, 0.0], [1.0, 0.0]], [0.5, 0.5]),
    "midpoint": ([[0.0, 0.0], [0.5, 0.0]], [0.0, 1.0]),
    "heun3": ([[0.0, 0.0, 0.0], [1.0 / 3.0, 0.0, 0.0], [0.0, 2.0 / 3.0, 0.0]],
              [0.25, 0.0, 0.75]),
    "rk4": ([[0.0, 0.0, 0.0, 0.0], [0.5, 0.0, 0.0, 0.0], [0.0, 0.5, 0.0, 0.0],
             [0.0, 0.0, 1.0, 0.0]],
            [1.0 / 6.0, 1.0 / 3.0, 1.0 / 3.0, 1.0 / 6.0]),
    # Ralston's minimum-error-bound methods (named in the paper's outlook,
    # Sec. 5 / App. D): second order c2 = 2/3, third order c = (0, 1/2, 3/4)
    "ralston2": ([[0.0, 0.0], [2.0 / 3.0, 0.0]], [0.25, 0.75]),
    "ralston3": ([[0.0, 0.0, 0.0], [0.5, 0.0, 0.0], [0.0, 0.75, 0.0]],
                 [2.0 / 9.0, 1.0 / 3.0, 4.0 / 9.0]),
}


def integrate_step(g, params, scheme, static, y, efeat, mp_steps, latent=128,
                   keep=False, model=None):
    """One explicit Runge-Kutta step with MGN as the scaled derivative:
    K_i = MGN([static, y + sum_j a_ij K_j]),  y' = y + sum_i b_i K_i.
    ``model`` (tests only) replaces the MGN call by any function of the stage
    state y_i -> K_i."""
    a, b = TABLEAUS[scheme]
    y = np.asarray(y, dtype=np.float64)
    st = np.asarray(static, dtype=np.float64)
    K, tapes = [], []
    for i in range(len(b)):
        yi = y.copy()
        for j in range(i):
            if a[i][j] != 0.0:
                yi = yi + a[i][j] * K[j]
        if model is not None:
            K.append(model(yi))
            continue
        x = np.concatenate([st, yi], axis=1)
        if keep:
            k_i, t = mgn_forward(g, params, x, efeat, mp_steps, latent, keep=True)
            tapes.append(t)
        else:
            k_i = mgn_forward(g, params, x, efeat, mp_steps, latent)
        K.append(k_i)
    y_next = y.copy()
    for i in range(len(b)):
        if b[i] != 0.0:
            y_next = y_next + b[i] * K[i]
    if keep:
        return y_next, (scheme, tapes)
    return y_next


def integrate_backward(tape, grad_y_next, n_static=4):
    """Reverse mode of integrate_step: returns (flat parameter gradient,
    gradient with respect to y)."""
    scheme, tapes = tape
    a, b = TABLEAUS[scheme]
    gy = np.asarray(grad_y_next, dtype=np.float64)
    s = len(b)
    ybar_stage = [None] * s
    gp_total = None
    for i in reversed(range(s)):
        kbar = b[i] * gy
        for j in range(i + 1, s):
            if a[j][i] != 0.0:
                kbar = kbar + a[j][i] * ybar_stage[j]
        gp, gin = mgn_backward(tapes[i], kbar)
        gp_total = gp if gp_total is None else gp_total + gp
        ybar_stage[i] = gin[:, n_static:]
    ybar = gy.copy()
    for i in range(s):
        ybar = ybar + ybar_stage[i]
    return gp_total, ybar


# --------------------------------------------------------------------------
# Predict-evaluate-correct at inference (the paper's outlook: a higher-order
# update for the cost of one MGN evaluation per step).  Reading: two-step
# Adams-Bashforth predictor, trapezoidal (Adams-Moulton) corrector, no
# re-evaluation at the corrected state, MGN in place of h*f:
#   y_p   = y_n + 3/2 K_n - 1/2 K_{n-1}
#   K_p   = MGN([static, y_p])
#   y_n+1 = y_n + 1/2 (K_p + K_n),   then (K_n+1, K_n) = (K_p, K_n).
# The history starts as K_0 = K_-1 = MGN(y_0), so the first step is
# Heun's second-order step.
# --------------------------------------------------------------------------
def pec_step(g, params, static, y, K, K_prev, efeat, mp_steps, latent=128, model=None):
    """One PEC step from y_n with history (K_n, K_n-1); returns
    (y_n+1, K_p), the new history being (K_p, K_n)."""
    y = np.asarray(y, dtype=np.float64)
    yp = y + 1.5 * K - 0.5 * K_prev
    if model is not None:
        Kp = model(yp)
    else:
        Kp = mgn_forward(g, params, np.concatenate([np.asarray(static, np.float64), yp], axis=1), efeat,
                         mp_steps, latent)
    return y + 0.5 * (Kp + K), Kp


def pec_rollout(g, params, static, y0, efeat, mp_steps, n_steps, latent=128, model=None):
    """n_steps PEC steps from y0 (history bootstrapped with MGN(y0));
    returns the list of states y_1 .. y_n."""
    y = np.asarray(y0, dtype=np.float64)
    if model is not None:
        K = model(y)
    else:
        K = mgn_forward(g, params, np.concatenate([np.asarray(static, np.float64), y], axis=1), efeat,
                        mp_steps, latent)
    K_prev = K
    out = []
    for _ in range(n_steps):
        y, Kp = pec_step(g, params, static, y, K, K_prev, efeat, mp_steps, latent, model)
        K_prev, K = K, Kp
        out.append(y)
    return out


# --------------------------------------------------------------------------
# Patch training step (Sec. 2.2 conditions 2 and 3; App. C: input noise,
# Adam, learning rate decaying exponentially from 1e-3 to 1e-7 over 4e6
# steps).  Readings: the noisy input is y + std * n with n standard normal
# and std = (0.02, 0.02, 0.03, 0.05) for (x, y momentum, vertical momentum,
# volume fraction), the target state is not perturbed; the loss is the mean
# squared error of the stepped state over the subdomain nodes of the sampled
# patches (normalised by 4 x their count); Adam with beta = (0.9, 0.999),
# eps = 1e-8; the k-th update (k = 1, 2, ...) uses lr(k - 1) with
# lr(t) = lr_start (lr_end / lr_start)^(t / decay_steps).
# --------------------------------------------------------------------------
NOISE_STD_3D = (0.02, 0.02, 0.03, 0.05)


def lr_schedule(t, lr_start=1e-3, lr_end=1e-7, decay_steps=4_000_000):
    return lr_start * (lr_end / lr_start) ** (float(t) / float(decay_steps))


def adam_update(p, g, m, v, k, lr, beta1=0.9, beta2=0.999, eps=1e-8):
    """The k-th Adam update (k >= 1) of p with gradient g; returns (p, m, v)."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mh = m / (1.0 - beta1 ** k)
    vh = v / (1.0 - beta2 ** k)
    return p - lr * mh / (np.sqrt(vh) + eps), m, v


def masked_mse(out, target, interior, n_norm=None):
    """mean((out - target)^2) over the subdomain nodes; n_norm nodes in the
    normaliser (default: the interior count)."""
    out = np.asarray(out, dtype=np.float64)
    mask = np.asarray(interior, dtype=np.float64)[:, None]
    n = float(mask.sum()) if n_norm is None else float(n_norm)
    return float((((out - np.asarray(target, np.float64)) ** 2) * mask).sum() / max(1.0, n * out.shape[1]))


def train_step(patches, params, scheme, static, y, y_target, noise, mp_steps, adam_m, adam_v, k,
               noise_std=NOISE_STD_3D, n_loss_nodes=None, latent=128):
    """One patch-training step: noisy input, one integration step per patch,
    masked MSE over the patches' subdomain nodes, gradients summed over the
    patches (condition 3), one Adam update.  patches: list of Patch.
    Returns (params, adam_m, adam_v, loss, grad)."""
    y_noisy = np.asarray(y, np.float64) + np.asarray(noise, np.float64) * np.asarray(noise_std, np.float64)
    if n_loss_nodes is None:
        n_loss_nodes = sum(int(pt.n_interior) for pt in patches)
    grad = np.zeros(np.asarray(params).size, dtype=np.float64)
    loss = 0.0
    for pt in patches:
        l2g = pt.node_l2g
        yn, tape = integrate_step(pt, params, scheme, np.asarray(static)[l2g], y_noisy[l2g], pt.efeat, mp_steps,
                                  latent, keep=True)
        it = pt.interior
        tgt = np.asarray(y_target, np.float64)[l2g]
        loss += masked_mse(yn, tgt, it, n_loss_nodes)
        gout = masked_mse_grad(yn, tgt, it) * (float(it.sum()) / float(n_loss_nodes))
        gp, _ = integrate_backward(tape, gout)
        grad += gp
    p2, m2, v2 = adam_update(np.asarray(params, np.float64), grad, adam_m, adam_v, k, lr_schedule(k - 1))
    return p2, m2, v2, loss, grad


def masked_mse_grad(out, target, interior):
    """Gradient of mean((out - target)^2) over the subdomain (interior) nodes
    only (condition 2 of Sec. 2.2)."""
    out = np.asarray(out, dtype=np.float64)
    mask = np.asarray(interior, dtype=np.float64)[:, None]
    n = max(1.0, float(mask.sum()) * out.shape[1])
    return 2.0 * (out - np.asarray(target, np.float64)) * mask / n
