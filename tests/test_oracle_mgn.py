"""Pins for the oracle's MGN forward/backward and integrators.

* MLP/LayerNorm against torch's textbook implementations (fp64).
* A dense brute force of the whole MGN call written with one-hot incidence
  matrices in torch (no index gathers, no sparse sums), and its autograd
  gradients against the oracle's hand-written reverse mode.
* fp64 central finite differences.
* Permutation equivariance, locality (m-hop receptive field, Sec. 2.1), the
  in-degree special case of the aggregation.
* Patch equivalence conditions (1)-(3) of Sec. 2.2.
* Integrators: the paper's H2 formula (App. A, equation heun), Taylor
  closed forms with a linear stand-in, and observed local-error orders
  (Sec. 2.3, equation FE_HUEN).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_facts.json")


def small(shape=(5, 4), m=2, seed=0, randomize=True, latent=128):
    M = synth.mesh(shape, seed)
    g = O.build_graph(M["cells"], M["pos"])
    P = synth.xavier_params(m, seed, latent=latent, randomize_norm=randomize)
    return M, g, P


# ---------------------------------------------------------------- MLP / LN
def test_mlp_ln_vs_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((7, 12))
    p = {"W1": rng.standard_normal((16, 12)), "b1": rng.standard_normal(16),
         "W2": rng.standard_normal((5, 16)), "b2": rng.standard_normal(5),
         "gamma": rng.standard_normal(5), "beta": rng.standard_normal(5)}
    y, _ = O.mlp(x, p)
    T = {k: torch.tensor(v) for k, v in p.items()}
    ref = torch.nn.functional.linear(
        torch.relu(torch.nn.functional.linear(torch.tensor(x), T["W1"], T["b1"])),
        T["W2"], T["b2"])
    assert np.allclose(y, ref.numpy(), rtol=1e-13, atol=1e-13)
    ln, _ = O.layer_norm(y, p["gamma"], p["beta"])
    ref_ln = torch.nn.functional.layer_norm(ref, (5,), T["gamma"], T["beta"], 1e-5)
    assert np.allclose(ln, ref_ln.numpy(), rtol=1e-12, atol=1e-12)


def test_layer_norm_constant_gives_beta():
    beta = np.linspace(-1, 1, 128)
    gamma = np.full(128, 3.0)
    y, _ = O.layer_norm(np.full((3, 128), 7.25), gamma, beta)
    assert np.array_equal(y, np.broadcast_to(beta, (3, 128)))
    z = np.random.default_rng(1).standard_normal((4, 128)) * 5
    y, _ = O.layer_norm(z, np.ones(128), np.zeros(128))
    var = z.var(axis=1)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-13)
    assert np.allclose(y.var(axis=1), var / (var + 1e-5), rtol=1e-12)


# ----------------------------------------------- dense brute force (torch)
def dense_mgn(g, P, node_in, efeat, m, D=128):
    """Whole MGN call with dense one-hot incidence matrices (torch fp64)."""
    N, E = g.n_nodes, g.n_edges
    S = torch.zeros(E, N, dtype=torch.float64)
    S[torch.arange(E), torch.tensor(g.senders)] = 1.0
    R = torch.zeros(E, N, dtype=torch.float64)
    R[torch.arange(E), torch.tensor(g.receivers)] = 1.0
    F = torch.nn.functional
    off = [0]
    flat = P

    def take(*shape):
        n = int(np.prod(shape))
        v = flat[off[0]:off[0] + n].reshape(shape)
        off[0] += n
        return v

    def block(din, dout, ln):
        W1, b1, W2, b2 = take(D, din), take(D), take(dout, D), take(dout)
        gb = (take(dout), take(dout)) if ln else None

        def f(x):
            y = F.linear(F.relu(F.linear(x, W1, b1)), W2, b2)
            return F.layer_norm(y, (dout,), gb[0], gb[1], 1e-5) if ln else y
        return f

    enc_n, enc_e = block(8, D, True), block(4, D, True)
    blocks = [(block(3 * D, D, True), block(2 * D, D, True)) for _ in range(m)]
    dec = block(D, 4, False)
    h = enc_n(node_in)
    e = enc_e(efeat)
    for fe, fn in blocks:
        msg = fe(torch.cat([e, S @ h, R @ h], dim=1))
        agg = R.T @ msg
        h, e = h + fn(torch.cat([h, agg], dim=1)), e + msg
    return dec(h)


@pytest.mark.parametrize("shape,m", [((4, 3), 1), ((5, 4), 2), ((3, 3, 3), 2)])
def test_dense_brute_force_forward_and_autograd(shape, m):
    M, g, P = small(shape, m, seed=3)
    w = synth.loss_weights(g.n_nodes, 3)
    out, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, m, keep=True)
    gp, gin = O.mgn_backward(tape, w)
    Pt = torch.tensor(P.astype(np.float64), requires_grad=True)
    xt = torch.tensor(M["node_in"].astype(np.float64), requires_grad=True)
    ref = dense_mgn(g, Pt, xt, torch.tensor(g.efeat.astype(np.float64)), m)
    assert np.allclose(out, ref.detach().numpy(), rtol=1e-11, atol=1e-11)
    (ref * torch.tensor(w.astype(np.float64))).sum().backward()
    assert np.allclose(gp, Pt.grad.numpy(), rtol=1e-9, atol=1e-9)
    assert np.allclose(gin, xt.grad.numpy(), rtol=1e-9, atol=1e-9)


def test_dense_brute_force_latent150():
    """The 3D model's width (App. C: latent 150, 3 MP steps): the oracle at
    latent 150 against the dense torch MGN of that width, outputs and
    autograd gradients."""
    m, D = 3, 150
    M, g, P = small((3, 3, 2), m, seed=9, latent=D)
    assert P.size == O.n_params(m, D)
    w = synth.loss_weights(g.n_nodes, 9)
    out, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, m, latent=D, keep=True)
    gp, gin = O.mgn_backward(tape, w)
    Pt = torch.tensor(P.astype(np.float64), requires_grad=True)
    xt = torch.tensor(M["node_in"].astype(np.float64), requires_grad=True)
    ref = dense_mgn(g, Pt, xt, torch.tensor(g.efeat.astype(np.float64)), m, D=D)
    assert np.allclose(out, ref.detach().numpy(), rtol=1e-11, atol=1e-11)
    (ref * torch.tensor(w.astype(np.float64))).sum().backward()
    assert np.allclose(gp, Pt.grad.numpy(), rtol=1e-9, atol=1e-9)
    assert np.allclose(gin, xt.grad.numpy(), rtol=1e-9, atol=1e-9)


def test_finite_differences():
    m = 2
    M, g, P = small((4, 4), m, seed=5)
    P = P.astype(np.float64)
    w = synth.loss_weights(g.n_nodes, 5).astype(np.float64)
    x = M["node_in"].astype(np.float64)

    def loss(Pv, xv):
        return float((O.mgn_forward(g, Pv, xv, g.efeat, m) * w).sum())

    _, tape = O.mgn_forward(g, P, x, g.efeat, m, keep=True)
    gp, gin = O.mgn_backward(tape, w)
    rng = np.random.default_rng(9)
    idx = rng.choice(P.size, 24, replace=False)
    h = 1e-6
    for i in idx:
        Pp, Pm = P.copy(), P.copy()
        Pp[i] += h
        Pm[i] -= h
        fd = (loss(Pp, x) - loss(Pm, x)) / (2 * h)
        assert abs(fd - gp[i]) <= 1e-6 * max(1.0, abs(gp[i])), (i, fd, gp[i])
    for (v, c) in [(0, 4), (5, 6), (11, 7), (15, 5)]:
        xp, xm = x.copy(), x.copy()
        xp[v, c] += h
        xm[v, c] -= h
        fd = (loss(P, xp) - loss(P, xm)) / (2 * h)
        assert abs(fd - gin[v, c]) <= 1e-6 * max(1.0, abs(gin[v, c]))


def test_backward_linear_in_grad_out():
    M, g, P = small((4, 3), 1, seed=2)
    _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, 1, keep=True)
    w1 = synth.loss_weights(g.n_nodes, 1).astype(np.float64)
    w2 = synth.loss_weights(g.n_nodes, 2).astype(np.float64)
    a, _ = O.mgn_backward(tape, w1)
    b, _ = O.mgn_backward(tape, w2)
    c, _ = O.mgn_backward(tape, 2.0 * w1 - 3.0 * w2)
    assert np.allclose(c, 2 * a - 3 * b, rtol=1e-10, atol=1e-10)


# ----------------------------------------------------- structural pins
def test_aggregate_is_in_degree():
    """Edge MLP weights zero and LayerNorm offset one: every message is the
    all-ones vector, so the aggregate of a node is its in-degree."""
    m = 1
    M, g, P = small((5, 4, 3), m, seed=1)
    Pd = O.unpack_params(P, m)
    P64 = P.astype(np.float64).copy()
    off = 0
    for name, fields in O.param_layout(m):
        for f, shape in fields:
            n = int(np.prod(shape))
            if name == "block0.edge":
                if f in ("W1", "W2", "b1", "b2"):
                    P64[off:off + n] = 0.0
                if f == "beta":
                    P64[off:off + n] = 1.0
            off += n
    del Pd
    _, tape = O.mgn_forward(g, P64, M["node_in"], g.efeat, m, keep=True)
    (x_mlp, _, _), _ = tape["blocks"][0][1]
    agg = x_mlp[:, 128:]
    deg = np.diff(g.rowptr).astype(np.float64)
    assert np.array_equal(agg, np.repeat(deg[:, None], 128, axis=1))


def test_permutation_equivariance():
    m = 2
    shape = (5, 4, 3)
    M, g, P = small(shape, m, seed=4)
    out = O.mgn_forward(g, P, M["node_in"], g.efeat, m)
    perm = synth.relabel(g.n_nodes, 4)  # new id of old node i
    pos2 = np.empty_like(M["pos"])
    pos2[perm] = M["pos"]
    x2 = np.empty_like(M["node_in"])
    x2[perm] = M["node_in"]
    g2 = O.build_graph(perm[M["cells"]], pos2)
    out2 = O.mgn_forward(g2, P, x2, g2.efeat, m)
    assert np.allclose(out2[perm], out, rtol=1e-11, atol=1e-11)


def test_locality_receptive_field():
    """After m steps a node sees exactly its m-hop neighbourhood (Sec. 2.1)."""
    m = 2
    M, g, P = small((9, 3), m, seed=6)
    x = M["node_in"].astype(np.float64)
    out = O.mgn_forward(g, P, x, g.efeat, m)
    src = np.zeros(g.n_nodes, bool)
    src[0] = True
    hop = O.hop_distance(g, src, g.n_nodes)
    x2 = x.copy()
    x2[0, 4:] += 0.5
    out2 = O.mgn_forward(g, P, x2, g.efeat, m)
    far = hop > m
    assert far.any()
    assert np.array_equal(out2[far], out[far])
    near = (hop >= 0) & (hop <= m)
    assert np.all(np.abs(out2[near] - out[near]).max(axis=1) > 0)


# --------------------------------------------------- patch equivalence
def _patch_inputs(M, pt):
    return M["node_in"][pt.node_l2g]


def test_mlp_row_results_independent_of_row_count():
    """The oracle's MLP gives a row bitwise the same result whatever rows are
    multiplied with it, which the bitwise condition-1 pin below relies on
    (a matrix-matrix BLAS product need not)."""
    rng = np.random.default_rng(3)
    p = {"W1": rng.standard_normal((128, 384)), "b1": rng.standard_normal(128),
         "W2": rng.standard_normal((128, 128)), "b2": rng.standard_normal(128)}
    x = rng.standard_normal((5000, 384))
    full, _ = O.mlp(x, p)
    for lo, hi in ((0, 1), (7, 29), (1000, 1333), (4990, 5000)):
        part, _ = O.mlp(x[lo:hi].copy(), p)
        assert np.array_equal(part, full[lo:hi])


@pytest.mark.parametrize("shape,splits,m,k", [((9, 8), (3, 2), 2, 2),
                                              ((5, 5, 6), (1, 1, 3), 2, 3)])
def test_condition1_interior_outputs_bitwise(shape, splits, m, k):
    M, g, P = small(shape, m, seed=7)
    out = O.mgn_forward(g, P, M["node_in"], g.efeat, m)
    part = O.partition(M["pos"], splits)
    for p in range(int(part.max()) + 1):
        pt = O.extract_patch(g, part, p, k)
        if pt.n_nodes == 0:
            continue
        o = O.mgn_forward(pt, P, _patch_inputs(M, pt), pt.efeat, m)
        it = pt.hop == 0
        assert np.array_equal(o[it], out[pt.node_l2g[it]])


def test_condition1_violated_differs():
    m = 3
    M, g, P = small((10, 6), m, seed=8)
    out = O.mgn_forward(g, P, M["node_in"], g.efeat, m)
    part = O.partition(M["pos"], (2, 1))
    pt = O.extract_patch(g, part, 0, 1)  # k = 1 < m
    o = O.mgn_forward(pt, P, _patch_inputs(M, pt), pt.efeat, m)
    it = pt.hop == 0
    assert not np.allclose(o[it], out[pt.node_l2g[it]], rtol=1e-6, atol=1e-6)


def test_conditions_2_3_gradient_accumulation():
    """Summing, over all patches, gradients of the loss on subdomain nodes
    equals the whole-mesh gradient (Sec. 2.2 conditions 2 and 3)."""
    m = 2
    M, g, P = small((8, 7), m, seed=9)
    w = synth.loss_weights(g.n_nodes, 9)
    _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, m, keep=True)
    gw, _ = O.mgn_backward(tape, w)
    part = O.partition(M["pos"], (2, 2))
    acc = np.zeros_like(gw)
    for p in range(4):
        pt = O.extract_patch(g, part, p, m)
        _, t = O.mgn_forward(pt, P, _patch_inputs(M, pt), pt.efeat, m, keep=True)
        wp = w[pt.node_l2g] * (pt.hop == 0)[:, None]
        gp, _ = O.mgn_backward(t, wp)
        acc += gp
    assert np.allclose(acc, gw, rtol=1e-10, atol=1e-10 * np.abs(gw).max())


# --------------------------------------------------------- integrators
def test_heun2_matches_paper_formula():
    """App. A, equation heun: y + 1/2 (MGN(y) + MGN(y + MGN(y)))."""
    m = 1
    M, g, P = small((4, 4), m, seed=10)
    st, y = M["onehot"].astype(np.float64), M["states"].astype(np.float64)

    def mgn(v):
        return O.mgn_forward(g, P, np.concatenate([st, v], 1), g.efeat, m)
    ref = y + 0.5 * (mgn(y) + mgn(y + mgn(y)))
    got = O.integrate_step(g, P, "heun2", st, y, g.efeat, m)
    assert np.allclose(got, ref, rtol=1e-14, atol=1e-14)
    fe = O.integrate_step(g, P, "euler", st, y, g.efeat, m)
    assert np.array_equal(fe, y + mgn(y))


@pytest.mark.parametrize("scheme,order", [("euler", 1), ("heun2", 2),
                                          ("midpoint", 2), ("heun3", 3),
                                          ("rk4", 4), ("ralston2", 2), ("ralston3", 3)])
def test_linear_standin_taylor(scheme, order):
    """With K(y) = y A the step is the Taylor polynomial sum_j y A^j / j!
    up to the method's order."""
    rng = np.random.default_rng(11)
    A = rng.standard_normal((4, 4)) * 0.3
    y = rng.standard_normal((6, 4))
    got = O.integrate_step(None, None, scheme, np.zeros((6, 4)), y, None, 0,
                           model=lambda v: v @ A)
    ref, term = y.copy(), y.copy()
    for j in range(1, order + 1):
        term = term @ A / j
        ref = ref + term
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("scheme", ["euler", "heun2", "heun3", "rk4", "midpoint", "ralston2", "ralston3"])
def test_observed_local_error_order(scheme):
    """y' = -y^2 (exact y(t) = y0/(1+y0 t)): halving h divides the one-step
    error by 2^(p+1).  Paper: FE O(h^2), H2 O(h^3), H3 O(h^4)."""
    facts = json.load(open(GOLD))
    p_expect = {"euler": 2, "heun2": 3, "midpoint": 3, "heun3": 4, "rk4": 5, "ralston2": 3, "ralston3": 4}[scheme]
    if scheme in facts["local_error_order"]:
        assert facts["local_error_order"][scheme] == p_expect
    y0 = np.array([[0.7, 1.1, 0.3, 1.5]])
    errs = []
    for h in (0.02, 0.01, 0.005):
        got = O.integrate_step(None, None, scheme, np.zeros_like(y0), y0, None, 0,
                               model=lambda v, h=h: -h * v * v)
        errs.append(np.abs(got - y0 / (1 + y0 * h)).max())
    orders = np.log2(np.array(errs[:-1]) / np.array(errs[1:]))
    assert np.all(np.abs(orders - p_expect) < 0.25), orders


def test_linear_standin_taylor_is_not_exceeded():
    """A wrong Ralston coefficient shows up one order higher: the methods
    match the Taylor polynomial to their order but not beyond (the next
    term differs), so the order pins above are tight."""
    rng = np.random.default_rng(12)
    A = rng.standard_normal((4, 4)) * 0.3
    y = rng.standard_normal((6, 4))
    for scheme, order in (("ralston2", 2), ("ralston3", 3)):
        got = O.integrate_step(None, None, scheme, np.zeros((6, 4)), y, None, 0, model=lambda v: v @ A)
        ref, term = y.copy(), y.copy()
        for j in range(1, order + 2):
            term = term @ A / j
            ref = ref + term
        assert not np.allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_pec_first_step_is_heun2_and_one_evaluation_per_step():
    """PEC bootstraps with K_-1 = K_0, so its first step is Heun's step; each
    later step calls the model once."""
    calls = []

    def model(v):
        calls.append(1)
        return -0.1 * v * v
    y0 = np.array([[0.7, 1.1, 0.3, 1.5]])
    ys = O.pec_rollout(None, None, np.zeros_like(y0), y0, None, 0, 4, model=model)
    h2 = O.integrate_step(None, None, "heun2", np.zeros_like(y0), y0, None, 0, model=lambda v: -0.1 * v * v)
    assert np.allclose(ys[0], h2, rtol=1e-15, atol=1e-15)
    assert len(calls) == 1 + 4


def test_pec_first_step_closed_form():
    """With K(y) = y A the bootstrap step is y0 (I + A + A^2/2), the
    second-order Taylor polynomial, and the new history value is the
    predicted derivative y0 (A + A^2)."""
    rng = np.random.default_rng(13)
    A = rng.standard_normal((4, 4)) * 0.2
    y0 = rng.standard_normal((3, 4))
    y1, Kp = O.pec_step(None, None, np.zeros_like(y0), y0, y0 @ A, y0 @ A, None, 0, model=lambda v: v @ A)
    I = np.eye(4)
    assert np.allclose(y1, y0 @ (I + A + A @ A / 2), rtol=1e-14, atol=1e-14)
    assert np.allclose(Kp, y0 @ (A + A @ A), rtol=1e-14, atol=1e-14)


def test_pec_error_approaches_trapezoidal_rule():
    """The corrector is the trapezoidal rule; with the two-step
    Adams-Bashforth predictor the predictor's (and the unevaluated
    corrected state's) contribution to the global error is one order higher,
    so PEC's error approaches that of the implicit trapezoidal rule (solved
    here to convergence by fixed-point iteration) as h -> 0.  A first-order
    predictor would leave an O(h^2) difference."""
    y0 = np.array([[0.7, 1.1, 0.3, 1.5]])
    exact = y0 / (1 + y0)
    ratios = []
    for n in (40, 80, 160):
        h = 1.0 / n
        ys = O.pec_rollout(None, None, np.zeros_like(y0), y0, None, 0, n, model=lambda v, h=h: -h * v * v)
        y = y0.copy()
        for _ in range(n):
            z = y.copy()
            for _ in range(200):
                z = y + 0.5 * h * (-y * y - z * z)
            y = z
        ratios.append(np.abs(ys[-1] - exact).max() / np.abs(y - exact).max())
    assert abs(ratios[-1] - 1.0) < 0.03, ratios
    assert abs(ratios[-1] - 1.0) < abs(ratios[0] - 1.0), ratios


def test_pec_observed_global_order():
    """AB2 predictor + trapezoidal corrector is a second-order method: on
    y' = -y^2 over t in [0, 1] the global error falls by 2^2 per halving of h."""
    y0 = np.array([[0.7, 1.1, 0.3, 1.5]])
    errs = []
    for n in (20, 40, 80):
        h = 1.0 / n
        ys = O.pec_rollout(None, None, np.zeros_like(y0), y0, None, 0, n, model=lambda v, h=h: -h * v * v)
        errs.append(np.abs(ys[-1] - y0 / (1 + y0)).max())
    orders = np.log2(np.array(errs[:-1]) / np.array(errs[1:]))
    assert np.all(np.abs(orders - 2.0) < 0.2), orders


def test_integrator_backward_fd():
    m = 1
    M, g, P = small((4, 3), m, seed=12)
    st, y = M["onehot"].astype(np.float64), M["states"].astype(np.float64)
    w = synth.loss_weights(g.n_nodes, 12).astype(np.float64)
    for scheme in ("heun2", "rk4", "heun3"):
        yn, tape = O.integrate_step(g, P, scheme, st, y, g.efeat, m, keep=True)
        gp, gy = O.integrate_backward(tape, w)

        def L(Pv, yv):
            return float((O.integrate_step(g, Pv, scheme, st, yv, g.efeat, m) * w).sum())
        h = 1e-6
        for (v, c) in [(0, 0), (3, 2), (7, 3)]:
            yp, ym = y.copy(), y.copy()
            yp[v, c] += h
            ym[v, c] -= h
            fd = (L(P, yp) - L(P, ym)) / (2 * h)
            assert abs(fd - gy[v, c]) <= 1e-6 * max(1, abs(fd))
        P64 = P.astype(np.float64)
        for i in (5, 20000, 60000, P.size - 3):
            Pp, Pm = P64.copy(), P64.copy()
            Pp[i] += h
            Pm[i] -= h
            fd = (L(Pp, y) - L(Pm, y)) / (2 * h)
            assert abs(fd - gp[i]) <= 1e-6 * max(1, abs(fd))


def test_param_layout_matches_generator():
    """The oracle's unpacking order agrees with the generator's field list and
    the documented total (1,788,036 floats at 15 steps, latent 128)."""
    assert O.n_params(15) == 1788036
    names = [(f"{n}.{f}", s) for n, fs in O.param_layout(15) for f, s in fs]
    gen = [(n, s) for n, _, s in synth.param_shapes(15)]
    assert names == gen


def test_masked_mse_grad():
    out = np.array([[1.0, 2, 3, 4], [0, 0, 0, 0]])
    tgt = np.zeros((2, 4))
    gr = O.masked_mse_grad(out, tgt, np.array([1, 0]))
    assert np.allclose(gr[0], 2 * out[0] / 4) and np.all(gr[1] == 0)


# --------------------------------------------------------- training step
def test_lr_schedule_and_noise_match_paper():
    """App. C: exponential decay 1e-3 -> 1e-7 over 4e6 steps (so 1e-5, the
    geometric mean, half way) and the per-channel input noise."""
    f = json.load(open(GOLD))
    lr = lambda t: O.lr_schedule(t, f["lr_start"], f["lr_end"], f["lr_decay_steps"])
    assert abs(lr(0) - 1e-3) < 1e-18 and abs(lr(4_000_000) / 1e-7 - 1) < 1e-12
    assert abs(lr(2_000_000) / 1e-5 - 1) < 1e-12
    assert abs(O.lr_schedule(4_000_000) / f["lr_end"] - 1) < 1e-12
    assert list(O.NOISE_STD_3D) == f["noise_std_3d"]


def test_adam_matches_torch():
    """Three updates of the oracle's Adam against torch.optim.Adam (fp64),
    with the scheduled learning rate set before every update."""
    rng = np.random.default_rng(21)
    p0 = rng.standard_normal(50)
    grads = [rng.standard_normal(50) * s for s in (1.0, 0.1, 3.0)]
    tp = torch.tensor(p0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([tp], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    p, m, v = p0.copy(), np.zeros(50), np.zeros(50)
    for k, g in enumerate(grads, start=1):
        lr = O.lr_schedule(k - 1, 1e-3, 1e-7, 10)  # a fast schedule, so the rate changes
        for grp in opt.param_groups:
            grp["lr"] = lr
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = O.adam_update(p, g, m, v, k, lr)
    st = opt.state[tp]
    assert np.allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)
    assert np.allclose(m, st["exp_avg"].numpy(), rtol=1e-13) and np.allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13)


def test_masked_mse_matches_torch_and_fd():
    rng = np.random.default_rng(22)
    out, tgt = rng.standard_normal((9, 4)), rng.standard_normal((9, 4))
    it = (rng.random(9) < 0.6).astype(np.uint8)
    ref = torch.nn.functional.mse_loss(torch.tensor(out[it == 1]), torch.tensor(tgt[it == 1])).item()
    assert abs(O.masked_mse(out, tgt, it) - ref) < 1e-14
    g = O.masked_mse_grad(out, tgt, it)
    h = 1e-6
    for (r, c) in [(0, 0), (4, 2), (8, 3), (int(np.argmin(it)), 1)]:
        op, om = out.copy(), out.copy()
        op[r, c] += h
        om[r, c] -= h
        fd = (O.masked_mse(op, tgt, it) - O.masked_mse(om, tgt, it)) / (2 * h)
        assert abs(fd - g[r, c]) < 1e-8


def _train_problem(shape, m, seed, k, splits):
    M, g, P = small(shape, m, seed=seed)
    st = M["onehot"].astype(np.float64)
    y = M["states"].astype(np.float64)
    tgt = synth.next_states(M["states"], seed).astype(np.float64)
    nz = synth.standard_noise(g.n_nodes, seed).astype(np.float64)
    part = O.partition(M["pos"], splits)
    pts = [O.extract_patch(g, part, p, k) for p in range(int(np.prod(splits)))]
    return M, g, P, st, y, tgt, nz, pts


def test_train_step_patches_equal_whole_mesh():
    """Conditions 2 and 3 through the integrator and the noisy input: the
    step over all patches (k = s m) has the whole-mesh loss, gradient and
    update; the whole mesh is the single patch of a one-part partition."""
    m = 1
    M, g, P, st, y, tgt, nz, pts = _train_problem((6, 5), m, 23, 2, (2, 2))
    whole = O.extract_patch(g, np.zeros(g.n_nodes, np.int32), 0, 0)
    z = np.zeros(P.size)
    a = O.train_step(pts, P, "heun2", st, y, tgt, nz, m, z, z, 1)
    b = O.train_step([whole], P, "heun2", st, y, tgt, nz, m, z, z, 1)
    assert abs(a[3] - b[3]) < 1e-12 * abs(b[3])
    assert np.allclose(a[4], b[4], rtol=1e-10, atol=1e-12 * np.abs(b[4]).max())
    assert np.allclose(a[0], b[0], rtol=1e-12, atol=1e-12)


def test_train_step_gradient_fd():
    """The summed gradient is the derivative of the loss (fp64 central
    differences), and the update is Adam's first step with lr(0) = 1e-3."""
    m = 1
    M, g, P, st, y, tgt, nz, pts = _train_problem((5, 4), m, 24, 2, (2, 1))
    z = np.zeros(P.size)
    p1, m1, v1, loss, grad = O.train_step(pts, P, "euler", st, y, tgt, nz, m, z, z, 1)

    def L(Pv):
        return O.train_step(pts, Pv, "euler", st, y, tgt, nz, m, z, z, 1)[3]
    P64, h = P.astype(np.float64), 1e-6
    for i in (7, 3000, 20000, P.size - 2):
        Pp, Pm = P64.copy(), P64.copy()
        Pp[i] += h
        Pm[i] -= h
        fd = (L(Pp) - L(Pm)) / (2 * h)
        assert abs(fd - grad[i]) <= 1e-6 * max(1e-3, abs(fd))
    # first update: lr g / (|g| + eps), within 1e-4 of lr sign(g) where |g| > 1e-4
    nzg = np.abs(grad) > 1e-4
    assert np.allclose((P64 - p1)[nzg], 1e-3 * np.sign(grad[nzg]), rtol=1e-3)


def test_subgradient_flip_matches_autograd():
    """oracle.mgn_backward(flips=...) takes the other one-sided derivative at
    the listed ReLU inputs: compare with autograd on the dense brute force
    where those units' derivative is changed without changing values."""
    m = 1
    M, g, P = small((4, 3), m, seed=13)
    w = synth.loss_weights(g.n_nodes, 13).astype(np.float64)
    _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, m, keep=True)
    z1 = tape["blocks"][0][0][0][1]
    # one inactive and one active unit of the edge MLP, one of the decoder
    r0, u0 = np.argwhere(z1 < 0)[3]
    r1, u1 = np.argwhere(z1 > 0)[5]
    zd = tape["dec"][0][1]
    r2, u2 = np.argwhere(zd > 0)[2]
    flips = [("block0.edge", int(r0), int(u0)), ("block0.edge", int(r1), int(u1)),
             ("dec", int(r2), int(u2))]
    gp, gin = O.mgn_backward(tape, w, flips=flips)
    assert O.relu_kinks(tape, 0.0) == []
    assert len(O.relu_kinks(tape, np.inf)) > 0

    F = torch.nn.functional
    orig_relu = F.relu
    calls = {"n": 0}

    def relu_with_flips(z):
        # call order in dense_mgn: enc_n, enc_e, block0.edge, block0.node, dec
        k = calls["n"]
        calls["n"] += 1
        y = orig_relu(z)
        sel = torch.zeros_like(z)
        if k == 2:
            sel[r0, u0] = 1.0
            sel[r1, u1] = -1.0
        if k == 4:
            sel[r2, u2] = -1.0
        return y + sel * (z - z.detach())

    Pt = torch.tensor(P.astype(np.float64), requires_grad=True)
    xt = torch.tensor(M["node_in"].astype(np.float64), requires_grad=True)
    F.relu = relu_with_flips
    try:
        ref = dense_mgn(g, Pt, xt, torch.tensor(g.efeat.astype(np.float64)), m)
    finally:
        F.relu = orig_relu
    (ref * torch.tensor(w)).sum().backward()
    assert np.allclose(gp, Pt.grad.numpy(), rtol=1e-9, atol=1e-9)
    assert np.allclose(gin, xt.grad.numpy(), rtol=1e-9, atol=1e-9)
    g0, _ = O.mgn_backward(tape, w)
    assert not np.allclose(g0, gp)


def test_bf16_gradient_conditioning():
    """Why bf16 gradients get a looser bound than bf16 outputs: even in fp64,
    a 2^-9 relative perturbation of the weights (one bf16 rounding) moves
    the gradient by several percent because ReLU inputs near their kink
    switch branch, while the outputs move by well under 1%."""
    m = 2
    M, g, P = small((32, 32), m, seed=11)
    w = synth.loss_weights(g.n_nodes, 11)
    P = P.astype(np.float64)
    o0, t0 = O.mgn_forward(g, P, M["node_in"], g.efeat, m, keep=True)
    g0, _ = O.mgn_backward(t0, w)
    P1 = P * (1 + np.random.default_rng(0).uniform(-2.0 ** -9, 2.0 ** -9, P.shape))
    o1, t1 = O.mgn_forward(g, P1, M["node_in"], g.efeat, m, keep=True)
    g1, _ = O.mgn_backward(t1, w)
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    assert rel(o1, o0) < 1e-2
    assert rel(g1, g0) > 3e-2
    # with every ReLU far from its kink the same perturbation moves the
    # gradient by about as much as the outputs
    S = synth.smooth_params(m, 11).astype(np.float64)
    s0, ts0 = O.mgn_forward(g, S, M["node_in"], g.efeat, m, keep=True)
    assert O.relu_kinks(ts0, 1e-2) == []
    gs0, _ = O.mgn_backward(ts0, w)
    S1 = S * (1 + np.random.default_rng(0).uniform(-2.0 ** -9, 2.0 ** -9, S.shape))
    s1, ts1 = O.mgn_forward(g, S1, M["node_in"], g.efeat, m, keep=True)
    gs1, _ = O.mgn_backward(ts1, w)
    assert rel(gs1, gs0) < 2e-2


def test_ball_output_equals_whole_mesh():
    """The full-size GPU tests read oracle outputs at single nodes from the
    m-hop ball inside a grid box (tests/fullsize_util.py): on a small mesh
    that equals the whole-mesh oracle output at a corner, a face and an
    interior point, up to fp64 rounding (the BLAS products of the MLPs may
    block rows differently for different matrix sizes)."""
    from fullsize_util import oracle_node_output, node_id
    shape, m = (11, 10, 12), 3
    M = synth.mesh(shape, 4)
    g = O.build_graph(M["cells"], M["pos"])
    P = synth.xavier_params(m, 4, randomize_norm=True)
    whole = O.mgn_forward(g, P, M["node_in"], g.efeat, m)
    for c in [(0, 0, 0), (5, 0, 7), (5, 4, 6), (10, 9, 11)]:
        got = oracle_node_output(M, shape, c, P, m)
        w = whole[node_id(shape, c)]
        assert np.max(np.abs(got - w) / np.abs(w)) < 1e-12, c
