"""GPU parity at the 3D model's shape (App. C: latent width 150, 3 MP steps;
Sec. 2.3: Heun's second-order step): fp32 and bf16, whose kernels run 160
columns wide with zero padding, against the fp64 oracle at latent 150, on
the same seeded inputs; gradients in the caller's latent-150 layout; patch
equivalence (condition 1 of Sec. 2.2) and the training step at that width."""
import numpy as np
import pytest

import oracle as O
import synth
from gpu_util import BF16_TOL, FP32_TOL, Problem, bf16_grad_tols, kink_resolved, rel_l2, segments

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2304_00338_amd import mgn  # noqa: E402

LAT = 150


PRECS = ["fp32", "bf16"]


def tol_of(prec):
    return FP32_TOL if prec == "fp32" else BF16_TOL


def run_fwd_bwd(pb, prec="fp32"):
    N, E = pb.g.n_nodes, pb.g.n_edges
    ctx = mgn.Context(pb.m, N, E, prec, save=True, latent=LAT)
    out = mgn.mgn_forward(ctx, pb.dg, pb.d_params, pb.d_node_in, pb.dg.efeat, save=True)
    gp = torch.zeros_like(pb.d_params)
    gi = torch.zeros((N, 8), dtype=torch.float32, device="cuda")
    mgn.mgn_backward(ctx, pb.d_w, gp, gi)
    torch.cuda.synchronize()
    return out.cpu().numpy(), gp.cpu().numpy(), gi.cpu().numpy()


def check(res, ref, m, tol, gtol):
    """gtol: one tolerance for every gradient, or {segment: tol, 'gin': tol}."""
    out, gp, gi = res
    ro, rgp, rgi = ref
    gt = gtol if isinstance(gtol, dict) else {"gin": gtol}
    assert rel_l2(out, ro) < tol, rel_l2(out, ro)
    for name, a, b in segments(m, LAT):
        assert rel_l2(gp[a:b], rgp[a:b]) < gt.get(name, gtol), (name, rel_l2(gp[a:b], rgp[a:b]))
    assert rel_l2(gi, rgi) < gt["gin"], rel_l2(gi, rgi)


@pytest.mark.parametrize("shape,m", [((9, 8, 7), 3), ((32, 32), 3), ((5, 4, 3), 1), ((12, 12, 12), 3)])
@pytest.mark.parametrize("prec", PRECS)
def test_forward_backward_latent150(shape, m, prec):
    """Output and every parameter segment's gradient at latent 150: fp32
    against the valid subgradient nearest the GPU result (kinks resolved),
    bf16 against the oracle with the ordinary-point bf16 gradient bounds."""
    pb = Problem(shape, m, seed=21, latent=LAT).device()
    assert pb.d_params.numel() == mgn.param_count(m, LAT)
    res = run_fwd_bwd(pb, prec)
    out, tape = O.mgn_forward(pb.go, pb.params, pb.node_in, pb.go.efeat, m, latent=LAT, keep=True)
    if prec == "fp32":
        gp, gi, _ = kink_resolved(tape, pb.w, res[1], res[2])
        check(res, (out, gp, gi), m, FP32_TOL, FP32_TOL)
    else:
        check(res, (out, *O.mgn_backward(tape, pb.w)), m, BF16_TOL, bf16_grad_tols(pb))


@pytest.mark.parametrize("prec", PRECS)
def test_smooth_point_latent150(prec):
    """Every ReLU input far from its kink: the gradient is unique, so both
    precisions are held to their output tolerance."""
    pb = Problem((10, 9, 8), 3, seed=22, smooth=True, latent=LAT).device()
    res = run_fwd_bwd(pb, prec)
    out, tape = O.mgn_forward(pb.go, pb.params, pb.node_in, pb.go.efeat, 3, latent=LAT, keep=True)
    assert O.relu_kinks(tape, 0.5) == []
    check(res, (out, *O.mgn_backward(tape, pb.w)), 3, tol_of(prec), tol_of(prec))


@pytest.mark.parametrize("prec", PRECS)
def test_bitwise_determinism_latent150(prec):
    pb = Problem((8, 7, 6), 3, seed=23, latent=LAT).device()
    a, b = run_fwd_bwd(pb, prec), run_fwd_bwd(pb, prec)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("scheme", ["heun2", "euler"])
def test_integrate_step_latent150(scheme, prec):
    """The paper's 3D configuration (latent 150, m = 3, H2): the step's
    increment and its gradients through both stages at a smooth point."""
    tol = tol_of(prec)
    pb = Problem((7, 6, 5), 3, seed=24, smooth=True, latent=LAT).device()
    N, E = pb.g.n_nodes, pb.g.n_edges
    ctx = mgn.Context(3, N, E, prec, max_stages=2, save=True, latent=LAT)
    yn = mgn.mgn_integrate_step(ctx, pb.dg, pb.d_params, scheme, pb.d_onehot, pb.d_states, pb.dg.efeat,
                                save=True)
    gp = torch.zeros_like(pb.d_params)
    gy = torch.zeros((N, 4), dtype=torch.float32, device="cuda")
    mgn.mgn_backward(ctx, pb.d_w, gp, gy)
    ryn, tape = O.integrate_step(pb.go, pb.params, scheme, pb.onehot, pb.states, pb.go.efeat, 3, latent=LAT,
                                 keep=True)
    rgp, rgy = O.integrate_backward(tape, pb.w)
    yn = yn.cpu().numpy()
    assert rel_l2(yn - pb.states, ryn - pb.states) < tol
    assert rel_l2(gp.cpu().numpy(), rgp) < tol
    assert rel_l2(gy.cpu().numpy(), rgy) < tol


def test_gradient_accumulates_latent150():
    """Condition 3 of Sec. 2.2: a second backward adds to the caller's
    latent-150 gradient buffer."""
    pb = Problem((6, 5, 4), 3, seed=25, latent=LAT).device()
    N, E = pb.g.n_nodes, pb.g.n_edges
    ctx = mgn.Context(3, N, E, "fp32", save=True, latent=LAT)
    mgn.mgn_forward(ctx, pb.dg, pb.d_params, pb.d_node_in, pb.dg.efeat, save=True)
    g1 = torch.zeros_like(pb.d_params)
    mgn.mgn_backward(ctx, pb.d_w, g1, None)
    g2 = g1.clone()
    mgn.mgn_backward(ctx, pb.d_w, g2, None)
    assert torch.equal(g2, g1 + g1)


@pytest.mark.parametrize("prec", PRECS)
def test_patch_equivalence_latent150(prec):
    """Condition 1 at the paper's 3D setting m = k = 3: every patch's
    subdomain nodes get bitwise the whole-mesh outputs."""
    m, k = 3, 3
    pb = Problem((8, 7, 12), m, seed=26, latent=LAT).device()
    ctx = mgn.Context(m, pb.g.n_nodes, pb.g.n_edges, prec, latent=LAT)
    whole = mgn.mgn_forward(ctx, pb.dg, pb.d_params, pb.d_node_in, pb.dg.efeat).cpu().numpy()
    part = O.partition(pb.pos, (2, 1, 3)).astype(np.int32)
    for p in range(6):
        pt = mgn.extract_patch(pb.g, part, p, k)
        mp = pt.patch_maps()
        dpt = mgn.DeviceGraph(pt)
        x = torch.from_numpy(pb.node_in[mp["node_l2g"]]).cuda()
        o = mgn.mgn_forward(ctx, dpt, pb.d_params, x, dpt.efeat).cpu().numpy()
        it = mp["interior"] == 1
        assert np.array_equal(o[it].view(np.uint32), whole[mp["node_l2g"][it]].view(np.uint32)), p


@pytest.mark.parametrize("prec", PRECS)
def test_patch_rollout_latent150(prec):
    """Patch-decomposed Heun rollout (ghost depth 2m = 6) equals the
    whole-mesh rollout bitwise for two steps."""
    m, k, shape = 3, 6, (6, 5, 16)
    M = synth.mesh(shape, 27)
    g = mgn.build_graph(M["cells"], M["pos"])
    part = synth.slab_part(shape, 2)
    patches = [mgn.DevicePatch(mgn.extract_patch(g, part, p, k)) for p in range(2)]
    ctx_p = mgn.Context(m, max(p.n_nodes for p in patches), max(p.n_edges for p in patches), prec,
                        max_stages=2, latent=LAT)
    ctx_w = mgn.Context(m, g.n_nodes, g.n_edges, prec, max_stages=2, latent=LAT)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    st, params = d(M["onehot"]), d(synth.xavier_params(m, 27, LAT))
    dg = mgn.DeviceGraph(g)
    yw = yp = d(M["states"])
    for t in range(2):
        yw = mgn.mgn_integrate_step(ctx_w, dg, params, "heun2", st, yw, dg.efeat)
        yp = mgn.mgn_patch_step(ctx_p, patches, params, "heun2", st, yp)
        assert torch.equal(yw, yp), t


@pytest.mark.parametrize("prec", PRECS)
def test_train_step_latent150(prec):
    """One patch-training step at the 3D shape (noise, Heun step per patch,
    masked MSE, gradients summed over the patches, Adam) against the oracle at
    a smooth point; the update equals the oracle's Adam applied to the GPU
    gradient."""
    tol = tol_of(prec)
    m, shape = 3, (6, 5, 14)
    M = synth.mesh(shape, 28)
    g = mgn.build_graph(M["cells"], M["pos"])
    go = O.build_graph(M["cells"], M["pos"])
    part = synth.slab_part(shape, 2)
    patches = [mgn.DevicePatch(mgn.extract_patch(g, part, p, 2 * m)) for p in range(2)]
    opatches = [O.extract_patch(go, part, p, 2 * m) for p in range(2)]
    P = synth.smooth_params(m, 28, LAT)
    tgt = synth.next_states(M["states"], 28)
    nz = synth.standard_noise(g.n_nodes, 28)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    ctx = mgn.Context(m, max(p.n_nodes for p in patches), max(p.n_edges for p in patches), prec, max_stages=2,
                      save=True, latent=LAT)
    params = d(P)
    grad, mm, vv = torch.zeros_like(params), torch.zeros_like(params), torch.zeros_like(params)
    loss = mgn.mgn_train_step(ctx, patches, params, "heun2", d(M["onehot"]), d(M["states"]), d(tgt), d(nz), grad,
                              mm, vv, mgn.Adam(), 1)
    z = np.zeros(P.size)
    _, _, _, rloss, rgrad = O.train_step(opatches, P, "heun2", M["onehot"], M["states"], tgt, nz, m, z, z, 1,
                                         latent=LAT)
    assert abs(loss.item() - rloss) < tol * abs(rloss)
    gg = grad.cpu().numpy()
    assert rel_l2(gg, rgrad) < tol
    rp, _, _ = O.adam_update(P.astype(np.float64), gg.astype(np.float64), z, z, 1, 1e-3)
    pg = params.cpu().numpy().astype(np.float64)
    bound = np.spacing(np.abs(rp).astype(np.float32)).astype(np.float64) + 1e-5 * np.abs(rp - P).max()
    assert np.all(np.abs(pg - rp) <= bound)


def _oracle_check(pb, prec, res):
    out, tape = O.mgn_forward(pb.go, pb.params, pb.node_in, pb.go.efeat, pb.m, latent=LAT, keep=True)
    if prec == "fp32":
        gp, gi, _ = kink_resolved(tape, pb.w, res[1], res[2])
        check(res, (out, gp, gi), pb.m, FP32_TOL, FP32_TOL)
    else:
        check(res, (out, *O.mgn_backward(tape, pb.w)), pb.m, BF16_TOL, bf16_grad_tols(pb))


@pytest.mark.parametrize("prec", PRECS)
def test_long_segment_hub_latent150(prec):
    """A centre node with 300 in-edges at width 160: its in-segment spans
    several chunk tiles whose slot sums are added in chunk order."""
    k = 300
    ang = np.linspace(0, 2 * np.pi, k, endpoint=False)
    rim = np.stack([np.cos(ang), np.sin(ang)], 1)
    pos = np.concatenate([[[0.0, 0.0]], rim, 2 * rim]).astype(np.float32)
    cells = np.array([[0, 1 + j, 1 + (j + 1) % k] for j in range(k)] +
                     [[1 + j, 1 + k + j, 1 + (j + 1) % k] for j in range(k)])
    rng = np.random.default_rng(31)
    node_in = np.concatenate([np.eye(4)[rng.integers(0, 4, pos.shape[0])],
                              rng.standard_normal((pos.shape[0], 4))], 1).astype(np.float32)
    pb = Problem(None, 2, seed=31, cells=cells, pos=pos, node_in=node_in, latent=LAT).device()
    assert pb.dg.n_long == 1
    _oracle_check(pb, prec, run_fwd_bwd(pb, prec))


def test_isolated_nodes_and_duplicates_latent150():
    rng = np.random.default_rng(32)
    n = 150
    cells = rng.integers(0, n - 20, size=(200, 3))
    cells = np.concatenate([cells, cells[:30]])
    pos = rng.standard_normal((n, 3)).astype(np.float32)
    node_in = np.concatenate([np.eye(4)[rng.integers(0, 4, n)], rng.standard_normal((n, 4))], 1)
    pb = Problem(None, 2, seed=32, cells=cells, pos=pos, node_in=node_in, latent=LAT).device()
    _oracle_check(pb, "fp32", run_fwd_bwd(pb, "fp32"))


@pytest.mark.parametrize("prec", PRECS)
def test_edgeless_graph_latent150(prec):
    """No edges: every aggregate is zero and the edge MLPs (in the caller's
    latent-150 layout) get exactly zero gradient."""
    rng = np.random.default_rng(33)
    n = 45
    pos = rng.standard_normal((n, 3)).astype(np.float32)
    node_in = np.concatenate([np.eye(4)[rng.integers(0, 4, n)], rng.standard_normal((n, 4))], 1)
    pb = Problem(None, 2, seed=33, cells=np.zeros((0, 3), np.int64), pos=pos, node_in=node_in, latent=LAT)
    assert pb.g.n_edges == 0
    pb.device()
    res = run_fwd_bwd(pb, prec)
    for name, a, b in segments(pb.m, LAT):
        if ".edge" in name or name == "enc_edge":
            assert np.all(res[1][a:b] == 0.0), name
    _oracle_check(pb, prec, res)


def test_empty_graph_latent150():
    pb = Problem((6, 6), 1, seed=34, latent=LAT)
    part = np.zeros(pb.g.n_nodes, np.int32)
    part[:3] = 2
    pt = mgn.extract_patch(pb.g, part, 1, 1)
    dpt = mgn.DeviceGraph(pt)
    ctx = mgn.Context(1, 10, 10, "fp32", save=True, latent=LAT)
    params = torch.from_numpy(pb.params).cuda()
    out = mgn.mgn_forward(ctx, dpt, params, torch.zeros((0, 8), dtype=torch.float32, device="cuda"), dpt.efeat,
                          save=True)
    assert out.shape == (0, 4)
    gp = torch.zeros_like(params)
    mgn.mgn_backward(ctx, torch.zeros((0, 4), device="cuda"), gp)
    assert float(gp.abs().sum()) == 0.0


@pytest.mark.parametrize("prec", PRECS)
def test_patch_union_multi_unit_latent150(prec):
    """Past one unit per wave: on the disjoint union of four slab patches
    (about 49k nodes, so the node and encoder kernels walk several 16-row
    units or rounds per wave, and the edge kernels several tiles), the
    forward output and the input gradient equal those of each patch computed
    alone (under 1,000 units each, at most one per wave) bitwise, and the
    parameter gradient equals the sum of the patches' gradients up to the
    order of the fp32 block sums."""
    import synth
    m, shape = 2, (36, 36, 32)
    M = synth.mesh(shape, 43)
    g = mgn.build_graph(M["cells"], M["pos"])
    part = synth.slab_part(shape, 4)
    hp = [mgn.extract_patch(g, part, p, m) for p in range(4)]
    u = mgn.patch_union(hp)
    l2g = [p.patch_maps()["node_l2g"] for p in hp]
    assert np.array_equal(u.patch_maps()["node_l2g"], np.concatenate(l2g))
    assert u.n_nodes > 16 * 2048 and max(p.n_nodes for p in hp) < 16 * 1000
    node_in = M["node_in"]
    params = torch.from_numpy(synth.smooth_params(m, 43, LAT)).cuda()
    gout = np.random.default_rng(43).standard_normal((u.n_nodes, 4)).astype(np.float32)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()

    def fwd_bwd(graph, rows, go):
        dg = mgn.DeviceGraph(graph)
        ctx = mgn.Context(m, graph.n_nodes, graph.n_edges, prec, save=True, latent=LAT)
        out = mgn.mgn_forward(ctx, dg, params, d(node_in[rows]), dg.efeat, save=True)
        gp = torch.zeros_like(params)
        gi = torch.zeros((graph.n_nodes, 8), dtype=torch.float32, device="cuda")
        mgn.mgn_backward(ctx, d(go), gp, gi)
        torch.cuda.synchronize()
        return out.cpu().numpy(), gp.cpu().numpy(), gi.cpu().numpy()

    ou, gpu_, giu = fwd_bwd(u, np.concatenate(l2g), gout)
    gsum = np.zeros_like(gpu_, dtype=np.float64)
    off = 0
    for p, ids in zip(hp, l2g):
        n = p.n_nodes
        op, gp, gi = fwd_bwd(p, ids, gout[off:off + n])
        assert np.array_equal(ou[off:off + n], op)
        assert np.array_equal(giu[off:off + n], gi)
        gsum += gp
        off += n
    assert rel_l2(gpu_, gsum) < 1e-5, rel_l2(gpu_, gsum)
