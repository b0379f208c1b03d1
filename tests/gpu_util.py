"""Shared helpers of the GPU parity tests: seeded problem set-up on both
sides (the oracle builds its own graph from the same cells and positions)
and error metrics."""
import numpy as np

import oracle as O
import synth

FP32_TOL = 1e-4   # relative L2, fp32 outputs and gradients
BF16_TOL = 2e-2   # relative L2, bf16-MLP outputs; also bf16 gradients at a
                  # smooth point (every ReLU input far from its kink)
# Relative L2 of bf16 gradients at an ordinary point: the gradient there is
# not a smooth function of the weights (ReLU inputs near zero switch branch),
# so no fixed tolerance fits every case.  The bf16 path rounds the weights
# and every activation operand once per GEMM (relative 2^-9 each); the bound
# per MLP segment is twice the largest change of the oracle's own gradient
# under random relative 2^-8 sign perturbations of all weights (see
# bf16_grad_tols).  Measured errors are 0.28-0.54 of that bound on every
# segment of the small-mesh cases and about 0.3 on the 32^3 mesh; the floor
# is only the output contract, for segments whose gradient is zero.
BF16_GRAD_TOL = BF16_TOL
KINK_TAU = 3e-6   # |ReLU input| below which fp32 and fp64 may take different branches


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def segments(m, latent=128):
    """(name, start, stop) of every MLP in the flat parameter buffer."""
    out, off = [], 0
    for name, fields in O.param_layout(m, latent):
        n = sum(int(np.prod(s)) for _, s in fields)
        out.append((name, off, off + n))
        off += n
    return out


def kink_resolved(tape, w, gp, gi, tau=KINK_TAU, max_kinks=48):
    """Gradients at a ReLU kink are not unique: at an input within tau of
    zero both one-sided derivatives are valid results within fp32 rounding.
    The valid set is {oracle gradient with the other branch taken on a
    subset S of the oracle's kinks}.  Find the member closest to the GPU
    result (additive model over single flips, fitted by least squares) and
    return the oracle's exact gradient for that subset.  Returns
    (grad_params, grad_in, S)."""
    g0, gi0 = O.mgn_backward(tape, w)
    kinks = O.relu_kinks(tape, tau)
    if not kinks:
        return g0, gi0, []
    assert len(kinks) <= max_kinks, f"{len(kinks)} kinks within {tau}"
    base = np.concatenate([g0, gi0.ravel()])
    target = np.concatenate([np.asarray(gp, np.float64), np.asarray(gi, np.float64).ravel()])
    cols = []
    for k in kinks:
        gk, gik = O.mgn_backward(tape, w, flips=[k])
        cols.append(np.concatenate([gk, gik.ravel()]) - base)
    c, *_ = np.linalg.lstsq(np.stack(cols, 1), target - base, rcond=None)
    S = [k for k, ci in zip(kinks, c) if ci > 0.5]
    if not S:
        return g0, gi0, []
    gS, giS = O.mgn_backward(tape, w, flips=S)
    return gS, giS, S


def grad_tols(pb, rel, floor, trials=2, scale=2.0):
    """Per-segment tolerances {name: tol, 'gin': tol} for gradients at an
    ordinary point: scale times the largest change of the oracle's own
    gradient under random relative +-rel perturbations of all weights,
    never below floor.  Oracle-only computation."""
    lat = getattr(pb, "latent", 128)
    _, tape = O.mgn_forward(pb.go, pb.params, pb.node_in, pb.go.efeat, pb.m, latent=lat, keep=True)
    g0, gi0 = O.mgn_backward(tape, pb.w)
    del tape
    worst = {}
    for t in range(trials):
        xi = np.random.default_rng(1000 + t).choice([-1.0, 1.0], size=pb.params.shape)
        _, t1 = O.mgn_forward(pb.go, pb.params * (1 + rel * xi), pb.node_in, pb.go.efeat, pb.m,
                              latent=lat, keep=True)
        g1, gi1 = O.mgn_backward(t1, pb.w)
        del t1
        for name, a, b in segments(pb.m, lat):
            worst[name] = max(worst.get(name, 0.0), rel_l2(g1[a:b], g0[a:b]))
        worst["gin"] = max(worst.get("gin", 0.0), rel_l2(gi1, gi0))
    return {k: max(floor, scale * v) for k, v in worst.items()}


def bf16_grad_tols(pb, trials=2, scale=2.0, floor=BF16_GRAD_TOL):
    """Tolerances for bf16 gradients at an ordinary point (see
    BF16_GRAD_TOL): the bf16 path rounds weights and activation operands to
    8 significant bits, so the perturbation is relative 2^-8."""
    return grad_tols(pb, 2.0 ** -8, floor, trials, scale)


def fp32_grad_tols(pb, trials=2, scale=2.0):
    """Tolerances for fp32 gradients at an ordinary point of a mesh too large
    to resolve its ReLU kinks one by one (kink_resolved): the fp32 forward's
    accumulated rounding in a K = 384 product is about sqrt(K) 2^-24 ~ 2^-20
    relative, so the valid subgradients spread like the oracle's gradient
    under relative 2^-20 weight perturbations; never below FP32_TOL."""
    return grad_tols(pb, 2.0 ** -20, FP32_TOL, trials, scale)


class Problem:
    def __init__(self, shape=None, m=2, seed=0, randomize=True, cells=None, pos=None, node_in=None,
                 smooth=False, latent=128):
        from paper_2304_00338_amd import mgn
        if shape is not None:
            M = synth.mesh(shape, seed)
            cells, pos, node_in = M["cells"], M["pos"], M["node_in"]
            self.onehot, self.states = M["onehot"], M["states"]
        else:
            self.onehot = node_in[:, :4]
            self.states = node_in[:, 4:]
        self.cells, self.pos, self.node_in = cells, pos, node_in.astype(np.float32)
        self.m = m
        self.seed = seed
        self.latent = latent
        self.g = mgn.build_graph(cells, pos)
        self.go = O.build_graph(cells, pos)
        self.params = (synth.smooth_params(m, seed, latent) if smooth
                       else synth.xavier_params(m, seed, latent, randomize_norm=randomize))
        self.w = synth.loss_weights(self.g.n_nodes, seed)

    def device(self):
        import torch
        from paper_2304_00338_amd import mgn
        self.dg = mgn.DeviceGraph(self.g)
        d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
        self.d_params = d(self.params)
        self.d_node_in = d(self.node_in)
        self.d_onehot = d(self.onehot)
        self.d_states = d(self.states)
        self.d_w = d(self.w)
        return self
