"""Shared helpers of the GPU parity tests: seeded problem set-up on both
sides (the oracle builds its own graph from the same cells and positions)
and error metrics."""
import numpy as np

import oracle as O
import synth

FP32_TOL = 1e-4   # relative L2, fp32 outputs and gradients
BF16_TOL = 2e-2   # relative L2, bf16-MLP outputs; also bf16 gradients at a
                  # smooth point (every ReLU input far from its kink)
# Relative L2 of bf16 gradients at an ordinary point.  The fp64 oracle's own
# gradient moves by 5-9% under a single 2^-9 (one bf16 rounding) relative
# perturbation of the weights and by 7.5-11% under 2^-8, because ReLU inputs
# near zero switch branch; the bf16 path rounds weights and every activation
# operand once per GEMM, so its gradient error is of the 2^-8 size.
BF16_GRAD_TOL = 0.15
KINK_TAU = 3e-6   # |ReLU input| below which fp32 and fp64 may take different branches


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def segments(m):
    """(name, start, stop) of every MLP in the flat parameter buffer."""
    out, off = [], 0
    for name, fields in O.param_layout(m):
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


class Problem:
    def __init__(self, shape=None, m=2, seed=0, randomize=True, cells=None, pos=None, node_in=None,
                 smooth=False):
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
        self.g = mgn.build_graph(cells, pos)
        self.go = O.build_graph(cells, pos)
        self.params = (synth.smooth_params(m, seed) if smooth
                       else synth.xavier_params(m, seed, randomize_norm=randomize))
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
