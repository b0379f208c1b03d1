"""mgn_forward_noalloc (the forward on the library's static device scratch)
against mgn_forward on the same inputs: two calls in a row on one context,
the second on a smaller graph, both bitwise equal to mgn_forward with a
caller workspace (same kernels, same launch shapes) and within the output
tolerances of the fp64 oracle; a context planned beyond the scratch is
rejected before any device work."""
import numpy as np
import pytest

import oracle as O
import synth
from gpu_util import BF16_TOL, FP32_TOL, rel_l2

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2304_00338_amd import mgn  # noqa: E402


def problem(shape, m, seed):
    M = synth.mesh(shape, seed)
    g = mgn.build_graph(M["cells"], M["pos"])
    go = O.build_graph(M["cells"], M["pos"])
    return M, g, go, mgn.DeviceGraph(g)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_noalloc_forward_matches_forward(prec):
    m = 3
    big = problem((14, 12, 10), m, 21)
    small = problem((9, 7, 6), m, 22)
    params = synth.xavier_params(m, 23, randomize_norm=True)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    dparams = d(params)
    Mb, gb = big[0], big[1]
    ctx_na = mgn.Context(m, gb.n_nodes, gb.n_edges, prec, allocate=False)
    assert 0 < ctx_na.ws_bytes <= mgn.NOALLOC_SCRATCH_BYTES
    ctx_ws = mgn.Context(m, gb.n_nodes, gb.n_edges, prec)
    tol = FP32_TOL if prec == "fp32" else BF16_TOL
    for M, g, go, dg in (big, small):
        x = d(M["node_in"])
        # poison the outputs so a call that skipped a row could not pass
        out_na = torch.full((g.n_nodes, 4), float("nan"), dtype=torch.float32, device="cuda")
        mgn.mgn_forward_noalloc(ctx_na, dg, dparams, x, dg.efeat, out_na)
        out_ws = mgn.mgn_forward(ctx_ws, dg, dparams, x, dg.efeat)
        torch.cuda.synchronize()
        a, b = out_na.cpu().numpy(), out_ws.cpu().numpy()
        assert np.isfinite(a).all()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
        ref = O.mgn_forward(go, params, M["node_in"], go.efeat, m)
        assert rel_l2(a, ref) < tol, rel_l2(a, ref)


def test_noalloc_rejects_oversized_context():
    m = 15
    ctx = mgn.Context(m, 852640, 11674318, "bf16", allocate=False)
    assert ctx.ws_bytes > mgn.NOALLOC_SCRATCH_BYTES
    M, g, go, dg = problem((5, 4, 3), m, 1)
    params = torch.zeros(mgn.param_count(m), dtype=torch.float32, device="cuda")
    x = torch.zeros((g.n_nodes, 8), dtype=torch.float32, device="cuda")
    out = torch.zeros((g.n_nodes, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(mgn.MgnError) as ei:
        mgn.mgn_forward_noalloc(ctx, dg, params, x, dg.efeat, out)
    assert ei.value.code == mgn.ERR_WORKSPACE
    assert "static scratch" in str(ei.value)
