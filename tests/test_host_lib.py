"""CPU tests of libmgn's host side: the library loads and exports every
symbol of include/mgn.h; graph construction, partition, patch extraction
and the tile schedule are bit-exact with the oracle; error paths.
No device call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import synth
from paper_2304_00338_amd import mgn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "mgn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mgn_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_header_symbols():
    L = ctypes.CDLL(mgn.LIB_PATH)
    names = header_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(L, n), n
    assert sorted(mgn.EXPORTS) == names
    assert mgn.version().startswith("mgn-gfx950")


def test_param_count():
    assert mgn.param_count(15) == 1788036 == O.n_params(15)
    for m in (0, 1, 2, 7):
        assert mgn.param_count(m) == O.n_params(m)


def compare_graph(g, go):
    a = g.arrays()
    for k in ("rowptr", "senders", "receivers", "rev"):
        assert np.array_equal(a[k], getattr(go, k)), k
    assert a["efeat"].dtype == np.float32
    assert np.array_equal(a["efeat"].view(np.uint32), go.efeat.view(np.uint32))


def check_schedule(g):
    a = g.arrays()
    tiles, longn = g.schedule()
    rp = a["rowptr"]
    TE = mgn.tile_edges()
    N = g.n_nodes
    covered = np.zeros(N, np.int64)
    edges = np.zeros(g.n_edges, np.int64)
    slots = {}
    for nb, ne, eb, ee in tiles:
        assert 0 <= ee - eb <= TE
        if ne >= 0:
            assert ne > nb and ne - nb <= TE
            assert eb == rp[nb] and ee == rp[ne]
            covered[nb:ne] += 1
        else:
            slots[-1 - ne] = (nb, eb, ee)
        edges[eb:ee] += 1
    for v, s0, nch, _ in longn:
        assert rp[v + 1] - rp[v] > TE
        covered[v] += 1
        spans = [slots[s0 + c] for c in range(nch)]
        assert all(sv == v for sv, _, _ in spans)
        assert spans[0][1] == rp[v] and spans[-1][2] == rp[v + 1]
        assert all(spans[c][2] == spans[c + 1][1] for c in range(nch - 1))
    assert np.all(covered == 1)
    assert np.all(edges == 1)
    # tiles are in node order
    starts = [t[0] for t in tiles]
    assert starts == sorted(starts)


@pytest.mark.parametrize("shape", [(32, 32), (7, 5), (6, 5, 4), (12, 11, 10), (2, 2, 2)])
def test_graph_bit_exact(shape):
    M = synth.mesh(shape, 3)
    g = mgn.build_graph(M["cells"], M["pos"])
    compare_graph(g, O.build_graph(M["cells"], M["pos"]))
    check_schedule(g)


@pytest.mark.parametrize("vpc,seed", [(2, 0), (3, 1), (4, 2), (3, 3)])
def test_graph_random_cells(vpc, seed):
    rng = np.random.default_rng(seed)
    n = 40
    cells = rng.integers(0, n - 5, size=(60, vpc))  # last 5 nodes isolated
    cells = np.concatenate([cells, cells[:7]])
    pos = rng.standard_normal((n, 3)).astype(np.float32)
    g = mgn.build_graph(cells, pos)
    compare_graph(g, O.build_graph(cells, pos))
    check_schedule(g)


def test_hub_node_long_segment():
    """A fan of 300 triangles around one centre: degree 300 > one tile, so the
    centre's in-segment is split into chunk tiles."""
    k = 300
    ang = np.linspace(0, 2 * np.pi, k, endpoint=False)
    pos = np.concatenate([[[0.0, 0.0]], np.stack([np.cos(ang), np.sin(ang)], 1)]).astype(np.float32)
    cells = np.array([[0, 1 + j, 1 + (j + 1) % k] for j in range(k)])
    g = mgn.build_graph(cells, pos)
    compare_graph(g, O.build_graph(cells, pos))
    tiles, longn = g.schedule()
    assert longn.shape[0] == 1 and longn[0, 0] == 0 and longn[0, 2] == -(-300 // mgn.tile_edges())
    check_schedule(g)


def test_partition_bit_exact():
    for shape, splits in [((30, 40), (3, 4)), ((13, 9, 11), (4, 3, 2)), ((36, 36, 45), (12, 12, 15))]:
        M = synth.mesh(shape, 1)
        assert np.array_equal(mgn.partition(M["pos"], splits), O.partition(M["pos"], splits))


@pytest.mark.parametrize("shape,splits,k", [((9, 8), (3, 2), 2), ((6, 7, 8), (2, 1, 3), 3),
                                            ((6, 5, 30), (1, 1, 4), 5)])
def test_patch_bit_exact(shape, splits, k):
    M = synth.mesh(shape, 2)
    g = mgn.build_graph(M["cells"], M["pos"])
    go = O.build_graph(M["cells"], M["pos"])
    part = O.partition(M["pos"], splits).astype(np.int32)
    for p in range(int(part.max()) + 1):
        pt = mgn.extract_patch(g, part, p, k)
        po = O.extract_patch(go, part, p, k)
        compare_graph(pt, po)
        mp = pt.patch_maps()
        assert np.array_equal(mp["node_l2g"], po.node_l2g)
        assert np.array_equal(mp["hop"], po.hop)
        assert np.array_equal(mp["interior"], po.interior)
        assert np.array_equal(mp["edge_l2g"], po.edge_l2g)
        assert mp["n_interior"] == po.n_interior
        check_schedule(pt)


def test_empty_patch_and_errors():
    M = synth.mesh((5, 5), 0)
    g = mgn.build_graph(M["cells"], M["pos"])
    part = np.zeros(g.n_nodes, np.int32)
    part[:4] = 2
    pt = mgn.extract_patch(g, part, 1, 2)
    assert pt.n_nodes == 0 and pt.n_edges == 0
    assert pt.schedule()[0].shape == (0, 4)
    with pytest.raises(mgn.MgnError) as e:
        mgn.extract_patch(g, part, 1, -1)
    assert e.value.code == mgn.ERR_ARG
    with pytest.raises(mgn.MgnError) as e:
        mgn.extract_patch(g, part, 3, 1)
    assert e.value.code == mgn.ERR_RANGE
    bad = part.copy()
    bad[7] = -4
    with pytest.raises(mgn.MgnError) as e:
        mgn.extract_patch(g, bad, 0, 1)
    assert e.value.code == mgn.ERR_RANGE
    with pytest.raises(mgn.MgnError) as e:
        mgn.build_graph(np.array([[0, 1, 99]]), M["pos"])
    assert e.value.code == mgn.ERR_RANGE
    with pytest.raises(mgn.MgnError) as e:
        mgn.build_graph(np.array([[0, 1, 2, 3, 4]]), M["pos"])
    assert e.value.code == mgn.ERR_ARG
    with pytest.raises(mgn.MgnError):
        mgn.partition(M["pos"], (0, 2))
    with pytest.raises(mgn.MgnError) as e:
        mgn.Graph(0)
    assert e.value.code == mgn.ERR_ARG


def test_ctx_planning_and_errors():
    c1 = mgn.Context(15, 1000, 20000, "fp32", allocate=False)
    c2 = mgn.Context(15, 1000, 20000, "bf16", allocate=False)
    c3 = mgn.Context(15, 1000, 20000, "bf16", save=True, max_stages=4, allocate=False)
    assert c1.ws_bytes > c2.ws_bytes > 0
    assert c3.ws_bytes > c2.ws_bytes
    # pure function of the arguments
    assert mgn.Context(15, 1000, 20000, "bf16", allocate=False).ws_bytes == c2.ws_bytes
    with pytest.raises(mgn.MgnError) as e:
        mgn.Context(15, 10, 10, "fp32", max_stages=5, allocate=False)
    assert e.value.code == mgn.ERR_ARG
    ws, h = ctypes.c_size_t(), ctypes.c_void_p()
    for lat, prec in ((140, "fp32"), (256, "bf16"), (160, "fp32")):
        cfg = mgn.config(3, prec, latent=lat)  # latents 128 and 150 only
        rc = mgn.lib().mgn_ctx_create(ctypes.byref(cfg), 10, 10, 1, 0, ctypes.byref(ws), ctypes.byref(h))
        assert rc == mgn.ERR_SHAPE, (lat, prec)
    # latent 150 (the 3D model, kernels padded to 160): parameter count in the
    # oracle's layout, a larger workspace than latent 128
    assert mgn.param_count(3, 150) == O.n_params(3, 150)
    c150 = mgn.Context(3, 1000, 20000, "fp32", save=True, max_stages=2, latent=150, allocate=False)
    c128 = mgn.Context(3, 1000, 20000, "fp32", save=True, max_stages=2, allocate=False)
    assert c150.ws_bytes > c128.ws_bytes
    assert mgn.scheme_stages("rk4") == 4 and mgn.scheme_stages("heun3") == 3
    assert mgn.lib().mgn_scheme_stages(9) == mgn.ERR_ARG
    # backward without a saved call
    rc = mgn.lib().mgn_backward(c1._h, None, None, None, None)
    assert rc == mgn.ERR_STATE


def test_c3_patch_closed_form():
    """The 146^3 mesh split in 16 z-slabs with a 15-hop ghost zone: slab 8
    has 213,160 interior nodes, 852,640 patch nodes and 11,674,318 edges."""
    shape = (146, 146, 146)
    M = synth.mesh(shape, 0)
    g = mgn.build_graph(M["cells"], M["pos"])
    assert g.n_nodes == 3112136 and g.n_edges == 43060070
    part = synth.slab_part(shape, 16)
    pt = mgn.extract_patch(g, part, 8, 15)
    mp = pt.patch_maps()
    assert pt.n_nodes == 852640 and pt.n_edges == 11674318
    assert mp["n_interior"] == 213160
    z = synth.grid_index(shape)[mp["node_l2g"], 2]
    assert z.min() == 58 and z.max() == 97
    dist = np.maximum(0, np.maximum(73 - z, z - 82))
    assert np.array_equal(mp["hop"], dist)
    check_schedule(pt)


def test_patch_union_is_block_diagonal():
    """mgn_patch_union: the parts' arrays concatenated with node / edge
    offsets (senders, receivers, rev shifted, rowptr continued), features and
    maps concatenated, no edge between parts, a valid tile schedule; errors
    for non-patches and null parts."""
    shape = (9, 8, 10)
    M = synth.mesh(shape, 3)
    g = mgn.build_graph(M["cells"], M["pos"])
    part = synth.slab_part(shape, 3)
    ps = [mgn.extract_patch(g, part, p, 2) for p in range(3)]
    u = mgn.patch_union(ps)
    a, mu = u.arrays(), u.patch_maps()
    nb = eb = 0
    for p in ps:
        b, mp = p.arrays(), p.patch_maps()
        n, e = p.n_nodes, p.n_edges
        assert np.array_equal(a["rowptr"][nb:nb + n + 1], b["rowptr"] + eb)
        for k in ("senders", "receivers"):
            assert np.array_equal(a[k][eb:eb + e], b[k] + nb)
        assert np.array_equal(a["rev"][eb:eb + e], b["rev"] + eb)
        assert np.array_equal(a["efeat"][eb:eb + e], b["efeat"])
        for k in ("node_l2g", "hop", "interior"):
            assert np.array_equal(mu[k][nb:nb + n], mp[k])
        assert np.array_equal(mu["edge_l2g"][eb:eb + e], mp["edge_l2g"])
        nb, eb = nb + n, eb + e
    assert (u.n_nodes, u.n_edges) == (nb, eb)
    assert mu["n_interior"] == g.n_nodes  # the slabs partition the mesh
    check_schedule(u)
    assert mgn.patch_union([]).n_nodes == 0
    with pytest.raises(mgn.MgnError) as e:
        mgn.patch_union([ps[0], g])
    assert e.value.code == mgn.ERR_STATE
    rc = mgn.lib().mgn_patch_union(None, 2, ctypes.byref(ctypes.c_void_p()))
    assert rc == mgn.ERR_ARG
