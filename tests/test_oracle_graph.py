"""Pins for the oracle's graph construction, partition and patch extraction.

Each check ties the oracle to something other than itself: closed-form edge
counts of the Kuhn split, brute-force set enumeration, adjacency-matrix
powers for hop distances, the paper's subdomain counts (App. C) and
geometric properties of the equal split (Sec. 2.2).
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle as O
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_facts.json")


def kuhn_undirected(shape):
    """Closed form: one undirected edge per grid point p and direction
    d in {0,1}^dim minus 0 with p + d inside the grid."""
    tot = 0
    for d in itertools.product((0, 1), repeat=len(shape)):
        if any(d):
            tot += int(np.prod([n - di for n, di in zip(shape, d)]))
    return tot


@pytest.mark.parametrize("shape,expect", [((32, 32), 5890), ((32, 32, 32), 434558)])
def test_config_edge_counts(shape, expect):
    assert 2 * kuhn_undirected(shape) == expect
    M = synth.mesh(shape, 0)
    g = O.build_graph(M["cells"], M["pos"])
    assert g.n_nodes == int(np.prod(shape))
    assert g.n_edges == expect


def test_full_mesh_closed_form():
    # 146^3 jittered grid (3,112,136 nodes): directed edges by the formula
    assert 146 ** 3 == 3112136
    assert 2 * kuhn_undirected((146, 146, 146)) == 43060070


@pytest.mark.parametrize("shape", [(5, 7), (3, 4, 5), (6, 6, 6), (2, 2), (2, 3, 2)])
def test_counts_and_degrees(shape):
    M = synth.mesh(shape, 1)
    g = O.build_graph(M["cells"], M["pos"])
    assert g.n_edges == 2 * kuhn_undirected(shape)
    deg = np.diff(g.rowptr)
    idx = synth.grid_index(shape)
    inner = np.all((idx > 0) & (idx < np.array(shape) - 1), axis=1)
    if inner.any():
        assert np.all(deg[inner] == (6 if len(shape) == 2 else 14))


def _brute_edges(cells, n):
    """O(n^2) brute force: a and b are adjacent iff some cell holds both."""
    adj = set()
    for a in range(n):
        for b in range(n):
            if a == b:
                continue
            for c in cells:
                if a in c and b in c:
                    adj.add((b, a))  # (receiver, sender)
                    break
    return sorted(adj)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_brute_force_random_cells(seed):
    rng = np.random.default_rng(100 + seed)
    n = 12
    vpc = [2, 3, 4, 3][seed]
    cells = rng.integers(0, n, size=(9, vpc))
    cells = np.concatenate([cells, cells[:2]])  # duplicate cells are merged
    pos = rng.standard_normal((n, 3)).astype(np.float32)
    g = O.build_graph(cells, pos)
    want = _brute_edges([set(c) for c in cells.tolist()], n)
    got = list(zip(g.receivers.tolist(), g.senders.tolist()))
    assert got == want
    # rowptr consistent with receivers; isolated nodes get empty segments
    for v in range(n):
        seg = g.receivers[g.rowptr[v]:g.rowptr[v + 1]]
        assert np.all(seg == v)
    assert g.rowptr[-1] == g.n_edges


def test_rev_and_features():
    M = synth.mesh((6, 5, 4), 3)
    g = O.build_graph(M["cells"], M["pos"])
    e = np.arange(g.n_edges)
    assert np.all(g.rev[g.rev] == e)
    assert np.all(g.senders[g.rev] == g.receivers)
    assert np.all(g.receivers[g.rev] == g.senders)
    f, fr = g.efeat, g.efeat[g.rev]
    assert np.array_equal(fr[:, :3], -f[:, :3])
    assert np.array_equal(fr[:, 3], f[:, 3])
    # displacement and length against an independent fp64 evaluation
    d = M["pos"][g.senders].astype(np.float64) - M["pos"][g.receivers]
    assert np.allclose(f[:, :3], d, rtol=1e-7, atol=0)
    assert np.allclose(f[:, 3], np.linalg.norm(d, axis=1), rtol=1e-7, atol=0)
    assert f.dtype == np.float32


def test_2d_features_padded():
    M = synth.mesh((4, 3), 0)
    g = O.build_graph(M["cells"], M["pos"])
    assert np.all(g.efeat[:, 3] == 0)
    d = M["pos"][g.senders].astype(np.float64) - M["pos"][g.receivers]
    assert np.allclose(g.efeat[:, 2], np.hypot(d[:, 0], d[:, 1]), rtol=1e-7)


def test_graph_errors():
    with pytest.raises(ValueError):
        O.build_graph(np.array([[0, 5, 1]]), np.zeros((3, 2), np.float32))
    with pytest.raises(ValueError):
        O.build_graph(np.array([[0, 1, 2, 3, 4]]), np.zeros((5, 2), np.float32))
    with pytest.raises(ValueError):
        O.build_graph(np.array([[0, 1, 2]]), np.zeros((3, 5), np.float32))


def test_paper_subdomain_counts():
    facts = json.load(open(GOLD))
    M2 = synth.mesh((30, 40), 0)
    part2 = O.partition(M2["pos"], facts["splits_2d"])
    assert len(np.unique(part2)) == facts["n_subdomains_2d"]
    assert part2.min() == 0 and part2.max() == facts["n_subdomains_2d"] - 1
    M3 = synth.mesh((36, 36, 45), 0)
    part3 = O.partition(M3["pos"], facts["splits_3d"])
    assert len(np.unique(part3)) == facts["n_subdomains_3d"]


def test_partition_geometry():
    """Every node lies inside the box of its subdomain (equal split)."""
    M = synth.mesh((9, 11, 7), 5)
    splits = (3, 2, 4)
    part = O.partition(M["pos"], splits)
    p = M["pos"].astype(np.float64)
    lo, hi = p.min(0), p.max(0)
    w = (hi - lo) / np.array(splits)
    ids = np.stack([part % 3, (part // 3) % 2, part // 6], axis=1)
    assert np.all(p >= lo + ids * w - 1e-12)
    assert np.all(p <= lo + (ids + 1) * w + 1e-12)


def test_partition_regular_grid_equal_parts():
    # unjittered 12-point axis split in 3: parts of exactly 4 points
    x = np.linspace(0, 1, 12, dtype=np.float32)
    pos = np.stack([x, np.zeros_like(x)], axis=1)
    part = O.partition(pos, (3, 1))
    assert np.array_equal(np.bincount(part), [4, 4, 4])


def _hops_by_matrix_powers(g, src, k):
    n = g.n_nodes
    A = np.zeros((n, n), dtype=np.int64)
    A[g.receivers, g.senders] = 1
    reach = np.zeros(n, dtype=bool)
    reach[src] = True
    hop = np.where(reach, 0, -1)
    B = np.eye(n, dtype=np.int64)
    for d in range(1, k + 1):
        B = np.minimum(B @ (A + np.eye(n, dtype=np.int64)), 1)
        r = B[:, src].any(axis=1) if src.any() else np.zeros(n, bool)
        hop[(hop < 0) & r] = d
    return hop


@pytest.mark.parametrize("shape,k", [((7, 6), 2), ((5, 4, 4), 1), ((5, 4, 4), 3)])
def test_patch_brute_force(shape, k):
    M = synth.mesh(shape, 2)
    g = O.build_graph(M["cells"], M["pos"])
    part = O.partition(M["pos"], (2,) * len(shape))
    for p in range(int(part.max()) + 1):
        pt = O.extract_patch(g, part, p, k)
        hop = _hops_by_matrix_powers(g, part == p, k)
        assert np.array_equal(pt.node_l2g, np.nonzero(hop >= 0)[0])
        assert np.array_equal(pt.hop, hop[hop >= 0])
        # induced subgraph: exactly the global edges with both ends inside
        inside = np.zeros(g.n_nodes, bool)
        inside[pt.node_l2g] = True
        want = np.nonzero(inside[g.senders] & inside[g.receivers])[0]
        assert np.array_equal(np.sort(pt.edge_l2g), want)
        assert np.array_equal(pt.node_l2g[pt.receivers], g.receivers[pt.edge_l2g])
        assert np.array_equal(pt.node_l2g[pt.senders], g.senders[pt.edge_l2g])
        assert np.array_equal(pt.efeat, g.efeat[pt.edge_l2g])
        assert np.all(pt.rev[pt.rev] == np.arange(pt.n_edges))
        key = pt.receivers * pt.n_nodes + pt.senders
        assert np.all(np.diff(key) > 0)


def test_slab_patch_closed_form():
    """z-slab subdomains of a Kuhn grid: hop distance = layer distance, so the
    patch is the clipped layer range [lo-k, hi+k] and its edges those of a
    Kuhn grid with that many layers.  Same layer structure as the 146^3 mesh
    split in 16 slabs with a 15-hop ghost zone, on a narrower cross-section."""
    shape = (6, 5, 146)
    M = synth.mesh(shape, 0)
    g = O.build_graph(M["cells"], M["pos"])
    part = synth.slab_part(shape, 16)
    nxy = shape[0] * shape[1]
    for p, k in [(8, 15), (7, 15), (0, 15), (15, 4)]:
        layers = np.nonzero(np.bincount(part[::nxy], minlength=16) >= 0)[0]
        kz = np.nonzero(part[::nxy] == p)[0]
        lo, hi = max(0, kz.min() - k), min(shape[2] - 1, kz.max() + k)
        L = hi - lo + 1
        pt = O.extract_patch(g, part, p, k)
        assert pt.n_nodes == nxy * L
        assert pt.n_interior == nxy * kz.size
        assert pt.n_edges == 2 * kuhn_undirected((shape[0], shape[1], L))
        z = synth.grid_index(shape)[pt.node_l2g, 2]
        dist = np.maximum(0, np.maximum(kz.min() - z, z - kz.max()))
        assert np.array_equal(pt.hop, dist)
        del layers
    # the 146^3 mesh itself, from the same closed form
    kz8 = [kz for kz in range(146) if (16 * kz) // 146 == 8]
    assert len(kz8) == 10
    L = min(145, kz8[-1] + 15) - max(0, kz8[0] - 15) + 1
    assert 146 * 146 * L == 852640
    assert 2 * kuhn_undirected((146, 146, L)) == 11674318


def test_empty_subdomain_and_errors():
    M = synth.mesh((4, 4), 0)
    g = O.build_graph(M["cells"], M["pos"])
    part = np.zeros(g.n_nodes, dtype=np.int64)
    part[:3] = 2  # subdomain 1 is empty
    pt = O.extract_patch(g, part, 1, 3)
    assert pt.n_nodes == 0 and pt.n_edges == 0 and pt.rowptr.tolist() == [0]
    with pytest.raises(ValueError):
        O.extract_patch(g, part, 0, -1)
    with pytest.raises(ValueError):
        O.extract_patch(g, part, 3, 1)
