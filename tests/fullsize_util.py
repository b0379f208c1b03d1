"""Helpers of the full-size GPU tests: oracle outputs at single nodes of a
large structured mesh.

By patch equivalence (Sec. 2.2, condition 1, pinned on the oracle in
tests/test_oracle_mgn.py) the output of an m-step MGN call at node v depends
only on the m-hop ball around v, and the oracle evaluated on that ball gives
exactly its whole-mesh output at v.  On a Kuhn grid two adjacent nodes differ
by at most one in every grid coordinate, so the m-hop ball lies inside the
L-infinity box of radius m, and every edge between two of its nodes belongs
to a cell inside the box of radius m + 1: the oracle only needs that box."""
import numpy as np

import oracle as O
import synth


def grid_strides(shape):
    st = [1]
    for s in shape[:-1]:
        st.append(st[-1] * int(s))
    return np.array(st, dtype=np.int64)


def node_id(shape, coord):
    return int(np.dot(np.asarray(coord, np.int64), grid_strides(shape)))


def box_submesh(shape, center, r):
    """Global ids (ascending) and local Kuhn cells of the grid box of
    L-infinity radius r around grid point `center`, clipped to the grid."""
    shape = np.asarray(shape, np.int64)
    c = np.asarray(center, np.int64)
    lo = np.maximum(c - r, 0)
    hi = np.minimum(c + r, shape - 1)
    sub = tuple(int(x) for x in hi - lo + 1)
    gidx = synth.grid_index(sub) + lo
    gids = gidx @ grid_strides(shape)
    return gids, synth.kuhn_cells(sub)


def oracle_node_output(M, shape, center, params, m, node_in=None):
    """fp64 oracle output [4] of one MGN call at grid point `center` of the
    mesh bundle M (synth.mesh), from the m-hop ball around it."""
    gids, cells = box_submesh(shape, center, m + 1)
    pos = M["pos"][gids]
    x = (M["node_in"] if node_in is None else node_in)[gids]
    go = O.build_graph(cells, pos)
    part = np.ones(gids.size, np.int32)
    v = int(np.searchsorted(gids, node_id(shape, center)))
    assert gids[v] == node_id(shape, center)
    part[v] = 0
    pt = O.extract_patch(go, part, 0, m)
    out = O.mgn_forward(pt, params, x[pt.node_l2g], pt.efeat, m)
    (iv,) = np.nonzero(pt.interior)
    assert iv.size == 1
    return out[iv[0]]
