"""Seeded synthetic inputs for the MeshGraphNets message-passing path.

This module only draws inputs: jittered structured meshes (vertex positions
and simplex cells), node types, node states, model parameters and gradient
seeds.  It holds none of the method's arithmetic (no edge construction, no
features derived from the mesh, no network evaluation), so both the CPU oracle
and the GPU path can take their inputs from here without sharing any of the
computation under test.

Recipe (stands in for the paper's 3D CO2-capture CFD meshes, Sec. 3 and
App. B, which are not available here):

* mesh: unit square / cube, ``n`` points per axis, spacing ``1/(n-1)``; every
  coordinate jittered by ``U(-0.2, 0.2) * spacing``; connectivity is the Kuhn
  split of each grid cell (2D: two triangles on the (0,0)-(1,1) diagonal;
  3D: six tetrahedra around the main diagonal).  Node ids run x fastest.
* node type (4-way one-hot): 0 interior, 1 on the min face of the last axis,
  2 on the max face of the last axis, 3 any other boundary node.
* node states: 2D four N(0,1) values; 3D velocity xyz ~ N(0,1) and a
  volume-fraction-like scalar ~ U[0,1].
* parameters: Xavier-uniform weights, zero biases, LayerNorm gain 1 and
  offset 0, laid out in the flat order documented in ``include/mgn.h``.
* seeds: sub-streams ``seed`` (jitter), ``seed+1`` (states), ``seed+2``
  (parameters), ``seed+3`` (gradient seeds / loss weights), NumPy PCG64.
"""
from __future__ import annotations

import itertools

import numpy as np

LATENT = 128
NODE_IN = 8
EDGE_IN = 4
OUT = 4
N_TYPES = 4


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(int(seed)))


def grid_ids(shape):
    """Node id of every grid point, x fastest (array indexed [.., y, x] order
    reversed: ids[i0, i1, ...] with axis 0 = x)."""
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape))
    return np.arange(n, dtype=np.int64).reshape(shape[::-1]).transpose(
        tuple(range(len(shape) - 1, -1, -1)))


def kuhn_cells(shape) -> np.ndarray:
    """Simplices of the Kuhn split of a structured grid with ``shape`` points
    per axis.  2D: triangles; 3D: tetrahedra.  int32 [n_cells, dim+1]."""
    shape = tuple(int(s) for s in shape)
    dim = len(shape)
    ids = grid_ids(shape)
    lo = tuple(slice(0, s - 1) for s in shape)
    cells = []
    for perm in itertools.permutations(range(dim)):
        corner = [0] * dim
        verts = []
        base = ids[tuple(slice(c, c + s - 1) for c, s in zip(corner, shape))]
        verts.append(base.reshape(-1))
        for ax in perm:
            corner[ax] = 1
            sl = tuple(slice(c, c + s - 1) for c, s in zip(corner, shape))
            verts.append(ids[sl].reshape(-1))
        cells.append(np.stack(verts, axis=1))
    del lo
    return np.concatenate(cells, axis=0).astype(np.int32)


def jittered_positions(shape, seed: int, jitter: float = 0.2) -> np.ndarray:
    """Unit-box grid points, spacing 1/(n-1) per axis, each coordinate moved by
    U(-jitter, jitter) * spacing.  float32 [N, dim], node ids x fastest."""
    shape = tuple(int(s) for s in shape)
    dim = len(shape)
    n = int(np.prod(shape))
    ids = grid_ids(shape).reshape(-1)
    # coordinates of node id: decompose id with x fastest
    idx = np.empty((n, dim), dtype=np.int64)
    rem = np.arange(n, dtype=np.int64)
    for ax in range(dim):
        idx[:, ax] = rem % shape[ax]
        rem //= shape[ax]
    del ids
    spacing = np.array([1.0 / (s - 1) for s in shape])
    rng = _rng(seed)
    jit = rng.uniform(-jitter, jitter, size=(n, dim))
    pos = idx * spacing + jit * spacing
    return pos.astype(np.float32)


def grid_index(shape) -> np.ndarray:
    """Integer grid coordinates of each node id (x fastest). int64 [N, dim]."""
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape))
    idx = np.empty((n, len(shape)), dtype=np.int64)
    rem = np.arange(n, dtype=np.int64)
    for ax in range(len(shape)):
        idx[:, ax] = rem % shape[ax]
        rem //= shape[ax]
    return idx


def node_types(shape) -> np.ndarray:
    """Type id per node: 0 interior, 1 min face of the last axis ('inlet'),
    2 max face of the last axis ('outlet'), 3 other boundary ('wall').
    Inlet/outlet take precedence over wall.  int32 [N]."""
    shape = tuple(int(s) for s in shape)
    idx = grid_index(shape)
    last = len(shape) - 1
    t = np.zeros(idx.shape[0], dtype=np.int32)
    on_bnd = np.zeros(idx.shape[0], dtype=bool)
    for ax, s in enumerate(shape):
        on_bnd |= (idx[:, ax] == 0) | (idx[:, ax] == s - 1)
    t[on_bnd] = 3
    t[idx[:, last] == 0] = 1
    t[idx[:, last] == shape[last] - 1] = 2
    return t


def one_hot(types: np.ndarray, n: int = N_TYPES) -> np.ndarray:
    oh = np.zeros((types.shape[0], n), dtype=np.float32)
    oh[np.arange(types.shape[0]), types] = 1.0
    return oh


def node_states(n_nodes: int, dim: int, seed: int) -> np.ndarray:
    """Four state values per node.  2D: N(0,1) x4.  3D: velocity N(0,1) x3 and
    a volume fraction U[0,1].  float32 [N, 4]."""
    rng = _rng(seed + 1)
    if dim == 2:
        return rng.standard_normal((n_nodes, 4)).astype(np.float32)
    v = rng.standard_normal((n_nodes, 3))
    a = rng.uniform(0.0, 1.0, size=(n_nodes, 1))
    return np.concatenate([v, a], axis=1).astype(np.float32)


def param_shapes(mp_steps: int, latent: int = LATENT, node_in: int = NODE_IN,
                 edge_in: int = EDGE_IN, out: int = OUT):
    """(name, kind, shape) in flat-buffer order.  kind: 'w' weight [out, in],
    'b' bias, 'g' LayerNorm gain, 'z' LayerNorm offset."""
    D = latent
    spec = []

    def mlp(prefix, din, dout, ln):
        spec.append((prefix + ".W1", "w", (D, din)))
        spec.append((prefix + ".b1", "b", (D,)))
        spec.append((prefix + ".W2", "w", (dout, D)))
        spec.append((prefix + ".b2", "b", (dout,)))
        if ln:
            spec.append((prefix + ".gamma", "g", (dout,)))
            spec.append((prefix + ".beta", "z", (dout,)))

    mlp("enc_node", node_in, D, True)
    mlp("enc_edge", edge_in, D, True)
    for i in range(mp_steps):
        mlp(f"block{i}.edge", 3 * D, D, True)
        mlp(f"block{i}.node", 2 * D, D, True)
    mlp("dec", D, out, False)
    return spec


def xavier_params(mp_steps: int, seed: int, latent: int = LATENT,
                  randomize_norm: bool = False) -> np.ndarray:
    """Flat float32 parameter buffer: Xavier-uniform U(+-sqrt(6/(fan_in+fan_out)))
    weights, zero biases, gain 1, offset 0.  With ``randomize_norm`` the biases,
    gains and offsets are drawn too (small random values), which exercises every
    parameter in gradient checks."""
    rng = _rng(seed + 2)
    chunks = []
    for _, kind, shape in param_shapes(mp_steps, latent):
        if kind == "w":
            fo, fi = shape
            lim = np.sqrt(6.0 / (fi + fo))
            chunks.append(rng.uniform(-lim, lim, size=shape).reshape(-1))
        elif kind == "g":
            v = np.ones(shape)
            if randomize_norm:
                v = v + rng.uniform(-0.5, 0.5, size=shape)
            chunks.append(v)
        else:
            v = np.zeros(shape)
            if randomize_norm:
                v = rng.uniform(-0.3, 0.3, size=shape)
            chunks.append(v)
    return np.concatenate(chunks).astype(np.float32)


def smooth_params(mp_steps: int, seed: int, latent: int = LATENT,
                  bias: float = 6.0, w1_scale: float = 0.05) -> np.ndarray:
    """Like xavier_params(randomize_norm=True) but every first-layer weight is
    scaled by ``w1_scale`` and every first-layer bias is ``bias``.  With the
    defaults every ReLU input stays several units above its kink on the
    synthetic meshes used here, so the network is smooth at this point and
    its gradient is unique."""
    flat = xavier_params(mp_steps, seed, latent, randomize_norm=True)
    off = 0
    for name, _, shape in param_shapes(mp_steps, latent):
        n = int(np.prod(shape))
        if name.endswith(".b1"):
            flat[off:off + n] = bias
        if name.endswith(".W1"):
            flat[off:off + n] *= w1_scale
        off += n
    return flat.astype(np.float32)


def loss_weights(n_nodes: int, seed: int, n_out: int = OUT) -> np.ndarray:
    """Fixed random weights w for the linear test loss sum(w * out). [N, 4]."""
    return _rng(seed + 3).standard_normal((n_nodes, n_out)).astype(np.float32)


def standard_noise(n_nodes: int, seed: int, n_out: int = OUT) -> np.ndarray:
    """Standard-normal draws [N, 4] for input noise (scaled per channel by the
    consumer).  Sub-stream seed + 5."""
    return _rng(seed + 5).standard_normal((n_nodes, n_out)).astype(np.float32)


def next_states(states: np.ndarray, seed: int, scale: float = 0.1) -> np.ndarray:
    """Synthetic next-step states: states plus N(0, scale^2) changes.
    Sub-stream seed + 6."""
    d = _rng(seed + 6).standard_normal(states.shape) * scale
    return (np.asarray(states, np.float64) + d).astype(np.float32)


def relabel(n_nodes: int, seed: int) -> np.ndarray:
    """Seeded random node permutation (new id of old node i is perm[i])."""
    return _rng(seed + 7).permutation(n_nodes).astype(np.int64)


def mesh(shape, seed: int = 0):
    """Convenience bundle: positions, cells, one-hot types, states, node_in."""
    shape = tuple(int(s) for s in shape)
    pos = jittered_positions(shape, seed)
    cells = kuhn_cells(shape)
    types = node_types(shape)
    states = node_states(pos.shape[0], len(shape), seed)
    oh = one_hot(types)
    node_in = np.concatenate([oh, states], axis=1).astype(np.float32)
    return {"shape": shape, "pos": pos, "cells": cells, "types": types,
            "onehot": oh, "states": states, "node_in": node_in}


def slab_part(shape, n_slabs: int) -> np.ndarray:
    """Grid-layer subdomain ids along the last axis: floor(P * k / n_last).
    int32 [N]."""
    shape = tuple(int(s) for s in shape)
    idx = grid_index(shape)
    kz = idx[:, -1]
    return ((n_slabs * kz) // shape[-1]).astype(np.int32)
