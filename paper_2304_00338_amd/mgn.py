"""Python binding of libmgn (argument marshalling only).

Every entry point of ``include/mgn.h`` is wrapped with the same name.  Host
arrays are NumPy; device buffers are torch tensors (torch supplies device
memory and the current HIP stream, nothing else).  All computation runs in
the HIP library; if ``libmgn.so`` is missing the import of any entry point
raises, there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# MGN_LIB selects another build of the same library (the host-sanitizer
# build of build_sanitized.py); by default the in-tree libmgn.so
LIB_PATH = os.environ.get("MGN_LIB") or os.path.join(HERE, "libmgn.so")

OK, ERR_ARG, ERR_RANGE, ERR_SHAPE, ERR_WORKSPACE, ERR_STATE, ERR_DEVICE, ERR_NOMEM = 0, -1, -2, -3, -4, -5, -6, -7
FP32, BF16 = 0, 1
EULER, HEUN2, MIDPOINT, HEUN3, RK4, RALSTON2, RALSTON3 = 0, 1, 2, 3, 4, 5, 6
SCHEMES = {"euler": EULER, "heun2": HEUN2, "midpoint": MIDPOINT, "heun3": HEUN3, "rk4": RK4,
           "ralston2": RALSTON2, "ralston3": RALSTON3}
PRECISIONS = {"fp32": FP32, "bf16": BF16}


class MgnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libmgn error {code}: {msg}")
        self.code = code


class Config(C.Structure):
    _fields_ = [("node_in", C.c_int32), ("edge_in", C.c_int32), ("latent", C.c_int32),
                ("out", C.c_int32), ("mp_steps", C.c_int32), ("mlp_layers", C.c_int32),
                ("ln_eps", C.c_float), ("precision", C.c_int32)]


class DGraph(C.Structure):
    _fields_ = [("n_nodes", C.c_int64), ("n_edges", C.c_int64), ("rowptr", C.c_void_p),
                ("senders", C.c_void_p), ("receivers", C.c_void_p), ("rev", C.c_void_p),
                ("tiles", C.c_void_p),
                ("n_tiles", C.c_int64), ("long_nodes", C.c_void_p), ("n_long", C.c_int64)]


class DPatch(C.Structure):
    _fields_ = [("g", DGraph), ("efeat", C.c_void_p), ("node_l2g", C.c_void_p), ("interior", C.c_void_p)]


class Adam(C.Structure):
    """mgn_adam: the paper's schedule (App. C) by default."""
    _fields_ = [("lr_start", C.c_double), ("lr_end", C.c_double), ("decay_steps", C.c_int64),
                ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double)]

    def __init__(self, lr_start=1e-3, lr_end=1e-7, decay_steps=4_000_000, beta1=0.9, beta2=0.999, eps=1e-8):
        super().__init__(lr_start, lr_end, decay_steps, beta1, beta2, eps)


_lib = None

EXPORTS = [
    "mgn_param_count", "mgn_build_graph", "mgn_graph_info", "mgn_graph_copy",
    "mgn_graph_schedule", "mgn_tile_edges", "mgn_tile_nodes", "mgn_graph_destroy",
    "mgn_partition", "mgn_extract_patch", "mgn_patch_union", "mgn_patch_copy_maps", "mgn_ctx_create",
    "mgn_ctx_destroy", "mgn_forward", "mgn_forward_noalloc", "mgn_backward", "mgn_integrate_step",
    "mgn_pec_step", "mgn_patch_step", "mgn_adam_lr", "mgn_adam_step", "mgn_train_step", "mgn_scheme_stages", "mgn_version", "mgn_last_error", "mgn_profile_enable",
    "mgn_profile_collect",
]


def lib():
    """Load libmgn.so (built in-tree); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build()")
    L = C.CDLL(LIB_PATH)
    P, i32, i64, vp = C.POINTER, C.c_int32, C.c_int64, C.c_void_p
    sig = {
        "mgn_param_count": (i64, [P(Config)]),
        "mgn_build_graph": (C.c_int, [vp, i64, i32, vp, i64, i32, P(vp)]),
        "mgn_graph_info": (C.c_int, [vp, P(i64), P(i64)]),
        "mgn_graph_copy": (C.c_int, [vp, vp, vp, vp, vp, vp]),
        "mgn_graph_schedule": (C.c_int, [vp, vp, P(i64), vp, P(i64)]),
        "mgn_tile_edges": (i32, []),
        "mgn_tile_nodes": (i32, []),
        "mgn_graph_destroy": (None, [vp]),
        "mgn_partition": (C.c_int, [vp, i64, i32, vp, vp]),
        "mgn_extract_patch": (C.c_int, [vp, vp, i32, i32, P(vp)]),
        "mgn_patch_union": (C.c_int, [vp, i32, P(vp)]),
        "mgn_patch_copy_maps": (C.c_int, [vp, vp, vp, vp, vp, P(i64)]),
        "mgn_ctx_create": (C.c_int, [P(Config), i64, i64, i32, i32, P(C.c_size_t), P(vp)]),
        "mgn_ctx_destroy": (None, [vp]),
        "mgn_forward": (C.c_int, [vp, P(DGraph), vp, vp, vp, vp, i32, vp, C.c_size_t, vp]),
        "mgn_forward_noalloc": (C.c_int, [vp, P(DGraph), vp, vp, vp, vp, vp]),
        "mgn_backward": (C.c_int, [vp, vp, vp, vp, vp]),
        "mgn_integrate_step": (C.c_int, [vp, P(DGraph), vp, i32, vp, vp, vp, vp, i32, vp, C.c_size_t, vp]),
        "mgn_pec_step": (C.c_int, [vp, P(DGraph), vp, vp, vp, vp, vp, vp, i32, vp, C.c_size_t, vp]),
        "mgn_patch_step": (C.c_int, [vp, i32, P(DPatch), vp, i32, vp, vp, vp, i64, vp, C.c_size_t, vp]),
        "mgn_adam_lr": (C.c_double, [P(Adam), i64]),
        "mgn_adam_step": (C.c_int, [P(Adam), i64, vp, vp, vp, vp, i64, vp]),
        "mgn_train_step": (C.c_int, [vp, i32, P(DPatch), vp, i32, vp, vp, vp, vp, vp, i64, vp, vp, vp, P(Adam), i64,
                                     vp, i64, vp, C.c_size_t, vp]),
        "mgn_scheme_stages": (C.c_int, [i32]),
        "mgn_version": (C.c_char_p, []),
        "mgn_last_error": (C.c_char_p, []),
        "mgn_profile_enable": (C.c_int, [vp, i32]),
        "mgn_profile_collect": (C.c_int, [vp, i32, vp, vp, vp, P(i32)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(rc):
    if rc != OK:
        raise MgnError(rc, lib().mgn_last_error().decode())
    return rc


def version():
    return lib().mgn_version().decode()


def last_error():
    return lib().mgn_last_error().decode()


def tile_edges():
    return lib().mgn_tile_edges()


def config(mp_steps, precision="fp32", ln_eps=1e-5, latent=128):
    prec = PRECISIONS[precision] if isinstance(precision, str) else int(precision)
    return Config(8, 4, latent, 4, int(mp_steps), 2, float(ln_eps), prec)


def param_count(mp_steps, latent=128):
    cfg = config(mp_steps, latent=latent)
    n = lib().mgn_param_count(C.byref(cfg))
    if n < 0:
        raise MgnError(ERR_SHAPE, last_error())
    return n


def _np(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.c_void_p)


# ------------------------------------------------------------ host graphs
class Graph:
    """Host mesh graph or patch (owns an mgn_graph handle)."""

    def __init__(self, handle, is_patch=False):
        self._h = C.c_void_p(handle)
        self.is_patch = is_patch
        n, e = C.c_int64(), C.c_int64()
        _check(lib().mgn_graph_info(self._h, C.byref(n), C.byref(e)))
        self.n_nodes, self.n_edges = n.value, e.value

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.mgn_graph_destroy(self._h)
            self._h = None

    def arrays(self):
        N, E = self.n_nodes, self.n_edges
        rowptr = np.empty(N + 1, np.int32)
        s = np.empty(E, np.int32)
        r = np.empty(E, np.int32)
        rev = np.empty(E, np.int32)
        f = np.empty((E, 4), np.float32)
        _check(lib().mgn_graph_copy(self._h, rowptr.ctypes.data, s.ctypes.data, r.ctypes.data,
                                    rev.ctypes.data, f.ctypes.data))
        return {"rowptr": rowptr, "senders": s, "receivers": r, "rev": rev, "efeat": f}

    def schedule(self):
        nt, nl = C.c_int64(), C.c_int64()
        _check(lib().mgn_graph_schedule(self._h, None, C.byref(nt), None, C.byref(nl)))
        tiles = np.empty((nt.value, 4), np.int32)
        longn = np.empty((nl.value, 4), np.int32)
        _check(lib().mgn_graph_schedule(self._h, tiles.ctypes.data, C.byref(nt),
                                        longn.ctypes.data, C.byref(nl)))
        return tiles, longn

    def patch_maps(self):
        N, E = self.n_nodes, self.n_edges
        l2g = np.empty(N, np.int32)
        hop = np.empty(N, np.int32)
        it = np.empty(N, np.uint8)
        el2g = np.empty(E, np.int64)
        ni = C.c_int64()
        _check(lib().mgn_patch_copy_maps(self._h, l2g.ctypes.data, hop.ctypes.data, it.ctypes.data,
                                         el2g.ctypes.data, C.byref(ni)))
        return {"node_l2g": l2g, "hop": hop, "interior": it, "edge_l2g": el2g,
                "n_interior": ni.value}


def build_graph(cells, pos):
    cells, pc = _np(cells, np.int32)
    pos, pp = _np(pos, np.float32)
    if cells.ndim != 2 or pos.ndim != 2:
        raise MgnError(ERR_ARG, "cells and pos must be 2-D")
    out = C.c_void_p()
    _check(lib().mgn_build_graph(pc, cells.shape[0], cells.shape[1], pp, pos.shape[0], pos.shape[1],
                                 C.byref(out)))
    return Graph(out.value)


def partition(pos, splits):
    pos, pp = _np(pos, np.float32)
    sp, spp = _np(splits, np.int32)
    part = np.empty(pos.shape[0], np.int32)
    _check(lib().mgn_partition(pp, pos.shape[0], pos.shape[1], spp, part.ctypes.data))
    return part


def extract_patch(g: Graph, part, p, k):
    part, pp = _np(part, np.int32)
    if part.shape != (g.n_nodes,):
        raise MgnError(ERR_ARG, "part must have one id per node")
    out = C.c_void_p()
    _check(lib().mgn_extract_patch(g._h, pp, int(p), int(k), C.byref(out)))
    return Graph(out.value, is_patch=True)


def patch_union(patches):
    """Disjoint union of patches as one patch-like graph (see include/mgn.h)."""
    arr = (C.c_void_p * max(1, len(patches)))(*[p._h.value for p in patches])
    out = C.c_void_p()
    _check(lib().mgn_patch_union(arr, len(patches), C.byref(out)))
    return Graph(out.value, is_patch=True)


# --------------------------------------------------------- device side
def _torch():
    import torch
    return torch


def _dptr(t, dtype=None, shape=None, name="tensor"):
    torch = _torch()
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise MgnError(ERR_ARG, f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise MgnError(ERR_ARG, f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise MgnError(ERR_ARG, f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise MgnError(ERR_ARG, f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


class DeviceGraph:
    """Device copies of a graph's CSR arrays and tile schedule."""

    def __init__(self, g: Graph, device="cuda"):
        torch = _torch()
        a = g.arrays()
        tiles, longn = g.schedule()
        dev = torch.device(device)
        self.n_nodes, self.n_edges = g.n_nodes, g.n_edges
        self.rowptr = torch.from_numpy(a["rowptr"]).to(dev)
        self.senders = torch.from_numpy(a["senders"]).to(dev)
        self.receivers = torch.from_numpy(a["receivers"]).to(dev)
        self.rev = torch.from_numpy(a["rev"]).to(dev)
        self.tiles = torch.from_numpy(tiles.reshape(-1)).to(dev)
        self.long_nodes = torch.from_numpy(longn.reshape(-1)).to(dev)
        self.efeat = torch.from_numpy(a["efeat"]).to(dev)
        self.n_tiles, self.n_long = tiles.shape[0], longn.shape[0]
        self.struct = DGraph(self.n_nodes, self.n_edges, self.rowptr.data_ptr(),
                             self.senders.data_ptr(), self.receivers.data_ptr(),
                             self.rev.data_ptr(), self.tiles.data_ptr(),
                             self.n_tiles,
                             self.long_nodes.data_ptr() if self.n_long else None, self.n_long)


class DevicePatch:
    """A patch on the device: its local graph (DeviceGraph) and the maps
    node_l2g / interior of mgn_patch_copy_maps."""

    def __init__(self, patch: Graph, device="cuda"):
        torch = _torch()
        mp = patch.patch_maps()
        self.dg = DeviceGraph(patch, device)
        self.node_l2g = torch.from_numpy(mp["node_l2g"]).to(device)
        self.interior = torch.from_numpy(mp["interior"]).to(device)
        self.n_nodes, self.n_edges, self.n_interior = patch.n_nodes, patch.n_edges, mp["n_interior"]
        self.struct = DPatch(self.dg.struct, self.dg.efeat.data_ptr(), self.node_l2g.data_ptr(),
                             self.interior.data_ptr())


class Context:
    """mgn_ctx plus a workspace tensor of the size the library asks for."""

    def __init__(self, mp_steps, max_nodes, max_edges, precision="fp32", max_stages=1,
                 save=False, ln_eps=1e-5, device="cuda", allocate=True, latent=128):
        self.cfg = config(mp_steps, precision, ln_eps, latent)
        self.mp_steps = int(mp_steps)
        self.latent = int(latent)
        ws = C.c_size_t()
        h = C.c_void_p()
        _check(lib().mgn_ctx_create(C.byref(self.cfg), int(max_nodes), int(max_edges),
                                    int(max_stages), 1 if save else 0, C.byref(ws), C.byref(h)))
        self._h = h
        self.ws_bytes = ws.value
        self.ws = None
        if allocate:
            torch = _torch()
            self.ws = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=device)

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.mgn_ctx_destroy(self._h)
            self._h = None


def mgn_forward(ctx: Context, g: DeviceGraph, params, node_in, efeat, out=None, save=False,
                stream=None):
    torch = _torch()
    N, E = g.n_nodes, g.n_edges
    if out is None:
        out = torch.empty((N, 4), dtype=torch.float32, device=node_in.device)
    _check(lib().mgn_forward(ctx._h, C.byref(g.struct), _dptr(params, torch.float32, name="params"),
                             _dptr(node_in, torch.float32, (N, 8), "node_in"),
                             _dptr(efeat, torch.float32, (E, 4), "efeat"),
                             _dptr(out, torch.float32, (N, 4), "out"), 1 if save else 0,
                             _dptr(ctx.ws, name="workspace"), ctx.ws_bytes, _stream(stream)))
    return out


NOALLOC_SCRATCH_BYTES = 128 << 20  # MGN_NOALLOC_SCRATCH_BYTES of include/mgn.h


def mgn_forward_noalloc(ctx: Context, g: DeviceGraph, params, node_in, efeat, out, stream=None):
    """mgn_forward (no saved activations) on the library's static device
    scratch instead of ctx's workspace: the context may be created with
    allocate=False; `out` must be given (nothing is allocated)."""
    torch = _torch()
    N, E = g.n_nodes, g.n_edges
    _check(lib().mgn_forward_noalloc(ctx._h, C.byref(g.struct), _dptr(params, torch.float32, name="params"),
                                     _dptr(node_in, torch.float32, (N, 8), "node_in"),
                                     _dptr(efeat, torch.float32, (E, 4), "efeat"),
                                     _dptr(out, torch.float32, (N, 4), "out"), _stream(stream)))
    return out


def mgn_backward(ctx: Context, grad_out, grad_params, grad_in=None, stream=None):
    torch = _torch()
    _check(lib().mgn_backward(ctx._h, _dptr(grad_out, torch.float32, name="grad_out"),
                              _dptr(grad_params, torch.float32, name="grad_params"),
                              _dptr(grad_in, torch.float32, name="grad_in") if grad_in is not None else None,
                              _stream(stream)))
    return grad_params


def mgn_integrate_step(ctx: Context, g: DeviceGraph, params, scheme, static, y, efeat,
                       y_next=None, save=False, stream=None):
    torch = _torch()
    N, E = g.n_nodes, g.n_edges
    sc = SCHEMES[scheme] if isinstance(scheme, str) else int(scheme)
    if y_next is None:
        y_next = torch.empty((N, 4), dtype=torch.float32, device=y.device)
    _check(lib().mgn_integrate_step(ctx._h, C.byref(g.struct), _dptr(params, torch.float32, name="params"),
                                    sc, _dptr(static, torch.float32, (N, 4), "static"),
                                    _dptr(y, torch.float32, (N, 4), "y"),
                                    _dptr(efeat, torch.float32, (E, 4), "efeat"),
                                    _dptr(y_next, torch.float32, (N, 4), "y_next"), 1 if save else 0,
                                    _dptr(ctx.ws, name="workspace"), ctx.ws_bytes, _stream(stream)))
    return y_next


def mgn_patch_step(ctx: Context, patches, params, scheme, static, y, y_next=None, stream=None):
    """One integration step of the whole mesh computed patch by patch with
    ghost refresh (see include/mgn.h); patches: list of DevicePatch."""
    torch = _torch()
    n = y.shape[0]
    sc = SCHEMES[scheme] if isinstance(scheme, str) else int(scheme)
    if y_next is None:
        y_next = torch.empty((n, 4), dtype=torch.float32, device=y.device)
    arr = (DPatch * max(1, len(patches)))(*[p.struct for p in patches])
    _check(lib().mgn_patch_step(ctx._h, len(patches), arr, _dptr(params, torch.float32, name="params"), sc,
                                _dptr(static, torch.float32, (n, 4), "static"), _dptr(y, torch.float32, (n, 4), "y"),
                                _dptr(y_next, torch.float32, (n, 4), "y_next"), n,
                                _dptr(ctx.ws, name="workspace"), ctx.ws_bytes, _stream(stream)))
    return y_next


def mgn_adam_lr(adam, k):
    return lib().mgn_adam_lr(C.byref(adam), int(k))


def mgn_adam_step(adam, k, params, grad, m, v, stream=None):
    """The k-th Adam update of params in place (see include/mgn.h)."""
    torch = _torch()
    n = params.numel()
    _check(lib().mgn_adam_step(C.byref(adam), int(k), _dptr(params, torch.float32, name="params"),
                               _dptr(grad, torch.float32, (n,), "grad"), _dptr(m, torch.float32, (n,), "m"),
                               _dptr(v, torch.float32, (n,), "v"), n, _stream(stream)))


def mgn_train_step(ctx: Context, patches, params, scheme, static, y, y_target, noise, grad, m, v, adam, k,
                   n_loss_nodes=None, noise_std=None, loss=None, stream=None):
    """One patch-training step (see include/mgn.h); returns the device loss
    (a 1-element tensor)."""
    torch = _torch()
    n = y.shape[0]
    sc = SCHEMES[scheme] if isinstance(scheme, str) else int(scheme)
    if loss is None:
        loss = torch.zeros(1, dtype=torch.float32, device=y.device)
    if n_loss_nodes is None:
        n_loss_nodes = sum(int(p.n_interior) for p in patches)
    sd = None if noise_std is None else (C.c_float * 4)(*[float(x) for x in noise_std])
    arr = (DPatch * max(1, len(patches)))(*[p.struct for p in patches])
    npar = params.numel()
    _check(lib().mgn_train_step(ctx._h, len(patches), arr, _dptr(params, torch.float32, name="params"), sc,
                                _dptr(static, torch.float32, (n, 4), "static"), _dptr(y, torch.float32, (n, 4), "y"),
                                _dptr(y_target, torch.float32, (n, 4), "y_target"),
                                _dptr(noise, torch.float32, (n, 4), "noise") if noise is not None else None,
                                C.cast(sd, C.c_void_p) if sd is not None else None, int(n_loss_nodes),
                                _dptr(grad, torch.float32, (npar,), "grad"), _dptr(m, torch.float32, (npar,), "m"),
                                _dptr(v, torch.float32, (npar,), "v"), C.byref(adam), int(k),
                                _dptr(loss, torch.float32, (1,), "loss"), n,
                                _dptr(ctx.ws, name="workspace"), ctx.ws_bytes, _stream(stream)))
    return loss


def mgn_pec_step(ctx: Context, g: DeviceGraph, params, static, y, khist, efeat, first=False,
                 y_next=None, stream=None):
    """One predict-evaluate-correct inference step; khist [2][N][4] is the
    derivative history, updated in place (see include/mgn.h)."""
    torch = _torch()
    N, E = g.n_nodes, g.n_edges
    if y_next is None:
        y_next = torch.empty((N, 4), dtype=torch.float32, device=y.device)
    _check(lib().mgn_pec_step(ctx._h, C.byref(g.struct), _dptr(params, torch.float32, name="params"),
                              _dptr(static, torch.float32, (N, 4), "static"),
                              _dptr(y, torch.float32, (N, 4), "y"),
                              _dptr(khist, torch.float32, (2, N, 4), "khist"),
                              _dptr(efeat, torch.float32, (E, 4), "efeat"),
                              _dptr(y_next, torch.float32, (N, 4), "y_next"), 1 if first else 0,
                              _dptr(ctx.ws, name="workspace"), ctx.ws_bytes, _stream(stream)))
    return y_next


def mgn_profile_enable(ctx: Context, enable=True):
    _check(lib().mgn_profile_enable(ctx._h, 1 if enable else 0))


def mgn_profile_collect(ctx: Context, max_kernels=32):
    """{kernel kind: (total_ms, launches)} since the last collect."""
    names = C.create_string_buffer(32 * max_kernels)
    ms = np.zeros(max_kernels, np.float64)
    cnt = np.zeros(max_kernels, np.int64)
    n = C.c_int32()
    _check(lib().mgn_profile_collect(ctx._h, max_kernels, names, ms.ctypes.data, cnt.ctypes.data,
                                     C.byref(n)))
    out = {}
    for k in range(min(n.value, max_kernels)):
        nm = names.raw[32 * k:32 * k + 32].split(b"\0")[0].decode()
        out[nm] = (float(ms[k]), int(cnt[k]))
    return out


def scheme_stages(scheme):
    sc = SCHEMES[scheme] if isinstance(scheme, str) else int(scheme)
    n = lib().mgn_scheme_stages(sc)
    if n < 0:
        raise MgnError(n, last_error())
    return n


# short aliases
forward = mgn_forward
backward = mgn_backward
integrate_step = mgn_integrate_step
