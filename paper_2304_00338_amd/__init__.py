"""MI355X (gfx950) MeshGraphNets message-passing library: HIP kernels behind
the C ABI in include/mgn.h, with a thin ctypes binding in ``mgn``."""
from . import mgn  # noqa: F401
from .mgn import (Context, DeviceGraph, Graph, MgnError, build_graph,  # noqa: F401
                  extract_patch, integrate_step, mgn_backward, mgn_forward,
                  mgn_integrate_step, partition)
