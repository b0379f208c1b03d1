"""Benchmark of the MGN message-passing hot path on one MI355X.

One step = one explicit-Euler MGN call (encode, 15 message-passing steps,
decode) on a 3D mesh patch plus its full reverse mode, with the loss on the
subdomain nodes only (Sec. 2.1 update rule; Sec. 2.2 patches and
condition 2).  The workload is slab 8 of 16 of a jittered 146^3 Kuhn
tetrahedral mesh with a 15-hop ghost zone: 852,640 nodes, 11,674,318
directed edges, latent 128, bf16 MFMA operands with fp32 accumulation.

Prints one JSON line: MP-step edges/s (fwd+bwd) = E * m / step time, plus
the roofline of the dominant kernel (average launch time measured with HIP
events on the library's stream during the timed region) and the CPU
oracle's throughput on a bounded sample of the same kind of mesh.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
D = 128


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_bytes(kind, N, E, n_tiles, se, have_ebar=True, write_e=True):
    """Algorithmic HBM bytes of one launch: every input read once and every
    output written once (P holds two fp32 node products, the latents of the
    edge stream have se bytes per element)."""
    if kind == "edge_fwd":
        return (E * (D * se * (2 if write_e else 1) + 4)
                + N * (2 * D * 4 + D * 4 + 4) + n_tiles * 16)
    if kind == "edge_bwd":
        return (E * (D * se + (D * 4 if have_ebar else 0) + D * 4 + D * se + 4)
                + N * (2 * D * 4 + D * 4 + D * 4 + 4) + n_tiles * 16)
    if kind == "node_srcsum":
        return E * (D * se + 4) + N * (4 + 4 * D * 4)
    if kind == "node_fwd":
        return N * (D * 4 * 3 + 2 * D * 4)
    if kind == "node_bwd":
        return N * (D * 4 * 5)
    return None


def setup(args):
    import torch
    import synth
    from paper_2304_00338_amd import mgn
    t0 = time.time()
    n = args.grid
    shape = (n, n, n)
    M = synth.mesh(shape, 0)
    log(f"mesh {shape}: {M['pos'].shape[0]} nodes, {M['cells'].shape[0]} cells ({time.time()-t0:.1f}s)")
    g = mgn.build_graph(M["cells"], M["pos"])
    log(f"graph: {g.n_edges} directed edges ({time.time()-t0:.1f}s)")
    part = synth.slab_part(shape, args.slabs)
    pt = mgn.extract_patch(g, part, args.slab, args.ghost)
    mp = pt.patch_maps()
    log(f"patch {args.slab}: {pt.n_nodes} nodes ({mp['n_interior']} interior), {pt.n_edges} edges "
        f"({time.time()-t0:.1f}s)")
    del g
    dg = mgn.DeviceGraph(pt)
    l2g = mp["node_l2g"]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    st = dev(M["onehot"][l2g])
    y = dev(M["states"][l2g])
    params = dev(synth.xavier_params(args.mp_steps, 0))
    # loss on the subdomain nodes only (condition 2): linear loss seed
    w = synth.loss_weights(pt.n_nodes, 0) * mp["interior"][:, None]
    gout = dev(w)
    ctx = mgn.Context(args.mp_steps, pt.n_nodes, pt.n_edges, args.precision, max_stages=1, save=True)
    log(f"workspace {ctx.ws_bytes / 2**30:.1f} GiB ({time.time()-t0:.1f}s)")
    return {"pt": pt, "mp": mp, "dg": dg, "st": st, "y": y, "params": params, "gout": gout,
            "ctx": ctx, "gp": torch.zeros_like(params), "ynext": torch.empty_like(y)}


def step(S, mgn, fwd_only=False):
    S["gp"].zero_()
    mgn.mgn_integrate_step(S["ctx"], S["dg"], S["params"], "euler", S["st"], S["y"], S["dg"].efeat,
                           S["ynext"], save=not fwd_only)
    if not fwd_only:
        mgn.mgn_backward(S["ctx"], S["gout"], S["gp"])


def cpu_baseline(args):
    """The fp64 oracle, as it stands, on a bounded sample: one MGN call
    (15 MP steps) forward and backward on a jittered Kuhn mesh of the same
    kind (16^3 grid)."""
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    shape = (args.cpu_grid,) * 3
    M = synth.mesh(shape, 0)
    g = O.build_graph(M["cells"], M["pos"])
    P = synth.xavier_params(args.mp_steps, 0)
    w = synth.loss_weights(g.n_nodes, 0)
    t0 = time.time()
    _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, args.mp_steps, keep=True)
    O.mgn_backward(tape, w)
    dt = time.time() - t0
    return {"value": g.n_edges * args.mp_steps / dt, "unit": "edges/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"one fp64 MGN call fwd+bwd, {args.mp_steps} MP steps, on a jittered "
                      f"{shape[0]}^3 Kuhn mesh ({g.n_nodes} nodes, {g.n_edges} edges): {dt:.1f}s",
            "seconds": dt}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--precision", default="bf16")
    ap.add_argument("--grid", type=int, default=146)
    ap.add_argument("--slabs", type=int, default=16)
    ap.add_argument("--slab", type=int, default=8)
    ap.add_argument("--ghost", type=int, default=15)
    ap.add_argument("--mp-steps", type=int, default=15)
    ap.add_argument("--cpu-grid", type=int, default=13)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibrate", action="store_true",
                    help="only run a plain device copy of known size (for counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the patch-parallel design is described in DESIGN.md); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2304_00338_amd import mgn
    mgn.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibrate:
        n = 1 << 28  # 1 GiB of fp32
        a = torch.ones(n, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 3}))
        return

    S = setup(args)
    N, E, m = S["pt"].n_nodes, S["pt"].n_edges, args.mp_steps
    ctx = S["ctx"]
    for _ in range(args.warmup):
        step(S, mgn)
    torch.cuda.synchronize()

    # forward-only throughput (context information)
    t0 = time.perf_counter()
    for _ in range(max(1, args.steps)):
        step(S, mgn, fwd_only=True)
    torch.cuda.synchronize()
    fwd_ms = (time.perf_counter() - t0) * 1e3 / max(1, args.steps)

    # timed region: K fwd+bwd steps, per-kernel HIP events on the same stream
    mgn.mgn_profile_enable(ctx, True)
    mgn.mgn_profile_collect(ctx)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(S, mgn)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    prof = mgn.mgn_profile_collect(ctx)
    mgn.mgn_profile_enable(ctx, False)

    kern_ms = {k: v[0] / args.steps for k, v in prof.items()}
    dom = max(prof, key=lambda k: prof[k][0])
    tot, cnt = prof[dom]
    avg_ms = tot / cnt
    se = 2 if args.precision == "bf16" else 4
    n_tiles = S["dg"].n_tiles
    if dom == "edge_bwd":
        per = [kernel_bytes(dom, N, E, n_tiles, se, have_ebar=(l < m - 1)) for l in range(m)]
    elif dom == "edge_fwd":
        per = [kernel_bytes(dom, N, E, n_tiles, se, write_e=(l < m - 1)) for l in range(m)]
    else:
        per = [kernel_bytes(dom, N, E, n_tiles, se)]
    bytes_per_launch = float(np.mean(per)) if per[0] is not None else None
    roof = None
    if bytes_per_launch is not None:
        ach = bytes_per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None, "kernel": dom,
                "avg_launch_ms": round(avg_ms, 4), "launches_per_step": cnt // args.steps,
                "algorithmic_bytes_per_launch": int(bytes_per_launch)}

    value = E * m / (ms * 1e-3)
    out = {
        "metric": "MP-step edges/sec (fwd+bwd) on 3D mesh patch; % of MFMA / HBM roofline",
        "value": round(value, 1), "unit": "edges/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.precision, "data": "synthetic",
        "config": {
            "workload": (f"patch {args.slab} of {args.slabs} z-slabs of a jittered {args.grid}^3 "
                         f"Kuhn-tetrahedral mesh, {args.ghost}-hop ghost zone, {m} MP steps, "
                         f"latent 128, one Euler step fwd+bwd, loss on subdomain nodes"),
            "n_nodes": N, "n_edges": E, "n_interior": int(S["mp"]["n_interior"]),
            "mp_steps": m, "latent": 128, "precision": args.precision, "parallelism": "none"},
        "roofline": roof,
        "fwd_edges_per_s": round(E * m / (fwd_ms * 1e-3), 1),
        "fwd_ms_per_call": round(fwd_ms, 3),
        "mgn_calls_per_s_fwd": round(1e3 / fwd_ms, 3),
        "mgn_calls_per_s_fwdbwd": round(1e3 / ms, 3),
        "kernel_ms_per_step": {k: round(v, 3) for k, v in sorted(kern_ms.items(), key=lambda x: -x[1])},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
