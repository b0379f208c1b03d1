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


# Executed bf16 MFMA work per edge of the bf16 edge kernels (16x16x32 MFMAs
# at 16,384 flop each over a 16-row block, counted as issued, select
# operands included): the edge forward runs the K = 128 products of W1e e
# and W2 a1, 16 + 8 selection MFMAs for P_s + P_r and e + m per 16 rows; the
# backward the three 128 x 128 products W2 a1 (recomputed z2), W2^T dz2 and
# W1e^T zbar.
MFMA_FLOP_PER_EDGE = {"edge_fwd": 2 * 128 * 128 * 2 + 24 * 16384 // 16,
                      "edge_bwd": 3 * 2 * 128 * 128}
MFMA_PEAK_BF16_TFLOPS = 2500.0
MFMA_PEAK_FP32_TFLOPS = 157.3


def edge_bwd_split_roofline(prec, D, N, E, m, avg_ms):
    """Position of the edge backward at latent width D (one launch per MP
    block) against both roofs: algorithmic bytes and executed MFMA flop per
    launch, each divided by the average launch time.
    fp32 (feature-split kernel): per edge e, the incoming edge gradient (not
    in the last block), the outgoing one and z-bar (fp32), sender / receiver
    ids; per node P, the gathered aggregate gradient and R; 5 products of
    D x D per edge (the recomputed W1e e and W2 a1, W2^T dz2, W1e^T zbar and
    the dW2 accumulation).
    bf16 (row-per-wave kernel): per edge the saved a1, the incoming edge
    gradient (not in the last block), the outgoing one, zbar and dz2 (bf16),
    the receiver id; per node the gathered aggregate gradient and R (fp32);
    3 products of D x D per edge (W2 a1, W2^T dz2, W1e^T zbar)."""
    if prec == "bf16":
        per_edge = [D * 2 + (D * 2 if l < m - 1 else 0) + 3 * D * 2 + 4 for l in range(m)]
        per_node = 2 * D * 4
        flop = 6.0 * D * D * E
        peak = MFMA_PEAK_BF16_TFLOPS
    else:
        per_edge = [D * 4 + (D * 4 if l < m - 1 else 0) + D * 4 + D * 4 + 8 for l in range(m)]
        per_node = 2 * D * 4 + D * 4 + D * 4
        flop = 10.0 * D * D * E
        peak = MFMA_PEAK_FP32_TFLOPS
    nbytes = float(np.mean(per_edge)) * E + N * per_node
    gbs = nbytes / (avg_ms * 1e-3) / 1e9
    tfs = flop / (avg_ms * 1e-3) / 1e12
    return {"kernel": "edge_bwd", "avg_launch_ms": round(avg_ms, 4),
            "hbm": {"algorithmic_bytes_per_launch": int(nbytes), "achieved_gbs": round(gbs, 1),
                    "frac": round(gbs / HBM_PEAK_GBS, 4)},
            "mfma": {"flop_per_launch": int(flop), "achieved_tflops": round(tfs, 1), "peak_tflops": peak,
                     "frac": round(tfs / peak, 4)}}


def kernel_bytes(kind, N, E, n_tiles, prec, have_ebar=True, write_e=True, keep_a1=True):
    """Algorithmic HBM bytes of one launch of the kernels this build runs:
    every input read once and every output written once.  In bf16 the edge
    latents, their gradient stream, node products P ([N][2D]) and the a1 /
    zbar / dz streams are 2 bytes per element; node latents, aggregates and
    node gradients are fp32 throughout."""
    se = 2 if prec == "bf16" else 4
    row, frow = D * se, D * 4
    erow = row if prec == "bf16" else frow  # edge-gradient stream
    tiles = n_tiles * 16 + 4 * (N + 1)
    bf = prec == "bf16"
    if kind == "edge_fwd":
        return (E * (row + 8 + (row if write_e else 0) + (row if keep_a1 and bf else 0))
                + N * (2 * row + frow) + tiles)
    if kind == "edge_bwd":
        if bf:  # from the saved a1: reads a1, ebar_in, aggbar; writes ebar_out, zbar, dz2, R
            return (E * (row + (erow if have_ebar else 0) + 4 + erow + 2 * row)
                    + N * (frow + frow) + tiles)
        return (E * (row + (frow if have_ebar else 0) + frow + row + 8)
                + N * (2 * row + frow + frow) + tiles)
    if kind == "wgrad":
        return E * row * (4 if bf else 2)
    if kind == "node_srcsum":
        return E * (row + 4) + N * (4 + 4 * frow)
    if kind == "node_fwd":
        return N * 3 * frow if bf else N * (3 * frow + 2 * row)
    if kind == "emit_p":
        return N * (frow + 2 * row)
    if kind == "node_bwd":
        return N * (5 * frow + (3 * row if bf else 0))
    if kind == "wgrad_node":
        return N * (2 * frow + 3 * row)
    if kind == "edge_enc":
        return E * (16 + row)
    if kind == "edge_enc_bwd":
        return E * (16 + erow)
    if kind == "node_enc":
        return N * (32 + frow + 2 * row)
    if kind == "decoder":
        return N * (frow + 16)
    return None


def step_bytes(kind, N, E, n_tiles, prec, m):
    """Algorithmic bytes of every launch of `kind` in one fwd+bwd step (one
    saving MGN call and its backward), or None."""
    if kind == "edge_fwd":
        return sum(kernel_bytes(kind, N, E, n_tiles, prec, write_e=(l < m - 1)) for l in range(m))
    if kind == "edge_bwd":
        return sum(kernel_bytes(kind, N, E, n_tiles, prec, have_ebar=(l < m - 1)) for l in range(m))
    if kind == "emit_p":
        return (m - 1) * kernel_bytes(kind, N, E, n_tiles, prec)
    if kind in ("wgrad", "node_srcsum", "node_fwd", "node_bwd", "wgrad_node"):
        return m * kernel_bytes(kind, N, E, n_tiles, prec)
    b = kernel_bytes(kind, N, E, n_tiles, prec)
    return b


# Device sources of each profiled kernel: its own file and the device
# headers it includes (launch.hpp only declares host launchers).
KERNEL_SOURCES = {"edge_bwd": ("edge_rows.hip", "rows_common.hpp", "dev_common.hpp")}
# The kernel symbol a profiled kernel kind runs as on the benchmark patch
# (bf16): the fp32 kernel of the same kind must not be taken for it.
KERNEL_SYMBOL = {"edge_bwd": "k_edge_bwd_rows", "edge_fwd": "k_edge_fwd_rows"}


def source_digest(kernel="edge_bwd"):
    """Digest of a kernel's device sources: counter-derived traffic is
    reported only for the kernel sources it was measured on."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2304_00338_amd", "csrc")
    for f in KERNEL_SOURCES[kernel]:
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_file(kernel):
    return os.path.join(ROOT, "profiles", f"{kernel}_c3_patch_traffic.json")


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None when it is absent or the kernel sources changed since."""
    try:
        t = json.load(open(traffic_file(kernel)))
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest(kernel):
        return None
    return t.get("bytes_per_launch")


def summarize_profile(d, kernel):
    """Summary of a profiling directory made by the commands listed in the
    output (kernel trace, FETCH_SIZE and WRITE_SIZE passes over one bench
    step, and the same two counters over a 1 GiB device copy): markdown on
    stdout, and the traffic of `kernel` written next to the summaries."""
    import glob
    import re
    import sqlite3

    def db(sub):
        f = glob.glob(os.path.join(d, sub, "*_results.db"))
        return sqlite3.connect(f[0]) if f else None

    def short(n):
        m = re.search(r"(k_[a-z0-9_]+?)(?:I|<|\()(.*)", n) or re.search(r"(k_[a-z0-9_]+)", n)
        if not m:
            return "copy" if "copy" in n.lower() else n[:40]
        t = re.match(r"<([^>]*)>", n[m.end(1):])
        if not t:
            return m.group(1)
        args = [a.strip() for a in t.group(1).split(",")]
        args[0] = {"1": "bf16", "0": "fp32"}.get(args[0], args[0])
        return m.group(1) + "<" + ", ".join(args) + ">"

    def pmc(con, counter):
        agg = {}
        for n, v in con.execute("select kernel_name, value from counters_collection where counter_name=?",
                                (counter,)):
            agg.setdefault(short(n), []).append(v)
        return {k: sum(v) / len(v) for k, v in agg.items()}

    tr = db("prof_trace")
    rows = list(tr.execute("select name, total_calls, total_duration, average, percentage from top_kernels"))
    fetch, write = pmc(db("prof_fetch"), "FETCH_SIZE"), pmc(db("prof_write"), "WRITE_SIZE")
    cf, cw = pmc(db("prof_copyf"), "FETCH_SIZE"), pmc(db("prof_copyw"), "WRITE_SIZE")
    copy_bytes = float(1 << 30)
    kf = max((k for k in cf if k == "copy" or "copy" in k), key=lambda k: cf[k])
    kw = max((k for k in cw if k == "copy" or "copy" in k), key=lambda k: cw[k])
    sf, sw = copy_bytes / (cf[kf] * 1024), copy_bytes / (cw[kw] * 1024)
    print("| kernel | calls | total ms | avg ms | % | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM GB (scaled) |")
    print("|---|---|---|---|---|---|---|---|")
    for n, c, tot, avg, pct in rows:
        k = short(n)
        f, w = fetch.get(k), write.get(k)
        hbm = f"{(f * sf + w * sw) * 1024 / 1e9:.2f}" if f is not None and w is not None else ""
        print(f"| {k} | {c} | {tot / 1e3:.3f} | {avg / 1e3:.4f} | {pct:.1f} | "
              f"{'' if f is None else f'{f:,.0f}'} | {'' if w is None else f'{w:,.0f}'} | {hbm} |")
    print(f"\nCopy calibration (1 GiB read and written): FETCH_SIZE {cf[kf]:,.1f} KiB -> scale {sf:.3f}; "
          f"WRITE_SIZE {cw[kw]:,.1f} KiB -> scale {sw:.3f}")
    if os.path.isdir(os.path.join(d, "prof_mfma")):
        mops, busy = pmc(db("prof_mfma"), "SQ_INSTS_VALU_MFMA_MOPS_BF16"), pmc(db("prof_mfma"), "SQ_VALU_MFMA_BUSY_CYCLES")
        avg_ms = {short(n): avg / 1e3 for n, c, tot, avg, pct in rows}
        print("\n| kernel | bf16 MFMA TFLOP per launch (counter) | TFLOP/s at the traced avg | % of 2.5 PFLOP/s |")
        print("|---|---|---|---|")
        for n, *_ in rows:
            k = short(n)
            if mops.get(k):
                tf = mops[k] * 512 / 1e12
                rate = tf / (avg_ms[k] * 1e-3)
                print(f"| {k} | {tf:.3f} | {rate:.0f} | {100 * rate / MFMA_PEAK_BF16_TFLOPS:.1f} |")
    sym = KERNEL_SYMBOL.get(kernel, "k_" + kernel)
    k = next((short(n) for n, *_ in rows if short(n) == sym), None)
    if k is not None and k in fetch and k in write:
        out = {"kernel": kernel, "profiled_as": k, "source_digest": source_digest(kernel),
               "fetch_kib_per_launch": fetch[k], "write_kib_per_launch": write[k],
               "fetch_scale": sf, "write_scale": sw,
               "bytes_per_launch": (fetch[k] * sf + write[k] * sw) * 1024}
        with open(traffic_file(kernel), "w") as fh:
            json.dump(out, fh, indent=1)
        print(f"\n{k}: {out['bytes_per_launch'] / 1e9:.2f} GB of HBM traffic per launch "
              f"(written to {os.path.relpath(traffic_file(kernel), ROOT)})")


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
            "ctx": ctx, "gp": torch.zeros_like(params), "ynext": torch.empty_like(y), "mesh": M, "g": g}


def c4_rollout(S, args, steps=10):
    """Whole-mesh inference rollout (the full 146^3 mesh, bf16, no saved
    activations): `steps` explicit-Euler MGN calls after one warm-up call."""
    import torch
    from paper_2304_00338_amd import mgn
    M, g = S["mesh"], S["g"]
    dg = mgn.DeviceGraph(g)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    st, y = dev(M["onehot"]), dev(M["states"])
    ctx = mgn.Context(args.mp_steps, g.n_nodes, g.n_edges, args.precision, max_stages=1)
    y = mgn.mgn_integrate_step(ctx, dg, S["params"], "euler", st, y, dg.efeat)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        y = mgn.mgn_integrate_step(ctx, dg, S["params"], "euler", st, y, dg.efeat)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    ok = bool(torch.isfinite(y).all().item())
    y_whole = y
    del ctx, dg
    res = {"workload": f"whole {args.grid}^3 mesh, {steps} explicit-Euler MGN calls, {args.mp_steps} MP steps, "
                       f"no saved activations", "n_nodes": g.n_nodes, "n_edges": g.n_edges,
           "ms_per_call": round(dt * 1e3, 3), "mgn_calls_per_s": round(1.0 / dt, 3),
           "fwd_edges_per_s": round(g.n_edges * args.mp_steps / dt, 1), "finite": ok}
    # the same rollout computed patch by patch (ghost rows refreshed from
    # their owners every step)
    import synth
    part = synth.slab_part((args.grid,) * 3, args.slabs)
    patches = [mgn.DevicePatch(mgn.extract_patch(g, part, p, args.ghost)) for p in range(args.slabs)]
    ctx = mgn.Context(args.mp_steps, max(p.n_nodes for p in patches), max(p.n_edges for p in patches),
                      args.precision, max_stages=1)
    y = mgn.mgn_patch_step(ctx, patches, S["params"], "euler", st, dev(M["states"]))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        y = mgn.mgn_patch_step(ctx, patches, S["params"], "euler", st, y)
    torch.cuda.synchronize()
    dtp = (time.perf_counter() - t0) / steps
    pe = sum(p.n_edges for p in patches)
    res["patch_decomposed"] = {
        "workload": f"{args.slabs} z-slab patches, {args.ghost}-hop ghost zones, ghost refresh every step",
        "patch_edges": pe, "redundancy": round(pe / g.n_edges, 3), "ms_per_step": round(dtp * 1e3, 3),
        "equals_whole_mesh": bool(torch.equal(y, y_whole))}
    del ctx, patches
    return res


def c3_relabelled(S, args, reps=3, seed=7):
    """The benchmark's fwd+bwd step on the same patch of the same mesh with
    the mesh's nodes relabelled by a seeded random permutation, so the
    patch's node order (and its gathers) lose the grid's locality: the
    worst case for the sender gathers and node-product reads."""
    import torch
    import synth
    from paper_2304_00338_amd import mgn
    M, n = S["mesh"], args.grid
    nn = M["pos"].shape[0]
    perm = np.random.default_rng(seed).permutation(nn).astype(np.int64)  # old id -> new id
    inv = np.argsort(perm)                                               # new id -> old id
    g2 = mgn.build_graph(perm[M["cells"]], M["pos"][inv])
    part = synth.slab_part((n, n, n), args.slabs)[inv]
    pt = mgn.extract_patch(g2, part, args.slab, args.ghost)
    mp = pt.patch_maps()
    old = inv[mp["node_l2g"]]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    R = dict(S)
    R.update({"dg": mgn.DeviceGraph(pt), "st": dev(M["onehot"][old]), "y": dev(M["states"][old]),
              "gout": dev(synth.loss_weights(pt.n_nodes, 0) * mp["interior"][:, None])})
    R["ynext"] = torch.empty_like(R["y"])
    step(R, mgn)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        step(R, mgn)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    res = {"workload": f"the benchmark patch with the mesh's nodes relabelled by a seeded random permutation "
                       f"(seed {seed})", "n_nodes": pt.n_nodes, "n_edges": pt.n_edges,
           "ms_per_step": round(dt * 1e3, 3),
           "mp_edges_per_s_fwdbwd": round(pt.n_edges * args.mp_steps / dt, 1)}
    del R, g2, pt
    return res


def step(S, mgn, fwd_only=False):
    S["gp"].zero_()
    mgn.mgn_integrate_step(S["ctx"], S["dg"], S["params"], "euler", S["st"], S["y"], S["dg"].efeat,
                           S["ynext"], save=not fwd_only)
    if not fwd_only:
        mgn.mgn_backward(S["ctx"], S["gout"], S["gp"])


def train_steps(S, args, reps=3):
    """The patch-training step on the benchmark patch: noisy input (the
    paper's 3D noise levels), one Euler step with saved activations, masked
    MSE on the subdomain nodes, backward, Adam (paper schedule)."""
    import torch
    import synth
    from paper_2304_00338_amd import mgn
    M = S["mesh"]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    patch = mgn.DevicePatch(S["pt"])
    st, y = dev(M["onehot"]), dev(M["states"])
    tgt, nz = dev(synth.next_states(M["states"], 0)), dev(synth.standard_noise(M["states"].shape[0], 0))
    params = S["params"].clone()
    grad, m, v = torch.zeros_like(params), torch.zeros_like(params), torch.zeros_like(params)
    adam = mgn.Adam()
    loss = mgn.mgn_train_step(S["ctx"], [patch], params, "euler", st, y, tgt, nz, grad, m, v, adam, 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(2, 2 + reps):
        loss = mgn.mgn_train_step(S["ctx"], [patch], params, "euler", st, y, tgt, nz, grad, m, v, adam, k)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    return {"workload": "one patch per step (the benchmark patch), Euler, input noise, masked MSE, Adam",
            "ms_per_step": round(dt * 1e3, 3), "steps_per_s": round(1.0 / dt, 3),
            "loss_finite": bool(np.isfinite(loss.item()))}


def paper_3d_train(S, args, n_patches=32, k=6, m=3, reps=3):
    """The paper's 3D training configuration (App. C) on one GPU: the mesh split
    into 12 x 12 x 15 subdomains, 32 of them sampled per step (the effective
    batch of 32 patches), ghost depth k = 2m so that Heun's two stages are
    exact on each patch, latent 150, m = 3 MP steps; one training step =
    input noise, one H2 step fwd+bwd per patch, masked MSE, gradients summed
    over the patches, Adam.  The 32 patches run as one disjoint-union graph
    (one launch per kernel); the same step over the list of patches (one
    launch per kernel and patch) is timed beside it."""
    import torch
    import synth
    from paper_2304_00338_amd import mgn
    M, g = S["mesh"], S["g"]
    part = mgn.partition(M["pos"], (12, 12, 15))
    ids = np.random.default_rng(0).choice(int(part.max()) + 1, n_patches, replace=False)
    hp = [mgn.extract_patch(g, part, int(p), k) for p in ids]
    un = mgn.patch_union(hp)
    batches = {"union": [mgn.DevicePatch(un)], "list": [mgn.DevicePatch(p) for p in hp]}
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    st, y = dev(M["onehot"]), dev(M["states"])
    tgt, nz = dev(synth.next_states(M["states"], 1)), dev(synth.standard_noise(M["states"].shape[0], 1))
    pe = un.n_edges
    res = {"workload": (f"{n_patches} of the 12x12x15 subdomains of the {args.grid}^3 mesh per step as one "
                        f"disjoint-union graph, {k}-hop ghost zones, latent 150, {m} MP steps, Heun 2 fwd+bwd, "
                        f"noise, masked MSE, Adam"),
           "patch_nodes": un.n_nodes, "patch_edges": pe, "interior_nodes": int(un.patch_maps()["n_interior"])}
    for prec in args.paper3d_precs.split(","):
        r = {}
        for mode in ("union", "list"):
            patches = batches[mode]
            params = dev(synth.xavier_params(m, 1, 150))
            ctx = mgn.Context(m, max(p.n_nodes for p in patches), max(p.n_edges for p in patches), prec,
                              max_stages=2, save=True, latent=150)
            grad, mm, vv = torch.zeros_like(params), torch.zeros_like(params), torch.zeros_like(params)
            adam = mgn.Adam()
            loss = mgn.mgn_train_step(ctx, patches, params, "heun2", st, y, tgt, nz, grad, mm, vv, adam, 1)
            torch.cuda.synchronize()
            mgn.mgn_profile_enable(ctx, True)
            mgn.mgn_profile_collect(ctx)
            t0 = time.perf_counter()
            for it in range(2, 2 + reps):
                loss = mgn.mgn_train_step(ctx, patches, params, "heun2", st, y, tgt, nz, grad, mm, vv, adam, it)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / reps
            prof = mgn.mgn_profile_collect(ctx)
            mgn.mgn_profile_enable(ctx, False)
            if mode == "union":
                eb = prof.get("edge_bwd")
                if eb:
                    r["edge_bwd_roofs"] = edge_bwd_split_roofline(prec, 160, un.n_nodes, pe, m, eb[0] / eb[1])
                r.update({"ms_per_step": round(dt * 1e3, 3), "steps_per_s": round(1.0 / dt, 3),
                          "mp_edges_per_s_fwdbwd": round(pe * m * 2 / dt, 1),
                          "kernel_ms_per_step": {kk: round(v[0] / reps, 3)
                                                 for kk, v in sorted(prof.items(), key=lambda x: -x[1][0])},
                          "loss_finite": bool(np.isfinite(loss.item()))})
            else:
                r["ms_per_step_patch_list"] = round(dt * 1e3, 3)
            del ctx
        res[prec] = r
    del batches
    return res


def integrator_steps(S, args, reps=3):
    """Forward-only time of one integration step of each scheme on the
    patch (no saved activations), and of one predict-evaluate-correct step."""
    import torch
    from paper_2304_00338_amd import mgn
    pt = S["pt"]
    ctx = mgn.Context(args.mp_steps, pt.n_nodes, pt.n_edges, args.precision, max_stages=4)
    out = {}
    for sc in ("euler", "heun2", "midpoint", "ralston2", "heun3", "ralston3", "rk4"):
        mgn.mgn_integrate_step(ctx, S["dg"], S["params"], sc, S["st"], S["y"], S["dg"].efeat, S["ynext"])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            mgn.mgn_integrate_step(ctx, S["dg"], S["params"], sc, S["st"], S["y"], S["dg"].efeat, S["ynext"])
        torch.cuda.synchronize()
        out[sc] = round((time.perf_counter() - t0) * 1e3 / reps, 3)
    kh = torch.zeros((2, pt.n_nodes, 4), dtype=torch.float32, device="cuda")
    y = mgn.mgn_pec_step(ctx, S["dg"], S["params"], S["st"], S["y"], kh, S["dg"].efeat, first=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        y = mgn.mgn_pec_step(ctx, S["dg"], S["params"], S["st"], y, kh, S["dg"].efeat)
    torch.cuda.synchronize()
    out["pec"] = round((time.perf_counter() - t0) * 1e3 / reps, 3)
    del ctx
    return out


def cpu_baseline(args, min_seconds=10.0, max_calls=50):
    """The fp64 oracle, as it stands, on a bounded sample: MGN calls (15 MP
    steps) forward and backward on a jittered Kuhn mesh of the same kind
    (13^3 grid), repeated until at least min_seconds of CPU work."""
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
    calls = 0
    t0 = time.time()
    while calls < max_calls and (calls == 0 or time.time() - t0 < min_seconds):
        _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, args.mp_steps, keep=True)
        O.mgn_backward(tape, w)
        del tape
        calls += 1
    dt = time.time() - t0
    return {"value": g.n_edges * args.mp_steps * calls / dt, "unit": "edges/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{calls} fp64 MGN calls fwd+bwd, {args.mp_steps} MP steps, on a jittered "
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
    ap.add_argument("--no-c4", action="store_true", help="skip the whole-mesh rollout measurement")
    ap.add_argument("--no-paper3d", action="store_true", help="skip the latent-150 3D training-step measurement")
    ap.add_argument("--no-relabelled", action="store_true",
                    help="skip the benchmark step on the randomly relabelled mesh")
    ap.add_argument("--paper3d-precs", default="fp32,bf16", help="precisions of the 3D training-step measurement")
    ap.add_argument("--paper3d-only", action="store_true",
                    help="only the latent-150 3D training-step measurement (one JSON object)")
    ap.add_argument("--copy-calibrate", action="store_true",
                    help="only run a plain device copy of known size (for counter scaling)")
    ap.add_argument("--summarize-profile", metavar="DIR",
                    help="summarize a rocprofv3 output directory (no GPU needed)")
    ap.add_argument("--profile-kernel", default="edge_bwd",
                    help="kernel whose counter traffic --summarize-profile records")
    args = ap.parse_args()
    if args.summarize_profile:
        summarize_profile(args.summarize_profile, args.profile_kernel)
        return
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

    if args.paper3d_only:
        import synth
        M = synth.mesh((args.grid,) * 3, 0)
        print(json.dumps(paper_3d_train({"mesh": M, "g": mgn.build_graph(M["cells"], M["pos"])}, args)), flush=True)
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
    n_tiles = S["dg"].n_tiles
    if dom == "edge_bwd":
        per = [kernel_bytes(dom, N, E, n_tiles, args.precision, have_ebar=(l < m - 1)) for l in range(m)]
    elif dom == "edge_fwd":
        per = [kernel_bytes(dom, N, E, n_tiles, args.precision, write_e=(l < m - 1)) for l in range(m)]
    else:
        per = [kernel_bytes(dom, N, E, n_tiles, args.precision)]
    bytes_per_launch = float(np.mean(per)) if per[0] is not None else None
    roof = None
    if bytes_per_launch is not None:
        ach = bytes_per_launch / (avg_ms * 1e-3) / 1e9
        traffic = measured_traffic(dom) if args.precision == "bf16" else None
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": None if traffic is None else int(traffic), "kernel": dom,
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
        "kernel_hbm_gbs": {k: round(sb / (kern_ms[k] * 1e-3) / 1e9, 1)
                           for k in sorted(kern_ms, key=lambda x: -kern_ms[x])
                           if (sb := step_bytes(k, N, E, n_tiles, args.precision, m)) is not None},
    }
    if dom in MFMA_FLOP_PER_EDGE and args.precision == "bf16":
        fl = MFMA_FLOP_PER_EDGE[dom] * E
        out["mfma"] = {"kernel": dom, "executed_flop_per_launch": fl,
                       "achieved_tflops": round(fl / (avg_ms * 1e-3) / 1e12, 1),
                       "peak_tflops": MFMA_PEAK_BF16_TFLOPS,
                       "frac": round(fl / (avg_ms * 1e-3) / 1e12 / MFMA_PEAK_BF16_TFLOPS, 4)}
    out["train_step"] = train_steps(S, args)
    if not args.no_relabelled:
        out["c3_relabelled"] = c3_relabelled(S, args)
    if not args.no_paper3d:
        out["paper_3d_train"] = paper_3d_train(S, args)
    if not args.no_c4:
        out["integrator_fwd_ms_per_step"] = integrator_steps(S, args)
        out["c4_rollout"] = c4_rollout(S, args)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
