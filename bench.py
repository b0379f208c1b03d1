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


# Executed MFMA work per edge (flop, counted per edge row; 16x16x32 bf16
# MFMAs at 16,384 flop over a 16-row block, select operands included).
# bf16 edge forward: W1e e and W2 a1 (K = 128) plus 16 + 8 selection MFMAs
# per 16 rows for P_s + P_r and e + m.  bf16 fused edge backward: the row
# waves' three 128 x 128 products (W2 a1 recomputed, W2^T dz2, W1e^T zbar),
# the gradient waves' dW2 = dz2^T a1 and dW1e = zbar^T e, and their ones
# columns (8 MFMAs per 64-row round and gradient wave, 4 waves).
# fp32 row-layout kernels (v_mfma_f32_16x16x4_f32, 2,048 flop each): the
# forward's two 128 x 128 products (W1e e, W2 a1); the fused backward's four
# (W1e e and W2 a1 recomputed, W2^T dz2, W1e^T zbar), dW2 and dW1e, and the
# ones columns of db2 / db1 (64 MFMAs per 64-row round and wave, 4 waves).
MFMA_FLOP_PER_EDGE = {"bf16": {"edge_fwd": 2 * 128 * 128 * 2 + 24 * 16384 // 16,
                               "edge_bwd": 5 * 2 * 128 * 128 + 4 * 8 * 16384 // 64},
                      "fp32": {"edge_fwd": 2 * 2 * 128 * 128,
                               "edge_bwd": 6 * 2 * 128 * 128 + 4 * 64 * 2048 // 64}}
MFMA_PEAK_BF16_TFLOPS = 2500.0
MFMA_PEAK_FP32_TFLOPS = 157.3


def edge_bwd_split_roofline(prec, D, N, E, m, avg_ms):
    """Position of the edge backward at latent width D (one launch per MP
    block) against both roofs: algorithmic bytes and executed MFMA flop per
    launch, each divided by the average launch time.
    fp32 (row-layout kernel at width 160): per edge e, the incoming edge
    gradient (not in the last block), the outgoing one and z-bar (fp32),
    sender / receiver ids; per node P, the gathered aggregate gradient and
    R; 5 products of D x D per edge (the recomputed W1e e and W2 a1, W2^T
    dz2, W1e^T zbar and the dW2 accumulation; dW1e is a separate pass).
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


def kernel_bytes(kind, N, E, n_tiles, prec, have_ebar=True, write_e=True, keep_a1=True, method=False):
    """HBM bytes of one launch of the library's kernels: every input
    read once and every output written once.  In bf16 the edge latents,
    their gradient stream, node products P ([N][2D]) and the a1 / zbar
    streams are 2 bytes per element; node latents, aggregates and node
    gradients are fp32 throughout.  method=True counts only the method's
    bytes (the MP step's own streams: edge latents in and out, the edge
    gradient in and out, the sender-side intermediate zbar, indices and
    node-level rows), leaving out the design's extra streams: the bf16
    path's saved first-layer activations a1 (written by the forward, read
    by the backward instead of a recompute)."""
    se = 2 if prec == "bf16" else 4
    row, frow = D * se, D * 4
    erow = row if prec == "bf16" else frow  # edge-gradient stream
    tiles = n_tiles * 16 + 4 * (N + 1)
    bf = prec == "bf16"
    a1 = row if (keep_a1 and bf and not method) else 0
    if kind == "edge_fwd":
        return (E * (row + 8 + (row if write_e else 0) + a1)
                + N * (2 * row + frow) + tiles)
    if kind == "edge_bwd":
        if bf:  # fused: reads a1, e, ebar_in, aggbar; writes ebar_out, zbar, R
            return (E * (a1 + row + (erow if have_ebar else 0) + 4 + erow + row)
                    + N * (frow + frow) + tiles)
        return (E * (row + (frow if have_ebar else 0) + frow + row + 8)
                + N * (2 * row + frow + frow) + tiles)
    if kind == "wgrad":  # fp32 dW1e pass (bf16 computes it inside the fused backward)
        return E * row * 2
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


def step_bytes(kind, N, E, n_tiles, prec, m, method=False):
    """Bytes of every launch of `kind` in one fwd+bwd step (one saving MGN
    call and its backward), or None."""
    if kind == "edge_fwd":
        return sum(kernel_bytes(kind, N, E, n_tiles, prec, write_e=(l < m - 1), method=method) for l in range(m))
    if kind == "edge_bwd":
        return sum(kernel_bytes(kind, N, E, n_tiles, prec, have_ebar=(l < m - 1), method=method)
                   for l in range(m))
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
KERNEL_SYMBOL = {"edge_bwd": "k_edge_bwd_fused", "edge_fwd": "k_edge_fwd_rows"}


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
    # wave-state counters (passes of at most four counters each): per-launch
    # averages, as fractions of the waves' lifetime (SQ_WAVE_CYCLES)
    sq = {}
    for sub in ("prof_sq1", "prof_sq2", "prof_sq3", "prof_mfma"):
        con = db(sub)
        if con is None:
            continue
        for n, c, v in con.execute("select kernel_name, counter_name, value from counters_collection"):
            sq.setdefault(short(n), {}).setdefault(c, []).append(v)
    sq = {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in sq.items()}
    if any("SQ_WAVE_CYCLES" in cs for cs in sq.values()):
        avg_ms = {short(n): avg / 1e3 for n, c, tot, avg, pct in rows}
        print("\nWave-state counters per launch (fractions of SQ_WAVE_CYCLES, the summed lifetime of the "
              "kernel's waves): issuing any instruction / VALU / VMEM / LDS, waiting on a dependency "
              "(SQ_WAIT_INST_ANY) and waiting at all (SQ_WAIT_ANY); LDS bank-conflict cycles per LDS instruction; "
              "MFMA pipe busy as a fraction of the kernel's SIMD-cycles (SQ_VALU_MFMA_BUSY_CYCLES / (avg time x "
              "2.4 GHz x 1024 SIMDs)).\n")
        print("| kernel | waves | issue any | VALU | VMEM | LDS | wait dep | wait any | LDS conflict / inst "
              "| MFMA busy |")
        print("|---|---|---|---|---|---|---|---|---|---|")
        for n, *_ in rows[:12]:
            k = short(n)
            cs = sq.get(k, {})
            wc = cs.get("SQ_WAVE_CYCLES")
            if not wc:
                continue
            fr = lambda c: f"{cs[c] / wc:.3f}" if c in cs else ""
            conf = (f"{cs['SQ_LDS_BANK_CONFLICT'] / cs['SQ_INSTS_LDS']:.2f}"
                    if cs.get("SQ_INSTS_LDS") and "SQ_LDS_BANK_CONFLICT" in cs else "")
            mb = (f"{cs['SQ_VALU_MFMA_BUSY_CYCLES'] / (avg_ms[k] * 1e-3 * 2.4e9 * 1024):.3f}"
                  if "SQ_VALU_MFMA_BUSY_CYCLES" in cs and avg_ms.get(k) else "")
            print(f"| {k} | {cs.get('SQ_WAVES', 0):,.0f} | {fr('SQ_ACTIVE_INST_ANY')} | {fr('SQ_ACTIVE_INST_VALU')} | "
                  f"{fr('SQ_ACTIVE_INST_VMEM')} | {fr('SQ_ACTIVE_INST_LDS')} | {fr('SQ_WAIT_INST_ANY')} | "
                  f"{fr('SQ_WAIT_ANY')} | {conf} | {mb} |")
        with open(os.path.join(d, "counters_per_launch.json"), "w") as fh:
            json.dump({"trace_avg_ms": {short(n): avg / 1e3 for n, c, tot, avg, pct in rows},
                       "fetch_kib": fetch, "write_kib": write, "fetch_scale": sf, "write_scale": sw,
                       "sq": sq}, fh, indent=1)
    # the kernel's instances (template specialisations), weighted by their
    # launches, as the bench's per-launch time averages over all of them
    sym = KERNEL_SYMBOL.get(kernel, "k_" + kernel)
    inst = [(short(n), c) for n, c, *_ in rows if short(n) == sym or short(n).startswith(sym + "<")]
    if inst and all(k in fetch and k in write for k, _ in inst):
        calls = sum(c for _, c in inst)
        fk = sum(fetch[k] * c for k, c in inst) / calls
        wk = sum(write[k] * c for k, c in inst) / calls
        k = " + ".join(f"{k} ({c} calls)" for k, c in inst)
        out = {"kernel": kernel, "profiled_as": k, "source_digest": source_digest(kernel),
               "fetch_kib_per_launch": fk, "write_kib_per_launch": wk,
               "fetch_scale": sf, "write_scale": sw,
               "bytes_per_launch": (fk * sf + wk * sw) * 1024}
        for f in (traffic_file(kernel), os.path.join(d, os.path.basename(traffic_file(kernel)))):
            with open(f, "w") as fh:
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


def launch_bytes(kind, N, E, n_tiles, prec, m, method=False):
    """Mean bytes per launch of `kind` over one fwd+bwd step, or None."""
    if kind == "edge_bwd":
        per = [kernel_bytes(kind, N, E, n_tiles, prec, have_ebar=(l < m - 1), method=method) for l in range(m)]
    elif kind == "edge_fwd":
        per = [kernel_bytes(kind, N, E, n_tiles, prec, write_e=(l < m - 1), method=method) for l in range(m)]
    else:
        per = [kernel_bytes(kind, N, E, n_tiles, prec, method=method)]
    return float(np.mean(per)) if per[0] is not None else None


def c3_other_slab(S, args, slab, reps=3):
    """The benchmark's fwd+bwd step on another slab patch of the same mesh
    (slab 7: 9 grid layers instead of 10), on the benchmark's context."""
    import torch
    import synth
    from paper_2304_00338_amd import mgn
    M, g, n = S["mesh"], S["g"], args.grid
    part = synth.slab_part((n, n, n), args.slabs)
    pt = mgn.extract_patch(g, part, slab, args.ghost)
    mp = pt.patch_maps()
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    R = dict(S)
    R.update({"dg": mgn.DeviceGraph(pt), "st": dev(M["onehot"][mp["node_l2g"]]),
              "y": dev(M["states"][mp["node_l2g"]]),
              "gout": dev(synth.loss_weights(pt.n_nodes, 0) * mp["interior"][:, None])})
    R["ynext"] = torch.empty_like(R["y"])
    step(R, mgn)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        step(R, mgn)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    res = {"workload": f"patch {slab} of {args.slabs} z-slabs, {args.ghost}-hop ghost zone, {args.mp_steps} MP "
                       f"steps, {args.precision}, one Euler step fwd+bwd", "n_nodes": pt.n_nodes,
           "n_interior": int(mp["n_interior"]), "n_edges": pt.n_edges, "ms_per_step": round(dt * 1e3, 3),
           "mp_edges_per_s_fwdbwd": round(pt.n_edges * args.mp_steps / dt, 1)}
    del R
    return res


def mesh_run(mgn, M, g, m, prec, scheme="euler", reps=5, warmup=2, profile=False):
    """fwd+bwd integration steps of `scheme` on a whole mesh: the MGN calls
    of every stage with saved activations, then the reverse through all of
    them (loss on every node).  Returns the mean step time (ms) and, with
    profile, the per-kernel event times of the timed steps."""
    import torch
    import synth
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    dg = mgn.DeviceGraph(g)
    st, y = dev(M["onehot"]), dev(M["states"])
    params = dev(synth.xavier_params(m, 0))
    gout = dev(synth.loss_weights(g.n_nodes, 0))
    stages = mgn.scheme_stages(scheme)
    ctx = mgn.Context(m, g.n_nodes, g.n_edges, prec, max_stages=stages, save=True)
    gp, ynext = torch.zeros_like(params), torch.empty_like(y)

    def one():
        gp.zero_()
        mgn.mgn_integrate_step(ctx, dg, params, scheme, st, y, dg.efeat, ynext, save=True)
        mgn.mgn_backward(ctx, gout, gp)
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    if profile:
        mgn.mgn_profile_enable(ctx, True)
        mgn.mgn_profile_collect(ctx)
    t0 = time.perf_counter()
    for _ in range(reps):
        one()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    prof = None
    if profile:
        prof = mgn.mgn_profile_collect(ctx)
        mgn.mgn_profile_enable(ctx, False)
    del ctx
    return ms, prof


def mfma_roofline(prof, prec, E, reps):
    """The dominant kernel of a profiled fwd+bwd run placed against the MFMA
    roof of its precision: executed MFMA flop per launch (per-edge count of
    MFMA_FLOP_PER_EDGE times E) / its average launch time."""
    dom = max(prof, key=lambda k: prof[k][0])
    tot, cnt = prof[dom]
    avg = tot / cnt
    fpe = MFMA_FLOP_PER_EDGE[prec].get(dom)
    peak = MFMA_PEAK_FP32_TFLOPS if prec == "fp32" else MFMA_PEAK_BF16_TFLOPS
    r = {"bound": "mfma", "kernel": dom, "avg_launch_ms": round(avg, 4), "launches_per_step": cnt // reps,
         "peak": peak, "unit": "TFLOP/s"}
    if fpe is not None:
        ach = fpe * E / (avg * 1e-3) / 1e12
        r.update({"flop_per_launch": int(fpe * E), "achieved": round(ach, 1), "frac": round(ach / peak, 4)})
    return r


def config_lines(args):
    """The other configurations at their full sizes: C1 (2D 32 x 32, 2 MP
    steps, fp32), C2 (3D 32^3, 15 MP steps, fp32 and bf16, with the dominant
    kernel against its MFMA roof) and C5 (the C2 mesh, Euler / midpoint
    (RK2) / RK4 steps fwd+bwd through all stages, fp32 and bf16)."""
    import synth
    from paper_2304_00338_amd import mgn
    out = {}
    M1 = synth.mesh((32, 32), 0)
    g1 = mgn.build_graph(M1["cells"], M1["pos"])
    ms, prof = mesh_run(mgn, M1, g1, 2, "fp32", reps=20, warmup=3)
    out["c1"] = {"workload": "2D 32x32 jittered triangulated mesh, 2 MP steps, fp32, one Euler step fwd+bwd",
                 "n_nodes": g1.n_nodes, "n_edges": g1.n_edges, "ms_per_step": round(ms, 3),
                 "mp_edges_per_s_fwdbwd": round(g1.n_edges * 2 / (ms * 1e-3), 1),
                 "mgn_calls_per_s_fwdbwd": round(1e3 / ms, 2)}
    M2 = synth.mesh((32, 32, 32), 0)
    g2 = mgn.build_graph(M2["cells"], M2["pos"])
    m = args.mp_steps
    c2 = {"workload": f"3D 32^3 jittered Kuhn-tetrahedral mesh, {m} MP steps, one Euler step fwd+bwd",
          "n_nodes": g2.n_nodes, "n_edges": g2.n_edges}
    for prec in ("fp32", "bf16"):
        ms, prof = mesh_run(mgn, M2, g2, m, prec, reps=5, warmup=2, profile=True)
        c2[prec] = {"ms_per_step": round(ms, 3), "mp_edges_per_s_fwdbwd": round(g2.n_edges * m / (ms * 1e-3), 1),
                    "mgn_calls_per_s_fwdbwd": round(1e3 / ms, 3),
                    "roofline": mfma_roofline(prof, prec, g2.n_edges, 5),
                    "kernel_ms_per_step": {k: round(v[0] / 5, 3)
                                           for k, v in sorted(prof.items(), key=lambda x: -x[1][0])}}
    out["c2"] = c2
    c5 = {"workload": f"C2 mesh, one integration step fwd+bwd through every stage, {m} MP steps"}
    for prec in ("fp32", "bf16"):
        r = {}
        for sc in ("euler", "midpoint", "rk4"):
            ms, _ = mesh_run(mgn, M2, g2, m, prec, scheme=sc, reps=3, warmup=1)
            st = mgn.scheme_stages(sc)
            r[sc] = {"stages": st, "ms_per_step": round(ms, 3), "mgn_calls_per_s_fwdbwd": round(st * 1e3 / ms, 2)}
        c5[prec] = r
    out["c5"] = c5
    return out


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


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args, c3_edges=None):
    """The fp64 oracle, as it stands, on a bounded sample of the C2 mesh (the
    3D 32^3 jittered Kuhn mesh, 434,558 edges): one MGN call fwd+bwd with
    1 MP step and one with 2; their difference is one MP step fwd+bwd, so
    value = E / (t2 - t1) MP-step edges/s.  Run with the host's BLAS threads
    (all usable cores) and again limited to one thread; the 15-step C2 call
    and the C3 patch call (11,674,318 edges) are extrapolated from these
    (encoder and decoder cost t1 - (t2 - t1), plus 15 MP steps scaled by
    the edge count), labelled as such."""
    import oracle as O
    import synth
    from threadpoolctl import threadpool_info, threadpool_limits
    M = synth.mesh((32, 32, 32), 0)
    g = O.build_graph(M["cells"], M["pos"])
    w = synth.loss_weights(g.n_nodes, 0)
    E, m_full = g.n_edges, args.mp_steps

    def call(m):
        P = synth.xavier_params(m, 0)
        t0 = time.time()
        _, tape = O.mgn_forward(g, P, M["node_in"], g.efeat, m, keep=True)
        O.mgn_backward(tape, w)
        del tape
        return time.time() - t0

    def measure():
        t1, t2 = call(1), call(2)
        per = max(t2 - t1, 1e-9)
        fixed = max(t1 - per, 0.0)
        return {"t_1step_s": round(t1, 3), "t_2step_s": round(t2, 3), "mp_step_fwdbwd_s": round(per, 3),
                "edges_per_s": E / per,
                "c2_call_fwdbwd_s_extrapolated": round(fixed + m_full * per, 2),
                "c3_call_fwdbwd_s_extrapolated": (round(fixed + m_full * per * c3_edges / E, 1)
                                                  if c3_edges else None)}
    blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    full = measure()
    with threadpool_limits(limits=1):
        one = measure()
    return {"value": round(full["edges_per_s"], 1), "unit": "edges/s", "cores": int(blas), "kind": "oracle",
            "sample": (f"fp64 oracle on the C2 mesh ({g.n_nodes} nodes, {E} edges): one MGN call fwd+bwd with 1 MP "
                       f"step ({full['t_1step_s']} s) and with 2 ({full['t_2step_s']} s); value = E / their "
                       f"difference, {blas} BLAS threads"),
            "cpu_model": cpu_model(), "usable_cores": len(os.sched_getaffinity(0)),
            "all_threads": full,
            "one_thread": dict(one, value=round(one["edges_per_s"], 1), cores=1)}


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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-c4", action="store_true", help="skip the whole-mesh rollout measurement")
    ap.add_argument("--no-paper3d", action="store_true", help="skip the latent-150 3D training-step measurement")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the C1 / C2 / C5 and slab-7 lines")
    ap.add_argument("--configs-only", action="store_true",
                    help="only the C1 / C2 / C5 lines (one JSON object)")
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
        print("bench.py measures one GPU: the library runs on one GPU only "
              "(patch-parallel sharding across GPUs is not implemented); run with --gpus 1",
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

    if args.configs_only:
        print(json.dumps(config_lines(args)), flush=True)
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
    bytes_method = launch_bytes(dom, N, E, n_tiles, args.precision, m, method=True)
    bytes_io = launch_bytes(dom, N, E, n_tiles, args.precision, m)
    roof = None
    if bytes_method is not None:
        ach = bytes_method / (avg_ms * 1e-3) / 1e9
        traffic = measured_traffic(dom) if args.precision == "bf16" else None
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": None if traffic is None else int(traffic), "kernel": dom,
                "avg_launch_ms": round(avg_ms, 4), "launches_per_step": cnt // args.steps,
                "algorithmic_bytes_per_launch": int(bytes_method),
                "kernel_io_bytes_per_launch": int(bytes_io),
                "kernel_io_gbs": round(bytes_io / (avg_ms * 1e-3) / 1e9, 1)}

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
    if dom in MFMA_FLOP_PER_EDGE[args.precision] and args.precision == "bf16":
        fl = MFMA_FLOP_PER_EDGE[args.precision][dom] * E
        out["mfma"] = {"kernel": dom, "executed_flop_per_launch": fl,
                       "achieved_tflops": round(fl / (avg_ms * 1e-3) / 1e12, 1),
                       "peak_tflops": MFMA_PEAK_BF16_TFLOPS,
                       "frac": round(fl / (avg_ms * 1e-3) / 1e12 / MFMA_PEAK_BF16_TFLOPS, 4)}
    out["train_step"] = train_steps(S, args)
    if not args.no_relabelled:
        out["c3_relabelled"] = c3_relabelled(S, args)
    if not args.no_configs:
        out["c3_slab7"] = c3_other_slab(S, args, 7)
    # the benchmark's context (111 GiB) is released before the other runs
    S["ctx"] = None
    del ctx
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_configs:
        out.update(config_lines(args))
    if not args.no_paper3d:
        out["paper_3d_train"] = paper_3d_train(S, args)
    if not args.no_c4:
        out["integrator_fwd_ms_per_step"] = integrator_steps(S, args)
        out["c4_rollout"] = c4_rollout(S, args)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, c3_edges=E)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
