#!/usr/bin/env python3
"""Benchmark: batched forward pass of 64 binary TreeLSTMs (N-ary, N = 2,
leaves U[10, 50], E = H = 256, fp32) on one MI355X.

A step is one pass of the whole hot path over one mini-batch: graph ingest,
batching schedule (Algorithm 1), memory plan, launch preparation and the
device execution (x staging, then per batch the fused gather -> MFMA cell GEMM
-> gate epilogue -> scatter kernel).  Inputs (x, packed weights) are resident
in HBM before the timed region.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--config 2]
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

METRIC = "node-cells/sec on 1 MI355X + % of MFMA/HBM roofline, TreeLSTM h=256"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}   # dense MFMA peaks (fp32, bf16)
# --policy names -> edb policy kinds (a learned table runs as a table policy)
POLICIES = {"table": 0, "learned": 0, "agenda": 1, "depth": 2, "sufficient": 3}
PEAK_HBM_GBS = 8000.0

WORKLOAD_TEXT = {
    1: "chain LSTM forward fp32: 8 sequences, lengths U[5,20], E=H=64",
    2: "binary TreeLSTM (N=2) forward fp32: 64 trees, leaves U[10,50], E=H=256",
    3: "lattice LSTM forward fp32: 32 lattices, lengths U[20,60], word p=0.3 span 2-4, E=100, H=200",
    4: "2-D grid RNN forward fp32: 32 grids 16x16, E=128, H=256",
    5: "child-sum TreeLSTM forward bf16 (fp32 accumulate): 256 trees, leaves U[20,200], arity U{1..4}, E=H=512",
    6: "binary TreeLSTM with two internal cell types forward fp32: 64 trees, leaves U[10,50], E=H=256",
    7: "binary TreeGRU forward fp32: 64 trees, leaves U[10,50], E=H=256",
    8: "MV-RNN forward fp32: 64 binary trees, leaves U[10,50], d=64 (a vector and a d x d matrix per node)",
    9: "lattice GRU forward fp32: 32 lattices, lengths U[20,60], word p=0.3 span 2-4, E=100, H=200",
}


def algorithmic_work(w, f):
    """Per batch (main flops, per-child flops, bytes) of the work the method
    must do: 2*K*N flops per node over the present operands (x, present
    children) and N = gates*H; per-child flops are the GEMMs of child-sum
    forget gates and lattice link gates; bytes = x rows, present children's h
    and c read, own h and c written (weights are counted once per forward,
    separately)."""
    from paper_2302_03851_amd import workloads as WL
    H, E = w.hidden, w.in_dim
    esz = 2 if w.dtype == "bf16" else 4
    G = {WL.LSTM_CHAIN: 4, WL.NARY_LEAF: 3, WL.NARY_INTERNAL: 5, WL.GRID: 5, WL.CS_LEAF: 3,
         WL.CS_INTERNAL: 3, WL.LAT_CHAR: 4, WL.LAT_WORD: 3, WL.GRU_LEAF: 2, WL.GRU_INTERNAL: 3,
         WL.LINEAR: 1, WL.MV_MAT: 1, WL.MV_VEC: 1, WL.LGRU_EDGE: 3, WL.POOL_MEAN: 1}
    mv = (WL.LINEAR, WL.MV_MAT, WL.MV_VEC)
    # an identity LINEAR map (an MV-RNN leaf) is no work
    ident = [w.kinds[t] == WL.LINEAR and w.weights[t]["W"].shape[0] == w.weights[t]["W"].shape[1] and
             np.array_equal(w.weights[t]["W"], np.eye(w.weights[t]["W"].shape[0], dtype=np.float32))
             for t in range(len(w.kinds))]
    out = []
    for b in range(f.sched.n_batches):
        t = int(f.sched.batch_type[b])
        k = w.kinds[t]
        nf = w.shapes()[t][0]
        fl = flr = by = 0
        for v in f.sched.batch_nodes[f.sched.batch_ptr[b]:f.sched.batch_ptr[b + 1]]:
            ch = w.children(int(v))
            fixed = [c for c in ch[:nf] if c >= 0]
            rag = [c for c in ch[nf:] if c >= 0]
            hasx = w.x_row[v] >= 0 and WL.KIND_SHAPE[k][2]
            Kp = (E if hasx else 0) + H * len(fixed)
            if k == WL.CS_INTERNAL:
                Kp = H
                flr += 2 * H * H * len(rag)                # h_k U_f
            if k == WL.LAT_CHAR and rag:
                fl += 2 * E * H
                flr += 2 * H * H * len(rag)                # x W_lx, c_w W_lc
            if k == WL.GRU_INTERNAL:
                fl += 2 * H * H * len(fixed)               # each candidate n_k reads its own child
            if k == WL.POOL_MEAN:
                # the mean of the edges' states (an identity map is no work)
                if not np.array_equal(w.weights[t]["W"], np.eye(H, dtype=np.float32)):
                    fl += 2 * H * H
                by += len(rag) * H * esz + H * esz
                continue
            if k in mv:
                # MV-RNN: h rows only (c mirrors h); the vector cell's two d x d
                # matrix-vector products count as per-child work
                if k == WL.MV_VEC:
                    flr += 4 * H * H
                if not ident[t]:
                    fl += 2 * Kp * H
                by += (E * esz if hasx else 0) + (len(fixed) + len(rag)) * H * esz + H * esz
                continue
            fl += 2 * Kp * G[k] * H
            by += (E * esz if hasx else 0) + len(fixed) * H * (esz + 4) + len(rag) * H * (esz + 4)
            by += H * (esz + 4)
        out.append((fl, flr, by))
    return out


def launch_work(info, work, split):
    """Algorithmic flops of one launch: the whole batch, or for a batch run in
    parts (its batch index in `split`): a child-sum batch on the large tile,
    part 2 the per-child forget GEMM, part 1 the per-parent sums (no flops),
    part 0 the parents' main GEMM; an MV-RNN vector batch, part 1 the
    matrix-vector products, part 0 its GEMM."""
    fl, flr, _ = work[info["batch"]]
    part = info["part"]
    if part == 2:
        return flr
    if part == 1:
        return flr if info["kind"] == 12 else 0
    return fl if info["batch"] in split else fl + flr


# small-tile variants (rows 16*RT, units 16*WU, split-K WK), in the library's order
SMALL_VARIANTS = [(2, 4, 1), (1, 4, 1), (1, 2, 2), (1, 1, 4), (1, 1, 8), (1, 1, 16), (2, 1, 4), (2, 2, 2)]
STREAM_SHAPES = {11: (1, 4), 12: (2, 4), 13: (1, 8), 14: (1, 16)}   # streamed tile: (rows / 16, waves)
LARGE_CLASS = {8: 0, 9: 1, 10: 2, 15: 3, 16: 4}                     # large tile: size class
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


KIND_NAMES = {0: "LSTM_CHAIN", 1: "NARY_LEAF", 2: "NARY_INTERNAL", 3: "GRID", 4: "CS_LEAF", 5: "CS_INTERNAL",
              6: "LAT_CHAR", 7: "LAT_WORD", 8: "GRU_LEAF", 9: "GRU_INTERNAL", 10: "LINEAR", 11: "MV_MAT",
              12: "MV_VEC", 13: "LGRU_EDGE", 14: "POOL_MEAN"}


def kernel_name(kind, variant, part, dtype):
    """A readable name of the kernel a launch runs (kind, tile family, variant)."""
    from paper_2302_03851_amd import _lib as L
    kname = KIND_NAMES[kind]
    if part == 1:
        return "mv_matvec_kernel" if kind == 12 else "child_reduce_kernel"
    if variant == L.WS_VARIANT:
        return f"ws_kernel<{kname}, bf16>"
    if variant in L.LARGE_VARIANTS:
        kk = "CS_FORGET" if part == 2 else ("CS_PARENT" if kind == 5 else kname)
        return f"big_kernel<{kk}, {dtype}, size class {LARGE_CLASS[variant]}>"
    if variant in STREAM_SHAPES:
        return f"stream_kernel<{kname}, {dtype}, variant {variant}>"
    return f"cell_kernel<{kname}, {dtype}, variant {variant}>"


def kernel_symbol(kind, dtype, variant, part):
    """The kernel a launch runs, as rocprofv3 prints its name (prefix)."""
    if part == 1:
        return "edbk::mv_matvec_kernel" if kind == 12 else "edbk::child_reduce_kernel"
    t = 'float' if dtype == 'f32' else '__bf16'
    from paper_2302_03851_amd import _lib as L
    if variant == L.WS_VARIANT:
        return f"edbk::ws_kernel<{kind}>"
    if variant in STREAM_SHAPES:
        rt, wk = STREAM_SHAPES[variant]
        return f"edbk::stream_kernel<{kind}, {t}, {rt}, {wk}>"
    if variant in LARGE_CLASS:
        kk = 15 if part == 2 else (16 if kind == 5 else kind)   # the child-sum forget / parent GEMMs
        return f"edbk::big_kernel<{kk}, {t}, {LARGE_CLASS[variant]}>"
    rt, wu, wk = SMALL_VARIANTS[variant]
    return f"edbk::cell_kernel<{kind}, {t}, {rt}, {wu}, {wk}>"


def source_digest():
    """SHA-256 over the kernel sources (counters taken on other code are stale)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2302_03851_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".h", ".hip", ".cpp")):
            h.update(f.encode())
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def traffic_from(d, workload):
    """Reduce rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs (KiB per dispatch)
    to HBM bytes per dispatch per kernel, scaled by what the same counters
    read for a plain copy of known size, into profiles/traffic.json."""
    import csv
    import glob

    def per_kernel(path):
        acc = {}
        for r in csv.DictReader(open(path)):
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return acc

    def one(pattern):
        m = glob.glob(os.path.join(d, pattern))
        if len(m) != 1:
            raise SystemExit(f"expected one file for {pattern} under {d}, found {m}")
        return m[0]

    # bytes per counted KiB for each calibration kernel (2 GiB per dispatch);
    # the elementwise kernel's 16-byte lane accesses match this library's
    # kernels, so its factor is the one applied
    scale, scale_copy = {}, {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        cp = per_kernel(one(f"copy_{ctr}/*counter_collection.csv"))
        for name, pat, dst in (("copy", "copyBuffer", scale_copy), ("elementwise", "MulFunctor", scale)):
            vals = [v for k, vs in cp.items() if pat in k for v in vs]
            if not vals:
                raise SystemExit(f"no {name} calibration dispatches in copy_{ctr}")
            dst[ctr] = (2048 << 10) / (sum(vals) / len(vals))
    fetch = per_kernel(one("c2_FETCH_SIZE/*counter_collection.csv"))
    write = per_kernel(one("c2_WRITE_SIZE/*counter_collection.csv"))
    out = {"workload": workload, "source_sha256": source_digest(),
           "fetch_scale": round(scale["FETCH_SIZE"], 4), "write_scale": round(scale["WRITE_SIZE"], 4),
           "copy_fetch_scale": round(scale_copy["FETCH_SIZE"], 4),
           "copy_write_scale": round(scale_copy["WRITE_SIZE"], 4),
           "calibration": "torch elementwise multiply (16-byte lane loads and stores), 2 GiB per dispatch",
           "kernels": {}}
    for k in sorted(set(fetch) & set(write)):
        f, w_ = fetch[k], write[k]
        out["kernels"][k] = {"dispatches": len(f),
                             "fetch_bytes": round(sum(f) / len(f) * 1024 * scale["FETCH_SIZE"]),
                             "write_bytes": round(sum(w_) / len(w_) * 1024 * scale["WRITE_SIZE"])}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(out, fh, indent=1)
    print(f"wrote {TRAFFIC_FILE}: {len(out['kernels'])} kernels, scales {scale} (device copy: {scale_copy})")


def trace_summary(d, symbol=None, last=0):
    """Markdown summary of a rocprofv3 --kernel-trace run under directory d:
    per kernel the calls, average / min / max duration and share of the
    summed time; with `symbol` and `last`, also the average of that kernel's
    last `last` dispatches (by start time): the roofline pass of this
    benchmark, which runs after every other launch of the path's kernels."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one kernel_trace.csv under {d}, found {files}")
    rows = [(r["Kernel_Name"], int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
            for r in csv.DictReader(open(files[0]))]
    per = {}
    for name, t0, t1 in rows:
        per.setdefault(name, []).append((t0, (t1 - t0) * 1e-3))
    total = sum(dt for v in per.values() for _, dt in v)
    out = ["| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for name, v in sorted(per.items(), key=lambda kv: -sum(dt for _, dt in kv[1])):
        ds = [dt for _, dt in v]
        nm = name if len(name) <= 90 else name[:87] + "..."
        out.append(f"| `{nm}` | {len(ds)} | {np.mean(ds):.2f} | {min(ds):.2f} | {max(ds):.2f} | "
                   f"{100 * sum(ds) / total:.1f}% |")
    if symbol:
        match = [v for name, v in per.items() if name.startswith("void " + symbol) or name.startswith(symbol)]
        if len(match) != 1:
            raise SystemExit(f"{symbol}: {len(match)} kernels match")
        v = sorted(match[0])
        tail = [dt for _, dt in v[-last:]] if last else [dt for _, dt in v]
        out.append("")
        out.append(f"`{symbol}`: average of its last {len(tail)} dispatches {np.mean(tail):.2f} us "
                   f"(min {min(tail):.2f}, max {max(tail):.2f}); all {len(v)} dispatches {np.mean([dt for _, dt in v]):.2f} us.")
    return "\n".join(out)


def traffic_of(symbol, workload):
    """HBM bytes per launch of a kernel from the committed counter record, or
    None when there is none for this workload or the sources have changed."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("source_sha256") != source_digest():
        return None
    for name, v in rec["kernels"].items():
        if name.startswith("void " + symbol) or name.startswith(symbol):
            return v["fetch_bytes"] + v["write_bytes"]
    return None


def weight_bytes(w):
    esz = 2 if w.dtype == "bf16" else 4
    return sum(int(np.prod(m.shape)) * (esz if m.ndim == 2 else 4) for d in w.weights for m in d.values())


def cpu_baseline(w, budget_s=12.0):
    """The oracle (numpy float64, node at a time) on the same workload: repeated
    full forwards until the time budget is spent, first with one BLAS thread,
    then with BLAS on every core this process may use (capped by
    OMP_NUM_THREADS when it is set)."""
    from threadpoolctl import threadpool_limits
    from oracle.evaluate import evaluate
    from oracle.mvrnn import mvrnn
    from oracle.latticegru import lattice_gru

    def forward():
        if w.aux is not None and "lattices" in w.aux:   # lattice GRU: the oracle runs the lattices
            a = w.aux
            for lat in a["lattices"]:
                lattice_gru(lat["length"], lat["words"], w.x[w.x_row[lat["char_edge"]]],
                            w.x[w.x_row[lat["word_edge"]]] if len(lat["words"]) else np.zeros((0, w.in_dim)),
                            a["Wx"], a["Wh"], a["bx"], a["bhn"])
        elif w.aux is not None:   # MV-RNN: the oracle evaluates the trees themselves
            a = w.aux
            mvrnn(a["tree_left"], a["tree_right"], a["leaf_vec"], a["leaf_mat"], w.weights[2]["W"].T,
                  w.weights[2]["b"], w.weights[1]["W_M"].T)
        else:
            evaluate(w.kinds, w.op_type, w.child_ptr, w.child_idx, w.x_row, w.x, w.weights, w.hidden,
                     n_fixed=w.n_children, dtype=w.dtype)

    def timed(threads):
        reps, t_total = 0, 0.0
        with threadpool_limits(limits=threads):
            while t_total < budget_s and reps < 20:
                t0 = time.perf_counter()
                forward()
                t_total += time.perf_counter() - t0
                reps += 1
        return reps, t_total

    reps, t_total = timed(1)
    cores = len(os.sched_getaffinity(0))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        cores = max(1, min(cores, int(os.environ["OMP_NUM_THREADS"])))
    reps_all, t_all = timed(cores)
    return {"value": round(w.n_nodes * reps / t_total, 1), "unit": "node-cells/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} full forward passes of the same {w.n_nodes}-node workload, "
                      f"{t_total:.1f} s, numpy float64 with BLAS limited to 1 thread",
            "all_cores": {"value": round(w.n_nodes * reps_all / t_all, 1), "cores": cores,
                          "sample": f"{reps_all} full forward passes, {t_all:.1f} s, BLAS on {cores} threads"}}


def probes(dtype_name, reps=3):
    """Measured denominators on this GPU: the matrix-core rate of the path's
    MFMA shape (edb_probe_mfma: 2048 work-groups of 4 waves, 8 independent
    accumulators per wave) and the device-memory copy rate (edb_probe_copy of
    1 GiB, 4x the last-level cache; read + written bytes), each the best of
    `reps` runs (the copy also over four grid sizes)."""
    import torch
    from paper_2302_03851_amd import _lib as L, edb
    st = torch.cuda.current_stream().cuda_stream
    bf16 = dtype_name == "bf16"
    n_wg, iters = 2048, (10000 if bf16 else 5000)
    out = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda:0")
    flops = n_wg * 4 * iters * 8 * (16384 if bf16 else 2048)
    ms = min(edb.probe_mfma(L.BF16 if bf16 else L.F32, n_wg, iters, out.data_ptr(), st) for _ in range(reps))
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    best = {}
    for wg in (8192, 16384, 32768, 65536):
        best[wg] = min(edb.probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, wg, st) for _ in range(reps))
    wg_best = min(best, key=best.get)
    del src, dst, out
    return {"mfma_tflops": round(flops / (ms * 1e-3) / 1e12, 1),
            "mfma_shape": "16x16x32 bf16" if bf16 else "16x16x4 f32",
            "copy_gbs": round(2 * nbytes / (best[wg_best] * 1e-3) / 1e9, 1), "copy_workgroups": wg_best}


def split_phase(configs, reps=5):
    """Split-phase diagnostic of each workload (one JSON line per workload):
    the gather and scatter of every batch as separate unfused copies
    (edb_split_phase), median over `reps` calls.  Algorithmic bytes: gather =
    the present operand rows read (x, present children's h and c), scatter =
    own h and c written; moved bytes = every row the copies read and write."""
    import torch
    from paper_2302_03851_amd import _lib as L
    from paper_2302_03851_amd import edb, workloads as WL

    pr = {}
    for spec in configs:
        k, _, mult = str(spec).partition("x")
        k, mult = int(k), int(mult or 1)
        w = WL.make_config(k, instances=DEFAULT_INSTANCES[k] * mult)
        if w.dtype not in pr:
            pr[w.dtype] = probes(w.dtype)
        rec = split_phase_record(w, k, mult, pr[w.dtype]["copy_gbs"], reps)
        rec["probes"] = pr[w.dtype]
        print(json.dumps(rec), flush=True)
        torch.cuda.empty_cache()


def split_phase_record(w, k, mult, copy_gbs, reps=5):
    """One workload's split-phase record (see split_phase)."""
    import torch
    from paper_2302_03851_amd import _lib as L
    from paper_2302_03851_amd import edb

    f = edb.Forward(w, flags=L.USE_GRAPH)
    f.run()
    torch.cuda.synchronize()
    B = f.sched.n_batches
    nb = f.exec.split_phase_bytes()
    buf = torch.empty(nb, dtype=torch.uint8, device="cuda:0")
    ms = np.median([f.exec.split_phase(f.x.data_ptr(), f.arena_h.data_ptr(), f.arena_c.data_ptr(),
                                       buf.data_ptr(), nb, f.stream.cuda_stream, B) for _ in range(reps)], axis=0)
    work = algorithmic_work(w, f)
    esz = 2 if w.dtype == "bf16" else 4
    H, E = w.hidden, w.in_dim
    shapes = edb.operand_shapes(w)
    rows = []
    for b in range(B):
        t = int(f.sched.batch_type[b])
        m = int(f.sched.batch_ptr[b + 1] - f.sched.batch_ptr[b])
        nf, rg, hx = shapes[t]
        segs = f.plan.segs[f.plan.seg_ptr[b]:f.plan.seg_ptr[b + 1]]
        moved_g = m * E * esz if hx else 0
        for kind_s, _base, _off, n in segs[1:]:
            if kind_s != L.SEG_NONE:
                moved_g += n * H * (esz + 4)
        own = m * H * (esz + 4)
        rows.append((m, work[b][2] - own, own, 2 * moved_g, 2 * own, ms[b, 0], ms[b, 1]))
    a = np.array(rows, dtype=np.float64)
    g_ms, s_ms = a[:, 5].sum(), a[:, 6].sum()
    alg = a[:, 1].sum() + a[:, 2].sum()
    moved = a[:, 3].sum() + a[:, 4].sum()
    big = int(np.argmax(a[:, 3]))
    peak, meas = PEAK_HBM_GBS, copy_gbs
    gbs = lambda by, t: by / (t * 1e-3) / 1e9
    rec = {"workload": WORKLOAD_TEXT[k], "instances_scale": mult, "nodes": w.n_nodes, "batches": B, "reps": reps,
           "gather_ms": round(g_ms, 4), "scatter_ms": round(s_ms, 4),
           "alg_bytes": int(alg), "moved_bytes": int(moved),
           "alg_gbs": round(gbs(alg, g_ms + s_ms), 1), "moved_gbs": round(gbs(moved, g_ms + s_ms), 1),
           "frac_alg": round(gbs(alg, g_ms + s_ms) / peak, 4),
           "frac_moved": round(gbs(moved, g_ms + s_ms) / peak, 4),
           "frac_moved_of_measured_copy": round(gbs(moved, g_ms + s_ms) / meas, 4) if meas else None,
           "largest_batch": {"batch": big, "rows": int(a[big, 0]),
                             "gather_us": round(a[big, 5] * 1e3, 2), "scatter_us": round(a[big, 6] * 1e3, 2),
                             "gather_moved_gbs": round(gbs(a[big, 3], a[big, 5]), 1),
                             "scatter_moved_gbs": round(gbs(a[big, 4], a[big, 6]), 1)},
           "peak_gbs": peak}
    del f, buf
    return rec


DEFAULT_INSTANCES = {1: 8, 2: 64, 3: 32, 4: 32, 5: 256, 6: 64, 7: 64, 8: 64, 9: 32}


def vendor_gemm(configs, reps=50):
    """Context for the large tile (one JSON line per workload): the longest
    launch of a leaf batch (x operand only, so the GEMM is m x E times E x
    gates*H) beside the vendor GEMM of the same shape and element type
    (torch.matmul, served by hipBLASLt), plain and after a row gather (torch
    indexing).  Our launch also gathers its rows, applies the gate epilogue
    and writes h (element type) and c (fp32); the vendor GEMM writes its
    product in the element type only.  Medians over `reps` runs; ours from the
    per-launch events of a profiled forward."""
    import torch
    from paper_2302_03851_amd import _lib as L
    from paper_2302_03851_amd import edb, workloads as WL

    gates = {WL.NARY_LEAF: 3, WL.CS_LEAF: 3, WL.GRU_LEAF: 2}
    for k in configs:
        w = WL.make_config(k)
        f = edb.Forward(w, flags=L.PROFILE)
        for _ in range(3):
            f.run()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            f.run()
            torch.cuda.synchronize()
            ts.append(f.exec.launch_times())
        t_us = np.median(np.array(ts), axis=0) * 1e3
        infos = [f.exec.launch_info(i) for i in range(f.exec.launches())]
        cand = [i for i in range(1, len(infos)) if infos[i]["kind"] in gates and infos[i]["part"] == 0]
        if not cand:
            print(json.dumps({"workload": WORKLOAD_TEXT[k], "leaf_launch": None}), flush=True)
            continue
        i = max(cand, key=lambda j: t_us[j])
        m, E, N = int(infos[i]["m"]), w.in_dim, gates[infos[i]["kind"]] * w.hidden
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        gen = torch.Generator(device="cuda:0").manual_seed(0)
        x = torch.randn(m, E, device="cuda:0", dtype=dt, generator=gen)
        W = torch.randn(E, N, device="cuda:0", dtype=dt, generator=gen)
        rows = torch.randperm(m, device="cuda:0", generator=gen)

        def timed(fn):
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
            out = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                e1.synchronize()
                out.append(e0.elapsed_time(e1) * 1e3)
            return float(np.median(out))

        flops = 2.0 * m * E * N
        peak = PEAK_TFLOPS[w.dtype]
        rec = {"workload": WORKLOAD_TEXT[k], "shape": {"m": m, "K": E, "N": N, "dtype": w.dtype},
               "ours": {"us": round(float(t_us[i]), 2), "variant": int(infos[i]["variant"]),
                        "work": "row gather + GEMM + gate epilogue, h and c written"}}
        for name, fn in (("vendor_mm", lambda: x @ W), ("vendor_gather_mm", lambda: x[rows] @ W)):
            us = timed(fn)
            rec[name] = {"us": round(us, 2)}
        for key in ("ours", "vendor_mm", "vendor_gather_mm"):
            rec[key]["tflops"] = round(flops / (rec[key]["us"] * 1e-6) / 1e12, 1)
            rec[key]["frac_of_peak"] = round(rec[key]["tflops"] / peak, 4)
        rec["peak_tflops"] = peak
        print(json.dumps(rec), flush=True)
        del f, x, W, rows
        torch.cuda.empty_cache()


def study(configs, replays=100):
    """Replay study of each workload (one JSON line per workload): warm and
    cold replays of the batch sequence's HIP graph (median, p10, p90; cold = a
    512 MB write before every replay, twice the last-level cache), the scale
    sweep at 1x, 4x and 16x the instances, and the end-to-end time of a new
    input graph (ingest + schedule + plan + prepare, then its run through the stream's kept
    graph of the same kernel sequence and the first replay)."""
    import torch
    from paper_2302_03851_amd import _lib as L
    from paper_2302_03851_amd import edb, workloads as WL

    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda:0")

    def replay_times(f, cold):
        ts = []
        for _ in range(replays):
            if cold:
                scratch.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(f.stream)
            f.run()
            e1.record(f.stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        ts = np.array(ts)
        return {"median_us": round(float(np.median(ts)), 2), "p10_us": round(float(np.percentile(ts, 10)), 2),
                "p90_us": round(float(np.percentile(ts, 90)), 2)}

    for k in configs:
        rec = {"workload": WORKLOAD_TEXT[k], "scale": {}}
        for mult in (1, 4, 16):
            w = WL.make_config(k, instances=DEFAULT_INSTANCES[k] * mult)
            f = edb.Forward(w, flags=L.USE_GRAPH)
            for _ in range(5):
                f.run()
            torch.cuda.synchronize()
            warm = replay_times(f, False)
            work = algorithmic_work(w, f)
            flops = sum(x[0] + x[1] for x in work)
            ent = {"instances": DEFAULT_INSTANCES[k] * mult, "nodes": w.n_nodes, "batches": f.sched.n_batches,
                   "warm": warm, "node_cells_per_s": round(w.n_nodes / (warm["median_us"] * 1e-6), 1),
                   "alg_tflops": round(flops / (warm["median_us"] * 1e-6) / 1e12, 3)}
            if mult == 1:
                ent["cold"] = replay_times(f, True)
                # a new input graph end to end (the mini-batch with its node ids
                # permuted: the same batch sizes): host objects, then the run
                # through the stream's kept HIP graph of the same kernel sequence
                # (its nodes updated in place) and the first replay
                w2, _ = WL.relabel(w, 7)
                s0 = edb.graph_stats()
                t0 = time.perf_counter()
                g = edb.Graph(w2.op_type, w2.child_ptr, w2.child_idx, w2.x_row, w2.n_types)
                sc = edb.Schedule(g, L.POLICY_TABLE, L.ENC_SORT, edb.LATTICE_TABLE if w.kinds == [6, 7] else None)
                pl = edb.Plan(g, sc, edb.operand_shapes(w2), L.PLAN_RC)
                ex = edb.Exec(g, sc, pl, f.cells, L.USE_GRAPH)
                t1 = time.perf_counter()
                ah = torch.empty((pl.n_slots, w.hidden), dtype=f.arena_h.dtype, device=f.arena_h.device)
                ac = torch.empty((pl.n_slots, w.hidden), dtype=torch.float32, device=f.arena_h.device)
                torch.cuda.synchronize()
                t2 = time.perf_counter()
                ex.execute([b.data_ptr() for b in f.weights], f.x.data_ptr(), ah.data_ptr(), ac.data_ptr(),
                           f.stream.cuda_stream)
                torch.cuda.synchronize()
                t3 = time.perf_counter()
                s1 = edb.graph_stats()
                ent["new_graph_ms"] = {"host": round((t1 - t0) * 1e3, 3),
                                       "graph_first_replay": round((t3 - t2) * 1e3, 3),
                                       "total": round((t1 - t0 + t3 - t2) * 1e3, 3),
                                       "graphs_instantiated": s1[0] - s0[0], "graphs_updated": s1[1] - s0[1]}
                del ex, pl, sc, g, ah, ac
            rec["scale"][f"x{mult}"] = ent
            print(f"study: workload {k} x{mult}: {w.n_nodes} nodes, warm median {warm['median_us']} us",
                  file=sys.stderr, flush=True)
            del f
            torch.cuda.empty_cache()
        print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--replays", type=int, default=200)
    ap.add_argument("--streams", type=int, default=None,
                    help="mini-batches in flight: host worker threads, each with its own stream and arena "
                         "(default: a third of the timed steps, at least 4 and at most 16, so that every "
                         "stream runs three or more of them)")
    ap.add_argument("--roofline-steps", type=int, default=50,
                    help="steps of the roofline pass (one mini-batch in flight, launches timed with HIP events)")
    ap.add_argument("--policy", default="table", choices=sorted(POLICIES),
                    help="batching policy: the configured FSM table (default), a table learned on the "
                         "workload's graph before timing (N-step Q-learning, E_sort), or a heuristic")
    ap.add_argument("--plan", default="rc", choices=["rc", "pq", "identity"],
                    help="arena layout: the reverse consumer-first pass (default), the PQ-tree layout, "
                         "or node ids (every operand indexed)")
    ap.add_argument("--study", metavar="CONFIGS",
                    help="instead of the benchmark: warm/cold replay, scale sweep and new-graph times of the "
                         "listed workloads (comma separated, e.g. 1,2,3,4,5)")
    ap.add_argument("--split-phase", metavar="CONFIGS",
                    help="instead of the benchmark: unfused gather and scatter times of the listed workloads "
                         "(comma separated; 'KxN' = workload K with N times its instances, e.g. 5,5x4,5x16)")
    ap.add_argument("--vendor-gemm", metavar="CONFIGS",
                    help="comma-separated workloads: the longest leaf-batch launch beside the vendor GEMM of its shape")
    ap.add_argument("--probes", action="store_true",
                    help="instead of the benchmark: measured MFMA and copy rates")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run plain copies of 2 GiB, 5 device copies and 5 elementwise (to scale HBM byte counters)")
    ap.add_argument("--traffic-from", metavar="DIR",
                    help="write profiles/traffic.json from rocprofv3 FETCH_SIZE/WRITE_SIZE runs under DIR "
                         "(c2_<counter>/ of this benchmark, copy_<counter>/ of --copy-calibration)")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="print a markdown summary of the rocprofv3 --kernel-trace run under DIR")
    ap.add_argument("--symbol", help="with --trace-summary: the kernel whose last --last dispatches are averaged")
    ap.add_argument("--last", type=int, default=0)
    args = ap.parse_args()
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.symbol, args.last))
        return
    if args.traffic_from:
        traffic_from(args.traffic_from, WORKLOAD_TEXT[args.config])
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested); the path shards by "
              "instance with no exchange, see the design notes", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2302_03851_amd import _lib as L
    from paper_2302_03851_amd import edb, workloads as WL

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.study:
        study([int(c) for c in args.study.split(",")])
        return
    if args.split_phase:
        split_phase(args.split_phase.split(","))
        return
    if args.probes:
        print(json.dumps({"f32": probes("f32"), "bf16": probes("bf16")}), flush=True)
        return
    if args.vendor_gemm:
        vendor_gemm([int(c) for c in args.vendor_gemm.split(",")])
        return
    if args.copy_calibration:
        # copies of known size, each dispatch reading and writing 2 GiB (8x the
        # 256 MB last-level cache, so that few reads hit it): the runtime's
        # device copy, and an elementwise kernel whose lanes load and store 16
        # bytes each (the access width of this library's kernels)
        src = torch.ones(512 << 20, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 4, "copy_bytes_written": dst.numel() * 4,
                          "copies": 5, "elementwise": 5}), flush=True)
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = WL.make_config(args.config)
    V = w.n_nodes

    # batching policy (a learned table is learned here, before any timing:
    # the paper learns one table per model offline)
    kind = POLICIES[args.policy]
    table = edb.LATTICE_TABLE if args.config == 3 else None
    policy_info = {"kind": args.policy}
    if args.policy == "learned":
        g0 = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
        tl = time.perf_counter()
        table, lstats, _ = edb.learn_policy(g0, L.ENC_SORT)
        policy_info.update(lstats, learn_ms=round((time.perf_counter() - tl) * 1e3, 2), encoding="E_sort")
        del g0
    elif kind != L.POLICY_TABLE:
        table = None

    # resident inputs: packed weights, x, arena
    plan_mode = {"rc": L.PLAN_RC, "pq": L.PLAN_PQ, "identity": L.PLAN_IDENTITY}[args.plan]
    base = edb.Forward(w, policy=kind, table=table, plan_mode=plan_mode, flags=L.USE_GRAPH)
    stream = base.stream.cuda_stream
    wptrs = [b.data_ptr() for b in base.weights]
    xp, ahp, acp = base.x.data_ptr(), base.arena_h.data_ptr(), base.arena_c.data_ptr()
    shapes = edb.operand_shapes(w)
    dt = base.dtype

    import threading

    # Mini-batches in flight.  Steady throughput rises up to about 16 (all
    # four hardware queues busy), but every stream's first and last steps run
    # with the pipeline filling or draining: with fewer than about three steps
    # per stream the run is mostly fill and drain, and fewer streams finish
    # the same steps sooner (20 steps: 6 streams take 0.10-0.11 ms a step, 16
    # streams 0.12-0.15)
    S = max(1, args.streams) if args.streams else min(16, max(4, args.steps // 3))
    streams = [base.stream] + [torch.cuda.Stream(device=dev) for _ in range(S - 1)]
    arenas = [(ahp, acp)] + [(torch.empty_like(base.arena_h), torch.empty_like(base.arena_c)) for _ in range(S - 1)]
    arena_ptrs = [arenas[0]] + [(a.data_ptr(), c.data_ptr()) for a, c in arenas[1:]]

    fwd = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, shapes, base.cells,
                          policy=kind, table=table, plan_mode=plan_mode)
    n_rows = base.plan.n_slots

    # a1 graph ingest, a2 schedule, a3 memory plan, descriptor upload and
    # a4..a8 device execution (asynchronous, eager launches), in one C call;
    # each worker's arguments (its stream and arena) marshalled once
    calls = [fwd.bind(wptrs, xp, arena_ptrs[i][0], arena_ptrs[i][1], n_rows, streams[i].cuda_stream)
             for i in range(S)]

    def step(i):
        calls[i]()

    class Workers:
        """S host threads, each with its own stream and arena, started once
        and parked at a barrier; run(n) releases them for n steps (each thread
        takes the next step when it is free) and returns when all are done."""

        def __init__(self):
            self.go = threading.Barrier(S + 1)
            self.end = threading.Barrier(S + 1)
            self.lock = threading.Lock()
            self.n = self.taken = 0
            self.quit = False
            self.errors = []
            self.threads = [threading.Thread(target=self.work, args=(i,), daemon=True) for i in range(S)]
            for t in self.threads:
                t.start()

        def work(self, i):
            while True:
                self.go.wait()
                if self.quit:
                    return
                try:
                    while True:
                        with self.lock:
                            if self.taken >= self.n:
                                break
                            self.taken += 1
                        step(i)
                except Exception as e:   # reported by run()
                    self.errors.append(e)
                self.end.wait()

        def run(self, n):
            self.n, self.taken = n, 0
            self.go.wait()
            self.end.wait()
            if self.errors:
                raise self.errors[0]

        def close(self):
            self.quit = True
            self.go.wait()
            for t in self.threads:
                t.join()

    # every worker stream has run a kernel before the first step (a stream's
    # first dispatch binds it to a hardware queue, a one-time cost)
    for st_ in streams:
        with torch.cuda.stream(st_):
            torch.zeros(1, device=dev).add_(1.0)
    torch.cuda.synchronize()
    pool = Workers()
    pool.run(args.warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pool.run(args.steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    pool.close()

    # device-only rate: the HIP graph of the same batch sequence replayed
    for _ in range(10):
        base.run()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.replays):
        base.run()
    ev1.record()
    torch.cuda.synchronize()
    ms_replay = ev0.elapsed_time(ev1) / args.replays

    # host part of a step (a1-a3 + descriptor upload), measured alone
    th = time.perf_counter()
    nh = 20
    parts = np.zeros(4)   # ingest, schedule, plan, prepare (ms, summed)
    for _ in range(nh):
        t0 = time.perf_counter()
        g = edb.Graph(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types)
        t1 = time.perf_counter()
        s = edb.Schedule(g, kind, L.ENC_SORT, table)
        t2 = time.perf_counter()
        p = edb.Plan(g, s, shapes, plan_mode)
        t3 = time.perf_counter()
        ex = edb.Exec(g, s, p, base.cells, 0)
        t4 = time.perf_counter()
        parts += np.array([t1 - t0, t2 - t1, t3 - t2, t4 - t3]) * 1e3
    ms_host = (time.perf_counter() - th) * 1e3 / nh
    host_parts = {k: round(float(v) / nh, 4) for k, v in zip(("ingest", "schedule", "plan", "prepare"), parts)}

    # gather and scatter as separate copies (split-phase diagnostic) at this
    # workload's size: the HBM side of the roofline
    sp = split_phase_record(w, args.config, 1, None)
    torch.cuda.empty_cache()

    # roofline pass: the same step with one mini-batch in flight, each step
    # alone on the GPU (synchronised), its launches recording start and stop
    # events in their dispatch packets; per-launch durations averaged over the
    # steps.  Nothing launches the path's kernels after this pass, so a
    # profiler trace of this command finds these dispatches as the last ones
    # of each kernel.
    fwd_prof = edb.ForwardCall(w.op_type, w.child_ptr, w.child_idx, w.x_row, w.n_types, shapes, base.cells,
                               policy=kind, table=table, plan_mode=plan_mode, flags=L.PROFILE)
    rec_times, rec_infos = [], None
    for _ in range(args.roofline_steps + 2):
        r = fwd_prof.call(wptrs, xp, ahp, acp, n_rows, stream, keep=True)
        torch.cuda.synchronize()
        if rec_infos is None:
            rec_infos = [r.launch_info(i) for i in range(r.launches())]
        rec_times.append(r.launch_times())
        del r
    rec_times = np.array(rec_times[2:])   # [steps][launches] ms; the first two steps warm the pass up
    n_profiled = rec_times.shape[0]

    times = rec_times.mean(axis=0)
    work = algorithmic_work(w, base)
    infos = rec_infos
    split = {inf["batch"] for inf in infos[1:] if inf["part"] != 0}
    # launches grouped by the kernel they run: (cell kind, tile variant, part)
    groups = {}
    for i, inf in enumerate(infos[1:], start=1):
        key = (inf["kind"], inf["variant"], inf["part"])
        gsum = groups.setdefault(key, [0.0, 0, 0])
        gsum[0] += times[i]
        gsum[1] += 1
        gsum[2] += launch_work(inf, work, split)
    dom = max(groups, key=lambda k: groups[k][0])
    tot_ms, nl, fl = groups[dom]
    avg_ms = tot_ms / nl
    tflops = (fl / nl) / (avg_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    # Launches with no algorithmic flops are bound by memory: the MV-RNN
    # matrix-vector launch (bytes per node: the two vector children and the 2H
    # matrix columns it reads) and a mean over children through the identity
    # map (the batch's algorithmic bytes)
    hbm_bound = dom == (WL.MV_VEC, -1, 1) or fl == 0
    if hbm_bound:
        esz_d = 2 if w.dtype == "bf16" else 4
        grp = [inf for inf in infos[1:] if (inf["kind"], inf["variant"], inf["part"]) == dom]
        if dom == (WL.MV_VEC, -1, 1):
            by_launch = sum(inf["m"] for inf in grp) * (2 * w.hidden + 2) * w.hidden * esz_d / nl
        else:
            by_launch = sum(work[inf["batch"]][2] for inf in grp) / nl
        gbs = by_launch / (avg_ms * 1e-3) / 1e9
    kind_v, var_v, part_v = dom
    kernel = kernel_name(kind_v, var_v, part_v, w.dtype)
    symbol = kernel_symbol(kind_v, w.dtype, var_v, part_v)
    # the largest contraction: the launch with the most algorithmic flops
    big_i = max(range(1, len(infos)), key=lambda i: launch_work(infos[i], work, split))
    big_inf, big_fl = infos[big_i], launch_work(infos[big_i], work, split)
    big_tflops = big_fl / (times[big_i] * 1e-3) / 1e12 if times[big_i] > 0 else 0.0
    largest = {"kernel": kernel_name(big_inf["kind"], big_inf["variant"], big_inf["part"], w.dtype),
               "symbol": kernel_symbol(big_inf["kind"], w.dtype, big_inf["variant"], big_inf["part"]),
               "launch": big_i, "rows": big_inf["m"], "alg_flops": int(big_fl),
               "avg_launch_us": round(float(times[big_i]) * 1e3, 2), "achieved": round(big_tflops, 3),
               "peak": peak, "unit": "TFLOP/s", "frac": round(big_tflops / peak, 4)}
    traffic = traffic_of(symbol, WORKLOAD_TEXT[args.config])
    tot_flops = sum(x[0] + x[1] for x in work)
    tot_bytes = sum(x[2] for x in work) + weight_bytes(w)

    result = {
        "metric": METRIC,
        "value": round(V / (ms_step * 1e-3), 1),
        "unit": "node-cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.config], "nodes": V, "batches": base.sched.n_batches,
                   "launches_per_step": sum(1 for i in range(base.exec.launches()) if base.exec.launch_info(i)["grid"] > 0), "mini_batches_in_flight": S,
                   "policy": policy_info, "plan": args.plan,
                   "step": "graph ingest + schedule + memory plan + launch prep + device execution"},
        "roofline": ({"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                      "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
                      "alg_bytes_per_launch": int(by_launch)} if hbm_bound else
                     {"bound": "mfma", "achieved": round(tflops, 3), "peak": peak, "unit": "TFLOP/s",
                      "frac": round(tflops / peak, 4), "traffic": traffic}) | {
                     "kernel": kernel, "symbol": symbol,
                     "launches": nl, "avg_launch_us": round(avg_ms * 1e3, 2),
                     "timing": f"HIP events in the dispatch packets, {n_profiled} steps with one mini-batch in "
                               "flight (each step alone on the GPU)",
                     "launches_timed": nl * n_profiled, "per_step_us": round(tot_ms * 1e3, 2),
                     "alg_flops_per_launch": int(fl / nl)},
        # the whole timed region's algorithmic work rate: every step's
        # flops over the region's wall time (mini-batches in flight share
        # the GPU, so this is the chip's rate, not one kernel's)
        "timed_region": {"alg_tflops": round(tot_flops / (ms_step * 1e-3) / 1e12, 3),
                         "frac_of_peak": round(tot_flops / (ms_step * 1e-3) / 1e12 / peak, 4),
                         "alg_hbm_gbs": round(tot_bytes / (ms_step * 1e-3) / 1e9, 1)},
        "device_replay": {"ms_per_forward": round(ms_replay, 4),
                          "node_cells_per_s": round(V / (ms_replay * 1e-3), 1),
                          "alg_tflops": round(tot_flops / (ms_replay * 1e-3) / 1e12, 3),
                          "alg_hbm_gbs": round(tot_bytes / (ms_replay * 1e-3) / 1e9, 1)},
        "host_ms_per_graph": round(ms_host, 4),
        "host_ms_parts": host_parts,
        "launch_us": [round(t * 1e3, 2) for t in times],
        "largest_launch": largest,
    }
    pm = probes(w.dtype)
    if hbm_bound:
        result["roofline"]["peak_measured"] = pm["copy_gbs"]
        result["roofline"]["frac_measured"] = round(gbs / pm["copy_gbs"], 4)
    else:
        result["roofline"]["peak_measured"] = pm["mfma_tflops"]
        result["roofline"]["frac_measured"] = round(tflops / pm["mfma_tflops"], 4)
    result["probes"] = pm
    result["roofline_hbm"] = {
        "bound": "hbm", "kernel": "copy_rows_kernel (split-phase gather and scatter of every batch)",
        "achieved": sp["alg_gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": sp["frac_alg"],
        "alg_bytes": sp["alg_bytes"], "moved_bytes": sp["moved_bytes"],
        "moved_gbs": sp["moved_gbs"], "frac_moved": sp["frac_moved"],
        "frac_moved_of_measured_copy": round(sp["moved_gbs"] / pm["copy_gbs"], 4),
        "gather_ms": sp["gather_ms"], "scatter_ms": sp["scatter_ms"], "launches": 2 * sp["batches"],
        "bytes": "algorithmic: present operand rows read (x, children's h and c) + own h and c written; "
                 "moved: every row the copies read and write (zero rows and the dense buffer included)",
        "largest_batch": sp["largest_batch"]}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
