#!/usr/bin/env python3
"""Benchmark of rollback-free GDN draft-tree verification on one MI355X.

One step = one pass of the whole hot path for one GDN layer over one batch of
synthetic draft trees: tree prepare, verify (every node's output from the
read-only cached state) and commit (state + conv state of the accepted node).
By default a step is timed as a decode loop runs it: prepare of the current
tree, then one fused launch that commits the previous step's accepted node
and verifies the current tree against the state it produces (--unfused: three
separate launches, prepare / verify / commit).
The default workload is the large one: 32 trees of 128 nodes (depth 16),
16 key / 48 value heads, dk = dv = 128, bf16 inputs, fp32 state.

The timed steps run eagerly (HIP events around every launch give the
per-kernel durations) with cold caches: a 512 MiB buffer is written before
every step (warm-up included), outside its events, so that L2 and the MALL
hold nothing the step reads, as in a model whose other layers run between two
steps of this one; the step time is the sum of its kernels' times.  --hot: no
eviction, and two consecutive steps are captured in a HIP graph and replayed
back to back; the replay time is the step time (--no-graph: the eager time).

Prints ONE JSON line on stdout: throughput in tree nodes verified per second
per GDN layer, the roofline of the dominant kernel (the fused step, or verify
with --unfused), the rate of a plain device copy on the same GPU, and the CPU
oracle's throughput on the same workload (all host threads and one thread).
--sweep instead prints one line with the fused, unfused and chunked step
times over tree sizes 32..512 (large recipe) and on 128 / 512-node chains.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
VERIFY_SOURCES = ("paper_2607_06763_amd/csrc/gdn_verify.hip", "paper_2607_06763_amd/csrc/gdn_internal.h")
PROFILES = os.path.join(ROOT, "profiles")


def verify_source_hash() -> str:
    h = hashlib.sha256()
    for rel in VERIFY_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(w) -> dict:
    """Bytes the method must move (each input read once, each output written
    once), per launch of each kernel."""
    import numpy as np
    B, T, Hk, Hv, dk, dv = w.B, w.T, w.Hk, w.Hv, w.dk, w.dv
    e = 2 if w.in_dtype == "bf16" else 4
    C = 2 * Hk * dk + Hv * dv
    meta_read = 4 * 4 * B * T + 8 * B            # order, depth, parent, pos + status, nvalid
    verify = (4 * B * Hv * dv * dk                # S0
              + e * B * T * (2 * Hk * dk + Hv * dv)  # q, k, v
              + e * 2 * B * T * Hv                 # alpha, beta
              + 4 * 3 * B * C + 4 * 4 * C          # conv state, conv weights
              + meta_read
              + 4 * B * T * Hv * dv)               # out
    # commit: S read + write, conv state read + write, raw inputs and gates of
    # the accepted paths, conv weights
    depth = np.zeros((B, T), int)
    for b in range(B):
        for i in range(T):
            p = w.parent[b, i]
            depth[b, i] = 0 if p < 0 else depth[b, p] + 1
    L = sum(depth[b, w.accepted[b]] + 1 for b in range(B) if w.accepted[b] >= 0)
    commit = (2 * 4 * B * Hv * dv * dk + 2 * 4 * 3 * B * C + int(L) * (e * C + 2 * e * Hv)
              + 4 * 4 * C + 8 * B * T + 8 * B)
    prepare = 4 * B * T + 8 * B * T * ((T + 63) // 64) + 4 * 4 * B * T + 8 * B
    # fused step: S, the conv state and the conv weights are read once
    fused = verify + commit - 4 * B * Hv * dv * dk - 4 * 3 * B * C - 4 * 4 * C
    return {"verify": int(verify), "commit": int(commit), "prepare": int(prepare),
            "step": int(fused)}


def measured_traffic(src_hash: str, kernel: str, workload: str):
    """HBM bytes per launch of kernel from the committed rocprofv3 counter
    summary (profiles/<kernel>_<workload>_hbm_traffic.md), if it was taken on
    the current kernel source; else None."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                vals[k.strip()] = v.strip().strip("`")
    if vals.get("verify_source_sha256_16") != src_hash or vals.get("kernel", "verify") != kernel:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, max_seconds: float = 20.0, one_thread_seconds: float = 8.0) -> dict:
    """The oracle (prepare + verify + commit) timed on this host's cores on
    whole trees of the same workload, with all threads and with one thread;
    as many trees as fit each time budget, estimated from the first tree."""
    import copy

    from oracle import oracle as orc

    def sub(nb):
        s = copy.copy(w)
        s.B = nb
        for n in ("parent", "q", "k", "v", "alpha", "beta", "S0", "conv_state", "accepted"):
            setattr(s, n, getattr(w, n)[:nb])
        return s

    def run(s):
        t0 = time.perf_counter()
        orc.prepare(s.parent)
        orc.verify(s)
        orc.commit(s)
        return time.perf_counter() - t0

    def rate(budget):
        t1 = run(sub(1))
        nb = max(1, min(w.B, int(budget / max(t1, 1e-6))))
        dt = run(sub(nb)) if nb > 1 else t1
        return nb, dt

    cores = orc.num_threads()
    nb, dt = rate(max_seconds)
    orc.set_num_threads(1)
    try:
        nb1, dt1 = rate(one_thread_seconds)
    finally:
        orc.set_num_threads(cores)
    return {"value": round(nb * w.T / dt, 2), "unit": "nodes/s", "cores": cores,
            "kind": "oracle",
            "value_1thread": round(nb1 * w.T / dt1, 2),
            "cpu_model": cpu_model(),
            "sample": f"{nb} of {w.B} trees x {w.T} nodes of the '{w.name}' workload, all "
                      f"{w.Hv} value heads; prepare+verify+commit; fp64 per-node path replay; "
                      f"{dt:.2f} s on {cores} threads; 1 thread: {nb1} trees in {dt1:.2f} s"}


def copy_rate_gbs(torch, mib: int = 512, reps: int = 5) -> float:
    """Device-to-device copy rate (read + write bytes / time) of a plain
    copy kernel on this GPU, timed with HIP events."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * 4 * n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return gbs


DTYPE = "bf16-in/f32 (S0 readout: fp16 MFMA operands, rows scaled by powers of two, fp32 accumulate)"


def measure(G, torch, np, w, form: str, steps: int, warmup: int, cold: bool, graph: bool) -> dict:
    """Times `steps` decode steps of workload w after `warmup` untimed ones.
    form: "fused" (prepare + gdn_tree_step), "unfused" (prepare, verify,
    commit) or "chunked" (prepare, chunked verify, commit).  Per-launch
    durations come from HIP events recorded on the launch stream around each
    entry point; with graph=True two steps are also captured in a HIP graph
    and the replay time is the step time."""
    dt = G.DeviceTree(w, device="cuda:0")
    S = dt.S0.clone()
    cs = dt.conv_state.clone()
    fused = form == "fused"
    # two metadata buffers and two conv-state buffers alternate between steps:
    # the fused launch reads the previous tree's metadata and conv state while
    # the current tree's are written
    metas = [dt.meta, torch.zeros_like(dt.meta)]
    css = [cs, torch.empty_like(cs)]
    # the previous step's raw inputs live in their own buffers (same values):
    # the commit reads them from HBM, not from what the verify just cached
    prev = {n: getattr(dt, n).clone() for n in ("q", "k", "v", "alpha", "beta")} if fused else {}
    nev = 3 if fused else 4

    def step(i, ev=None):
        if ev is not None:
            ev[0].record()
        if fused:
            cur, pmeta = metas[i % 2], metas[(i + 1) % 2]
            G.prepare(dt.dims, dt.parent, cur, dt.tree_status)
            if ev is not None:
                ev[1].record()
            G.step(dt.dims, pmeta, dt.accepted, prev["q"], prev["k"], prev["v"], prev["alpha"],
                   prev["beta"], dt.commit_status, cur, dt.q, dt.k, dt.v, dt.alpha, dt.beta,
                   dt.conv_w, css[i % 2], css[(i + 1) % 2], S, dt.out)
            if ev is not None:
                ev[2].record()
            return
        dt.prepare()
        if ev is not None:
            ev[1].record()
        dt.verify(S0=S, conv_state=cs, chunked=form == "chunked")
        if ev is not None:
            ev[2].record()
        dt.commit(S, cs)
        if ev is not None:
            ev[3].record()

    flush = torch.empty((512 << 20) // 4, dtype=torch.float32, device="cuda:0") if cold else None
    if cold:
        graph = False  # every launch of a cold run sees cold caches
    if fused:
        G.prepare(dt.dims, dt.parent, metas[1], dt.tree_status)  # the "previous" tree of step 0
    for i in range(warmup):
        if flush is not None:
            flush.fill_(float(i))
        step(i)
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if flush is not None:
            flush.fill_(float(i))
        step(warmup + i, events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps
    ms_eager = ms_step
    reps = 0
    if graph:
        # two consecutive steps (the metadata / conv-state buffers alternate)
        # captured once; warm-up launches on the capture stream first
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(0)
            step(1)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            step(0)
            step(1)
        for _ in range(max(1, warmup // 2)):
            g.replay()
        torch.cuda.synchronize()
        reps = max(1, (steps + 1) // 2)
        t0 = time.perf_counter()
        for _ in range(reps):
            g.replay()
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / (2 * reps)
    per = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(nev - 1)] for e in events]) * 1e3
    r = {"us_prep": float(per[:, 0].mean()), "us_main": float(per[:, 1].mean()),
         "us_main_p10_p50_p90": [float(x) for x in np.percentile(per[:, 1], [10, 50, 90])],
         "us_commit": float(per[:, 2].mean()) if not fused else None,
         "ms_eager": ms_eager, "reps": reps}
    if cold:  # the eager wall time includes the flushes: the kernels' own times
        ms_step = float(per.sum(1).mean()) * 1e-3
    r["ms_step"] = ms_step
    del dt, S, cs, metas, css, prev, flush
    return r


SWEEP_T = (32, 64, 128, 256, 512)


def sweep(G, torch, np, W, args) -> dict:
    """Pull-back (fused and unfused) and chunked step times over tree sizes on
    the large recipe, and at T = 128 / 512 on chains (depth T - 1): the
    crossover of the two verification forms."""
    rows = []
    cases = [("large", T) for T in SWEEP_T] + [("chain", 128), ("chain", 512)]
    for shape, T in cases:
        w = W.make_sweep(T, shape=shape)
        nb = algorithmic_bytes(w)
        row = {"shape": shape, "T": T, "B": w.B, "nodes": w.B * w.T}
        for form in ("fused", "unfused", "chunked"):
            r = measure(G, torch, np, w, form, args.steps, args.warmup, True, False)
            main_bytes = nb["step"] if form == "fused" else nb["verify"]
            row[form] = {"us_prepare": round(r["us_prep"], 2), "us_verify_or_step": round(r["us_main"], 2),
                         "us_commit": None if r["us_commit"] is None else round(r["us_commit"], 2),
                         "us_total": round(r["ms_step"] * 1e3, 2),
                         "nodes_per_s": round(w.B * w.T / (r["ms_step"] * 1e-3), 1),
                         "hbm_frac": round(main_bytes / (r["us_main"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
            print(f"[sweep] {shape} T={T} {form}: {row[form]}", file=sys.stderr, flush=True)
            torch.cuda.empty_cache()
        rows.append(row)
        del w
    return {"sweep": rows, "cold_caches": True, "steps": args.steps, "warmup": args.warmup}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4, help="workload index 0..4 (default: large)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tree-size", type=int, default=0,
                    help="run the large workload's recipe at this tree size T (16..512) instead of "
                         "the --config workload")
    ap.add_argument("--shape", default="large", choices=["large", "chain"],
                    help="tree shape for --tree-size: the large recipe, or single paths of T nodes")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="time eager launches only (with --hot: after the eager pass, two steps are "
                         "captured in a HIP graph and the replay time is the step time; per-kernel "
                         "durations always come from the eager pass)")
    ap.add_argument("--chunked", action="store_true",
                    help="verify with the chunked-form kernel (Eq. 9-13) instead of the pull-back; "
                         "implies --unfused")
    ap.add_argument("--hot", action="store_true",
                    help="back-to-back steps on warm caches: kernel times from eager steps, value from "
                         "the HIP-graph replay (default: cold, a 512 MiB buffer is written before every "
                         "step, outside its events, evicting L2 and the MALL; kernel times and value "
                         "from those steps)")
    ap.add_argument("--unfused", action="store_true",
                    help="time prepare, verify and commit as three launches (default: prepare + "
                         "the fused commit-then-verify step)")
    ap.add_argument("--sweep", action="store_true",
                    help="time fused, unfused and chunked steps over T in 32..512 on the large "
                         "recipe and on chains; prints one JSON line with the table")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="after timing, run 5 plain device copies of this many MiB (a known-size "
                         "kernel for scaling HBM counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU (asked for {max(args.gpus, world)}): every "
              "(sequence, head) unit is independent and there is no multi-GPU path.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2607_06763_amd import gdn_tree as G
    from paper_2607_06763_amd import workloads as W

    if not os.path.exists(G.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    torch.cuda.set_device(0)
    if args.sweep:
        res = sweep(G, torch, np, W, args)
        res["copy_GBs"] = round(copy_rate_gbs(torch), 1)
        print(json.dumps(res), flush=True)
        return 0
    w = W.make_sweep(args.tree_size, shape=args.shape) if args.tree_size else W.make_config(args.config)
    nbytes = algorithmic_bytes(w)
    nodes = w.B * w.T
    form = "chunked" if args.chunked else ("unfused" if args.unfused else "fused")
    fused = form == "fused"
    cold = not args.hot
    graph = args.graph and not cold
    r = measure(G, torch, np, w, form, args.steps, args.warmup, cold, graph)
    us_prep, us_main, ms_step = r["us_prep"], r["us_main"], r["ms_step"]
    p10, p50, p90 = r["us_main_p10_p50_p90"]
    src_hash = verify_source_hash()
    if fused:
        kname, kbytes = "step", nbytes["step"]
    else:
        kname, kbytes = ("verify_chunked" if args.chunked else "verify"), nbytes["verify"]
        us_com = r["us_commit"]
    ach = kbytes / (us_main * 1e-6) / 1e9
    copy_gbs = copy_rate_gbs(torch)
    traffic = measured_traffic(src_hash, kname, w.name)
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": kname, "algorithmic_bytes_per_launch": kbytes,
                "avg_launch_us": round(us_main, 3)}
    if fused:
        detail = {
            "us_prepare": round(us_prep, 3), "us_step": round(us_main, 3),
            "us_step_p10_p50_p90": [round(p10, 3), round(p50, 3), round(p90, 3)],
            "step_hbm_frac": round(ach / HBM_PEAK_GBS, 4),
        }
    else:
        detail = {
            "us_prepare": round(us_prep, 3), "us_verify": round(us_main, 3),
            "us_verify_p10_p50_p90": [round(p10, 3), round(p50, 3), round(p90, 3)],
            "us_commit": round(us_com, 3),
            "nodes_per_s_verify_only": round(nodes / (us_main * 1e-6), 1),
            "verify_hbm_frac": round(ach / HBM_PEAK_GBS, 4),
            "commit_GBs": round(nbytes["commit"] / (us_com * 1e-6) / 1e9, 1),
            "verify_plus_commit_hbm_frac": round(
                (nbytes["verify"] + nbytes["commit"]) / ((us_main + us_com) * 1e-6) / 1e9
                / HBM_PEAK_GBS, 4),
        }
    detail["copy_GBs"] = round(copy_gbs, 1)
    detail["frac_of_copy"] = round(ach / copy_gbs, 4)
    detail["algorithmic_bytes"] = nbytes
    detail["caches"] = ("cold: 512 MiB written before every timed step (outside its events); value = nodes / "
                        "the mean of the step's kernel times" if cold else
                        "hot: back-to-back steps" + ("; value from the HIP-graph replay" if graph else ""))
    if graph:
        detail["ms_per_step_eager"] = round(r["ms_eager"], 5)
    props = torch.cuda.get_device_properties(0)
    detail["device"] = f"{props.name} ({getattr(props, 'gcnArchName', '?')}, {props.multi_processor_count} CUs)"
    detail["verify_source_sha256_16"] = src_hash
    out = {
        "metric": "tree nodes verified/s per GDN layer",
        "value": round(nodes / (ms_step * 1e-3), 1),
        "unit": "nodes/s",
        "n_gpus": 1,
        "steps": 2 * r["reps"] if graph else args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.B} trees x T={w.T} nodes, Hk={w.Hk} Hv={w.Hv} "
                               f"dk={w.dk} dv={w.dv}, {w.in_dtype} inputs, fp32 state and output",
                   "global_batch": w.B, "seq_len": w.T, "parallelism": "none (1 GPU)",
                   "step": ("prepare + fused commit/verify" if fused else
                            "prepare + " + ("chunked " if args.chunked else "") + "verify + commit")
                           + (", HIP graph replay" if graph else ", cold caches" if cold else "")},
        "roofline": roofline,
        "detail": detail,
    }
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["detail"]["copy_calibration_bytes_each"] = 2 * 4 * n
        del src, dst
    if not args.no_cpu_baseline:
        cb = cpu_baseline(w)
        # part of this ratio is algorithmic: the oracle replays the full state
        # along every path, the GPU path pulls the query back
        cb["gpu_speedup_vs_naive_replay_oracle"] = {
            "all_threads": round(out["value"] / cb["value"], 1),
            "one_thread": round(out["value"] / cb["value_1thread"], 1)}
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
