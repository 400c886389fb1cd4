"""Per-phase clocks of the fused decode step up to 128 slots, or of the
chunked form's kernel (a diagnostic).

Not part of the verification path.  It copies csrc/ to a temporary
directory, inserts s_memtime stamps at the phase boundaries of the kernel
(lane 0 of a wave stores the counter to a buffer), builds that copy as a
separate library, points the binding at it and runs the kernel a few times
on a named workload.  It prints, per phase, the mean clocks over all
workgroups of the last launch.

    python3 -m paper_2607_06763_amd.phase_clocks [--config 4] [--launches 5]
    python3 -m paper_2607_06763_amd.phase_clocks --kernel chunked [--tree-size 512] [--shape large]

s_memtime counts shader clocks; a stamp lands in the buffer only if its
workgroup's linear index is below the buffer's capacity."""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

# (phase name, stamp before, stamp after); per-head stamps are k + 8 hh
PHASES = [
    ("prologue: metadata, q / k staging, conv, norms", 0, 1),
    ("commit of the previous path (window loads, features, replay)", 2, 3),
    ("raw v staging, gates, first row piece stored", 3, 4),
    ("v conv -> v~ in LDS", 4, 5),
    ("pull-back walk (this wave's nodes)", 5, 6),
    ("move to the MFMA layout + barrier", 6, 7),
    ("S0 plane, next head's loads + barrier", 7, 8),
    ("MFMA readout + output stores issued", 8, 9),
]
NSLOT = 64
WAVES = 8
CSLOT = 128  # stamps per workgroup of the chunked kernel (4 per 32-slot block)


def _instrument(src: str) -> str:
    def rep(old, new):
        nonlocal src
        if src.count(old) != 1:
            raise RuntimeError(f"phase_clocks: anchor not found once: {old[:70]!r}")
        src = src.replace(old, new)

    rep("  int32_t* commit_status;\n};", "  int32_t* commit_status;\n  unsigned long long* stamps;\n  long long stamp_cap;\n};")
    rep("namespace gdn {\n",
        "namespace gdn {\n"
        "#define TS(k) do { const long long lin_ = ((long long)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + "
        "blockIdx.x; if (p.stamps && lin_ < p.stamp_cap && (threadIdx.x & 63) == 0 && (threadIdx.x >> 6) < 8 && "
        "(k) < 64) p.stamps[lin_ * 512 + (threadIdx.x >> 6) * 64 + (k)] = __builtin_amdgcn_s_memtime(); } while (0)\n"
        "static unsigned long long* g_stamps = nullptr;\nstatic long long g_stamp_cap = 0;\n"
        "#define TR(k) do { const long long lin_ = ((long long)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + "
        "blockIdx.x; if (p.stamps && lin_ < p.stamp_cap && threadIdx.x == 0) "
        "p.stamps[lin_ * 512 + (k)] = __builtin_amdgcn_s_memrealtime(); } while (0)\n")
    rep("  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;\n",
        "  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;\n  TS(0);\n  TR(62);\n")
    rep("  // ---------------- phase 2: one value head at a time ----------------\n",
        "  TS(1);\n  // ---------------- phase 2: one value head at a time ----------------\n")
    rep("    if constexpr (FUSED) fused_commit<DK, DVS, TIn>(p, s_rv, s_ppath, Lp, b, g, h, c0, tid, sr);\n",
        "    TS(2 + 8 * hh);\n"
        "    if constexpr (FUSED) fused_commit<DK, DVS, TIn>(p, s_rv, s_ppath, Lp, b, g, h, c0, tid, sr);\n"
        "    TS(3 + 8 * hh);\n")
    rep("      if (Lp > 0) store_state_rows<DK, DVS, kSP>(p.S, b, Hv, DV, h, c0, tid, sr, 0);\n    __syncthreads();\n",
        "      if (Lp > 0) store_state_rows<DK, DVS, kSP>(p.S, b, Hv, DV, h, c0, tid, sr, 0);\n    __syncthreads();\n"
        "    TS(4 + 8 * hh);\n")
    rep("    // 2c: query pull-back along the path of each node", "    TS(5 + 8 * hh);\n    // 2c: query pull-back along the path of each node")
    rep("    // a_i x~_i and the value accumulators move to the MFMA layout:",
        "    TS(6 + 8 * hh);\n    // a_i x~_i and the value accumulators move to the MFMA layout:")
    rep("    __syncthreads();  // v~ consumed\n", "    __syncthreads();  // v~ consumed\n    TS(7 + 8 * hh);\n")
    rep("    lds_barrier();\n\n    // 2e: P^T", "    lds_barrier();\n    TS(8 + 8 * hh);\n\n    // 2e: P^T")
    rep("    lds_barrier();  // S0 planes consumed before the next head reuses the region\n  }\n",
        "    TS(9 + 8 * hh);\n    lds_barrier();  // S0 planes consumed before the next head reuses the region\n  }\n"
        "  TS(40);\n  TR(63);\n")
    rep("  p.commit_status = a.commit_status;\n",
        "  p.commit_status = a.commit_status;\n  p.stamps = g_stamps;\n  p.stamp_cap = g_stamp_cap;\n")
    src += ('\nextern "C" void gdn_phase_stamps(void* buf, long long cap_blocks) {\n'
            '  gdn::g_stamps = static_cast<unsigned long long*>(buf);\n'
            '  gdn::g_stamp_cap = buf ? cap_blocks : 0;\n}\n')
    return src


def _instrument_chunked(src: str) -> str:
    def rep(old, new):
        nonlocal src
        if src.count(old) != 1:
            raise RuntimeError(f"phase_clocks: anchor not found once: {old[:70]!r}")
        src = src.replace(old, new)

    rep("  float* U;        // [B][Hv][T][DV]: right-hand sides, then the solved rows\n};",
        "  float* U;        // [B][Hv][T][DV]: right-hand sides, then the solved rows\n"
        "  unsigned long long* stamps;\n  long long stamp_cap;\n};")
    rep("namespace gdn {\n",
        "namespace gdn {\n"
        "#define TS(k) do { const long long lin_ = (long long)blockIdx.y * gridDim.x + blockIdx.x; "
        "if (p.stamps && lin_ < p.stamp_cap && threadIdx.x == 0 && (k) < 128) "
        "p.stamps[lin_ * 128 + (k)] = __builtin_amdgcn_s_memtime(); } while (0)\n"
        "static unsigned long long* g_stamps = nullptr;\nstatic long long g_stamp_cap = 0;\n")
    rep("  // ---- metadata by position: node, parent position, log alpha, beta\n",
        "  TS(0);\n  // ---- metadata by position: node, parent position, log alpha, beta\n")
    rep("  // ---- phase A: a Q S0^T -> out, beta (V - a K S0^T) -> U\n",
        "  TS(1);\n  // ---- phase A: a Q S0^T -> out, beta (V - a K S0^T) -> U\n")
    rep("  // ---- phase B: forward substitution over the blocks\n",
        "  TS(2);\n  // ---- phase B: forward substitution over the blocks\n")
    rep("  for (int jb = 0; jb < NBv; ++jb) {\n    store_qk(jb);\n",
        "  for (int jb = 0; jb < NBv; ++jb) {\n    TS(4 + 4 * jb);\n    store_qk(jb);\n")
    rep("    // ---- diagonal block: A = -X_jj, M0 = I + A, Y_jj; R_j -> LDS\n",
        "    TS(5 + 4 * jb);\n    // ---- diagonal block: A = -X_jj, M0 = I + A, Y_jj; R_j -> LDS\n")
    rep("    // the inverse is in s_ma (M_4); U_j = M_4 R_j -> LDS and the workspace\n",
        "    TS(6 + 4 * jb);\n    // the inverse is in s_ma (M_4); U_j = M_4 R_j -> LDS and the workspace\n")
    rep("    // ---- O_j += Y_jj U_j, scaled and stored\n",
        "    TS(7 + 4 * jb);\n    // ---- O_j += Y_jj U_j, scaled and stored\n")
    rep("    __syncthreads();\n  }\n}\n\n// ---------------------------------------------------------------------------\n// Launch: features",
        "    __syncthreads();\n  }\n  TS(127);\n}\n\n// ---------------------------------------------------------------------------\n// Launch: features")
    rep("  hipLaunchKernelGGL((chunk_kernel<DK, DV, TIn>), dim3(p.Hv, p.B), dim3(kHT), SM::total, stream, p);",
        "  const_cast<ChunkParams&>(p).stamps = g_stamps;\n  const_cast<ChunkParams&>(p).stamp_cap = g_stamp_cap;\n"
        "  hipLaunchKernelGGL((chunk_kernel<DK, DV, TIn>), dim3(p.Hv, p.B), dim3(kHT), SM::total, stream, p);")
    src += ('\nextern "C" void gdn_chunk_stamps(void* buf, long long cap_blocks) {\n'
            '  gdn::g_stamps = static_cast<unsigned long long*>(buf);\n'
            '  gdn::g_stamp_cap = buf ? cap_blocks : 0;\n}\n')
    return src


def build_instrumented(workdir: str) -> str:
    """Copy of the library with stamps in the on-chip verify kernel and in
    the chunked form's kernel."""
    from . import build as B
    csrc = os.path.join(workdir, "csrc")
    shutil.copytree(B.CSRC, csrc)
    for name, fn in (("gdn_verify.hip", _instrument), ("gdn_chunked.hip", _instrument_chunked)):
        p = os.path.join(csrc, name)
        with open(p) as f:
            src = fn(f.read())
        with open(p, "w") as f:
            f.write(src)
    flags = [f if f != B.CSRC else csrc for f in B.CFLAGS]
    objs = []
    for name in sorted(os.listdir(csrc)):
        if name.endswith(".hip"):
            obj = os.path.join(workdir, name + ".o")
            r = subprocess.run([B.HIPCC, *flags, "-c", os.path.join(csrc, name), "-o", obj],
                               capture_output=True, text=True)
            if r.returncode:
                raise RuntimeError(f"hipcc failed for {name}:\n{r.stderr[-2000:]}")
            objs.append(obj)
    lib = os.path.join(workdir, "libgdntree_phases.so")
    subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, "-o", lib], check=True)
    return lib


def _run_chunked(args, G, W, np, torch, ctypes) -> int:
    L = G.lib()
    L.gdn_chunk_stamps.restype = None
    L.gdn_chunk_stamps.argtypes = [ctypes.c_void_p, ctypes.c_longlong]
    w = W.make_sweep(args.tree_size, B=32, shape=args.shape)
    dt = G.DeviceTree(w)
    dt.prepare()
    blocks = w.B * w.Hv
    stamps = torch.zeros(blocks * CSLOT, dtype=torch.int64, device="cuda")
    L.gdn_chunk_stamps(ctypes.c_void_p(stamps.data_ptr()), blocks)
    out = torch.empty_like(dt.out)
    for i in range(args.launches):
        stamps.zero_()
        dt.verify(out=out, chunked=True)
        torch.cuda.synchronize()
        print(f"[phase_clocks] launch {i + 1} done", flush=True)
    L.gdn_chunk_stamps(ctypes.c_void_p(0), 0)
    st = stamps.view(blocks, CSLOT).cpu().numpy().astype(np.float64)
    st = st[st[:, 0] > 0]
    nb = (w.T + 31) // 32
    rows = {"metadata": st[:, 1] - st[:, 0], "phase A (a Q S0^T, beta (V - a K S0^T))": st[:, 2] - st[:, 1]}
    acc = {"block tops and pairs with earlier blocks": 0.0, "diagonal block and its inverse": 0.0,
           "U_j": 0.0, "O_j stores (to the next block)": 0.0}
    for jb in range(nb):
        t4, t5, t6, t7 = (st[:, 4 + 4 * jb + k] for k in range(4))
        nxt = st[:, 4 + 4 * (jb + 1)] if jb + 1 < nb and 4 + 4 * (jb + 1) < CSLOT - 1 else st[:, CSLOT - 1]
        live = t4 > 0
        acc["block tops and pairs with earlier blocks"] += np.where(live, t5 - t4, 0)
        acc["diagonal block and its inverse"] += np.where(live, t6 - t5, 0)
        acc["U_j"] += np.where(live, t7 - t6, 0)
        acc["O_j stores (to the next block)"] += np.where(live & (nxt > 0), nxt - t7, 0)
    rows.update(acc)
    print(f"workload {w.name} ({args.shape}): B={w.B} T={w.T} Hk={w.Hk} Hv={w.Hv} dk={w.dk} dv={w.dv}; "
          f"{st.shape[0]} workgroups, {nb} blocks of 32 slots; clocks of the last launch")
    print("| phase | clocks per workgroup (mean) |")
    print("|---|---|")
    for k, v in rows.items():
        print(f"| {k} | {np.mean(v):.0f} |")
    print(f"| whole workgroup | {np.mean(st[:, CSLOT - 1] - st[:, 0]):.0f} |")
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--kernel", choices=("step", "chunked"), default="step")
    ap.add_argument("--config", type=int, default=4, help="named workload (step)")
    ap.add_argument("--tree-size", type=int, default=512, help="tree slots (chunked)")
    ap.add_argument("--shape", choices=("large", "chain"), default="large", help="tree shape (chunked)")
    ap.add_argument("--launches", type=int, default=5)
    ap.add_argument("--lib", default=None, help="an instrumented library built before (skips the build)")
    args = ap.parse_args()

    import ctypes

    import numpy as np
    import torch

    from . import gdn_tree as G
    from . import workloads as W

    workdir = None
    lib = args.lib
    if lib is None:
        workdir = tempfile.mkdtemp(prefix="gdn_phases_")
        print(f"[phase_clocks] building the instrumented copy in {workdir}", flush=True)
        lib = build_instrumented(workdir)
    G.LIB_PATH = lib
    try:
        if args.kernel == "chunked":
            return _run_chunked(args, G, W, np, torch, ctypes)
        return _run_step(args, G, W, np, torch, ctypes)
    finally:
        if workdir:
            shutil.rmtree(workdir, ignore_errors=True)


def _run_step(args, G, W, np, torch, ctypes) -> int:
    L = G.lib()
    L.gdn_phase_stamps.restype = None
    L.gdn_phase_stamps.argtypes = [ctypes.c_void_p, ctypes.c_longlong]

    w = W.make_config(args.config)
    if w.T > 128:
        raise SystemExit("phase_clocks times the on-chip kernel (T <= 128)")
    prev = G.DeviceTree(w)
    cur = G.DeviceTree(W.make_config(args.config))
    prev.prepare()
    cur.prepare()
    blocks = w.B * w.Hv * 8   # workgroups with room for stamps (more are not recorded)
    stamps = torch.zeros(blocks * WAVES * NSLOT, dtype=torch.int64, device="cuda")
    L.gdn_phase_stamps(ctypes.c_void_p(stamps.data_ptr()), blocks)
    S = prev.S0.clone()
    cs_in = prev.conv_state.clone()
    cs_out = torch.empty_like(cs_in)
    for i in range(args.launches):
        stamps.zero_()
        S.copy_(prev.S0)
        cur.step_from(prev, S, cs_in, cs_out)
        torch.cuda.synchronize()
        print(f"[phase_clocks] launch {i + 1} done", flush=True)
    L.gdn_phase_stamps(ctypes.c_void_p(0), 0)
    st = stamps.view(blocks, WAVES, NSLOT).cpu().numpy().astype(np.float64)
    live = st[:, 0, 0] > 0
    st = st[live]
    nblk = st.shape[0]
    heads = max(1, w.Hv // w.Hk) if w.B * w.Hk >= 256 else 1
    print(f"workload {w.name}: B={w.B} T={w.T} Hk={w.Hk} Hv={w.Hv} dk={w.dk} dv={w.dv}; "
          f"{nblk} workgroups, {heads} value head(s) each; clocks of the last launch")
    print("| phase | head | wave 0 | slowest wave |")
    print("|---|---|---|---|")
    total0 = st[:, 0, 40] - st[:, 0, 0]
    for name, a, b in PHASES:
        hs = [None] if a < 2 else range(heads)
        for hh in hs:
            ka, kb = (a, b) if hh is None else (a + 8 * hh, b + 8 * hh)
            d = st[:, :, kb] - st[:, :, ka]
            ok = (st[:, :, ka] > 0) & (st[:, :, kb] > 0)
            d0 = d[:, 0][ok[:, 0]]
            dm = np.where(ok, d, 0).max(axis=1)
            print(f"| {name} | {'' if hh is None else hh} | {d0.mean():.0f} | {dm.mean():.0f} |")
    print(f"| whole workgroup (wave 0) | | {total0.mean():.0f} | |")
    # s_memrealtime counts a constant 100 MHz: the ratio of the two counters
    # over the same span is the shader clock the stamps count
    real = st[:, 0, 63] - st[:, 0, 62]
    ok = real > 0
    if ok.any():
        ghz = (total0[ok] / real[ok]).mean() * 0.1
        print(f"shader clock over the workgroups' lifetimes: {ghz:.2f} GHz (s_memtime / s_memrealtime x 100 MHz)")
    return 0


if __name__ == "__main__":
    sys.exit(main())
