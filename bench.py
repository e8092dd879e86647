"""Benchmark: the range finder on the 16384 x 16384 fp64 workload, one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline]
    python bench.py --fixed-rank R[,R..] [--fixed-block B]
                                          fixed-rank mode (k_max = R, tol = 0,
                                          b = 128) against one-shot pipelines
                                          with the same sketch: QR and orgqr
                                          on this library's kernels, and
                                          rocSOLVER (Sec. 6 / Fig. 6)
    python bench.py --copy-probe MIB      one plain device copy of MIB MiB
                                          (calibrates the HBM byte counters)
    python bench.py --summarize DIR...    per-kernel summary of rocprofv3 CSVs
    python bench.py --pmc-report DIR... --copy-fetch D --copy-write D
                    [--traffic-out FILE --kernel NAME --workload W]
                                          counters per kernel, HBM bytes scaled
                                          by the copy probe, and the traffic
                                          record bench.py reads

A step is one rrf_run (Alg. 2 to the tolerance, then explicit Q and B) with A
already resident in HBM.  Prints one JSON line:
  value       algorithmic GFLOP/s of the whole run (flop counts of the method,
              no padding or speculative work), higher is better;
  ms_per_step wall time of one run;
  roofline    the dominant kernel (the fused update) against the fp64 MFMA
              peak, from HIP events on the plan's stream;
  gemm_wy     all GEMM-shaped stages together against the same peak;
  cpu_baseline the CPU oracle on a bounded sample of the same workload.
"""

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"float64": 78.6, "float32": 157.3}   # MI355X dense MFMA
HBM_GBS = 8000.0
METRIC = "range-finder wall time (s) + achieved GFLOP/s as % of MFMA peak"
GEMM_STAGES = ("sample", "reduce", "formw", "update", "orgqr")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="square_fp64_16384")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=3,
                    help="extra runs with per-kernel HIP-event timing")
    ap.add_argument("--fixed-rank", default=None, metavar="R[,R..]",
                    help="only the fixed-rank comparison at these ranks")
    ap.add_argument("--fixed-block", type=int, default=128,
                    help="block size b of the fixed-rank runs (Fig. 6: 128)")
    ap.add_argument("--subspace-map", action="store_true",
                    help="only time the GaLore subspace map (Sec. 7) on galore-sized bases")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run one device-to-device copy of MIB MiB")
    ap.add_argument("--summarize", nargs="+", default=None, metavar="DIR",
                    help="only summarise rocprofv3 CSV output (no GPU)")
    ap.add_argument("--pmc-report", nargs="+", default=None, metavar="DIR",
                    help="only report rocprofv3 --pmc CSV output (no GPU)")
    ap.add_argument("--copy-fetch", default=None, help="copy-probe FETCH_SIZE run")
    ap.add_argument("--copy-write", default=None, help="copy-probe WRITE_SIZE run")
    ap.add_argument("--traffic-out", default=None, help="write the traffic record here")
    ap.add_argument("--kernel", default=None, help="kernel of the traffic record")
    return ap.parse_args()


CSRC = os.path.join(ROOT, "paper_2608_28941_amd", "csrc")
COPY_PROBE_KERNEL = "copy_kernel<double>"


def sources_sha256():
    """Hash of the HIP/C++ sources: a traffic record is valid only for them."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def read_counters(dirs):
    """{kernel: {dispatch_id: {counter: value, "_ns": duration}}} from the
    counter_collection CSVs under dirs (values summed over instances)."""
    import csv
    import glob
    out = {}
    for d in dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                k = short_kernel(r["Kernel_Name"])
                disp = out.setdefault(k, {}).setdefault((f, r["Dispatch_Id"]), {})
                c = r["Counter_Name"]
                disp[c] = disp.get(c, 0.0) + float(r["Counter_Value"])
                disp["_ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    return out


def copy_scale(d, counter, known_bytes):
    """Bytes per counted byte, from the copy probe's single copy dispatch."""
    c = read_counters([d]).get(COPY_PROBE_KERNEL, {})
    vals = [v[counter] for v in c.values() if counter in v]
    if not vals:
        raise SystemExit(f"no {COPY_PROBE_KERNEL} {counter} in {d}")
    return known_bytes / (vals[0] * 1024.0)


def pmc_report(a):
    mib = 1024   # the copy probe that the calibration runs use
    known = mib * (1 << 20)
    fs = copy_scale(a.copy_fetch, "FETCH_SIZE", known) if a.copy_fetch else None
    ws = copy_scale(a.copy_write, "WRITE_SIZE", known) if a.copy_write else None
    cnt = read_counters(a.pmc_report)
    lines = ["| kernel | dispatches | avg us (counter run) | read GB/launch | write GB/launch | "
             "HBM GB/s | MFMA TFLOP/s | MFMA busy |", "|---|---:|---:|---:|---:|---:|---:|---:|"]
    rec = None
    for k in sorted(cnt, key=lambda x: -sum(v.get("_ns", 0) for v in cnt[x].values())):
        disp = list(cnt[k].values())
        def mean(c):
            v = [d[c] for d in disp if c in d]
            return sum(v) / len(v) if v else None
        ns = [d["_ns"] for d in disp if "FETCH_SIZE" in d or "WRITE_SIZE" in d] or \
             [d["_ns"] for d in disp]
        avg_ns = sum(ns) / len(ns)
        rd = mean("FETCH_SIZE")
        wr = mean("WRITE_SIZE")
        rd = rd * 1024.0 * fs if (rd is not None and fs) else None
        wr = wr * 1024.0 * ws if (wr is not None and ws) else None
        f64 = mean("SQ_INSTS_VALU_MFMA_MOPS_F64")
        f32 = mean("SQ_INSTS_VALU_MFMA_MOPS_F32")
        mops = (f64 or 0.0) + (f32 or 0.0)
        mfma_ns = [d["_ns"] for d in disp if "SQ_INSTS_VALU_MFMA_MOPS_F64" in d] or ns
        mfma_avg_ns = sum(mfma_ns) / len(mfma_ns)
        busy = mean("SQ_VALU_MFMA_BUSY_CYCLES")
        gui = mean("GRBM_GUI_ACTIVE")
        busy_frac = busy / (gui / 8.0 * 4 * 256) if (busy is not None and gui) else None
        gbs = ((rd or 0.0) + (wr or 0.0)) / avg_ns if (rd is not None or wr is not None) else None
        tf = mops * 512.0 / mfma_avg_ns / 1e3 if mops else None
        def fmt(x, f):
            return "" if x is None else f.format(x)
        lines.append(f"| {k} | {len(disp)} | {avg_ns / 1e3:.1f} | {fmt(rd and rd / 1e9, '{:.4f}')} | "
                     f"{fmt(wr and wr / 1e9, '{:.4f}')} | {fmt(gbs, '{:.0f}')} | {fmt(tf, '{:.2f}')} | "
                     f"{fmt(busy_frac, '{:.1%}')} |")
        if a.kernel and k == a.kernel:
            rec = {"rd": rd, "wr": wr, "n": sum(1 for d in disp if "FETCH_SIZE" in d)}
    print(f"copy-probe scale: FETCH_SIZE x{fs}, WRITE_SIZE x{ws} (bytes per counted byte)\n")
    print("\n".join(lines))
    if a.traffic_out:
        if not rec or rec["rd"] is None or rec["wr"] is None:
            raise SystemExit(f"no FETCH_SIZE/WRITE_SIZE for {a.kernel}")
        with open(a.traffic_out, "w") as f:
            f.write("# HBM traffic per launch of the dominant kernel: rocprofv3 --pmc FETCH_SIZE\n"
                    "# and WRITE_SIZE (KiB per dispatch) scaled by what the same counters read for a\n"
                    "# plain copy of known size (bench.py --copy-probe), averaged over the launches\n"
                    "# of one run.  Valid only for the sources with the hash below.\n")
            f.write(f"workload {a.workload}\nkernel {a.kernel}\nsources_sha256 {sources_sha256()}\n")
            f.write(f"fetch_scale {fs:.6f}\nwrite_scale {ws:.6f}\nlaunches {rec['n']}\n")
            f.write(f"fetch_bytes_per_launch {rec['rd']:.6e}\nwrite_bytes_per_launch {rec['wr']:.6e}\n")
            f.write(f"traffic_bytes_per_launch {rec['rd'] + rec['wr']:.6e}\n")


def read_traffic(workload):
    """Bytes per launch of the dominant kernel from the committed record, or
    None when there is none for this workload or the sources have changed."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        key, _, val = line.strip().partition(" ")
        rec[key] = val.strip()
    if rec.get("workload") != workload or rec.get("sources_sha256") != sources_sha256():
        return None
    try:
        return float(rec["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def short_kernel(name):
    """'void rrf::(anonymous namespace)::update_kernel<double, 64, 64>(...)'
    -> 'update_kernel<double, 64, 64>'."""
    name = re.sub(r"^void\s+", "", name)
    name = name.replace("rrf::(anonymous namespace)::", "").replace("rrf::", "")
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and i > 0:
            return name[:i]
    return name


def summarize(dirs):
    """Markdown tables of the kernel-trace statistics and of the per-dispatch
    counter values (mean over dispatches) found under ``dirs``."""
    import csv
    import glob
    lines = []
    for d in dirs:
        for f in sorted(glob.glob(os.path.join(d, "**", "*kernel_stats.csv"),
                                  recursive=True)):
            lines.append(f"### kernel statistics ({os.path.basename(f)})\n")
            lines.append("| kernel | calls | total ms | avg us | min us | max us | % |")
            lines.append("|---|---:|---:|---:|---:|---:|---:|")
            for r in csv.DictReader(open(f)):
                lines.append("| {} | {} | {:.3f} | {:.1f} | {:.1f} | {:.1f} | {} |".format(
                    short_kernel(r["Name"]), r["Calls"],
                    float(r["TotalDurationNs"]) / 1e6, float(r["AverageNs"]) / 1e3,
                    float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, r["Percentage"]))
            lines.append("")
        for f in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"),
                                  recursive=True)):
            acc = {}
            disp = {}
            for r in csv.DictReader(open(f)):
                k = short_kernel(r["Kernel_Name"])
                c = r["Counter_Name"]
                key = (k, c)
                acc.setdefault(key, {})
                did = r["Dispatch_Id"]
                acc[key][did] = acc[key].get(did, 0.0) + float(r["Counter_Value"])
                disp.setdefault(k, set()).add(did)
            counters = sorted({c for _, c in acc})
            lines.append(f"### counters, mean per dispatch ({os.path.basename(f)})\n")
            lines.append("| kernel | dispatches | " + " | ".join(counters) + " |")
            lines.append("|---|---:|" + "---:|" * len(counters))
            for k in sorted(disp):
                vals = []
                for c in counters:
                    v = acc.get((k, c))
                    vals.append("" if not v else "{:.6g}".format(sum(v.values()) / len(v)))
                lines.append(f"| {k} | {len(disp[k])} | " + " | ".join(vals) + " |")
            lines.append("")
    print("\n".join(lines))


def oneshot_lib(plan, A, Om, pb=64):
    """One-shot fixed-rank range finder on this library's kernels: Y = A Omega
    (one vendor GEMM), blocked Householder QR of Y with the library's panel QR
    (rrf_panel_qr) and block reflector (rrf_apply_block_reflector) in
    pb-column panels, Q = H_0 .. H_{r-1} [I_r; 0] backward with the same
    block reflector (orgqr), and B = Q^T A (one vendor GEMM).  A and Omega
    column-major; returns (Q, B) column-major / row-major."""
    import torch
    m = A.shape[0]
    r = Om.shape[1]
    Y = (Om.t() @ A.t()).t()                 # m x r, column-major
    refl = []
    for j in range(0, r, pb):
        jb = min(pb, r - j)
        V, T, _ = plan.panel_qr(Y[j:, j:j + jb])
        if j + jb < r:
            plan.apply_block_reflector(V, T, Y[j:, j + jb:], trans=True)
        refl.append((j, V, T))
    Q = torch.zeros(r, m, dtype=A.dtype, device=A.device).t()
    Q[:r, :r] = torch.eye(r, dtype=A.dtype, device=A.device)
    for j, V, T in reversed(refl):
        plan.apply_block_reflector(V, T, Q[j:, j:], trans=False)
    B = Q.t() @ A
    return Q, B


def fixed_rank(a):
    """Fixed-rank mode (Sec. 6, Fig. 6): rrf_run with k_max = r and tol = 0
    (r columns in r / b blocks, RRF_WARN_KMAX expected) at b = a.fixed_block
    against two one-shot fixed-rank range finders on the same GPU and the
    same sketch Omega (columns 0..r-1 of RRF-NORMAL-v1):
      lib:       Y = A Omega, blocked QR and orgqr on this library's panel
                 and block-reflector kernels, B = Q^T A (oneshot_lib);
      rocsolver: Y = A Omega, Q from torch.linalg.qr (rocSOLVER geqrf +
                 orgqr), B = Q^T A.
    Both comparators use the vendor GEMM for the two products.  Prints one
    JSON line."""
    import torch
    import paper_2608_28941_amd as rrf
    import workloads as W
    w = W.WORKLOADS[a.workload]
    A_host = W.build_matrix(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdt = torch.float64 if w.dtype == "float64" else torch.float32
    A = rrf.colmajor(torch.from_numpy(A_host).to(dev))
    del A_host
    normA = float(torch.linalg.norm(A.double()))
    ranks = [int(x) for x in a.fixed_rank.split(",")]
    b = a.fixed_block
    out = []

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            res = fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps, res

    def rel_res(Q, B):
        num = 0.0
        for c0 in range(0, A.shape[1], 2048):
            R = A[:, c0:c0 + 2048] - Q @ B[:, c0:c0 + 2048]
            num += float((R.double() ** 2).sum())
        return num ** 0.5 / normA

    with rrf.Plan(tdt, w.m, w.n, 64) as lib_plan:
        for r in ranks:
            print(f"[fixed-rank] r={r} b={b}", file=sys.stderr, flush=True)
            with rrf.Plan(tdt, w.m, w.n, b, k_max=r) as plan:
                t_ours, res = timed(lambda: plan.run_raw(A, 0.0, b, w.sketch_seed), a.steps)
                k = res[2]
                Q, B, _ = plan.run(A, 0.0, b, w.sketch_seed)
                res_ours = rel_res(Q, B)
                del Q, B
            Om = rrf.sketch(tdt, w.sketch_seed, w.n, 0, r)
            t_lib, (Ql, Bl) = timed(lambda: oneshot_lib(lib_plan, A, Om), a.steps)
            res_lib = rel_res(Ql, Bl)
            orth_lib = float(torch.linalg.norm(Ql.t() @ Ql - torch.eye(r, dtype=tdt, device=dev)))
            del Ql, Bl
            Ar = A.contiguous()

            def roc():
                Qo, _ = torch.linalg.qr(Ar @ Om)
                return Qo, Qo.t().contiguous() @ Ar
            t_roc, (Qo, Bo) = timed(roc, a.steps)
            del Ar
            res_roc = rel_res(Qo, Bo)
            del Qo, Bo, Om
            fl = algorithmic_flops(w.m, w.n, k, b)
            fl_one = (4.0 * w.m * w.n * r + 4.0 * w.m * r * r - 4.0 / 3.0 * r ** 3)
            out.append({"r": r, "k": k, "ours_ms": round(t_ours * 1e3, 3),
                        "ours_gflops": round(fl / t_ours / 1e9, 1),
                        "ours_residual": res_ours,
                        "oneshot_lib_ms": round(t_lib * 1e3, 3),
                        "oneshot_lib_gflops": round(fl_one / t_lib / 1e9, 1),
                        "oneshot_lib_residual": res_lib, "oneshot_lib_orth": orth_lib,
                        "rocsolver_ms": round(t_roc * 1e3, 3),
                        "rocsolver_gflops": round(fl_one / t_roc / 1e9, 1),
                        "rocsolver_residual": res_roc})
            print(f"[fixed-rank] r={r} ours {t_ours*1e3:.2f} ms, one-shot (library kernels) "
                  f"{t_lib*1e3:.2f} ms, one-shot (rocSOLVER) {t_roc*1e3:.2f} ms",
                  file=sys.stderr, flush=True)
    print(json.dumps({"metric": "fixed-rank wall time (ms): adaptive range finder with "
                                "k_max = r vs one-shot pipelines",
                      "workload": w.name, "dtype": w.dtype, "block_b": b,
                      "steps": a.steps, "results": out}))


def subspace_map_bench(a):
    """Time rrf_subspace_map (Q_new^T (Q_old M)) for the galore_fp32_4096x4096
    shape: 4096-row fp32 bases of ranks 512 and 448 and a 512 x 4096 state,
    random orthonormal bases (synthetic)."""
    import torch
    import paper_2608_28941_amd as rrf
    m, r0, r1, n = 4096, 512, 448, 4096
    g = torch.Generator(device="cpu").manual_seed(9)
    Q_old = torch.linalg.qr(torch.randn(m, r0, generator=g, dtype=torch.float64))[0]
    Q_new = torch.linalg.qr(torch.randn(m, r1, generator=g, dtype=torch.float64))[0]
    M = torch.randn(r0, n, generator=g, dtype=torch.float64)
    dev = [rrf.colmajor(t.to(torch.float32).to("cuda:0")) for t in (Q_new, Q_old, M)]
    with rrf.Plan(torch.float32, m, n, 64) as p:
        for _ in range(max(a.warmup, 1)):
            p.subspace_map(*dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(a.steps):
            out = p.subspace_map(*dev)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / a.steps
    flops = 2.0 * m * r1 * r0 + 2.0 * r1 * r0 * n
    ref = Q_new.T @ (Q_old @ M)
    err = float((out.double().cpu() - ref).abs().max())
    print(json.dumps({"op": "subspace_map", "m": m, "r_old": r0, "r_new": r1, "n": n,
                      "dtype": "f32", "ms": round(dt * 1e3, 4),
                      "tflops": round(flops / dt / 1e12, 2),
                      "frac_of_fp32_mfma_peak": round(flops / dt / 1e12 / PEAK_TFLOPS["float32"], 3),
                      "max_abs_err_vs_fp64": err, "data": "synthetic"}))


def copy_probe(mib):
    """One device copy of ``mib`` MiB through the library's copy kernel:
    reads and writes exactly mib MiB, the scale for FETCH_SIZE/WRITE_SIZE."""
    import ctypes
    import torch
    from paper_2608_28941_amd import _abi
    rows = 1 << 17                      # 1 MiB of float64 per column
    src = torch.ones(rows * mib, dtype=torch.float64, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    lib = _abi.load()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    _abi.check(lib.rrf_copy_matrix(_abi.RRF_F64,
                                   ctypes.c_void_p(src.data_ptr()), rows,
                                   ctypes.c_void_p(dst.data_ptr()), rows, rows, mib, s),
               "rrf_copy_matrix")
    torch.cuda.synchronize()
    ok = bool(torch.equal(src, dst))
    print(json.dumps({"copy_probe_mib": mib, "bytes_read": rows * mib * 8,
                      "bytes_written": rows * mib * 8, "equal": ok}))
    if not ok:
        sys.exit(1)


def algorithmic_flops(m, n, k, b):
    """Flops the method itself performs for rank k with block b (no padding,
    no speculative sample of the final block): per block, sample 2 m_i n b_i,
    block update 4 m_i n b_i + n b_i^2, panel 3 m_i b_i^2 - 2/3 b_i^3; then
    explicit Q 2 m k^2 - 2/3 k^3."""
    f = 0.0
    kk = 0
    while kk < k:
        bi = min(b, k - kk)
        mi = m - kk
        f += 2.0 * mi * n * bi + 4.0 * mi * n * bi + n * bi * bi
        f += 3.0 * mi * bi * bi - 2.0 / 3.0 * bi ** 3
        kk += bi
    f += 2.0 * m * k * k - 2.0 / 3.0 * k ** 3
    return f


def blas_info():
    """The BLAS library numpy runs on (threadpoolctl): vendor, version, threads."""
    try:
        import threadpoolctl
        for d in threadpoolctl.threadpool_info():
            if d.get("user_api") == "blas":
                return {"internal_api": d.get("internal_api"), "version": d.get("version"),
                        "num_threads": int(d.get("num_threads", 1))}
    except Exception:
        pass
    return {"internal_api": None, "version": None, "num_threads": os.cpu_count() or 1}


def cpu_baseline(A_host, w, budget_cols=1024, kmax=None):
    """The oracle (numpy, float64) on a bounded sample: the first block of
    Alg. 2 on the first ``budget_cols`` columns of the same matrix; next to
    it the whole oracle (Alg. 2 to the tolerance, explicit Q) on the
    500 x 300 fp64 workload, one warm-up and the mean of three runs."""
    import numpy as np
    import workloads as W
    from oracle import hbarrf
    blas = blas_info()
    nc = min(budget_cols, A_host.shape[1])
    As = np.asfortranarray(A_host[:, :nc])
    kmax = kmax or w.block_b
    t0 = time.perf_counter()
    r = hbarrf(As, 0.0, w.block_b, w.sketch_seed, k_max=kmax, dtype=w.np_dtype)
    dt = time.perf_counter() - t0
    fl = algorithmic_flops(As.shape[0], nc, r.k, w.block_b)
    wt = W.WORKLOADS["tiny_fp64_500x300"]
    At = W.build_matrix(wt)
    hbarrf(At, wt.tol, wt.block_b, wt.sketch_seed)
    t1 = time.perf_counter()
    for _ in range(3):
        rt = hbarrf(At, wt.tol, wt.block_b, wt.sketch_seed)
    dtt = (time.perf_counter() - t1) / 3
    flt = algorithmic_flops(wt.m, wt.n, rt.k, wt.block_b)
    return {"value": fl / dt / 1e9, "unit": "GFLOP/s", "cores": blas["num_threads"],
            "kind": "oracle", "seconds": dt, "blas": blas,
            "sample": (f"first block (k={r.k}) of Alg. 2 on A[:, :{nc}] of "
                       f"{w.name} ({As.shape[0]}x{nc}), numpy float64, "
                       f"one reflector at a time"),
            "whole_run_tiny": {"workload": wt.name, "k": rt.k, "ms": dtt * 1e3,
                               "gflops": flt / dtt / 1e9}}


def main():
    a = parse()
    if a.summarize:
        summarize(a.summarize)
        return
    if a.pmc_report:
        pmc_report(a)
        return
    if a.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {a.gpus});"
              " the sharded design is described in DESIGN.md", file=sys.stderr)
        sys.exit(2)
    if a.copy_probe > 0:
        copy_probe(a.copy_probe)
        return
    if a.subspace_map:
        subspace_map_bench(a)
        return
    if a.fixed_rank:
        fixed_rank(a)
        return
    import torch
    import paper_2608_28941_amd as rrf
    import workloads as W

    w = W.WORKLOADS[a.workload]
    print(f"[bench] building {w.name} ({w.m}x{w.n} {w.dtype})", file=sys.stderr,
          flush=True)
    A_host = W.build_matrix(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    A = rrf.colmajor(torch.from_numpy(A_host).to(dev))
    tdt = torch.float64 if w.dtype == "float64" else torch.float32
    plan = rrf.Plan(tdt, w.m, w.n, w.block_b)

    def step():
        return plan.run_raw(A, w.tol, w.block_b, w.sketch_seed)

    print("[bench] warmup", file=sys.stderr, flush=True)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] timing {a.steps} steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for _ in range(a.steps):
        _, _, k, _, _, status = step()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / max(a.steps, 1)
    tr = plan.trace()
    flops = algorithmic_flops(w.m, w.n, k, w.block_b)

    # Per-kernel timing (HIP events on the plan's stream) in separate runs.
    stages = None
    if a.profile_steps > 0:
        plan.set_timing(True)
        acc = {}
        for _ in range(a.profile_steps):
            step()
            for s, v in plan.stage_stats().items():
                d = acc.setdefault(s, {"ms": 0.0, "launches": 0, "flops": 0.0,
                                       "bytes": 0.0})
                for key in d:
                    d[key] += v[key]
        plan.set_timing(False)
        stages = {s: {"ms": v["ms"] / a.profile_steps,
                      "launches": v["launches"] // a.profile_steps,
                      "flops": v["flops"] / a.profile_steps,
                      "bytes": v["bytes"] / a.profile_steps}
                  for s, v in acc.items()}

    peak = PEAK_TFLOPS[w.dtype]
    roof = None
    gemm = None
    if stages:
        upd = stages["update"]
        ach = upd["flops"] / (upd["ms"] * 1e-3) / 1e12 if upd["ms"] > 0 else 0.0
        traffic = read_traffic(w.name)
        roof = {"bound": "mfma",
                "kernel": "update (B -= V W, next sample, norms; with look-ahead also "
                          "the next panel)",
                "achieved": round(ach, 3), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4),
                "traffic": None if traffic is None else round(traffic, 0),
                "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE)",
                "avg_launch_ms": upd["ms"] / max(upd["launches"], 1),
                "launches_per_step": upd["launches"]}
        gf = sum(stages[s]["flops"] for s in GEMM_STAGES)
        gm = sum(stages[s]["ms"] for s in GEMM_STAGES)
        gach = gf / (gm * 1e-3) / 1e12 if gm > 0 else 0.0
        gemm = {"achieved": round(gach, 3), "peak": peak, "unit": "TFLOP/s",
                "frac": round(gach / peak, 4), "ms": gm,
                "stage_ms": {s: round(v["ms"], 4) for s, v in stages.items()}}

    base = None
    if not a.no_cpu_baseline:
        print("[bench] cpu baseline (oracle, bounded sample)", file=sys.stderr,
              flush=True)
        base = cpu_baseline(A_host, w)

    out = {
        "metric": METRIC,
        "value": round(flops / wall / 1e9, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(wall * 1e3, 4),
        "wall_s": round(wall, 6),
        "pct_of_mfma_peak": round(100.0 * flops / wall / (peak * 1e12), 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64" if w.dtype == "float64" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "m": w.m, "n": w.n, "block_b": w.block_b,
                   "tol": w.tol, "k": k, "blocks": tr["nblocks"],
                   "algorithmic_flops": flops, "status": status,
                   "matrix_seed": w.matrix_seed, "sketch_seed": w.sketch_seed},
        "roofline": roof,
        "gemm_wy": gemm,
        "cpu_baseline": base,
    }
    print(json.dumps(out))
    plan.close()


if __name__ == "__main__":
    main()
