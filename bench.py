"""Benchmark: ExTernD factorization throughput on one MI355X.

A step is one complete factorization (every step of the hot path: staging,
selection, block ALS iterations, joint scale solves, deflations, packing)
of one synthetic matrix already resident in HBM.  Default workload: the
9728 x 2560 MLP down-projection-shaped matrix (Student-t(4), std 0.015,
log-normal(0, 0.3) row scales), mu = 3 (k = 7680), tau = 1.0, block = 64,
8 ALS iterations.

Prints one JSON line with the throughput (ALS components per second), the
roofline position of the dominant kernel (HIP events recorded around its
launches during the timed region) and the CPU oracle timed on a bounded
sample of the same workload.
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

import numpy as np  # noqa: E402

METRIC = "sec/matrix + ALS components/sec at 9728×2560 μ=3 τ=1.0; energy preserved E"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
INT8_PEAK_TOPS = 5000.0        # MI355X dense int8 MFMA, published
# The one-launch sequential path runs in a single workgroup, i.e. on one of
# the 256 compute units: its ceiling is one CU's share of the published fp32
# vector rate (157.3 TFLOP/s / 256).
CHIP_FP32_PEAK_GFLOPS = 157.3e3
CU_FP32_PEAK_GFLOPS = CHIP_FP32_PEAK_GFLOPS / 256
# the kernels and the launch geometry (grid sizes and workspace layout)
KERNEL_SOURCES = ["paper_2607_13511_amd/csrc/externd_kernels.hip", "paper_2607_13511_amd/csrc/externd_api.hip",
                  "paper_2607_13511_amd/csrc/externd_internal.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.json")


def workload(name: str):
    from paper_2607_13511_amd import synth
    if name == "down9728":
        return synth.down9728(weighted=False)
    if name == "down9728_imatrix":
        return synth.down9728(weighted=True)
    if name in ("down9728_b256", "down9728_b256_imatrix"):
        # the same matrix at the paper's default block width (Sec. 2.4)
        import dataclasses
        w = synth.down9728(weighted=name.endswith("_imatrix"))
        return dataclasses.replace(w, name=w.name.replace("_b64", "_b256"), block=256)
    if name == "attn2048":
        return synth.attn2048()
    if name == "gauss256":
        return synth.gauss256()
    if name == "block4b":
        return None      # the seven matrices of a transformer block: bench_block
    raise SystemExit(f"unknown workload {name}")


def sequential_gap(w, curve, block):
    """GPU energy minus that of the greedy sequential ALS oracle (one component
    at a time, Sec. 2.3) at the workload's checkpoints, taken from the stored
    full-size record of that oracle when one exists for this exact input (the
    record carries the sha256 of the matrix). None when there is no record."""
    path = os.path.join(ROOT, "tests", "golden", "seq", f"seq_{w.name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    A = np.ascontiguousarray(w.A, dtype=np.float32)
    if (rec["m"], rec["n"], rec["block"], rec["iters"]) != (A.shape[0], A.shape[1], w.block, w.iters) \
            or rec["mu"] != w.mu or rec["tau"] != w.tau or rec["weighted"] != (w.h is not None) \
            or hashlib.sha256(A.tobytes()).hexdigest() != rec["a_sha256"]:
        return None
    seq, stride = rec["seq_curve"], rec["seq_stride"]
    out = {"record": os.path.relpath(path, ROOT), "oracle_seconds": rec["seq_seconds"], "checkpoints": {}}
    for kc in rec["checkpoints_k"]:
        b, s = kc // block - 1, kc // stride - 1
        if 0 <= b < len(curve) and 0 <= s < len(seq):
            out["checkpoints"][f"k={kc}"] = {"gpu": float(curve[b]), "sequential": seq[s],
                                             "gpu_minus_sequential": float(curve[b]) - seq[s]}
    return out


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def vstep_row_groups(m: int, n: int) -> int:
    """Row groups of the V-step contraction (the library's layout rule:
    about 480 column-tile x row-group workgroups, at most 8)."""
    nct, nrt = -(-n // 32), -(-m // 32)
    return max(1, min(-(-480 // nct), min(nrt, 8)))


def seq_flops(m: int, n: int, k: int, iters: int) -> float:
    """Algorithmic flops of one factorization on the one-launch sequential
    path: per component, each ALS iteration contracts the residual twice
    (R^T u and R diag(h~) v: a multiply-add per entry, 2 m n flops each),
    and the deflation and the column energies take one more multiply-add
    per entry each (2 m n flops each)."""
    return float(k) * (4.0 * iters + 4.0) * m * n


def algorithmic_bytes(kclass: str, m: int, n: int) -> float:
    """Algorithmic HBM bytes per launch: the residual is read once by each
    contraction (4 m n) and read and written once by the deflation (8 m n);
    the ternary operands and outputs add < 2 % and are not counted.  The
    target kernels read the contraction's output (V: the row groups' int64
    partials of P, 64 x n each; U: Q, 64 x m fp64) and write the fp64
    target (64 x n or 64 x m).  The ternarizations read the fp64 target
    and write the factor in two int8 forms (component-major and MFMA-ready);
    the last U-step of a block also reads Q, which is not counted."""
    if kclass == "deflate":
        return 8.0 * m * n
    if kclass == "vstep_target":
        return (vstep_row_groups(m, n) + 1) * 64 * 8.0 * n
    if kclass == "ustep_target":
        return 2 * 64 * 8.0 * m
    if kclass == "ternarize_v":
        return 64 * (8.0 + 2.0) * n
    if kclass == "ternarize_u":
        return 64 * (8.0 + 2.0) * m
    return 4.0 * m * n


def traffic_from_counters(kclass: str):
    """Measured HBM bytes per launch from committed rocprofv3 counter data,
    or None when absent or taken on a different kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("kernel_source_sha256") != kernel_source_hash():
        return None
    ent = data.get("kernels", {}).get(kclass)
    if not ent:
        return None
    return float(ent["fetch_bytes"] + ent["write_bytes"])


def oracle_threads() -> tuple:
    """Threads the numpy oracle may use on this host: the cores this process
    may run on, capped by OMP_NUM_THREADS when the environment sets it.
    Returns (threads, cores in the affinity mask)."""
    avail = len(os.sched_getaffinity(0))
    try:
        cap = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        cap = 0
    return (min(avail, cap) if cap > 0 else avail), avail


def cpu_baseline(w, comps: int, blocks: int):
    """The CPU oracle as it stands, timed on a bounded sample of the same
    workload: the sequential greedy ALS (Sec. 2.3, one component at a time)
    on its first `comps` components, and the block ALS (Sec. 2.4) on its
    first `blocks` blocks.  Every component of a run costs the same (the
    iteration count is fixed and the residual stays dense), so the time per
    matrix is the sample time scaled to k.  The BLAS pool is limited to the
    threads reported."""
    import oracle
    threads, avail = oracle_threads()
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover - threadpoolctl missing
        threadpool_limits = None
    import contextlib
    ctx = threadpool_limits(limits=threads) if threadpool_limits else contextlib.nullcontext()
    m, n = w.A.shape
    k = oracle.rank_of(m, n, w.mu)
    with ctx:
        t0 = time.perf_counter()
        oracle.factorize_sequential(w.A, w.mu, w.tau, w.iters, h=w.h, k=comps)
        dt = time.perf_counter() - t0
        out = {"value": comps / dt, "unit": "components/s", "cores": int(threads), "kind": "oracle",
               "sample": f"first {comps} of {k} components of the sequential greedy ALS (oracle.factorize_sequential, "
                         f"fp64 numpy) on {w.name}", "seconds": dt, "sec_per_matrix_extrapolated": dt * k / comps,
               "host_cores_in_affinity": int(avail)}
        if blocks > 0:
            t0 = time.perf_counter()
            f = oracle.factorize_block(w.A, w.mu, w.tau, w.block, w.iters, h=w.h, max_blocks=blocks)
            db = time.perf_counter() - t0
            bc = blocks * f.block
            out["block_oracle"] = {"value": bc / db, "unit": "components/s", "seconds": db,
                                   "sample": f"first {blocks} blocks ({bc} of {f.k} components) of the block ALS "
                                             f"(oracle.factorize_block, fp64 numpy)",
                                   "sec_per_matrix_extrapolated": db * f.k / bc}
    return out


def sparsity_and_bpw(res, m: int, n: int, k: int) -> dict:
    """Zero fractions of the factors, decoded from the packed 2-bit trits
    (code 00 is zero), and the effective storage of Eq. (5): under mask+sign
    packing an element costs 2 - sparsity bits, and k (m + n) elements are
    stored for m n weights, i.e. mu (m + n) / max(m, n) (2 - sparsity) bits
    per original weight (mu = k / min(m, n))."""
    import torch

    def zeros(packed, rows, cols):
        p = packed.reshape(rows, -1)
        z = 0
        for t in range(4):
            code = (p >> (2 * t)) & 3
            valid = cols - t - 1 >= 4 * torch.arange(p.shape[1], device=p.device)
            z += int(((code == 0) & valid).sum().item())
        return z

    zb, zc = zeros(res.B_packed, m, k), zeros(res.C_packed, k, n)
    sp = (zb + zc) / float(k * (m + n))
    mu = k / min(m, n)
    return {"zero_fraction_B": zb / float(m * k), "zero_fraction_C": zc / float(k * n), "sparsity": sp,
            "bpw_eff": mu * (m + n) / max(m, n) * (2.0 - sp), "bpw_eff_rule": "Eq. (5): mu (m+n)/max(m,n) (2 - sparsity)"}


def calibrate_copy(nbytes: int, reps: int):
    """A plain device copy of known size, for scaling the FETCH_SIZE and
    WRITE_SIZE counters (run under rocprofv3 --pmc)."""
    import torch
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").uniform_()
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}))


def collect_traffic(dbs, copy_bytes: int):
    """Per-launch HBM bytes of the timed kernel classes from rocprofv3 --pmc
    databases (FETCH_SIZE run, WRITE_SIZE run, and the same two counters on
    a plain device copy of copy_bytes), each counter scaled by copy-bytes /
    the counter's reading for the copy.  Writes profiles/traffic_counters.json
    and a short markdown summary beside it."""
    import re
    import sqlite3

    def per_kernel(path, counter):
        con = sqlite3.connect(path)
        rows = con.execute("select kernel_name, count(*), avg(value) from counters_collection "
                           "where counter_name=? group by kernel_name", (counter,)).fetchall()
        return {re.sub(r"\(.*", "", k).replace("void ", "").replace("externd::", ""): (int(c), float(a) * 1024.0)
                for k, c, a in rows}

    fetch, write = per_kernel(dbs[0], "FETCH_SIZE"), per_kernel(dbs[1], "WRITE_SIZE")
    cfetch, cwrite = per_kernel(dbs[2], "FETCH_SIZE"), per_kernel(dbs[3], "WRITE_SIZE")
    copy_f = max(v[1] for k, v in cfetch.items() if "copyBuffer" in k)
    copy_w = max(v[1] for k, v in cwrite.items() if "copyBuffer" in k)
    ff, fw = copy_bytes / copy_f, copy_bytes / copy_w
    classes = {"vstep_contraction": "k_vstep", "ustep_contraction": "k_ustep<false>", "deflate": "k_deflate<false>",
               "vstep_target": "k_vtarget", "ustep_target": "k_utarget", "ternarize_v": "k_tern_v",
               "ternarize_u": "k_tern_u"}
    out = {"kernel_source_sha256": kernel_source_hash(), "copy_bytes": copy_bytes,
           "fetch_scale": ff, "write_scale": fw, "kernels": {}}
    lines = ["# HBM traffic per launch (rocprofv3 --pmc), 9728x2560 workload", "",
             "Commands (repository root, one MI355X):", "", "```",
             "rocprofv3 --pmc FETCH_SIZE -d gpurun_out/pmc_fetch -o pmc -- python bench.py --steps 1 --warmup 0 --cpu-comps 0",
             "rocprofv3 --pmc WRITE_SIZE -d gpurun_out/pmc_write -o pmc -- python bench.py --steps 1 --warmup 0 --cpu-comps 0",
             f"rocprofv3 --pmc FETCH_SIZE -d gpurun_out/pmc_copy_fetch -o pmc -- python bench.py --calibrate-copy {copy_bytes}",
             f"rocprofv3 --pmc WRITE_SIZE -d gpurun_out/pmc_copy_write -o pmc -- python bench.py --calibrate-copy {copy_bytes}",
             "python bench.py --collect-traffic gpurun_out/pmc_fetch/pmc_results.db gpurun_out/pmc_write/pmc_results.db "
             f"gpurun_out/pmc_copy_fetch/pmc_results.db gpurun_out/pmc_copy_write/pmc_results.db --copy-bytes {copy_bytes}",
             "```", "",
             f"Copy calibration: a {copy_bytes} B device copy reads FETCH_SIZE = {copy_f:.0f} B and WRITE_SIZE = "
             f"{copy_w:.0f} B, so fetch counts are scaled by {ff:.4f} and write counts by {fw:.4f}.", "",
             "| kernel | launches | fetch MB/launch | write MB/launch | algorithmic MB/launch |", "|---|---:|---:|---:|---:|"]
    m, n = 9728, 2560
    for cls, kname in classes.items():
        if kname not in fetch:
            continue
        fb, wb = fetch[kname][1] * ff, write.get(kname, (0, 0.0))[1] * fw
        out["kernels"][cls] = {"kernel": kname, "launches": fetch[kname][0], "fetch_bytes": fb, "write_bytes": wb}
        lines.append(f"| {kname} | {fetch[kname][0]} | {fb / 1e6:.1f} | {wb / 1e6:.1f} | "
                     f"{algorithmic_bytes(cls, m, n) / 1e6:.1f} |")
    lines += ["", "All kernels (unscaled counter averages, MiB per launch):", "",
              "| kernel | launches | FETCH_SIZE | WRITE_SIZE |", "|---|---:|---:|---:|"]
    for k in sorted(fetch, key=lambda k: -fetch[k][0] * fetch[k][1]):
        lines.append(f"| {k} | {fetch[k][0]} | {fetch[k][1] / 2**20:.2f} | {write.get(k, (0, 0.0))[1] / 2**20:.2f} |")
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    with open(os.path.join(ROOT, "profiles", "traffic_down9728x2560.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps(out))


KERNEL_CLASS = {"k_vstep": "vstep_contraction", "k_ustep": "ustep_contraction", "k_ustep<false>": "ustep_contraction",
                "k_ustep<true>": "ustep_contraction", "k_deflate": "deflate", "k_deflate<false>": "deflate",
                "k_deflate<true>": "deflate", "k_vtarget": "vstep_target", "k_utarget": "ustep_target",
                "k_tern_v": "ternarize_v", "k_tern_u": "ternarize_u"}


def _short_kernel(name: str) -> str:
    import re
    return re.sub(r"\(.*", "", name).replace("void ", "").replace("externd::", "")


def render_command() -> str:
    import shlex
    return "python " + " ".join(shlex.quote(a) for a in sys.argv)


def render_trace(db: str, out_path: str, title: str, command: str, shape=None):
    """Markdown summary of a rocprofv3 --kernel-trace database: calls, total
    and average duration per kernel; with the matrix shape, the algorithmic
    bytes per launch of each timed kernel class (the same rule as the bench
    line's roofline) over the rocprofv3 average, as GB/s and as a fraction
    of 8 TB/s."""
    import sqlite3
    con = sqlite3.connect(db)
    cols = [r[1] for r in con.execute("pragma table_info(kernels)")]
    name_col = "kernel_name" if "kernel_name" in cols else "name"
    agg = {}
    for k, c, tot in con.execute(f"select {name_col}, count(*), sum(end - start) from kernels group by {name_col}"):
        kk = _short_kernel(k)
        c0, s0 = agg.get(kk, (0, 0.0))
        agg[kk] = (c0 + c, s0 + tot)
    total = sum(v[1] for v in agg.values())
    lines = [f"# {title}", "", "Command (from the repository root, on one MI355X):", "", "```", command, "```", "",
             "Rendered with:", "", "```", render_command(), "```", "",
             f"Kernel dispatches summed over the whole run (warm-up and timed steps): {total / 1e6:.1f} ms of GPU time.",
             ""]
    if shape:
        m, n = shape
        lines += [f"Rates use the algorithmic bytes per launch at m = {m}, n = {n} (bench.py algorithmic_bytes) over "
                  "the average duration below.", "",
                  "| kernel | calls | total (us) | average (us) | share | algorithmic GB/s | of 8 TB/s |",
                  "|---|---:|---:|---:|---:|---:|---:|"]
    else:
        lines += ["| kernel | calls | total (us) | average (us) | share |", "|---|---:|---:|---:|---:|"]
    for k, (c, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        row = f"| {k} | {c} | {t / 1e3:.1f} | {t / c / 1e3:.2f} | {100 * t / total:.1f}% |"
        if shape:
            cls = KERNEL_CLASS.get(k)
            if cls:
                gbs = algorithmic_bytes(cls, *shape) / (t / c * 1e-9) / 1e9
                row += f" {gbs:.0f} | {gbs / HBM_PEAK_GBS:.3f} |"
            else:
                row += " | |"
        lines.append(row)
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def render_mfma(db: str, out_path: str, command: str, m: int = 9728, n: int = 2560):
    """Markdown summary of a rocprofv3 --pmc run over the MFMA counters
    (SQ_VALU_MFMA_BUSY_CYCLES and the int8 / bf16 / fp64 MOPS counters):
    MFMA operations issued per launch beside the algorithmic count, and the
    MFMA pipes' busy fraction over the launch."""
    import sqlite3
    con = sqlite3.connect(db)
    data = {}
    for k, c, v, d, cnt in con.execute("select kernel_name, counter_name, avg(value), avg(duration), count(*) "
                                      "from counters_collection group by kernel_name, counter_name"):
        e = data.setdefault(_short_kernel(k), {})
        e[c], e["dur"], e["n"] = v, d, cnt
    bb = 64
    alg = {"vstep_contraction": 4 * 2.0 * m * n * bb, "ustep_contraction": 4 * 2.0 * m * n * bb,
           "deflate": 3 * 2.0 * m * n * bb}
    lines = [f"# MFMA counters per launch (rocprofv3 --pmc), {m}x{n} workload (mu=3, tau=1.0, b=64, 8 iterations)",
             "", "Command (from the repository root, on one MI355X):", "", "```", command, "```", "",
             "Rendered with:", "", "```", render_command(), "```", "",
             "MOPS counters count MFMA math operations / 512. `busy` is SQ_VALU_MFMA_BUSY_CYCLES summed over the 1024 "
             "SIMDs; utilisation = busy / (dispatch duration under the counter run x 2.4 GHz x 1024 SIMDs). The int8 "
             "count of a contraction is 4 x 2 m n 64 operations per launch (four 8-bit digit planes of the fixed-point "
             "residual, block width 64); the deflation's bf16 work is 3 x 2 m n 64 (three exact bf16 parts of each "
             "scale).", "",
             "| kernel | launches | int8 ops | bf16 ops | fp64 ops | algorithmic MFMA ops | busy cycles | duration (us) "
             "| MFMA utilisation |", "|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for k in sorted(data, key=lambda k: -data[k].get("SQ_VALU_MFMA_BUSY_CYCLES", 0)):
        d = data[k]
        busy = d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0)
        if busy <= 0:
            continue
        i8, b16, f64 = (d.get(f"SQ_INSTS_VALU_MFMA_MOPS_{t}", 0) * 512 for t in ("I8", "BF16", "F64"))
        a = alg.get(KERNEL_CLASS.get(k, ""), None)
        util = busy / (d["dur"] * 1e-9 * 2.4e9 * 1024)
        lines.append(f"| {k} | {d['n']} | {i8:.4g} | {b16:.4g} | {f64:.4g} | {f'{a:.4g}' if a else '—'} | {busy:.4g} "
                     f"| {d['dur'] / 1e3:.1f} | {100 * util:.1f}% |")
    lines += ["", "The contractions and the deflation are bound by HBM bandwidth (a pass over the residual), not by "
              "the matrix cores: at the measured durations their MFMA pipes are busy for the fractions shown."]
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="down9728")
    ap.add_argument("--cpu-comps", type=int, default=96,
                    help="sequential-oracle sample in components (0 = skip the CPU baseline)")
    ap.add_argument("--cpu-blocks", type=int, default=32, help="block-oracle sample in blocks (0 = skip)")
    ap.add_argument("--calibrate-copy", type=int, default=0, help="run only a copy of this many bytes")
    ap.add_argument("--collect-traffic", nargs=4, metavar="DB",
                    help="rocprofv3 --pmc databases: FETCH_SIZE, WRITE_SIZE, copy FETCH_SIZE, copy WRITE_SIZE")
    ap.add_argument("--copy-bytes", type=int, default=268435456)
    ap.add_argument("--apply", action="store_true",
                    help="time inference with the workload's factorization (externd_apply, nb = 1 and 8)")
    ap.add_argument("--sweeps", type=int, default=None,
                    help="time externd_factorize_refined with this many refinement sweeps instead")
    ap.add_argument("--concurrency", type=int, default=4,
                    help="block4b: factorizations in flight at once (one HIP stream, host thread and "
                         "workspace each; the 21 jobs are dealt longest first)")
    ap.add_argument("--target-energy", type=float, default=None,
                    help="time the energy-target run instead (stop at the first block with E >= target, "
                         "mu of the workload as the maximum)")
    ap.add_argument("--render-trace", nargs=4, metavar=("DB", "OUT", "TITLE", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --kernel-trace database (rates for --workload)")
    ap.add_argument("--render-mfma", nargs=3, metavar=("DB", "OUT", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --pmc run over the MFMA counters")
    args = ap.parse_args()
    if args.render_trace:
        w = workload(args.workload)
        render_trace(*args.render_trace, shape=None if w is None else w.A.shape)
        return
    if args.render_mfma:
        render_mfma(*args.render_mfma)
        return
    if args.collect_traffic:
        collect_traffic(args.collect_traffic, args.copy_bytes)
        return

    if args.gpus != 1:
        print(json.dumps({"error": f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
                                   "this build has no multi-GPU path"}))
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy, 5)
        return

    from paper_2607_13511_amd import binding
    binding.lib()      # fails loudly when the HIP library is missing

    w = workload(args.workload)
    if w is None:
        return bench_block(binding, torch, args)
    m, n = w.A.shape
    dev = torch.device("cuda:0")
    if args.sweeps is not None:
        return bench_sweeps(binding, torch, w, args)
    if args.target_energy is not None:
        bench_target(binding, torch, w, args)
        return
    if args.apply:
        bench_apply(binding, torch, w, args)
        return
    A = torch.from_numpy(w.A).to(dev)
    h = torch.from_numpy(w.h).to(dev) if w.h is not None else None
    k = binding.rank(m, n, w.mu)
    ws = torch.empty(binding.workspace_bytes(m, n, k), dtype=torch.uint8, device=dev)
    print(f"bench: {w.name} m={m} n={n} k={k} block={w.block} iters={w.iters}", file=sys.stderr, flush=True)

    for i in range(args.warmup):
        r = binding.factorize(A, w.mu, w.tau, w.block, w.iters, h=h, workspace=ws)
        print(f"bench: warmup {i} E={r.E:.6f}", file=sys.stderr, flush=True)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ktot = {}
    res = None
    for i in range(args.steps):
        res = binding.factorize(A, w.mu, w.tau, w.block, w.iters, h=h, workspace=ws, timed=True)
        for kc, (ms, cnt, issued) in res.kernel_times.items():
            a, b, c = ktot.get(kc, (0.0, 0, 0))
            ktot[kc] = (a + ms, b + cnt, c + issued)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    sec_per_matrix = dt / args.steps
    print(f"bench: timed {args.steps} steps, {sec_per_matrix * 1e3:.2f} ms/matrix E={res.E:.6f}",
          file=sys.stderr, flush=True)

    ktot = {kc: v for kc, v in ktot.items() if v[1] > 0}      # classes this workload launches
    # dominant kernel class by summed duration
    dom = max(ktot, key=lambda kc: ktot[kc][0] / max(1, ktot[kc][1]) * ktot[kc][2])
    dom_ms, dom_cnt, _ = ktot[dom]
    avg_s = dom_ms / dom_cnt / 1e3
    if dom == "sequential_one_launch":
        flops = seq_flops(m, n, k, w.iters)
        achieved = flops / avg_s / 1e9
        roofline = {"bound": "alu", "achieved": achieved, "peak": CHIP_FP32_PEAK_GFLOPS, "unit": "GFLOP/s",
                    "frac": achieved / CHIP_FP32_PEAK_GFLOPS, "traffic": None, "kernel": dom,
                    "avg_launch_us": avg_s * 1e6, "algorithmic_flops_per_launch": flops,
                    "one_cu_peak": CU_FP32_PEAK_GFLOPS, "frac_of_one_cu": achieved / CU_FP32_PEAK_GFLOPS,
                    "note": "one workgroup on one compute unit: peak is the chip's fp32 vector rate "
                            "(157.3 TFLOP/s = 256 CUs x 2.4 GHz x 256 flop/clk); frac_of_one_cu against 1/256 of it"}
    else:
        abytes = algorithmic_bytes(dom, m, n)
        achieved = abytes / avg_s / 1e9
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, "traffic": traffic_from_counters(dom),
                    "kernel": dom, "avg_launch_us": avg_s * 1e6, "algorithmic_bytes_per_launch": abytes}
    per_kernel = {}
    for kc, (ms, cnt, issued) in ktot.items():
        avg = ms / cnt / 1e3
        if kc == "sequential_one_launch":
            per_kernel[kc] = {"launches_per_matrix": issued // args.steps, "avg_us": avg * 1e6,
                              "GFLOP_s": seq_flops(m, n, k, w.iters) / avg / 1e9, "share_of_step": avg * issued / dt}
            continue
        gbs = algorithmic_bytes(kc, m, n) / avg / 1e9
        # one launch in binding.TIMING_STRIDE is timed (events on the library's stream)
        per_kernel[kc] = {"timed_launches_per_matrix": cnt / args.steps,
                          "launches_per_matrix": issued // args.steps,
                          "avg_us": avg * 1e6, "GB_s": gbs,
                          "share_of_step": avg * issued / dt}
        if kc in ("vstep_contraction", "ustep_contraction"):
            # int8 MFMA work issued: 4 digit planes x 2 m n (block padded to 64)
            tops = 4 * 2.0 * m * n * 64 / avg / 1e12
            per_kernel[kc]["mfma_int8_tops"] = tops
            per_kernel[kc]["mfma_frac"] = tops / INT8_PEAK_TOPS
    checkpoints = {}
    for kk in w.checkpoints_k:
        b = kk // res.block - 1
        if 0 <= b < len(res.curve):
            checkpoints[f"k={kk}"] = float(res.curve[b])

    factors = sparsity_and_bpw(res, m, n, k)
    cpu = None
    if args.cpu_comps > 0:
        print(f"bench: CPU oracle on {args.cpu_comps} sequential components and {args.cpu_blocks} blocks",
              file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_comps, args.cpu_blocks)

    out = {
        "metric": METRIC,
        "value": k / sec_per_matrix,
        "unit": "components/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec_per_matrix * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": w.name, "m": m, "n": n, "mu": w.mu, "tau": w.tau, "block": res.block,
                   "iters": w.iters, "k": k, "importance": w.h is not None},
        "sec_per_matrix": sec_per_matrix,
        "energy": res.E,
        "energy_w": res.E_w,
        "energy_checkpoints": checkpoints,
        "sequential_oracle": sequential_gap(w, res.curve, res.block),
        "factors": factors,
        "arithmetic": ("fp32 residual in registers of one workgroup; fp32 per-thread partial sums combined in "
                       "fp64; fp64 thresholds, scales and energies") if dom == "sequential_one_launch" else
                      ("fp32 residual; exact int8-MFMA contractions of 32-bit fixed point; fp64 targets/solves; "
                       "bf16-MFMA deflation with fp32 accumulation"),
        "roofline": roofline,
        "kernels": per_kernel,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def bench_block(binding, torch, args):
    """The seven matrices of one synthetic ~4B transformer block (q 2560x4096,
    k and v 2560x1024, o 4096x2560, gate and up 2560x9728, down 9728x2560;
    Student-t(4) at std 0.02, importance weights exp(N(0, 1))), factorized
    matrix by matrix to mu = 3.5 at each tau in (0.7, 1.0, 2.0), block 64,
    8 ALS iterations, importance-weighted: the whole sweep is one step.
    Energies at mu = 2, 2.5 and 3.5 come from the per-block curve (every
    prefix of a greedy run is the run to that rank)."""
    from paper_2607_13511_amd import synth
    dev = torch.device("cuda:0")
    mats = []
    for idx in range(len(synth.BLOCK_SHAPES)):
        name, A, h = synth.transformer_block(idx)
        mats.append((name, torch.from_numpy(A).to(dev), torch.from_numpy(h).to(dev)))
    taus, mu, block, iters = (0.7, 1.0, 2.0), 3.5, 64, 8
    jobs = [(name, A, h, tau) for tau in taus for name, A, h in mats]
    # longest first: cost ~ k m n ~ mu min(m, n) m n
    jobs.sort(key=lambda j: -min(j[1].shape) * j[1].shape[0] * j[1].shape[1])
    nconc = max(1, args.concurrency)
    wsize = max(binding.workspace_bytes(A.shape[0], A.shape[1], binding.rank(A.shape[0], A.shape[1], mu))
                for _, A, _ in mats)
    lanes = []
    for _ in range(nconc):
        st = torch.cuda.Stream()      # default priority
        with torch.cuda.stream(st):
            lanes.append((st, torch.empty(wsize, dtype=torch.uint8, device=dev)))
    torch.cuda.synchronize()

    def run_job(lane, job):
        st, ws = lane
        name, A, h, tau = job
        with torch.cuda.stream(st):
            t0 = time.perf_counter()
            r = binding.factorize(A, mu, tau, block, iters, h=h, workspace=ws, stream=st)
            dt = time.perf_counter() - t0
        m, n = A.shape
        pts = {}
        for mu_c in (2.0, 2.5, 3.5):
            b = binding.rank(m, n, mu_c) // r.block - 1
            pts[str(mu_c)] = {"E": float(r.curve[b]), "E_w": float(r.curve_w[b])}
        return f"{name}@tau{tau}", {"m": m, "n": n, "k": r.k, "sec": dt, "components_per_s": r.k / dt,
                                    "checkpoints": pts}

    def one_step(record):
        import threading
        per, lock, nxt = {}, threading.Lock(), [0]

        def worker(i):
            while True:
                with lock:
                    if nxt[0] >= len(jobs):
                        return
                    job = jobs[nxt[0]]
                    nxt[0] += 1
                key, val = run_job(lanes[i], job)
                with lock:
                    per[key] = val

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(nconc)]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        torch.cuda.synchronize()
        return per if record else {}

    for _ in range(args.warmup):
        one_step(False)
    t0 = time.perf_counter()
    per = {}
    for _ in range(args.steps):
        per = one_step(True)
    sec = (time.perf_counter() - t0) / args.steps
    comps = sum(v["k"] for v in per.values())
    print(json.dumps({
        "metric": "sec per transformer block (7 matrices x 3 tau) + ALS components/sec", "value": comps / sec,
        "unit": "components/s", "higher_is_better": True, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "sec_per_step": sec, "data": "synthetic",
        "config": {"workload": "transformer_block_4b_7mat_mu3.5_tau0.7-1.0-2.0_b64_imatrix", "mu": mu,
                   "taus": list(taus), "block": block, "iters": iters, "importance": True,
                   "concurrency": nconc},
        "job_sec_sum_per_tau": {str(t): sum(v["sec"] for k2, v in per.items() if k2.endswith(f"tau{t}"))
                                for t in taus},
        "matrices": per,
    }), flush=True)


def bench_apply(binding, torch, w, args):
    """Time y = B (diag(D) (C x)) on the packed factors of the workload's
    factorization (HIP events on the current stream, 50 launches per batch
    size).  Algorithmic bytes per call: the packed B and C, D, the inputs and
    outputs and the k x nb fp32 intermediate diag(D) C X^T (written and
    read)."""
    m, n = w.A.shape
    dev = torch.device("cuda:0")
    A = torch.from_numpy(w.A).to(dev)
    res = binding.factorize(A, w.mu, w.tau, w.block, w.iters)
    k = res.k
    out = {"metric": "inference y = B(diag(D)(C x)) time per call", "unit": "us", "higher_is_better": False,
           "n_gpus": 1, "data": "synthetic", "config": {"workload": w.name, "m": m, "n": n, "k": k}, "batches": {}}
    for nb in (1, 8):
        X = torch.randn((nb, n), dtype=torch.float32, device=dev)
        ws = torch.empty(binding.lib().externd_apply_workspace_bytes(m, n, k, nb), dtype=torch.uint8, device=dev)
        for _ in range(3):
            binding.apply(res.B_packed, res.C_packed, res.D, m, n, X, workspace=ws)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 50
        a.record()
        for _ in range(reps):
            binding.apply(res.B_packed, res.C_packed, res.D, m, n, X, workspace=ws)
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / reps
        nbytes = m * ((k + 3) // 4) + k * ((n + 3) // 4) + 4 * k + 4 * nb * (n + m) + 2 * 4 * k * nb
        out["batches"][str(nb)] = {"us_per_call": us, "bytes_per_call": nbytes, "GB_s": nbytes / us / 1e3,
                                   "frac_of_8TBs": nbytes / us / 1e3 / HBM_PEAK_GBS,
                                   "trit_macs_per_s": nb * k * (m + n) / us / 1e-6}
    print(json.dumps(out), flush=True)


def bench_target(binding, torch, w, args):
    """Time externd_factorize_to_energy on the workload: the components needed
    to reach the target (effective mu) and the time per matrix."""
    m, n = w.A.shape
    dev = torch.device("cuda:0")
    A = torch.from_numpy(w.A).to(dev)
    h = torch.from_numpy(w.h).to(dev) if w.h is not None else None
    k = binding.rank(m, n, w.mu)
    ws = torch.empty(binding.workspace_bytes(m, n, k), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        binding.factorize_to_energy(A, w.mu, args.target_energy, w.tau, w.block, w.iters, h=h, workspace=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        res = binding.factorize_to_energy(A, w.mu, args.target_energy, w.tau, w.block, w.iters, h=h, workspace=ws)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    print(json.dumps({
        "metric": "sec/matrix to reach the energy target", "value": sec, "unit": "s", "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "data": "synthetic",
        "config": {"workload": w.name, "target_energy": args.target_energy, "mu_max": w.mu, "tau": w.tau,
                   "block": res.block, "iters": w.iters, "importance": w.h is not None},
        "k_used": res.k_used, "mu_effective": res.k_used / min(m, n), "energy": res.E, "energy_w": res.E_w,
        "components_per_s": res.k_used / sec,
    }), flush=True)


def bench_sweeps(binding, torch, w, args):
    """Time externd_factorize_refined on the workload: extraction plus
    ``--sweeps`` refinement sweeps, with the energy before and after."""
    m, n = w.A.shape
    dev = torch.device("cuda:0")
    A = torch.from_numpy(w.A).to(dev)
    h = torch.from_numpy(w.h).to(dev) if w.h is not None else None
    k = binding.rank(m, n, w.mu)
    ws = torch.empty(binding.workspace_bytes(m, n, k), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        binding.factorize_refined(A, w.mu, w.tau, w.block, w.iters, args.sweeps, h=h, workspace=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        res = binding.factorize_refined(A, w.mu, w.tau, w.block, w.iters, args.sweeps, h=h, workspace=ws)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    F = res.factorization
    print(json.dumps({
        "metric": "sec/matrix with refinement sweeps", "value": sec, "unit": "s", "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "data": "synthetic",
        "config": {"workload": w.name, "mu": w.mu, "tau": w.tau, "block": F.block, "iters": w.iters,
                   "sweeps": args.sweeps, "importance": w.h is not None},
        "energy_extraction": float(F.curve[-1]), "energy_w_extraction": float(F.curve_w[-1]),
        "sweep_energy": [float(x) for x in res.sweep_curve],
        "sweep_energy_w": [float(x) for x in res.sweep_curve_w],
        "accepted": res.accepted, "revisits": res.revisits,
    }), flush=True)


if __name__ == "__main__":
    main()
