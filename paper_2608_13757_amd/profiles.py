"""Profiler summaries for the kernels of this package.

Turns rocprofv3 output into the short records kept under ``profiles/``:

* ``traffic``: HBM bytes per launch of one kernel from two ``--pmc`` runs
  (``FETCH_SIZE`` then ``WRITE_SIZE``, KiB per dispatch), each scaled by the
  same counter's reading for a device copy of known size run in the same
  process (``bench.py --copy-calibration-mib``), next to the algorithmic
  bytes; stamped with a digest of the kernel's sources so that a stale record
  is never reported for a changed kernel.
* ``trace``: the per-kernel table of a ``--kernel-trace --stats`` run.
* ``sq``: shader-sequencer counters of the uninstrumented dispatches of both
  modes from ``--pmc`` runs (at most 8 SQ counters per run): wave cycles,
  cycles spent waiting, instruction mix, MFMA busy cycles and MFMA work, per
  dispatch, with the wait and issue shares of the wave cycles and, from
  ``GRBM_GUI_ACTIVE``, the shader clock and the MFMA and LDS busy shares.

Usage (from the repository root, after the rocprofv3 runs)::

    python -m paper_2608_13757_amd.profiles traffic --kernel gemm \\
        --fetch-dir OUT/pf --write-dir OUT/pw --copy-mib 1024 \\
        --algorithmic-bytes 100679680 --workload "..." --command "..." --command "..."
    python -m paper_2608_13757_amd.profiles trace --kernel gemm --stats-dir OUT/pt \\
        --workload "..." --command "..."
"""
import argparse
import csv
import glob
import hashlib
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PROFILES = os.path.join(ROOT, "profiles")

# sources whose text determines each kernel's code, and the name fragment of
# its barrier-free, uninstrumented dispatch in rocprofv3 output
KERNELS = {
    "stream3": (["kern_stream3.hip", "device_sync.h", "bfs_internal.h"], ["stream3_kernel<0, false"]),
    "gemm": (["kern_gemm.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"], ["gemm_kernel<0, false, 1, 0>"]),
    "attn": (["kern_attn.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"], ["attn_kernel<0, false>"]),
    "rms": (["kern_rms.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"], ["rms_kernel<0, false, 4>"]),
    "adamw": (["kern_adamw.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"], ["adamw_kernel<0, false>"]),
    "moe": (["kern_moe.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"],
            ["moe_kernel<1, 0, false, 256>", "moe_kernel<2, 0, false, 256>"]),
    "chain": (["kern_chain.hip", "engine_sync.h", "device_sync.h", "bfs_internal.h"], ["chain_kernel<0, false>"]),
}
COPY_NAMES = ("__amd_rocclr_copyBuffer",)   # the runtime's device-to-device copy


def digest(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNELS[kernel][0]:
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str):
    """HBM bytes per launch (per step for a multi-kernel step) from
    profiles/<kernel>_traffic.json, or None when absent or stale."""
    path = os.path.join(PROFILES, f"{kernel}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_source_digest") != digest(kernel):
        return None
    return rec.get("traffic_bytes_per_step")


def _counter_rows(d: str):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    with open(files[0]) as fh:
        return list(csv.DictReader(fh))


def _per_dispatch(rows, counter, match):
    """Mean over dispatches whose kernel name contains ``match`` of the
    counter summed over its instances (one row per dispatch and counter)."""
    by_dispatch = {}
    for r in rows:
        if r["Counter_Name"] != counter or match not in r["Kernel_Name"]:
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id") or len(by_dispatch)
        by_dispatch[key] = by_dispatch.get(key, 0.0) + float(r["Counter_Value"])
    if not by_dispatch:
        raise SystemExit(f"no {counter} rows for {match}")
    vals = list(by_dispatch.values())
    return sum(vals) / len(vals), len(vals)


def _copy_reading(rows, counter, copy_bytes):
    best = None
    for r in rows:
        if r["Counter_Name"] == counter and any(n in r["Kernel_Name"] for n in COPY_NAMES):
            v = float(r["Counter_Value"])
            best = v if best is None else max(best, v)
    if best is None:
        raise SystemExit(f"no copy dispatch with {counter}")
    return best


def traffic(args):
    _, names = KERNELS[args.kernel]
    copy_bytes = args.copy_mib << 20
    fr, wr = _counter_rows(args.fetch_dir), _counter_rows(args.write_dir)
    f_copy, w_copy = _copy_reading(fr, "FETCH_SIZE", copy_bytes), _copy_reading(wr, "WRITE_SIZE", copy_bytes)
    fetch_factor = copy_bytes / (f_copy * 1024.0)
    write_factor = copy_bytes / (w_copy * 1024.0)
    per_kernel = {}
    total = 0.0
    for n in names:
        f_kib, nf = _per_dispatch(fr, "FETCH_SIZE", n)
        w_kib, nw = _per_dispatch(wr, "WRITE_SIZE", n)
        rd, wt = f_kib * 1024.0 * fetch_factor, w_kib * 1024.0 * write_factor
        per_kernel[n] = {"FETCH_SIZE_KiB_per_dispatch": f_kib, "WRITE_SIZE_KiB_per_dispatch": w_kib,
                         "dispatches": [nf, nw], "read_bytes": rd, "write_bytes": wt}
        total += rd + wt
    rec = {
        "kernel": args.kernel, "workload": args.workload, "commands": args.command,
        "calibration": {"copy_bytes": copy_bytes, "copy_FETCH_SIZE_KiB": f_copy, "copy_WRITE_SIZE_KiB": w_copy,
                        "fetch_factor": fetch_factor, "write_factor": write_factor},
        "per_kernel": per_kernel,
        "traffic_bytes_per_step": total,
        "algorithmic_bytes_per_step": args.algorithmic_bytes,
        "traffic_over_algorithmic": total / args.algorithmic_bytes,
        "kernel_source_digest": digest(args.kernel),
    }
    out = os.path.join(PROFILES, f"{args.kernel}_traffic.json")
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(out, json.dumps({k: rec[k] for k in ("traffic_bytes_per_step", "traffic_over_algorithmic")}))


def trace(args):
    files = glob.glob(os.path.join(args.stats_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {args.stats_dir}")
    with open(files[0]) as fh:
        rows = list(csv.DictReader(fh))
    stem = args.kernel if args.kernel != "stream3" else "stream3"
    lines = [f"# {args.kernel} kernel: kernel trace ({args.workload})", "",
             "Command (run from the repository root on one MI355X, `TMPDIR=/tmp`):", ""]
    for c in args.command:
        lines += ["```", c, "```", ""]
    lines += ["Template arguments: <mode, instrumented> (mode 0 = barrier-free, 1 = barrier); "
              "MoE: <phase, mode, instrumented>.  `interp_kernel` is the generic interpreter "
              "(mode and instrumentation are run-time arguments there).", "",
              "| Kernel | Calls | Average ns | Min ns | Max ns |", "|---|---|---|---|---|"]
    stems = ("stream3_kernel<", "gemm_kernel<", "attn_kernel<", "moe_kernel<", "rms_kernel<", "adamw_kernel<",
             "chain_kernel<", "interp_kernel")
    for r in rows:
        name = r["Name"]
        if not any(t in name for t in stems):
            continue
        short = name[name.index("::") + 2:] if "::" in name else name
        short = short.split("(")[0]
        lines.append(f"| `{short}` | {r['Calls']} | {float(r['AverageNs']):.0f} | {float(r['MinNs']):.0f} | "
                     f"{float(r['MaxNs']):.0f} |")
    out = os.path.join(PROFILES, f"{stem}_kernel_trace.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(out)


SQ_DERIVED = [
    ("wait share of wave cycles", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES"),
    ("issue share of wave cycles", "SQ_ACTIVE_INST_ANY", "SQ_WAVE_CYCLES"),
    ("LDS instructions per wave", "SQ_INSTS_LDS", "SQ_WAVES"),
    ("SALU instructions per wave", "SQ_INSTS_SALU", "SQ_WAVES"),
    ("branches per wave", "SQ_INSTS_BRANCH", "SQ_WAVES"),
]


N_XCD, N_CU, N_SIMD = 8, 256, 1024     # MI355X: XCDs, compute units, SIMDs


def _mean_duration_s(rows, match):
    """Mean duration (s) of the dispatches whose kernel name contains
    ``match``, from the start and end timestamps (ns) of their rows."""
    spans = {}
    for r in rows:
        if match in r["Kernel_Name"] and r.get("Start_Timestamp") and r.get("End_Timestamp"):
            key = r.get("Dispatch_Id") or r.get("Correlation_Id")
            spans[key] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    return sum(spans.values()) / len(spans) if spans else None


def sq(args):
    """Per-dispatch means of every SQ counter of the runs, for each
    uninstrumented kernel instantiation of the family, with the shader clock
    (GRBM_GUI_ACTIVE per XCD over the dispatch's duration) and the MFMA and
    LDS busy shares of the clock cycles when those counters are present."""
    stem = {"stream3": "stream3_kernel<", "gemm": "gemm_kernel<", "attn": "attn_kernel<",
            "moe": "moe_kernel<", "rms": "rms_kernel<", "adamw": "adamw_kernel<",
            "chain": "chain_kernel<"}[args.kernel]
    table = {}          # kernel -> counter -> (mean, dispatches)
    clock = {}          # kernel -> (GRBM_GUI_ACTIVE per XCD, mean dispatch duration)
    for d in args.dir:
        rows = _counter_rows(d)
        names = sorted({r["Kernel_Name"] for r in rows if stem in r["Kernel_Name"]})
        counters = sorted({r["Counter_Name"] for r in rows})
        for n in names:
            short = n[n.index(stem):].split("(")[0]
            if ", true" in short:
                continue
            for c in counters:
                table.setdefault(short, {})[c] = _per_dispatch(rows, c, n)
            if "GRBM_GUI_ACTIVE" in counters:
                clock[short] = (table[short]["GRBM_GUI_ACTIVE"][0] / N_XCD, _mean_duration_s(rows, n))
    kernels = sorted(table)
    counters = sorted({c for k in kernels for c in table[k]})
    lines = [f"# {args.kernel} kernel: SQ counters, barrier-free vs barrier ({args.workload})", "",
             "Commands (run from the repository root on one MI355X, `TMPDIR=/tmp`):", ""]
    for c in args.command:
        lines += ["```", c, "```", ""]
    lines += ["Per-dispatch means over the timed and warm-up launches (counter values summed over the "
              "hardware instances).  Template arguments: <mode, instrumented, ...> (mode 0 = barrier-free, "
              "1 = barrier); MoE: <phase, mode, instrumented, M-tile rows>.  SQ_WAVE_CYCLES, SQ_BUSY_CYCLES, "
              "SQ_WAIT_ANY and SQ_ACTIVE_INST_ANY are in quad cycles (only their ratios are used); "
              "SQ_VALU_MFMA_BUSY_CYCLES counts shader-clock cycles per SIMD, SQ_LDS_IDX_ACTIVE per compute "
              "unit, and GRBM_GUI_ACTIVE per XCD.  The profiler serializes dispatches, so the clock row "
              "divides GRBM_GUI_ACTIVE per XCD by the dispatch's own duration.", "",
              "| Counter | " + " | ".join(f"`{k}`" for k in kernels) + " |",
              "|---|" + "---|" * len(kernels)]
    for c in counters:
        lines.append(f"| {c} | " + " | ".join(f"{table[k][c][0]:.4g}" if c in table[k] else "" for k in kernels)
                     + " |")
    for label, num, den in SQ_DERIVED + ([("MFMA bf16 FLOP (512 per MOP)", "SQ_INSTS_VALU_MFMA_MOPS_BF16", None)]):
        vals = []
        for k in kernels:
            t = table[k]
            if num not in t or (den is not None and den not in t):
                vals.append("")
            elif den is None:
                vals.append(f"{t[num][0] * 512:.4g}")
            else:
                vals.append(f"{t[num][0] / t[den][0]:.3f}")
        lines.append(f"| *{label}* | " + " | ".join(vals) + " |")
    if clock:
        def busy(counter, units):
            return [f"{table[k][counter][0] / (clock[k][0] * units):.3f}" if k in clock and counter in table[k]
                    else "" for k in kernels]
        # launches of a few microseconds are dominated by the time the GPU
        # stays active around the dispatch: no clock estimate for them
        lines.append("| *shader clock (GHz)* | " + " | ".join(
            f"{clock[k][0] / clock[k][1] / 1e9:.2f}" if k in clock and clock[k][1] and clock[k][1] > 50e-6 else ""
            for k in kernels) + " |")
        lines.append("| *MFMA busy share of SIMD cycles* | " + " | ".join(busy("SQ_VALU_MFMA_BUSY_CYCLES", N_SIMD))
                     + " |")
        lines.append("| *LDS busy share of CU cycles* | " + " | ".join(busy("SQ_LDS_IDX_ACTIVE", N_CU)) + " |")
    out = os.path.join(PROFILES, f"{args.kernel}_sq.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(out)


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--kernel", required=True, choices=sorted(KERNELS))
    t.add_argument("--fetch-dir", required=True)
    t.add_argument("--write-dir", required=True)
    t.add_argument("--copy-mib", type=int, default=1024)
    t.add_argument("--algorithmic-bytes", type=float, required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--command", action="append", default=[])
    k = sub.add_parser("trace")
    k.add_argument("--kernel", required=True, choices=sorted(KERNELS))
    k.add_argument("--stats-dir", required=True)
    k.add_argument("--workload", required=True)
    k.add_argument("--command", action="append", default=[])
    q = sub.add_parser("sq")
    q.add_argument("--kernel", required=True, choices=sorted(KERNELS))
    q.add_argument("--dir", action="append", required=True)
    q.add_argument("--workload", required=True)
    q.add_argument("--command", action="append", default=[])
    a = ap.parse_args()
    {"traffic": traffic, "trace": trace, "sq": sq}[a.cmd](a)


if __name__ == "__main__":
    main()
