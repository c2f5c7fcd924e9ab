"""Text summaries of rocprofv3 output for the repair kernels.

Three kinds of summary are written (short text files, a few KB):

* ``kernel_stats``: the ``--kernel-trace --stats`` table of one command, with
  the bench line of the same run appended;
* ``traffic``: HBM bytes per launch of one kernel class from two ``--pmc``
  passes (``FETCH_SIZE``, then ``WRITE_SIZE``; KiB per dispatch), each divided
  by the factor the same counter reads for a device-to-device copy of known
  size in the same process.  The file records a hash of the sources that
  build the kernel, so a reader can tell whether the counters still describe
  the current code;
* ``counters``: per kernel class, the means over its dispatches of one
  ``--pmc`` pass of SQ counters, and the ratios derived from them: MFMA-pipe
  busy time over CU-busy time (SQ_VALU_MFMA_BUSY_CYCLES counts one cycle per
  1,024 MFMA FLOPs of one SIMD, so it is divided by four SIMDs times
  SQ_BUSY_CU_CYCLES, the busy cycles summed over the CUs), MFMA FLOPs per
  launch (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512), the share of wave cycles spent
  waiting on any dependency, VALU-active cycles per wave cycle, and LDS bank
  conflict cycles per LDS-active cycle.

Usage::

    python -m paper_2609_35139_amd.profsum stats <kernel_stats.csv> <bench.json> <out.txt> <command...>
    python -m paper_2609_35139_amd.profsum traffic <fetch_counter_collection.csv> \
        <write_counter_collection.csv> <bench.json> <class> <out.txt> <command...>
    python -m paper_2609_35139_amd.profsum counters <counter_collection.csv> <bench.json> \
        <out.txt> <command...>
"""
import csv
import hashlib
import json
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")

# kernel class -> (substring of the device function name, sources that build it)
CLASS_KERNEL = {
    "attention": ("attention_kernel", ["attention.hip", "common.h", "launch.h"]),
    "layernorm": ("layernorm_kernel", ["rowops.hip", "common.h", "launch.h"]),
    "compress_segments": ("compress_segments_kernel", ["rowops.hip", "common.h", "launch.h"]),
    "gemm_expand": ("EpiExpand", ["gemm.hip", "common.h", "launch.h"]),
    "gemm_qkv": ("EpiQKV", ["gemm.hip", "common.h", "launch.h"]),   # EpiQKVh or EpiQKV
}
for _c in ("gemm_compress", "gemm_fuse", "gemm_oproj", "gemm_ffn1", "gemm_ffn2"):
    CLASS_KERNEL[_c] = ("EpiBias", ["gemm.hip", "common.h", "launch.h"])
# the bench's 8192^3 bf16 library GEMM (measured-peak reference; no sources here)
CLASS_KERNEL["library_gemm_8192"] = ("Cijk_", [])


def source_hash(cls):
    h = hashlib.sha256()
    for f in CLASS_KERNEL[cls][1]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def bench_line(path):
    with open(path) as fh:
        for line in fh:
            if line.startswith('{"metric"'):
                return json.loads(line)
    raise ValueError(f"no bench JSON line in {path}")


def short_name(n):
    n = re.sub(r"\(.*", "", n)
    for k in ("EpiBias", "EpiQKVh", "EpiQKV", "EpiExpandRope", "EpiExpand"):
        if k in n:
            return "gemm_nt_kernel<" + k + ">"
    m = re.search(r"cr::(\w+)|_ZN2cr\d+(\w+?)I|_ZN2cr\d+(\w+)E", n)
    return (m.group(1) or m.group(2) or m.group(3)) if m else n[:40]


def kernel_stats(stats_csv, bench_json, command):
    rows = list(csv.DictReader(open(stats_csv)))
    b = bench_line(bench_json)
    out = [f"# rocprofv3 kernel statistics: repair forward pass, workload {b['config']['workload']}",
           f"# command: {command}",
           "# (the bench runs warmup + timed + profiled passes; averages are per launch)",
           "%-36s %8s %12s %10s %7s" % ("kernel", "calls", "total_us", "avg_us", "pct")]
    for r in rows:
        out.append("%-36s %8s %12.1f %10.2f %7.2f" % (
            short_name(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e3,
            float(r["AverageNs"]) / 1e3, float(r["Percentage"])))
    # per class from the kernel trace of the same run (classes by launch order)
    trace = os.path.join(os.path.dirname(stats_csv), "run_kernel_trace.csv")
    if os.path.exists(trace):
        tr = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Dispatch_Id"]))
        durs = {}
        for r, cls in zip(tr, classify([r["Kernel_Name"] for r in tr], b)):
            if cls:
                durs.setdefault(cls, []).append(
                    (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        out += ["", "# per-class average launch from the kernel trace of the same run (us;",
                "# bias-epilogue GEMMs told apart by their place in the launch order):",
                "#   " + ", ".join("%s %.2f (%d)" % (c, sum(v) / len(v), len(v))
                                   for c, v in durs.items())]
    rf = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in b["roofline"].items()}
    out += ["", "# bench line of the same command (live HIP events on the library's stream;",
            "# under the tracer each interval also holds the tracer's own handling of",
            "# the dispatch, a few us per launch, so short kernels read long here and",
            "# the reported bench line is the one of an untraced run):",
            "#   ms_per_step %.3f, value %.4g tokens/s" % (b["ms_per_step"], b["value"]),
            "#   roofline " + json.dumps(rf),
            "#   per-class average launch (us): " +
            ", ".join("%s %.1f" % (k["class"], k["avg_us"]) for k in b["kernels"])]
    return "\n".join(out) + "\n"


def _dispatches(path, counter):
    """[(dispatch id, kernel name, value)] in dispatch order for one counter
    of a --pmc pass (values of one dispatch summed over its rows)."""
    vals, names = {}, {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        vals[d] = vals.get(d, 0.0) + float(r["Counter_Value"])
        names[d] = r["Kernel_Name"]
    return [(d, names[d], vals[d]) for d in sorted(vals)]


def _per_dispatch(path, counter):
    """{kernel name: [value per dispatch]} for one counter of a --pmc pass."""
    out = {}
    for _, name, v in _dispatches(path, counter):
        out.setdefault(name, []).append(v)
    return out


def gemm_sequence(n_blocks):
    """Classes of the bias-epilogue GEMMs of one repair, in launch order."""
    return (["gemm_compress", "gemm_fuse"] +
            ["gemm_oproj", "gemm_ffn1", "gemm_ffn2"] * n_blocks)


def _class_values(path, counter, cls, bench):
    """Counter values of the dispatches of one kernel class.  The GEMMs with
    a bias epilogue share one device function; they are told apart by their
    position in the repair's fixed launch order (the profiled command runs
    nothing else that launches them)."""
    ds = _dispatches(path, counter)
    return [v for (_, _, v), c in zip(ds, classify([n for _, n, _ in ds], bench)) if c == cls]


def _calibration(per_kernel, copy_bytes):
    """Counter bytes / true bytes of the device-to-device copy of copy_bytes."""
    best = None
    for name, vs in per_kernel.items():
        if "copy" not in name.lower():
            continue
        for v in vs:
            ratio = v * 1024.0 / copy_bytes
            if 0.25 < ratio < 4.0 and (best is None or abs(ratio - 1) < abs(best - 1)):
                best = ratio
    if best is None:
        raise ValueError("calibration copy not found among the profiled kernels")
    return best


def traffic(fetch_csv, write_csv, bench_json, cls, command):
    b = bench_line(bench_json)
    calib = b["calibration"]["copy_bytes"]
    sub = CLASS_KERNEL[cls][0]
    res = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        per = _per_dispatch(path, counter)
        factor = _calibration(per, calib)
        ks = _class_values(path, counter, cls, b)
        if not ks:
            raise ValueError(f"no dispatch of {sub} in {path}")
        kib = sum(ks) / len(ks)
        res[counter] = {"kib_per_dispatch": kib, "dispatches": len(ks), "copy_factor": factor,
                        "bytes_per_launch": kib * 1024.0 / factor}
    total = res["FETCH_SIZE"]["bytes_per_launch"] + res["WRITE_SIZE"]["bytes_per_launch"]
    algo = None
    for k in b["kernels"]:
        if k["class"] == cls and "gbs" in k:
            algo = k["gbs"] * 1e9 * k["avg_us"] * 1e-6
    out = [f"# HBM traffic per launch: {cls} ({sub}), workload {b['config']['workload']}",
           f"# command (one pass per counter): {command}",
           f"# calibration: device-to-device copy of {calib} bytes in the same process",
           f"class: {cls}",
           f"source_sha256: {source_hash(cls)}"]
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        r = res[counter]
        out.append(f"{counter.lower()}_kib_per_dispatch: {r['kib_per_dispatch']:.1f}"
                   f"  (mean of {r['dispatches']} dispatches; copy factor {r['copy_factor']:.4f})")
    out.append(f"fetch_bytes_per_launch: {res['FETCH_SIZE']['bytes_per_launch']:.0f}")
    out.append(f"write_bytes_per_launch: {res['WRITE_SIZE']['bytes_per_launch']:.0f}")
    out.append(f"traffic_bytes_per_launch: {total:.0f}")
    if algo:
        out.append(f"algorithmic_bytes_per_launch: {algo:.0f}  (ratio {total / algo:.3f})")
    return "\n".join(out) + "\n"


SQ_RATIOS = (
    ("mfma_busy_of_cu_busy", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", 4.0),
    ("wait_of_wave_cycles", "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES", 1.0),
    ("valu_active_of_wave_cycles", "SQ_ACTIVE_INST_VALU", "SQ_WAVE_CYCLES", 1.0),
    ("lds_conflict_of_lds_active", "SQ_LDS_BANK_CONFLICT", "SQ_ACTIVE_INST_LDS", 1.0),
)


def classify(names, bench):
    """Kernel class of each dispatch, given the dispatches' kernel names in
    dispatch order (None for kernels of no class).  Bias-epilogue GEMMs share
    device functions across classes and are assigned by their position in
    the repair's fixed launch order, after the weight preparation's own
    GEMMs (one or two, launched once before the first repair)."""
    per_step = {k["class"]: k["launches_per_step"] for k in bench["kernels"]}
    seq = gemm_sequence(per_step.get("gemm_oproj", 0))
    skip = sum("EpiBias" in n for n in names) % len(seq)
    out, k = [], 0
    for name in names:
        cls = None
        for c, (sub, _) in CLASS_KERNEL.items():
            if sub != "EpiBias" and sub in name and "EpiExpandRope" not in name:
                cls = c
        if "EpiBias" in name:
            cls = seq[(k - skip) % len(seq)] if k >= skip else None
            k += 1
        out.append(cls)
    return out


def counters(csv_path, bench_json, command, n_cus=256):
    """Per-class means of one --pmc pass (one row per dispatch and counter)
    and the derived ratios of SQ_RATIOS."""
    b = bench_line(bench_json)
    disp = {}
    for r in csv.DictReader(open(csv_path)):
        d = int(r["Dispatch_Id"])
        e = disp.setdefault(d, {"name": r["Kernel_Name"],
                                "dur_ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    order = sorted(disp)
    by_cls = {}
    for d, cls in zip(order, classify([disp[d]["name"] for d in order], b)):
        if cls:
            by_cls.setdefault(cls, []).append(disp[d])
    names = sorted({n for e in disp.values() for n in e if n.isupper() or n.startswith("SQ_")})
    out = [f"# SQ counters per kernel class, workload {b['config']['workload']}",
           f"# command: {command}",
           "# means over the class's dispatches of the profiled run; duration from the",
           "# dispatch timestamps of the same (serialised) run",
           f"# mfma_busy_of_cu_busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 * SQ_BUSY_CU_CYCLES); "
           f"SQ_BUSY_CU_CYCLES / {n_cus} / duration = mean CU-busy cycles per ns",
           ""]
    for cls in [c for c in CLASS_KERNEL if c in by_cls]:
        es = by_cls[cls]
        mean = {n: sum(e.get(n, 0.0) for e in es) / len(es) for n in names}
        dur = sum(e["dur_ns"] for e in es) / len(es)
        out.append(f"[{cls}] dispatches {len(es)}, duration_us {dur / 1e3:.2f}")
        for n in names:
            out.append(f"  {n}: {mean[n]:.6g}")
        if mean.get("SQ_INSTS_VALU_MFMA_MOPS_BF16"):
            out.append(f"  mfma_flops_per_launch: {mean['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512:.6g}")
        if mean.get("SQ_BUSY_CU_CYCLES"):
            out.append(f"  cu_busy_cycles_per_ns: {mean['SQ_BUSY_CU_CYCLES'] / n_cus / dur:.3f}")
        for label, num, den, f in SQ_RATIOS:
            if mean.get(den):
                out.append(f"  {label}: {mean.get(num, 0.0) / (f * mean[den]):.4f}")
    return "\n".join(out) + "\n"


def read_traffic(path, cls):
    """Traffic bytes per launch recorded for cls, or None when the file is
    missing or the kernel sources changed since the counters were taken."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.split()[0] if v.split() else ""
    if kv.get("class") != cls or kv.get("source_sha256") != source_hash(cls):
        return None
    return float(kv["traffic_bytes_per_launch"])


def main(argv):
    mode = argv[0]
    if mode == "stats":
        stats_csv, bench_json, out = argv[1:4]
        text = kernel_stats(stats_csv, bench_json, " ".join(argv[4:]))
    elif mode == "traffic":
        fetch_csv, write_csv, bench_json, cls, out = argv[1:6]
        text = traffic(fetch_csv, write_csv, bench_json, cls, " ".join(argv[6:]))
    elif mode == "counters":
        csv_path, bench_json, out = argv[1:4]
        text = counters(csv_path, bench_json, " ".join(argv[4:]))
    else:
        raise SystemExit(__doc__)
    with open(out, "w") as fh:
        fh.write(text)
    print(text)


if __name__ == "__main__":
    main(sys.argv[1:])
