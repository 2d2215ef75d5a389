"""rocprofv3 evidence for bench.py: per-kernel durations and HBM traffic of
the epoch kernel on one workload.

    python3 bench_profile.py --workload netflix [--scheme hogwild] [bench.py options ...]

runs four passes of bench.py under rocprofv3 (each a child process, each with
its own time limit):

  1. --kernel-trace --stats: average duration of every kernel;
  2. --pmc FETCH_SIZE and 3. --pmc WRITE_SIZE: bytes the L2 caches read from
     and write to the memory fabric per dispatch (KiB), with a plain 4 GiB
     device copy in the same run to calibrate both counters (the copy reads
     and writes exactly 4 GiB, so scale = 4 GiB / counter reading of the copy);
  4. --pmc with six SQ counters: wave instructions issued per dispatch
     (vector, scalar, vector memory reads and writes), waves and busy cycles.

and writes profiles/<kernel>_<workload>[_<scheme>].md (the summary, with the
commands) and profiles/traffic_<kernel>_<scheme>_<workload>.json (scaled HBM
bytes per launch and the digest of the kernel sources they were taken on;
bench.py reports them as roofline.traffic only while that digest matches).
Raw rocprofv3 output stays under --out (default profiles/raw/prof_<tag>, not
committed); the summary names that directory $OUT.
With --summarize-only the passes are not run again.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import shutil
import statistics
import subprocess
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (source_digest, PROFILE_DIR; imports nothing that touches the GPU)

COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_BYTES = 4 << 30
SQ_COUNTERS = ("SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_VMEM_WR", "SQ_WAVES",
               "SQ_BUSY_CYCLES")
# wave64 vector instructions the chip can issue per second: 256 CUs x 4 SIMDs, each
# taking 4 cycles (16 lanes) per wave64 instruction, at 2.4 GHz
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4


def say(msg):
    print(f"[bench_profile] {msg}", flush=True)


def run_pass(cmd, limit):
    say("running: " + " ".join(cmd))
    rc = subprocess.run(["timeout", "-k", "10", "-s", "KILL", str(limit)] + cmd, cwd="/tmp",
                        env=dict(os.environ, TMPDIR="/tmp")).returncode
    say(f"exit status {rc}")
    return rc


def find_csv(d, suffix):
    hits = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {d}")
    return hits[-1]


def rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


_DEMANGLED = {}


def demangle(name: str) -> str:
    """Itanium-mangled kernel names (rocprofv3 leaves some, e.g. _Float16
    instantiations, undemangled) through c++filt; else the nested name."""
    name = name.strip()
    if not name.startswith("_Z"):
        return name
    if name not in _DEMANGLED:
        out = ""
        if shutil.which("c++filt"):
            out = subprocess.run(["c++filt", name], capture_output=True, text=True).stdout.strip()
        if not out or out == name:
            # _ZN<len><id><len><id>...: keep the identifiers before the template arguments
            parts, i = [], 3 if name.startswith("_ZN") else 2
            while i < len(name) and name[i].isdigit():
                j = i
                while name[j].isdigit():
                    j += 1
                n = int(name[i:j])
                parts.append(name[j:j + n])
                i = j + n
            out = "::".join(parts) or name
        _DEMANGLED[name] = out
    return _DEMANGLED[name]


def short(name: str) -> str:
    # "void mfsgd::k_hogwild<128, float, 4, false>(...)" -> "mfsgd::k_hogwild<128, float, 4, false>"
    name = demangle(name)
    if name.startswith("void "):
        name = name[5:]
    depth, out = 0, []
    for ch in name:
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            break
        out.append(ch)
    return "".join(out).strip()


def counter_per_dispatch(d, counter):
    """{dispatch id: (kernel name, summed counter value)} of one --pmc pass."""
    out = {}
    for r in rows(find_csv(d, "counter_collection.csv")):
        if r.get("Counter_Name") != counter:
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id")
        name, val = out.get(key, (r.get("Kernel_Name", ""), 0.0))
        out[key] = (name, val + float(r["Counter_Value"]))
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="netflix")
    ap.add_argument("--scheme", default="hogwild", choices=["hogwild", "wavefront", "wavefront_det", "table"])
    ap.add_argument("--kernel", default="", help="epoch kernel name (default: whichever of k_hogwild, k_blocked "
                                                 "and k_table takes more time in the trace)")
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--out", default="")
    ap.add_argument("--limit", type=int, default=400, help="seconds per rocprofv3 pass")
    ap.add_argument("--summarize-only", action="store_true")
    ap.add_argument("bench_args", nargs=argparse.REMAINDER, help="after --: more bench.py options")
    a = ap.parse_args()
    extra = [x for x in a.bench_args if x != "--"]
    out = os.path.abspath(a.out or os.path.join(ROOT, "profiles", "raw", f"prof_{a.workload}_{a.scheme}"))
    py = sys.executable or "python3"
    base = [py, os.path.join(ROOT, "bench.py"), "--workload", a.workload, "--scheme", a.scheme,
            "--no-cpu-baseline", "--no-extra"] + extra
    cmds = {
        "trace": ["rocprofv3", "--kernel-trace", "--stats", "--output-format", "csv", "-d",
                  os.path.join(out, "trace"), "-o", "run", "--"] + base + ["--steps", str(a.steps), "--warmup", "1"],
    }
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        cmds[c] = ["rocprofv3", "--pmc", c, "--output-format", "csv", "-d", os.path.join(out, c), "-o", "run",
                   "--"] + base + ["--steps", "3", "--warmup", "1", "--copy-calibration"]
    # instruction issue: counts of issued wave instructions per dispatch (8 SQ counters, one pass)
    cmds["SQ"] = ["rocprofv3", "--pmc", *SQ_COUNTERS, "--output-format", "csv", "-d", os.path.join(out, "SQ"), "-o",
                  "run", "--"] + base + ["--steps", "2", "--warmup", "1"]
    passes = ("trace", "FETCH_SIZE", "WRITE_SIZE", "SQ")
    if not a.summarize_only:
        for key in passes:
            rc = run_pass(cmds[key], a.limit)
            if rc != 0:
                # rocprofv3 may end with a segmentation fault after the program has finished;
                # accept the pass only if its result files are there
                try:
                    find_csv(os.path.join(out, key), "kernel_stats.csv" if key == "trace" else
                         "counter_collection.csv")
                except SystemExit:
                    raise SystemExit(f"pass {key} failed with status {rc}")
                say(f"pass {key}: status {rc} but results are complete; using them")

    stats = rows(find_csv(os.path.join(out, "trace"), "kernel_stats.csv"))
    trace = rows(find_csv(os.path.join(out, "trace"), "kernel_trace.csv"))
    kernel = a.kernel
    if not kernel:
        tot = {k: sum(float(r["TotalDurationNs"]) for r in stats if short(r["Name"]).split("<")[0].endswith(k))
               for k in ("k_hogwild", "k_hogwild_half", "k_blocked", "k_table")}
        kernel = max(tot, key=tot.get)
    kw = int(extra[extra.index("--k") + 1]) if "--k" in extra else 0
    tag = f"{kernel}_{a.workload}" + ("" if a.scheme == "hogwild" else f"_{a.scheme}") + (f"_k{kw}" if kw else "")
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in trace
            if short(r["Kernel_Name"]).split("<")[0].endswith(kernel)]
    if not durs:
        raise SystemExit(f"kernel {kernel} not in the trace")
    timed = durs[1:] if len(durs) > 1 else durs  # the first launch is bench.py's warm-up epoch
    avg_ns = statistics.mean(timed)

    scale, per_launch = {}, {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        disp = counter_per_dispatch(os.path.join(out, c), c)
        copies = [v for n, v in disp.values() if COPY_KERNEL in n]
        big = max(copies) if copies else 0.0
        if big <= 0:
            raise SystemExit(f"no copy calibration dispatch in the {c} pass")
        scale[c] = COPY_BYTES / (big * 1024.0)
        vals = [v for n, v in disp.values() if short(n).split("<")[0].endswith(kernel)]
        vals = vals[1:] if len(vals) > 1 else vals
        per_launch[c] = (statistics.median(vals), statistics.median(vals) * 1024.0 * scale[c])

    sq = {}
    for c in SQ_COUNTERS:
        disp = counter_per_dispatch(os.path.join(out, "SQ"), c)
        vals = [v for n, v in disp.values() if short(n).split("<")[0].endswith(kernel)]
        vals = vals[1:] if len(vals) > 1 else vals
        sq[c] = statistics.median(vals) if vals else None

    w = None
    try:
        from paper_1610_05838_amd import datagen
        w = datagen.workload(a.workload)
    except Exception:  # the summary still stands without the workload's sizes
        pass
    nnz = w["ntrain"] if w else None
    if w and "--ntrain" in extra:
        nnz = int(extra[extra.index("--ntrain") + 1])
    k = kw or (w["k"] if w else 128)
    fb = 2 if (w and w["dtype"] == "fp16") else 4
    bpu = 4 * k * fb + 12
    hbm = per_launch["FETCH_SIZE"][1] + per_launch["WRITE_SIZE"][1]

    os.makedirs(bench.PROFILE_DIR, exist_ok=True)
    md = os.path.join(bench.PROFILE_DIR, f"{tag}.md")
    total = sum(float(r["TotalDurationNs"]) for r in stats) or 1.0
    L = [f"# {kernel} on the {a.workload} workload, {a.scheme} (rocprofv3 summaries)", "",
         "Made by `python3 bench_profile.py --workload " + a.workload + " --scheme " + a.scheme +
         (" -- " + " ".join(extra) if extra else "") + "`, which runs these passes (from /tmp):", ""]
    for key in passes:
        L.append("    " + " ".join(x.replace(out, "$OUT").replace(ROOT, "$REPO") for x in cmds[key]))
    L += ["", "$OUT is the directory the raw rocprofv3 output was written to (not committed).",
          "", "## Kernel statistics (kernel trace)", "",
          "| kernel | calls | average ms | min ms | max ms | share |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        L.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.3f} | "
                 f"{float(r['MinNs']) / 1e6:.3f} | {float(r['MaxNs']) / 1e6:.3f} | "
                 f"{100 * float(r['TotalDurationNs']) / total:.2f}% |")
    L += ["", f"Epoch kernel `{kernel}`: {len(timed)} timed launches (after the warm-up epoch), average "
              f"{avg_ns / 1e6:.3f} ms, min {min(timed) / 1e6:.3f}, max {max(timed) / 1e6:.3f}.", "",
          "## L2-to-fabric traffic (PMC)", "",
          "FETCH_SIZE and WRITE_SIZE count the bytes the L2 caches read from and write to the memory fabric; "
          "reads the Infinity Cache serves are included, so these are an upper bound on HBM bytes.", "",
          f"Calibration: `{COPY_KERNEL}` copies 4 GiB -> 4 GiB; scale FETCH_SIZE x{scale['FETCH_SIZE']:.4f}, "
          f"WRITE_SIZE x{scale['WRITE_SIZE']:.4f} (bytes = KiB x 1024 x scale).", "",
          f"| per launch of `{kernel}` | raw KiB (median of timed launches) | scaled bytes | bytes per update |",
          "|---|---|---|---|"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        raw, b = per_launch[c]
        L.append(f"| {c} | {raw:.0f} | {b:.4e} | {b / nnz:.1f} |" if nnz else f"| {c} | {raw:.0f} | {b:.4e} | |")
    L.append(f"| total L2-to-fabric | | {hbm:.4e} | {hbm / nnz:.1f} |" if nnz else
             f"| total L2-to-fabric | | {hbm:.4e} | |")
    if nnz:
        L += ["", f"Algorithmic bytes per update: {bpu} (4k*sizeof(feature)+12, k={k}); updates per launch {nnz}.",
              f"Average launch (trace): {avg_ns / 1e6:.3f} ms -> algorithmic {nnz * bpu / avg_ns:.1f} GB/s "
              f"({100 * nnz * bpu / avg_ns / bench.HBM_PEAK_GBS:.1f}% of 8 TB/s), measured L2-to-fabric "
              f"{hbm / avg_ns:.1f} GB/s ({100 * hbm / avg_ns / bench.HBM_PEAK_GBS:.1f}% of 8 TB/s)."]
    if sq.get("SQ_INSTS_VALU"):
        L += ["", "## Instruction issue (PMC)", "",
              f"Wave instructions issued per launch of `{kernel}` (median of timed launches) and per update.  "
              f"The chip issues at most {VALU_ISSUE_PEAK / 1e9:.1f} G wave64 vector instructions/s "
              "(256 CUs x 4 SIMDs, 4 cycles each per wave64 instruction, 2.4 GHz).", "",
              "| counter | per launch | per update |", "|---|---|---|"]
        for c in SQ_COUNTERS:
            if sq.get(c) is not None:
                L.append(f"| {c} | {sq[c]:.4e} | " + (f"{sq[c] / nnz:.2f} |" if nnz else "|"))
        rate = sq["SQ_INSTS_VALU"] / (avg_ns * 1e-9)
        L += ["", f"Vector instruction issue: {rate / 1e9:.1f} G/s over the average launch, "
                  f"{100 * rate / VALU_ISSUE_PEAK:.1f}% of {VALU_ISSUE_PEAK / 1e9:.1f} G/s."]
    with open(md, "w") as f:
        f.write("\n".join(L) + "\n")
    tj = os.path.join(bench.PROFILE_DIR, f"traffic_{kernel}_{a.scheme}_{a.workload}" + (f"_k{kw}" if kw else "") + ".json")
    with open(tj, "w") as f:
        json.dump({"kernel": kernel, "workload": a.workload, "scheme": a.scheme,
                   "bench_args": extra, "source_digest": bench.source_digest(),
                   "hbm_bytes_per_launch": hbm, "fetch_bytes_per_launch": per_launch["FETCH_SIZE"][1],
                   "write_bytes_per_launch": per_launch["WRITE_SIZE"][1],
                   "copy_scale_fetch": scale["FETCH_SIZE"], "copy_scale_write": scale["WRITE_SIZE"],
                   "avg_launch_ns_trace": avg_ns, "summary": os.path.basename(md),
                   "sq_per_launch": sq, "valu_issue_peak_per_s": VALU_ISSUE_PEAK}, f, indent=1)
    say(f"wrote {md} and {tj}")
    print("\n".join(L))


if __name__ == "__main__":
    main()
