"""Benchmark: SGD updates/s and achieved HBM GB/s of the SGD-MF epoch at k=128
on one MI355X.

Headline workload (default): the Hugewiki-shaped synthetic set, the largest
of the paper's data sets that one GPU holds -- m=50,082,603 users, n=39,780
items, 3,069,000,000 training ratings (+31,000,000 test, 36.8 GB of samples),
Zipf(1.0) users, uniform items, k=128, binary16 feature storage (12.8 GB of
P), lr 0.01, lambda 0.01, wavefront-update on a 64 x 64 grid (the paper's
schedule for it).  A step is one full epoch (every training rating updates P
and Q once) followed by the test RMSE, with all inputs resident in HBM; the
wavefront plan is made once before the timed steps.

Two more lines ride along in the same JSON object ("extra"): the
Netflix-shaped set (binary32, the default batch-Hogwild!) and the
Yahoo!Music-shaped set (binary32, 832 MB of factors, the default
batch-Hogwild!), each with its own epoch time, updates/s, algorithmic
bandwidth and test RMSE (--no-extra skips them).

Printed: one JSON line with the whole-run updates/s, the roofline of the
epoch kernel (algorithmic bytes per update 4k*sizeof(feature)+12 over the
kernel's HIP-event time, against 8 TB/s; measured HBM traffic from the
committed rocprofv3 counter summary when it was taken on the current
sources) and the CPU oracle timed on a bounded prefix of the same workload.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1610_05838_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def profile_record(kernel_key: str, variant: list):
    """The committed rocprofv3 counter record of this kernel and workload, if
    it was taken on the current kernel sources with the same bench options
    (`variant`: the options that change the launch); else None."""
    path = os.path.join(PROFILE_DIR, f"traffic_{kernel_key}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_digest") != source_digest() or d.get("bench_args", []) != variant:
        return None
    return d


def measured_traffic(kernel_key: str, variant: list):
    """L2-to-fabric bytes per launch from the committed counter record, or None."""
    d = profile_record(kernel_key, variant)
    return d.get("hbm_bytes_per_launch") if d else None


def _oracle_factors(w, S, dtype):
    """Initial factors for the oracle: all rows, or (for models too large to
    build on the host in seconds) the rows S touches, with S renumbered."""
    import numpy as np
    import oracle

    if w["m"] * w["k"] <= 1 << 30:
        P, Q = oracle.init_factors(w["m"], w["n"], w["k"], w["seed"], dtype)
        return P, Q, S, ""
    ur, uc = np.unique(S["u"], return_inverse=True)
    vr, vc = np.unique(S["v"], return_inverse=True)
    C = S.copy()
    C["u"], C["v"] = uc, vc
    P = oracle.init_rows(w["m"], w["k"], w["seed"], 0, ur, dtype)
    Q = oracle.init_rows(w["n"], w["k"], w["seed"], 1, vr, dtype)
    return P, Q, C, f" (on the {len(ur)} user and {len(vr)} item rows the sample touches)"


def cpu_baseline(w, S, target_s: float, threads: int):
    """The oracle (never tuned) on a bounded prefix of the same workload.
    S: a host prefix of the training samples, long enough for target_s."""
    import numpy as np

    # the OpenMP runtime the oracle loads reads these once: one thread per
    # physical core, spread over the sockets
    os.environ["OMP_PROC_BIND"] = "spread"
    os.environ["OMP_PLACES"] = "cores"
    import oracle

    dtype = np.float16 if w["dtype"] == "fp16" else np.float32
    P, Q, S, note = _oracle_factors(w, S, dtype)
    probe = min(len(S), 100_000 if dtype == np.float32 else 20_000)
    t0 = time.perf_counter()
    oracle.epoch_serial(P, Q, S[:probe], w["lr"], w["lam"], w["lam"])
    rate = probe / max(time.perf_counter() - t0, 1e-9)
    count = int(min(len(S) - probe, max(probe, rate * target_s)))
    t0 = time.perf_counter()
    oracle.epoch_serial(P, Q, S[probe:probe + count], w["lr"], w["lam"], w["lam"])
    dt = time.perf_counter() - t0
    serial = {"value": count / dt, "unit": "updates/s", "cores": 1, "kind": "oracle",
              "sample": f"serial binary64 oracle, samples {probe}..{probe + count - 1} of epoch 0 of the "
                        f"{w['name']} workload ({count} updates, {dt:.1f} s){note}"}
    omp = None
    if threads > 1:
        P, Q, S, note = _oracle_factors(w, S, dtype)
        n2 = int(min(len(S), count * threads))
        t0 = time.perf_counter()
        used = oracle.epoch_hogwild_omp(P, Q, S[:n2], w["lr"], w["lam"], w["lam"], 256, threads)
        dt = time.perf_counter() - t0
        omp = {"value": n2 / dt, "unit": "updates/s", "cores": used, "kind": "oracle-openmp-hogwild",
               "sample": f"first {n2} samples of epoch 0, batches of 256 claimed by {used} threads ({dt:.1f} s)"
                         f"{note}"}
    return serial, omp


XGMI_LINK_GBS = 153.0  # one MI355X xGMI link, per direction (published figure, not measured here)


def shard_share(args):
    """One GPU's share of a G-GPU epoch under the block partition of the
    paper's section 4.1, measured on this GPU at its real shape.  R is cut
    into G x G blocks by equal user and item ranges; GPU g keeps user segment
    g of P for the whole epoch and in wave w updates block (g, (g + w) mod G)
    while item segment (g + w) mod G of Q travels to it from its neighbour.
    Here g = 0: the share's samples are generated, bucketed by item segment,
    and each wave's block is one batch-Hogwild! epoch over that block's
    samples (the kernel touches only the rows of its segments).  The wave's
    Q-segment message is priced at one xGMI link's rate."""
    import numpy as np
    import torch

    from paper_1610_05838_amd import datagen, mfsgd

    G = args.shard
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = datagen.workload(args.workload)
    if args.ntrain:
        w["ntrain"] = args.ntrain
    m, n, k, nnz = w["m"], w["n"], w["k"], w["ntrain"]
    t0 = time.perf_counter()
    blocks = [[] for _ in range(G)]
    chunk = 1 << 25
    for c0 in range(0, nnz, chunk):
        S = datagen.draw(w, c0, min(chunk, nnz - c0)) if w["draw"] == "independent" else datagen.make(w)[0]
        mine = S[(S["u"].astype(np.int64) * G) // m == 0]
        seg = (mine["v"].astype(np.int64) * G) // n
        for j in range(G):
            blocks[j].append(mine[seg == j])
        if w["draw"] != "independent":
            break
    blocks = [np.concatenate(b) for b in blocks]
    share = sum(len(b) for b in blocks)
    log(f"share of GPU 0 of {G}: {share} of {nnz} samples in {time.perf_counter() - t0:.1f}s")
    dtype = 1 if w["dtype"] == "fp16" else 0
    feat = 2 if dtype else 4
    # one address space inside each block: its working set is one user and one item segment
    for key, val in dict(dtype=dtype, batch_f=256, workers=args.workers, depth=args.depth, partition=0,
                         debug=0).items():
        mfsgd.set_option(key, val)
    mfsgd.init(m, n, k, w["seed"])
    stream = torch.cuda.current_stream()
    dB = [mfsgd.samples_to_device(b, dev) for b in blocks]
    wave_ms = np.zeros(G)
    epochs = max(1, args.steps)
    for t in range(args.warmup + epochs):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(G)]
        for wv in range(G):  # GPU 0 works on item segment wv in wave wv
            ev[wv][0].record(stream)
            mfsgd.epoch(dB[wv], datagen.lr_at(w, t), w["lam"], w["lam"], "hogwild", stream)
            ev[wv][1].record(stream)
        torch.cuda.synchronize()
        if t >= args.warmup:
            wave_ms += np.array([a.elapsed_time(b) for a, b in ev]) / epochs
    q_bytes = -(-n // G) * k * feat
    xfer_ms = q_bytes / (XGMI_LINK_GBS * 1e9) * 1e3
    proj_ms = float(np.maximum(wave_ms, xfer_ms).sum())
    mfsgd.finalize()
    print(json.dumps({
        "mode": "shard", "workload": w["name"], "gpus_emulated": G, "rank": 0, "k": k, "dtype": w["dtype"],
        "share_samples": share, "total_samples": nnz, "wave_samples": [len(b) for b in blocks],
        "wave_ms": [round(x, 3) for x in wave_ms], "compute_ms_per_epoch": round(float(wave_ms.sum()), 3),
        "share_updates_per_s": share / (wave_ms.sum() / 1e3),
        "q_segment_bytes": q_bytes, "xgmi_link_gbs_assumed": XGMI_LINK_GBS, "transfer_ms_per_wave": round(xfer_ms, 4),
        "projected_epoch_ms": round(proj_ms, 3),
        "note": "rank 0's share only; under skewed data the ranks' shares differ, and the slowest sets the epoch"}),
        flush=True)


def oracle_threads():
    """Threads for the OpenMP oracle: the physical cores (lscpu's core ids)
    among the CPUs this process may run on, capped by OMP_NUM_THREADS when it
    is set (the machine's share for this job).  Returns (threads, physical
    cores seen)."""
    import subprocess

    cpus = set(os.sched_getaffinity(0))
    cores = set()
    try:
        out = subprocess.run(["lscpu", "-p=CPU,CORE,SOCKET"], capture_output=True, text=True, timeout=30).stdout
        for line in out.splitlines():
            if line.startswith("#") or not line.strip():
                continue
            cpu, core, sock = line.split(",")[:3]
            if int(cpu) in cpus:
                cores.add((sock, core))
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    physical = len(cores) or len(cpus)
    n = physical
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n), physical


def kernel_of(mfsgd, scheme, staged):
    """Name of the epoch kernel a launch runs."""
    if scheme == "table":
        return "k_table"
    if scheme != "hogwild" or (mfsgd.get_option("partitioned") == 1 and not staged):
        return "k_blocked"
    return "k_hogwild_half" if mfsgd.get_option("half_workers") else "k_hogwild"


def apply_options(mfsgd, args, dtype):
    mfsgd.reset_options()
    mfsgd.set_option("dtype", dtype)
    for key, val in (("workers", args.workers), ("depth", args.depth), ("team_waves", args.team_waves)):
        if val:
            mfsgd.set_option(key, val)
    if args.partition is not None:
        mfsgd.set_option("partition", args.partition)
    for kv in args.set:
        key, val = kv.split("=", 1)
        mfsgd.set_option(key, int(val))


def measure(args, name, scheme, steps, warmup, dev, host_prefix=0):
    """Generate the workload into HBM, run `warmup` then `steps` timed steps
    (epoch + test RMSE) of `scheme`, and return the measurements."""
    import numpy as np
    import torch

    from paper_1610_05838_amd import datagen, mfsgd

    w = datagen.workload(name)
    if args.ntrain:
        w["ntrain"] = args.ntrain
    t0 = time.perf_counter()
    S = None
    if args.staged:
        if scheme != "hogwild":
            raise SystemExit("--staged runs batch-Hogwild! only")
        S = datagen.draw(w, 0, w["ntrain"]) if w["draw"] == "independent" else datagen.make(w)[0]
        T = datagen.draw(w, w["ntrain"], w["ntest"]) if w["draw"] == "independent" else datagen.make(w)[1]
        dS = torch.from_numpy(S.view(np.int32).reshape(-1, 3)).pin_memory()
    elif w["draw"] == "independent":
        # generated chunk by chunk straight into HBM; the host keeps a prefix for the CPU baseline
        dS = datagen.draw_to_device(w, 0, w["ntrain"], dev, chunk=1 << 27, progress=lambda a, b: (
            log(f"  generated {a}/{b}") if a % (1 << 30) < (1 << 27) else None))
        T = datagen.draw(w, w["ntrain"], w["ntest"])
        if host_prefix:
            S = datagen.draw(w, 0, min(w["ntrain"], host_prefix))
    else:
        S, T = datagen.make(w)
        dS = mfsgd.samples_to_device(S, dev)
    dT = mfsgd.samples_to_device(T, dev)
    nnz = w["ntrain"]
    if args.k:
        w["k"] = args.k  # after generation: only the trained width changes
    log(f"generated {w['name']}: {nnz} train + {len(T)} test in {time.perf_counter() - t0:.1f}s")
    dtype = 1 if w["dtype"] == "fp16" else 0
    apply_options(mfsgd, args, dtype)
    mfsgd.init(w["m"], w["n"], w["k"], w["seed"])
    grid_s = args.grid_s or w.get("grid_s", 32)
    if scheme == "table":
        grid_s = mfsgd.get_option("table_grid")
        if warmup < 1:
            raise SystemExit("--scheme table plans in its first epoch: use --warmup 1 or more")
    elif scheme != "hogwild":
        t0 = time.perf_counter()
        mfsgd.plan(dS, grid_s)
        log(f"wavefront plan (s={grid_s}) {time.perf_counter() - t0:.3f}s")
    stream = torch.cuda.current_stream()

    def step(t, ev=None):
        lr = datagen.lr_at(w, t)
        if ev is not None:
            ev[0].record(stream)
        if args.staged:
            mfsgd.epoch_staged(dS, lr, w["lam"], w["lam"], stream)
        else:
            mfsgd.epoch(dS, lr, w["lam"], w["lam"], scheme, stream)
        if ev is not None:
            ev[1].record(stream)
        return mfsgd.rmse(dT, stream)

    rmses = []
    for t in range(warmup):
        rmses.append(step(t))
        log(f"{name} warmup epoch {t}: test rmse {rmses[-1]:.5f}")
    # the automatic batch-Hogwild! form is chosen per sample array at the first epoch
    kernel = kernel_of(mfsgd, scheme, args.staged)
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        rmses.append(step(warmup + i, events[i]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    epoch_ms = [a.elapsed_time(b) for a, b in events]
    log(f"{name}: timed {steps} steps in {wall:.3f}s; epoch kernel ms: " + ", ".join(f"{x:.2f}" for x in epoch_ms))
    log(f"{name}: test rmse after each epoch: " + ", ".join(f"{x:.4f}" for x in rmses))
    form = mfsgd.get_option("hogwild_form") if scheme == "hogwild" and not args.staged else -1
    atomic = mfsgd.get_option("hogwild_atomic") if form >= 0 else 0
    pairs = kernel == "k_blocked" and mfsgd.get_option("blocked_pairs") == 1
    r = dict(w=w, scheme=scheme, grid_s=grid_s, nnz=nnz, ntest=len(T), epoch_ms=epoch_ms, rmses=rmses, wall=wall,
             kernel=kernel, S=S, dtype=dtype, resident=mfsgd.get_option("resident_waves"),
             partitioned=scheme == "hogwild" and mfsgd.get_option("partitioned") == 1 and not args.staged,
             form=", ".join(x for x in ({-1: "", 0: "one address space", 1: "XCD-partitioned",
                                         3: "XCD-partitioned, free-running", 4: "one XCD"}.get(form, str(form)),
                                        "atomic adds" if atomic else "",
                                        "two batches per claim" if pairs else "") if x))
    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        for i in range(3):
            b.copy_(a)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(3)]
        log("copy calibration: 3 x 4 GiB device copies, " + ", ".join(
            f"{x:.2f} ms ({2 * a.numel() * 4 / x / 1e6:.0f} GB/s read+write)" for x in ms))
        del a, b
    mfsgd.finalize()
    del dS, dT
    torch.cuda.empty_cache()
    return r


def rates(r):
    """Epoch-kernel rates of one measurement."""
    w = r["w"]
    bpu = 4 * w["k"] * (2 if r["dtype"] else 4) + 12
    avg_s = sum(r["epoch_ms"]) / len(r["epoch_ms"]) / 1e3
    gbs = r["nnz"] * bpu / avg_s / 1e9
    return bpu, avg_s, gbs


def describe(r):
    w = r["w"]
    return (f"{w['name']}: m={w['m']} n={w['n']} k={w['k']} nnz={r['nnz']} ntest={r['ntest']} {w['dtype']} "
            f"{r['scheme']}" + (f" s={r['grid_s']}" if r["scheme"] != "hogwild" else " f=256"))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="hugewiki")
    ap.add_argument("--scheme", default="", choices=["", "hogwild", "wavefront", "wavefront_det", "table"],
                    help="default: wavefront-update for workloads that name a grid (hugewiki), else batch-Hogwild!; "
                         "table: the global scheduling table (LIBMF's policy; --set table_grid=S --set "
                         "table_workers=W), planned in the first warm-up epoch")
    ap.add_argument("--grid-s", type=int, default=0, help="wavefront grid side (0: the workload's, else 32)")
    ap.add_argument("--workers", type=int, default=0)
    ap.add_argument("--depth", type=int, default=0, help="samples in flight per wavefront (0: the library's choice)")
    ap.add_argument("--team-waves", type=int, default=0)
    ap.add_argument("--partition", type=int, default=None,
                    help="batch-Hogwild! form: 0 one address space, 1 XCD-partitioned, 2 one XCD (library default), "
                         "3 partitioned without tickets")
    ap.add_argument("--ntrain", type=int, default=0, help="override the training size (0: the workload's)")
    ap.add_argument("--k", type=int, default=0,
                    help="train at this width instead of the workload's (same samples; 0: the workload's k)")
    ap.add_argument("--set", action="append", default=[], metavar="KEY=VALUE",
                    help="further library option (mfsgd_set_option), applied before init")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="OpenMP oracle threads (0: the physical cores available, capped by OMP_NUM_THREADS)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the Netflix- and Yahoo-shaped extra lines")
    ap.add_argument("--extra-steps", type=int, default=5)
    ap.add_argument("--staged", action="store_true",
                    help="training samples stay in pinned host memory and stream through the GPU (mfsgd_epoch_staged, "
                         "batch-Hogwild!): value then includes the PCIe transfers and is not the resident rate")
    ap.add_argument("--log-jsonl", default="", metavar="PATH",
                    help="also write one JSON row per timed epoch (epoch, ms, updates/s, algorithmic GB/s, fraction "
                         "of the HBM peak, test RMSE) to PATH")
    ap.add_argument("--shard", type=int, default=0, metavar="G",
                    help="measure one GPU's share of a G-GPU run instead (the block partition of the paper's section "
                         "4.1: GPU 0 keeps user segment 0 and takes item segment w in wave w); prints its own JSON line")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 4 GiB device copy (for scaling rocprofv3 byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library runs the SGD hot path on a single MI355X "
              "(multi-GPU sharding is a design note, not implemented)", file=sys.stderr)
        sys.exit(2)

    if args.shard > 1:
        shard_share(args)
        return

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    # the paper runs Hugewiki under wavefront-update (its own section 3.2.3 grid), the others under batch-Hogwild!
    scheme = args.scheme or ("wavefront" if args.workload == "hugewiki" else "hogwild")
    threads, physical = oracle_threads()
    if args.cpu_threads:
        threads = args.cpu_threads
    r = measure(args, args.workload, scheme, args.steps, args.warmup, dev,
                host_prefix=0 if args.no_cpu_baseline else (50_000_000 if threads > 1 else 20_000_000))
    w = r["w"]
    if args.log_jsonl:
        bpu = rates(r)[0]
        with open(args.log_jsonl, "w") as f:
            for i, ms in enumerate(r["epoch_ms"]):
                ups = r["nnz"] / (ms / 1e3)
                f.write(json.dumps({"workload": w["name"], "scheme": scheme, "dtype": w["dtype"],
                                    "epoch": args.warmup + i + 1, "epoch_ms": ms, "updates_per_s": ups,
                                    "algorithmic_gbs": ups * bpu / 1e9, "frac_of_peak": ups * bpu / 1e9 / HBM_PEAK_GBS,
                                    "test_rmse": r["rmses"][args.warmup + i]}) + "\n")
    bytes_per_update, avg_epoch_s, achieved_gbs = rates(r)
    value = r["nnz"] * args.steps / r["wall"]
    kernel = r["kernel"]
    key = f"{kernel}_{scheme}_{w['name']}" + (f"_k{args.k}" if args.k else "")
    variant = [x for x in sys.argv[1:] if x not in ("--no-cpu-baseline", "--copy-calibration", "--no-extra")]
    drop = {"--steps", "--warmup", "--workload", "--scheme", "--cpu-seconds", "--cpu-threads", "--gpus", "--log-jsonl",
            "--extra-steps"}
    variant = [x for i, x in enumerate(variant) if x not in drop and (i == 0 or variant[i - 1] not in drop)]
    traffic = measured_traffic(key, variant)
    out = {
        "metric": f"SGD updates/sec and achieved HBM GB/s (% of peak) at k={w['k']}, 1 MI355X",
        "value": value,
        "unit": "updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["wall"] / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if r["dtype"] == 0 else "f16-storage/f32-math",
        "data": f"synthetic (seeded planted low-rank model with the {w['name']} shape)",
        "config": {"workload": describe(r), "scheme": scheme, "form": r["form"] or None,
                   "workers": args.workers or "auto", "staged": args.staged, "resident_waves": r["resident"],
                   "depth": args.depth or "auto", "epochs_timed": args.steps},
        "roofline": {"bound": "hbm", "achieved": achieved_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": kernel,
                     "bytes_per_update": bytes_per_update, "updates_per_launch": r["nnz"],
                     "avg_launch_ms": avg_epoch_s * 1e3,
                     "note": "achieved counts every row access at HBM cost (4k*sizeof+12 B per update); rows served "
                             "by the L2 or the Infinity Cache can push it past the peak.  traffic: L2-to-fabric bytes "
                             "per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a 4 GiB copy), null unless "
                             "taken on these kernel sources"},
        "epoch_updates_per_s": r["nnz"] / avg_epoch_s,
        "median_epoch_ms": sorted(r["epoch_ms"])[len(r["epoch_ms"]) // 2],
        "test_rmse": r["rmses"][-1],
    }
    if traffic:
        out["roofline"]["traffic_gbs"] = traffic / avg_epoch_s / 1e9
        out["roofline"]["traffic_frac"] = traffic / avg_epoch_s / 1e9 / HBM_PEAK_GBS
    rec = profile_record(key, variant)
    sq = (rec or {}).get("sq_per_launch") or {}
    if sq.get("SQ_INSTS_VALU"):
        # the bound that applies where the rows come from the caches: wave64
        # vector instructions issued per second against what the chip can issue
        peak = rec["valu_issue_peak_per_s"]
        rate = sq["SQ_INSTS_VALU"] / avg_epoch_s
        out["roofline_issue"] = {"bound": "valu-issue", "achieved": rate / 1e9, "peak": peak / 1e9,
                                 "unit": "G wave64 vector instructions/s", "frac": rate / peak,
                                 "valu_per_update": sq["SQ_INSTS_VALU"] / r["nnz"],
                                 "salu_per_update": (sq.get("SQ_INSTS_SALU") or 0) / r["nnz"],
                                 "note": "instruction counts per launch from the committed rocprofv3 SQ counters "
                                         "(same kernel sources), rate over this run's average launch"}
    if scheme == "table":
        out["config"]["table_grid"] = r["grid_s"]
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle on a bounded prefix ({threads} OpenMP threads; {physical} physical cores "
            f"available; OMP_PROC_BIND={os.environ.get('OMP_PROC_BIND')})")
        serial, omp = cpu_baseline(w, r["S"], args.cpu_seconds, threads)
        out["cpu_baseline"] = serial
        if omp:
            omp["physical_cores_available"] = physical
            out["cpu_baseline_openmp"] = omp
    r["S"] = None
    if not args.no_extra and not args.staged and args.workload == "hugewiki" and not args.ntrain and not args.k:
        extra = []
        for name in ("netflix", "yahoo"):
            e = measure(args, name, "hogwild", args.extra_steps, 1, dev)
            bpu, avg_s, gbs = rates(e)
            extra.append({"workload": describe(e), "scheme": "hogwild",
                          "form": e["form"], "kernel": e["kernel"],
                          "epochs_timed": args.extra_steps, "median_epoch_ms": sorted(e["epoch_ms"])[len(e["epoch_ms"]) // 2],
                          "epoch_updates_per_s": e["nnz"] / avg_s, "bytes_per_update": bpu,
                          "algorithmic_gbs": gbs, "frac": gbs / HBM_PEAK_GBS,
                          "test_rmse_after_epochs": [len(e["rmses"]), e["rmses"][-1]]})
        out["extra"] = extra
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
