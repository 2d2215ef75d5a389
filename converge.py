"""Convergence and scalability experiments on one MI355X (the analogues of the
paper's schedule comparison, section 3.2.4, and of its updates/s-versus-
workers figures).

  python converge.py curves  [--workload netflix_fp16] [--epochs 20] [--lr config|paper]
                             [--schemes hogwild,wavefront:8,wavefront:32] [--target 0.92]
      Test RMSE after every epoch and the cumulative epoch-kernel time, per
      schedule, from the same initial factors; prints the epoch and the time at
      which each schedule first reaches --target.

  python converge.py workers [--workload netflix_fp16] [--counts 64,128,...,8192]
                             [--schemes hogwild,wavefront:32,table] [--uniform]
      Updates/s of the epoch kernel against the number of concurrent workers
      (wavefronts), one warm-up and --epochs timed epochs per point; a count
      of 0 is the library's default launch.  "table" is the global scheduling
      table (LIBMF's policy, section 3.2.1) on a grid of twice as many row and
      column blocks as workers (at most 1024), "table:s" on a fixed grid of
      side s.  --uniform draws the workload's users and items uniformly
      instead of Zipf-like.

  python converge.py chain [--workload netflix_fp16] [--grid s]
      Where a pooled wavefront-update epoch goes: per-block claim and
      completion stamps of one traced epoch, summarised for the column block
      holding the most samples (whose blocks run one after another) and for
      the teams.

Learning rates: "config" is the workload's own schedule (lr * decay^t);
"paper" is the decaying schedule of the evaluation section,
s_t = alpha / (1 + beta * t^1.5), with the per-dataset alpha, beta and lambda
of its parameter table (the Netflix row for the Netflix-shaped sets).

Every run prints one JSON line per measurement, then a markdown table.  The
data are the seeded synthetic sets of paper_1610_05838_amd.datagen.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Parameter table of the evaluation section: (lambda, alpha, beta) per dataset.
PAPER_PARAMS = {"netflix": (0.05, 0.08, 0.3), "yahoo": (1.0, 0.08, 0.2), "hugewiki": (0.03, 0.08, 0.3)}


def log(msg):
    print(f"[converge] {msg}", file=sys.stderr, flush=True)


def stand_in(name: str) -> str:
    """The dataset a synthetic workload stands in for."""
    for d in PAPER_PARAMS:
        if name.startswith(d):
            return d
    raise SystemExit(f"no parameter row for workload {name!r}")


def lr_schedule(w: dict, kind: str):
    """(lr(t), lambda) for the chosen schedule."""
    from paper_1610_05838_amd import datagen

    if kind == "config":
        return (lambda t: datagen.lr_at(w, t)), w["lam"]
    lam, alpha, beta = PAPER_PARAMS[stand_in(w["name"])]
    return (lambda t: alpha / (1.0 + beta * t ** 1.5)), lam


def parse_schemes(text: str):
    out = []
    for item in text.split(","):
        name, _, s = item.partition(":")
        if name not in ("hogwild", "wavefront", "wavefront_det", "table"):
            raise SystemExit(f"unknown scheme {name!r}")
        out.append((name, int(s) if s else 0))
    return out


def label(scheme, s):
    if scheme == "table":
        return "global table" + (f" s={s}" if s else " s=2W")
    return scheme if scheme == "hogwild" else f"{scheme} s={s}"


class Runner:
    """Holds the device copies of one workload's train and test sets."""

    def __init__(self, workload: str, uniform: bool = False):
        import torch

        from paper_1610_05838_amd import datagen, mfsgd

        assert torch.cuda.is_available(), "converge.py needs a GPU"
        self.torch, self.datagen, self.M = torch, datagen, mfsgd
        self.dev = torch.device("cuda:0")
        torch.cuda.set_device(self.dev)
        w = datagen.workload(workload, **(dict(zipf_u=0.0, zipf_v=0.0) if uniform else {}))
        if uniform:
            w["name"] += " (uniform indices)"
        t0 = time.perf_counter()
        if w["draw"] == "independent":
            self.dS = datagen.draw_to_device(w, 0, w["ntrain"], self.dev)
            T = datagen.draw(w, w["ntrain"], w["ntest"])
        else:
            S, T = datagen.make(w)
            self.dS = mfsgd.samples_to_device(S, self.dev)
        self.dT = mfsgd.samples_to_device(T, self.dev)
        self.w = w
        log(f"generated {workload}: {w['ntrain']} train + {w['ntest']} test in {time.perf_counter() - t0:.1f}s")

    def setup(self, scheme, s, workers=0, partition=2):
        """Initialise (and plan); returns the number of concurrent workers
        (wavefronts) the launch will have, 0 for the library's default.
        A wavefront-update grid of side s runs s teams of team_waves
        wavefronts, grouped four to a workgroup (one-wavefront teams when
        workers == s)."""
        w, M = self.w, self.M
        # every option at the library's default except those named here
        M.reset_options()
        M.set_option("dtype", 1 if w["dtype"] == "fp16" else 0)
        if scheme == "table":
            W = workers or 128
            grid = s or min(1024, 2 * W)
            M.set_option("table_grid", grid)
            M.set_option("table_workers", W)
            M.init(w["m"], w["n"], w["k"], w["seed"])
            return W
        s = s or w.get("grid_s", 32)
        team = 0
        actual = workers
        if scheme != "hogwild" and workers > 0:
            team = max(1, workers // s)
            actual = s if team == 1 else s * 4 * ((team + 3) // 4)
        if scheme == "hogwild":
            M.set_option("workers", workers)
            M.set_option("partition", partition)
        else:
            M.set_option("team_waves", team)
        M.init(w["m"], w["n"], w["k"], w["seed"])
        if scheme != "hogwild":
            M.plan(self.dS, s)
        return actual

    def epoch_ms(self, scheme, lr, lam):
        torch, stream = self.torch, self.torch.cuda.current_stream()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        self.M.epoch(self.dS, lr, lam, lam, scheme, stream)
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b)


def curves(args):
    r = Runner(args.workload, args.uniform)
    w = r.w
    lr_t, lam = lr_schedule(w, args.lr)
    rows = []
    for scheme, s in parse_schemes(args.schemes):
        r.setup(scheme, s, partition=args.partition)
        s_eff = (s or 256) if scheme == "table" else (s or w.get("grid_s", 32))
        elapsed, hist, hit = 0.0, [], None
        for t in range(args.epochs):
            ms = r.epoch_ms(scheme, lr_t(t), lam)
            elapsed += ms
            e = r.M.rmse(r.dT)
            hist.append(e)
            if hit is None and e <= args.target:
                hit = (t + 1, elapsed)
            print(json.dumps({"exp": "curves", "workload": w["name"], "lr": args.lr, "scheme": label(scheme, s_eff),
                              "epoch": t + 1, "lr_t": round(lr_t(t), 6), "epoch_ms": round(ms, 3),
                              "elapsed_ms": round(elapsed, 3), "test_rmse": round(e, 6)}), flush=True)
        rows.append((label(scheme, s_eff), elapsed / args.epochs, hist, hit))
        r.M.finalize()
    marks = [t for t in (1, 2, 5, 10, 20, 40) if t <= args.epochs]
    print(f"\n{w['name']}, lr schedule {args.lr}, {args.epochs} epochs, target test RMSE {args.target}\n")
    print("| schedule | mean epoch ms | test RMSE after " + " / ".join(map(str, marks)) + " epochs | time to target |")
    print("|---|---|---|---|")
    for name, mean_ms, hist, hit in rows:
        tt = f"{hit[1]:.0f} ms ({hit[0]} epochs)" if hit else "not reached"
        print(f"| {name} | {mean_ms:.2f} | " + " / ".join(f"{hist[t - 1]:.4f}" for t in marks) + f" | {tt} |")


def workers(args):
    r = Runner(args.workload, args.uniform)
    w = r.w
    lr_t, lam = lr_schedule(w, "config")
    counts = [int(x) for x in args.counts.split(",")]
    table = {}
    for scheme, s in parse_schemes(args.schemes):
        for W in counts:
            s_eff = (s or min(1024, 2 * W)) if scheme == "table" else (s or w.get("grid_s", 32))
            actual = r.setup(scheme, s, workers=W, partition=args.partition)
            if actual != W:
                log(f"{label(scheme, s_eff)}: {W} workers is not a team shape (runs {actual}); skipped")
                r.M.finalize()
                continue
            resident = r.M.get_option("resident_waves")
            if W == 0 and scheme == "hogwild":
                W = resident
            r.epoch_ms(scheme, lr_t(0), lam)
            if scheme not in ("hogwild", "table"):
                # workgroups per team as laid out (capped by the co-resident
                # workgroups of the team's XCD); four wavefronts each, one for
                # one-wavefront teams
                _, sizes = r.M.debug_team_layout(s_eff)
                actual = int(sizes.sum().item()) * (1 if W == s_eff else 4)
                if actual != W:
                    log(f"{label(scheme, s_eff)}: {W} workers requested, {actual} launched")
                    W = actual
            ms = min(r.epoch_ms(scheme, lr_t(1 + i), lam) for i in range(args.epochs))
            ups = w["ntrain"] / (ms / 1e3)
            table[(label(scheme, s), W)] = ups
            print(json.dumps({"exp": "workers", "workload": w["name"], "scheme": label(scheme, s_eff), "workers": W,
                              "resident_waves": resident, "epoch_ms": round(ms, 3), "updates_per_s": ups}),
                  flush=True)
            r.M.finalize()
    names = list(dict.fromkeys(k[0] for k in table))
    print(f"\n{w['name']}: updates/s (10^9) of the epoch kernel against concurrent workers (wavefronts)\n")
    print("| workers | " + " | ".join(names) + " |")
    print("|---|" + "---|" * len(names))
    for W in sorted({k[1] for k in table}):
        print(f"| {W} | " + " | ".join(f"{table[(n, W)] / 1e9:.3f}" if (n, W) in table else "-" for n in names)
              + " |")


def chain(args):
    """Where a pooled wavefront-update epoch goes: the per-block claim and
    completion stamps (debug trace, 100 MHz clock) of one epoch after a
    warm-up epoch, summarised for the column block holding the most samples
    (its blocks run one after another) and for the teams."""
    import numpy as np

    r = Runner(args.workload, args.uniform)
    w, M = r.w, r.M
    lr_t, lam = lr_schedule(w, "config")
    s = args.grid or w.get("grid_s", 32)
    r.setup("wavefront", s)
    starts = M.debug_plan_starts(s).cpu().numpy()
    warm = r.epoch_ms("wavefront", lr_t(0), lam)
    M.set_option("debug", 2)
    traced = r.epoch_ms("wavefront", lr_t(1), lam)
    tr = M.debug_trace(5 * s * s).cpu().numpy().view(np.uint32)
    M.finalize()
    cols = tr[:s * s].reshape(s, s).astype(np.int64)                # [team, wave] -> column block
    clk = tr[3 * s * s:5 * s * s].reshape(s, s, 2).astype(np.int64)  # claim, completion (10 ns ticks)
    cnt = np.diff(starts).reshape(s, s)                              # [row block, column block] -> samples
    t0 = clk[:, :, 0].min()
    c0 = ((clk[:, :, 0] - t0) % (1 << 32)) / 100.0                   # microseconds
    c1 = ((clk[:, :, 1] - t0) % (1 << 32)) / 100.0
    n = np.array([[cnt[t, cols[t, x]] for x in range(s)] for t in range(s)])
    colsum = cnt.sum(axis=0)
    hot = int(np.argmax(colsum))
    links = sorted((c0[t, x], c1[t, x], t, x, n[t, x]) for t in range(s) for x in range(s) if cols[t, x] == hot)
    busy = sum(b - a for a, b, *_ in links)
    gaps = [links[i + 1][0] - links[i][1] for i in range(len(links) - 1)]
    rates = [c / (b - a) / 1e3 for a, b, _, _, c in links if b > a and c >= 10_000]
    span = c1.max()
    print(f"\n{w['name']}, wavefront-update s = {s}: warm-up epoch {warm:.2f} ms, traced epoch {traced:.2f} ms "
          f"(debug stamps on), stamped span {span / 1e3:.2f} ms\n")
    print("| measure | value |")
    print("|---|---|")
    print(f"| column block with the most samples | {hot}: {int(colsum[hot]):,} samples "
          f"({colsum[hot] / cnt.sum():.3f} of all, mean column {cnt.sum() / s / cnt.sum():.3f}) |")
    print(f"| its blocks busy (sum of claim-to-completion) | {busy / 1e3:.2f} ms ({busy / span:.2f} of the span) |")
    print(f"| hand-over gaps between its blocks | {sum(gaps) / 1e3:.3f} ms (largest {max(gaps):.1f} us) |")
    if rates:
        print(f"| its blocks of >= 10,000 samples: updates/s | median {np.median(rates):.3f} x 10^9, "
              f"min {min(rates):.3f}, max {max(rates):.3f} |")
    ends = c1.max(axis=1) / 1e3
    print(f"| teams' last completion | min {ends.min():.2f} ms, median {np.median(ends):.2f}, max {ends.max():.2f} |")
    print(f"\nBlocks of column block {hot} in wave order (claim and completion in us from the first claim):\n")
    print("| wave | team | samples | claimed | completed | updates/s (10^9) |")
    print("|---|---|---|---|---|---|")
    for a, b, t, x, c in links:
        rate = f"{c / (b - a) / 1e3:.3f}" if b > a else "-"
        print(f"| {x} | {t} | {int(c):,} | {a:.1f} | {b:.1f} | {rate} |")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("exp", choices=["curves", "workers", "chain"])
    ap.add_argument("--workload", default="netflix_fp16")
    ap.add_argument("--epochs", type=int, default=0, help="curves: epochs (default 20); workers: timed epochs (default 2)")
    ap.add_argument("--lr", choices=["config", "paper"], default="config")
    ap.add_argument("--schemes", default="")
    ap.add_argument("--target", type=float, default=0.92)
    ap.add_argument("--partition", type=int, default=2,
                    help="batch-Hogwild! form (the library's option): 2 automatic (default), 0 one address "
                         "space, 1 XCD-partitioned, 3 free-running partition, 4 one XCD")
    ap.add_argument("--counts", default="32,64,128,256,512,1024,2048,4096,8192")
    ap.add_argument("--uniform", action="store_true", help="users and items drawn uniformly (no Zipf skew)")
    ap.add_argument("--grid", type=int, default=0, help="chain: grid side (default: the workload's)")
    args = ap.parse_args()
    if args.exp == "curves":
        args.epochs = args.epochs or 20
        args.schemes = args.schemes or "hogwild,wavefront:8,wavefront:32"
        curves(args)
    elif args.exp == "chain":
        chain(args)
    else:
        args.epochs = args.epochs or 2
        args.schemes = args.schemes or "hogwild,wavefront:32"
        workers(args)


if __name__ == "__main__":
    main()
