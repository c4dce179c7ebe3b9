#!/usr/bin/env python3
"""Throughput of the population-fitness path on one MI355X.

A step is one GA generation of the 16384-genome workload (256 devices,
126-block model, 32-48 clusters per genome): e2_eval_population (cluster
extraction, the Algorithm 1 DP for every (genome, cluster) pair, Eq. 3-5
fitness) followed by e2_ga_step (elites, tournaments, crossover, mutation).
Inputs are resident in HBM before timing; the context (quantised tables) is
built once, outside the timed region.

Printed on one JSON line:
  value        DP cells/s: the Algorithm 1 table size m * sum_{k=1..m}(N-k+1)
               summed over every feasible (genome, cluster) problem of each
               timed generation, divided by the timed wall time
  fitness_evals_per_s   genomes scored per second
  roofline     the DP launch (extraction + DP + fitness kernels of one
               e2_eval_population call, timed with events on its stream)
               against the int32 VALU peak: 8 int32 VALU ops per j-candidate
               the kernel evaluates (64-bit subtract 2, 64-bit max 3,
               64-bit min 3)
  cpu_baseline the CPU oracle on a bounded sample of the same generation-0
               population, single-threaded
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2606_03770_amd as e2  # noqa: E402
from paper_2606_03770_amd import workload  # noqa: E402

METRIC = "partition-DP cells/sec and GA fitness evals/sec on 1 MI355X; % int-VALU peak"
INF = (1 << 64) - 1
# int32 VALU lane-ops per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
INT_VALU_PEAK = 256 * 4 * 16 * 2.4e9
OPS_PER_CANDIDATE = 8


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# Work accounting (host side, from the same integer inputs).
# ---------------------------------------------------------------------------
def window_tables(wl):
    """win[f][d][i]: smallest start j with blocks j..i (+ head if f) within
    device d's memory, 255 if none; cap[f][d]: longest stage that fits."""
    M, N = wl.n_dev, wl.n_layer
    wp = np.concatenate([[0], np.cumsum(wl.layer_bytes.astype(object))])
    win = np.full((2, M, N), 255, dtype=np.int64)
    cap = np.zeros((2, M), dtype=np.int64)
    for f in range(2):
        extra = int(wl.head_bytes) if f else 0
        for d in range(M):
            mem = int(wl.mem_bytes[d])
            j = 0
            for i in range(N):
                while j <= i and wp[i + 1] - wp[j] + extra > mem:
                    j += 1
                if j <= i:
                    win[f, d, i] = j
                    cap[f, d] = max(cap[f, d], i - j + 1)
    return win, cap


def row_candidates(win, N):
    """rc[f][d][k]: j-candidates of DP row k (k >= 2) on device d."""
    i = np.arange(N)
    rc = np.zeros(win.shape[:2] + (N + 1,), dtype=np.int64)
    for k in range(2, N + 1):
        lo = np.maximum(win, k - 1)
        c = np.where((win == 255) | (i < k - 1), 0, np.maximum(0, i - lo + 1))
        rc[:, :, k] = c.sum(axis=2)
    return rc


def generation_work(wl, labels, T, master, win_cap_rc):
    """(Algorithm 1 cells over feasible problems, j-candidates the DP kernel
    evaluates) for one population, vectorised over (genome, device)."""
    win, cap, rc = win_cap_rc
    N, K = wl.n_layer, wl.k_max
    P, M = labels.shape
    lab = labels.astype(np.int64)
    assigned = lab < K
    pp = np.repeat(np.arange(P), M).reshape(P, M)
    dd = np.tile(np.arange(M), (P, 1))
    key = (pp * 256 + np.where(assigned, lab, 255)).ravel()
    m = np.bincount(key, minlength=P * 256).reshape(P, 256)[:, :K]
    feasible = T != INF
    cells = int((m * (m * N - m * (m - 1) // 2))[feasible].sum())
    # chain position (1-based) of every device: rank by id within (genome, label)
    order = np.lexsort((dd.ravel(), key))
    sk = key[order]
    first = np.r_[0, np.nonzero(np.diff(sk))[0] + 1]
    start = np.repeat(first, np.diff(np.r_[first, len(sk)]))
    rank = np.empty(P * M, dtype=np.int64)
    rank[order] = np.arange(P * M) - start + 1
    rank = rank.reshape(P, M)
    c0 = cap[0][dd]
    csum = np.bincount(key, weights=c0.ravel(), minlength=P * 256).reshape(P, 256)[:, :K]
    cmin = np.full(P * 256, 1 << 30, dtype=np.int64)
    np.minimum.at(cmin, key, c0.ravel())
    cmin = cmin.reshape(P, 256)[:, :K]
    hmax = np.zeros(P * 256, dtype=np.int64)
    np.maximum.at(hmax, key, cap[1][dd].ravel())
    hmax = hmax.reshape(P, 256)[:, :K]
    listed = (m >= 1) & (m <= N) & (csum >= N) & (cmin >= 1) & (hmax >= 1)
    k = np.minimum(rank, N)
    r0 = np.where(rank >= 2, rc[0][dd, k], 0)
    r1 = np.where(rank >= 2, rc[1][dd, k], 0)
    mq = np.where(assigned, m[pp, np.minimum(lab, K - 1)], 0)
    per_dev = (mq - 1) * r0 + r1  # every master position
    # one more pass for the chosen master of feasible clusters
    safe_lab = np.minimum(lab, K - 1)
    mdev = master[pp, safe_lab].astype(np.int64)
    mrank = np.where(mdev >= 0, rank[pp, np.maximum(mdev, 0)], 0)
    per_dev += np.where(feasible[pp, safe_lab], np.where(rank == mrank, r1, r0), 0)
    use = assigned & listed[pp, safe_lab]
    cand = int(per_dev[use].sum())
    return cells, cand


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5_256dev_126L_ga", choices=workload.NAMES)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU-oracle sample (0 disables)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes 5 times "
                         "(reference for the HBM byte counters) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported in this build "
              f"(the evaluation shards by genome range; see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    e2.lib()

    wl = workload.make(args.workload)
    P, M, K = wl.population, wl.n_dev, wl.k_max
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    stream = torch.cuda.current_stream()
    L0 = torch.from_numpy(wl.labels).to(dev)
    R0 = torch.from_numpy(wl.roles).to(dev)
    Lb = [torch.empty_like(L0), torch.empty_like(L0)]
    Rb = [torch.empty_like(R0), torch.empty_like(R0)]
    fit = {k: torch.empty(P, dtype=torch.int64, device=dev) for k in ("w", "phase")}
    fp = wl.fitness_params()

    def reset():
        Lb[0].copy_(L0)
        Rb[0].copy_(R0)
        torch.cuda.synchronize()

    def run(n_steps, events=None):
        cur = 0
        for g in range(n_steps):
            if events is not None:
                events[g][0].record(stream)
            e2.e2_eval_population(ctx, Lb[cur], Rb[cur], fp, with_rates=False, out=fit)
            if events is not None:
                events[g][1].record(stream)
            e2.e2_ga_step(ctx, Lb[cur], Rb[cur], fit["w"], fit["phase"], wl.ga_params(g),
                          out=(Lb[1 - cur], Rb[1 - cur]))
            cur = 1 - cur

    log(f"workload {wl.name}: P={P} M={M} N={wl.n_layer} k_max={K}; warmup {args.warmup}")
    reset()
    run(args.warmup)
    torch.cuda.synchronize()
    reset()
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.steps, events)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    eval_ms = [a.elapsed_time(b) for a, b in events]
    log(f"timed {args.steps} steps: {elapsed * 1e3:.2f} ms; eval launches "
        f"{np.mean(eval_ms):.3f} ms avg")

    # replay the same generations to count the work (outside the timed region)
    wcr = window_tables(wl)
    wcr = (wcr[0], wcr[1], row_candidates(wcr[0], wl.n_layer))
    Lr, Rr = L0.clone(), R0.clone()
    cells = cand = 0
    for g in range(args.steps):
        sol = e2.e2_solve_partitions(ctx, Lr, Rr)
        f2 = e2.e2_eval_population(ctx, Lr, Rr, fp, with_rates=False)
        lo, ro = e2.e2_ga_step(ctx, Lr, Rr, f2["w"], f2["phase"], wl.ga_params(g))
        torch.cuda.synchronize()
        c1, c2 = generation_work(wl, Lr.cpu().numpy(), e2.u64(sol["T"]),
                                 sol["master"].cpu().numpy(), wcr)
        cells += c1
        cand += c2
        Lr, Rr = lo, ro
    value = cells / elapsed
    dp_time = sum(eval_ms) / 1e3
    achieved = cand * OPS_PER_CANDIDATE / dp_time
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "DP cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": wl.name, "devices": M, "layers": wl.n_layer,
                   "population": P, "clusters_per_genome": "32-48" if K == 48 else str(K),
                   "step": "one GA generation: e2_eval_population + e2_ga_step"},
        "fitness_evals_per_s": P * args.steps / elapsed,
        "dp_cells_per_step": cells / args.steps,
        "j_candidates_per_step": cand / args.steps,
        "roofline": {"bound": "alu", "kernel": "k_dp (e2_eval_population launch)",
                     "achieved": achieved / 1e12, "peak": INT_VALU_PEAK / 1e12,
                     "unit": "TOP/s (int32 VALU)", "frac": achieved / INT_VALU_PEAK,
                     "traffic": None,
                     "avg_launch_ms": dp_time * 1e3 / args.steps},
    }
    if args.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def copy_calibration(nbytes):
    """A plain copy of a known size: FETCH_SIZE / WRITE_SIZE per dispatch of
    this kernel, against nbytes, give the scale of the byte counters."""
    import torch
    src = torch.ones(nbytes // 8, dtype=torch.int64, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": (nbytes // 8) * 8, "launches": 5}), flush=True)


def cpu_baseline(wl, seconds):
    """The oracle, as it is, on the first S genomes of the generation-0
    population (S sized from a short probe to take about `seconds`)."""
    import oracle
    oracle._load()
    probe = 16
    t0 = time.perf_counter()
    oracle.eval_population(wl.subset(np.arange(probe)))
    dt = time.perf_counter() - t0
    S = int(min(wl.population, max(probe, probe * seconds / max(dt, 1e-6))))
    sub = wl.subset(np.arange(S))
    t0 = time.perf_counter()
    sol = oracle.eval_population(sub)
    dt = time.perf_counter() - t0
    cells = 0
    N = wl.n_layer
    for p in range(S):
        for q in range(wl.k_max):
            if sol["T"][p, q] != INF:
                m = int((sub.labels[p] == q).sum())
                cells += m * sum(N - k + 1 for k in range(1, m + 1))
    log(f"cpu oracle: {S} genomes in {dt:.2f} s")
    return {"value": cells / dt, "unit": "DP cells/s", "cores": 1, "kind": "oracle",
            "sample": f"first {S} of {wl.population} genomes of generation 0, "
                      f"full evaluation (quantise, DP per cluster, fitness)",
            "fitness_evals_per_s": S / dt, "seconds": dt}


if __name__ == "__main__":
    main()
