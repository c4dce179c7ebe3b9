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
  roofline     the DP kernel k_dp (timed with HIP events the library records
               around it on the call's stream) against the int32 VALU peak:
               VALU ops per useful j-candidate of the DP kernel, 3 with u32 or
               fp64 keys (subtract, max, min; fp64 vector ops issue at the
               int32 rate on MI355X) and 8 with the u64 keys of the reference
               path (64-bit subtract 2, max 3, min 3), candidates counted on
               the host from the same inputs; traffic = HBM bytes per launch
               from the committed rocprofv3 counters when they were taken on
               the current kernel sources
  cpu_baseline the CPU oracle on a bounded sample of the same generation-0
               population, single-threaded
  role_search  e2_search_roles on the 1024-genome, 64-device workload with
               its decode-slot model: per call, every cluster is solved for
               prefill and for 1..8 decode requests in flight, then roles are
               brute-forced per genome over its clusters with a decode rate;
               then a two-chromosome generation (search + App. A GA step)
  role_search_256_devices  the same on the 16384-genome, 256-device workload
               (32-48 clusters per genome)
  ablations    the two ablations of Sec. 4.2 on the same 1024-genome
               workload: finishing-time objective vs Algorithm 1, adapted
               SplitWise roles vs the brute-force search (time per call and
               how many genomes each side wins); and the idle-device
               relaxation (time per call, clusters it solves faster)
  two_chromosome  the same measurements for the paper's two-chromosome
               genomes (an ordering of the devices cut into replicas, App. A):
               e2_eval_population_ordered + e2_ga_step_ordered per generation
               on the same problem instance and population size
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
MAX_BANDED_CHAIN = 64  # longest chain the banded DP path takes (one device per lane)
LDS_TB_CELLS = 2048    # split-point bytes a DP wave keeps in LDS
PAIR_MAX_CELLS = 32    # widest band whose combine and forward row share one pass


def pool_cells(N):
    """Cells of a DP wave's forward-row pool: the largest band total
    (m - 1)(N - m + 1) of a chain the banded path takes."""
    best = max([(m - 1) * (N - m + 1) for m in range(2, min(MAX_BANDED_CHAIN, N) + 1)], default=0)
    return max(best, LDS_TB_CELLS)


U32_MAX_VALUE = 0xFFFFFE  # largest finite value of the u32-key path
F64_LIMIT = 1 << 45       # prefix sums, head and link times of an fp64-key problem stay below
OPS_PER_CANDIDATE_NARROW = 3  # u32 or fp64 keys: subtract, max, min



def window_tables(wl):
    """Per device: window starts win[f][d][i] (smallest j with blocks j..i,
    plus the head if f, within memory; 255 if none), reversed-block window
    starts winR[d][x], and the longest stage cap[f][d]."""
    M, N = wl.n_dev, wl.n_layer
    wp = np.concatenate([[0], np.cumsum(wl.layer_bytes.astype(object))])
    win = np.full((2, M, N), 255, dtype=np.int64)
    winR = np.full((M, N), 255, dtype=np.int64)
    cap = np.zeros((2, M), dtype=np.int64)
    for d in range(M):
        mem = int(wl.mem_bytes[d])
        for f in range(2):
            extra = int(wl.head_bytes) if f else 0
            j = 0
            for i in range(N):
                while j <= i and wp[i + 1] - wp[j] + extra > mem:
                    j += 1
                if j <= i:
                    win[f, d, i] = j
                    cap[f, d] = max(cap[f, d], i - j + 1)
        y = 0
        for x in range(N):
            while y <= x and wp[N - y] - wp[N - 1 - x] > mem:
                y += 1
            if y <= x:
                winR[d, x] = y
    return win, winR, cap


def count_tables(win, winR, N):
    """Prefix sums over cells of the window lengths i - max(w(i), kmin) + 1
    (0 where no stage fits), for every device and every kmin:
    C[f][d][kmin][i] (forward, f = head), CR[d][kmin][x] (reversed)."""
    def build(w):
        k = np.arange(N)[:, None]                  # kmin
        i = np.arange(N)[None, :]                  # cell
        lo = np.maximum(w[..., None, :], k)        # [..., kmin, cell]
        c = np.where(w[..., None, :] == 255, 0, np.maximum(0, i - lo + 1))
        out = np.zeros(c.shape[:-1] + (N + 1,), dtype=np.int64)
        np.cumsum(c, axis=-1, out=out[..., 1:])
        return out
    return build(win), build(winR)


def value_bounds(wl, win):
    """vmax[r][d]: the largest cost of a memory-fitting stage of device d in
    role r (plus the head time for stages holding the head bytes); vtot[r][d]:
    the time of all blocks plus the head; and the quantised link times
    tau[r][d][e] (INF for dead links)."""
    t, h, tau = e2.e2_quantise(wl.problem_arrays())
    M, N = wl.n_dev, wl.n_layer
    vtot = np.array([[int(t[r, d].sum(dtype=np.uint64)) + int(h[r, d]) for d in range(M)]
                     for r in range(2)], dtype=object)
    vmax = np.zeros((2, M), dtype=object)
    for r in range(2):
        P = np.concatenate([np.zeros((M, 1), np.uint64), np.cumsum(t[r], axis=1, dtype=np.uint64)],
                           1)
        for d in range(M):
            best = 0
            for f in range(2):
                ok = win[f, d] != 255
                if ok.any():
                    i = np.nonzero(ok)[0]
                    c = P[d, i + 1] - P[d, win[f, d, i]]
                    best = max(best, int(c.max()) + (int(h[r, d]) if f else 0))
            vmax[r, d] = best
    return vmax, vtot, tau


def label_problems(labels, k_max):
    """(genome, cluster, chain) of every non-empty cluster of labelled
    genomes; a chain lists the cluster's devices in ascending id."""
    out = []
    for p in range(labels.shape[0]):
        row = labels[p]
        for q in np.unique(row):
            if q < k_max:
                out.append((p, int(q), np.nonzero(row == q)[0]))
    return out


def ordered_problems(order, sizes):
    """(genome, replica, chain) of every non-empty replica of two-chromosome
    genomes; a chain is the replica's run of the ordering.  Replicas holding
    an id >= M are left out (the library rejects them before the DP)."""
    P, M = order.shape
    ends = np.minimum(np.cumsum(sizes.astype(np.int64), axis=1), M)
    starts = np.concatenate([np.zeros((P, 1), np.int64), ends[:, :-1]], axis=1)
    out = []
    for p in range(P):
        for q in np.nonzero(ends[p] > starts[p])[0]:
            chain = order[p, starts[p, q]:ends[p, q]].astype(np.int64)
            if chain.max() < M:
                out.append((p, int(q), chain))
    return out


def head_free(problem):
    """The same problem with no head time and no head bytes: every master
    then ties, and the DP's optimum is the optimum without a master."""
    return dict(problem, head_flops=np.zeros(2, dtype=np.uint64), head_bytes=0)


def generation_work(wl, problems, roles, T, master, tabs, T0):
    """(Algorithm 1 cells over feasible problems, useful j-candidates the DP
    kernel evaluates with u64 keys, those it evaluates with u32 or fp64 keys,
    Algorithm 1's own memory-feasible j-candidates over the problems that
    pass the pre-check: one full table per master, every cell scanning the
    split points its window allows)
    for one population, given as its (genome, cluster, chain) problems, their
    optima T, masters and optima T0 without a master (head_free).  The
    candidate count follows k_dp row by row: reversed rows, the last cell of
    the full reversed table (T0), then masters in ascending position with
    the forward row after each, up to the first master whose optimum is T0
    (every master when T0 < T, none when T0 is infinite; a stop in a pass
    that pairs the combine with the forward row evaluates that forward row
    too and keeps the combine's row as the chosen master's first), then the
    chosen master's rows and last cell (banded path); or one full table per master
    plus the chosen master's again (reference path, u64 keys).  A problem takes the
    banded path when its chain has at most 64 devices, its forward bands fit
    the pool and either every finite value it can produce (largest fitting
    stage cost of its devices, largest finite link time) is at most
    U32_MAX_VALUE (u32 keys) or its devices' total times and its link times
    are below F64_LIMIT (fp64 keys)."""
    win, winR, cap, C, CR, vmax, vtot, tau = tabs
    N = wl.n_layer
    feasible = T != INF
    cells = 0
    cand = 0
    cand32 = 0
    alg1 = 0

    def rows(f, d, kmin, lo, hi):
        """useful candidates of rows with cells lo..hi (arrays, broadcast)"""
        ok = hi >= lo
        lo_c = np.clip(lo, 0, N)
        hi_c = np.clip(hi + 1, 0, N)
        v = C[f, d, np.clip(kmin, 0, N - 1), hi_c] - C[f, d, np.clip(kmin, 0, N - 1), lo_c]
        return np.where(ok, v, 0)

    def rrows(d, kmin, lo, hi):
        ok = hi >= lo
        v = CR[d, np.clip(kmin, 0, N - 1), np.clip(hi + 1, 0, N)] - \
            CR[d, np.clip(kmin, 0, N - 1), np.clip(lo, 0, N)]
        return np.where(ok, v, 0)

    # group problems by chain length
    probs = {}
    for p, q, chain in problems:
        probs.setdefault(len(chain), []).append((p, q, chain))
    for m, lst in probs.items():
        n = len(lst)
        pq = np.array([(a, b) for a, b, _ in lst])
        ch = np.stack([c for _, _, c in lst])                      # [n, m]
        feas = feasible[pq[:, 0], pq[:, 1]]
        cells += int(feas.sum()) * m * (m * N - m * (m - 1) // 2)
        c0, cH = cap[0][ch], cap[1][ch]
        listed = (m <= N) & (c0.sum(1) >= N) & (c0.min(1) >= 1) & (cH.max(1) >= 1)
        if not listed.any():
            continue
        ch, c0, cH, feas, pq = ch[listed], c0[listed], cH[listed], feas[listed], pq[listed]
        n = len(ch)
        # Algorithm 1 as the paper states it: for each master, rows 2..m over
        # cells k-1..N-1, the master's row with its head window
        k_all = np.arange(1, m + 1)
        lo_a = np.broadcast_to(k_all - 1, ch.shape)
        hi_a = np.full(ch.shape, N - 1)
        a0 = rows(0, ch, lo_a, lo_a, hi_a)
        a1 = rows(1, ch, lo_a, lo_a, hi_a)
        alg1 += int(((m - 1) * a0 + a1)[:, 1:].sum())
        rr = (roles[pq[:, 0], pq[:, 1]] != 0).astype(np.int64)
        links = [[int(tau[rr[a], ch[a][k - 1], ch[a][k]]) for k in range(1, m)] for a in range(n)]
        links = [[x for x in lk if x != INF] for lk in links]
        b32 = [max([vmax[rr[a], d] for d in ch[a]] + links[a]) for a in range(n)]
        b64 = [max([vtot[rr[a], d] for d in ch[a]] + links[a]) for a in range(n)]
        narrow = np.array([b <= U32_MAX_VALUE or bt < F64_LIMIT for b, bt in zip(b32, b64)],
                          dtype=bool)
        mu = np.zeros(n, dtype=np.int64)
        t_opt = T[pq[:, 0], pq[:, 1]]
        t_free = T0[pq[:, 0], pq[:, 1]]
        mdev = master[pq[:, 0], pq[:, 1]].astype(np.int64)
        for a in range(n):
            if feas[a]:
                mu[a] = int(np.nonzero(ch[a] == mdev[a])[0][0]) + 1
        k = np.arange(1, m + 1)                                     # [m]
        pre = np.concatenate([np.zeros((n, 1), np.int64), np.cumsum(c0, 1)], 1)
        tot = pre[:, m:m + 1]
        flo = np.maximum(k - 1, N - 1 - (tot - pre[:, 1:]))
        fhi = np.minimum(N - 1 - (m - k), pre[:, 1:] - 1)
        sizes = np.where(fhi >= flo, fhi - flo + 1, 0)
        pool = sizes[:, :m - 1].sum(1)
        # chains of up to 64 devices whose forward bands fit the pool take the
        # banded path, the others one full table per master
        fast = (m <= MAX_BANDED_CHAIN) & (pool <= pool_cells(N)) & narrow
        # --- fast path
        if fast.any():
            chf, c0f, cHf = ch[fast], c0[fast], cH[fast]
            lof, hif, muf = flo[fast], fhi[fast], mu[fast]
            pref = pre[fast]
            kk = np.broadcast_to(k, lof.shape)
            jm0 = np.maximum(kk - 1, lof - c0f + 1)
            jmH = np.maximum(kk - 1, lof - cHf + 1)
            # masters 1..ex, forward rows 1..ex-1: ex is the first master
            # reaching T0 (the chosen one when T = T0), m when T0 < T, and 0
            # when T0 is infinite; rows and combines of position 1 scan nothing
            tf, t0f = t_opt[fast], t_free[fast]
            ex = np.where(t0f == INF, 0, np.where(tf == t0f, muf, m))[:, None]
            fwd = rows(0, chf, jm0, lof, hif)
            comb = np.where(cHf > 0, rows(1, chf, jmH, lof, hif), 0)
            tot_f = (fwd * ((kk >= 2) & (kk <= ex - 1) & (kk <= m - 1))).sum(1) + \
                (comb * ((kk >= 2) & (kk <= ex))).sum(1)
            # the last cell of the full reversed table (device 1, all blocks)
            if m >= 2:
                full = np.full(len(chf), N - 1)
                tot_f += rrows(chf[:, 0], np.maximum(m - 1, N - c0f[:, 0]), full, full)
            # reversed rows t = 2..m-1: device k = m+1-t
            for t in range(2, m):
                kd = m + 1 - t
                tt = pref[:, m]
                gl = np.maximum(kd - 1, N - (tt - pref[:, kd - 1]))
                gh = np.minimum(pref[:, kd - 1], N - (m - kd + 1))
                xlo, xhi = N - 1 - gh, N - 1 - gl
                d = chf[:, kd - 1]
                jm = np.maximum(t - 1, xlo - c0f[:, kd - 1] + 1)
                tot_f += np.where(gh >= gl, rrows(d, jm, xlo, xhi), 0)
            # chosen master's rows mu*..m-1 and the last cell
            ff = muf > 0
            for kk1 in range(2, m):
                isn = (kk1 == muf)
                sel = ff & (kk1 >= muf)
                f_arr = isn.astype(np.int64)
                jm = np.where(isn, jmH[:, kk1 - 1], jm0[:, kk1 - 1])
                v0 = rows(0, chf[:, kk1 - 1], jm, lof[:, kk1 - 1], hif[:, kk1 - 1])
                v1 = rows(1, chf[:, kk1 - 1], jm, lof[:, kk1 - 1], hif[:, kk1 - 1])
                tot_f += np.where(sel, np.where(f_arr == 1, v1, v0), 0)
            if m >= 2:
                isn = (muf == m)
                capl = np.where(isn, cHf[:, m - 1], c0f[:, m - 1])
                jm = np.maximum(m - 1, N - capl)
                v0 = rows(0, chf[:, m - 1], jm, np.full(len(chf), N - 1), np.full(len(chf), N - 1))
                v1 = rows(1, chf[:, m - 1], jm, np.full(len(chf), N - 1), np.full(len(chf), N - 1))
                tot_f += np.where(ff, np.where(isn, v1, v0), 0)
            # a sweep that stops at mu* in a paired pass (2 <= mu* <= m-1,
            # a band of at most 32 cells) also evaluates F_mu* in the other
            # half-wave and keeps the combine's row as the chosen master's
            # row mu*, which is then not computed again
            idx = np.clip(muf - 1, 0, m - 1)[:, None]
            n_mu = np.take_along_axis(np.where(hif >= lof, hif - lof + 1, 0), idx, 1)[:, 0]
            paired = (tf == t0f) & (t0f != INF) & (muf >= 2) & (muf <= m - 1) & \
                (n_mu >= 1) & (n_mu <= PAIR_MAX_CELLS)
            tot_f += np.where(paired, np.take_along_axis(fwd, idx, 1)[:, 0] -
                              np.take_along_axis(comb, idx, 1)[:, 0], 0)
            cand32 += int(tot_f.sum())
        # --- reference path
        if (~fast).any():
            chs, mus = ch[~fast], mu[~fast]
            lo = np.broadcast_to(k - 1, chs.shape)
            hi = np.full(chs.shape, N - 1)
            r0 = rows(0, chs, lo, lo, hi)
            r1 = rows(1, chs, lo, lo, hi)
            per = ((m - 1) * r0 + r1)[:, 1:].sum(1)
            extra = np.where(np.arange(1, m + 1)[None, :] == mus[:, None], r1, r0)[:, 1:].sum(1)
            cand += int((per + np.where(mus > 0, extra, 0)).sum())
    return cells, cand, cand32, alg1


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5_256dev_126L_ga", choices=workload.NAMES)
    ap.add_argument("--genomes", default="both", choices=("both", "labels", "two_chromosome"),
                    help="which genome kind(s) to time; the first is the headline")
    ap.add_argument("--ordered-steps", type=int, default=5,
                    help="timed generations of the two-chromosome GA after the headline "
                         "(with --genomes both; 0 disables)")
    ap.add_argument("--search-steps", type=int, default=5,
                    help="timed role and slot searches on the 1024-genome workload "
                         "(with --genomes both; 0 disables)")
    ap.add_argument("--config-steps", type=int, default=10,
                    help="timed evaluations of each of the 12- to 128-device workloads "
                         "(with --genomes both; 0 disables)")
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
    e2.e2_ctx_keep_scratch(ctx)  # a serving loop: scratch kept per stream
    ctx_free = e2.e2_ctx_create(head_free(wl.problem_arrays()))  # work accounting only
    stream = torch.cuda.current_stream()
    fp = wl.fitness_params()
    win, winR, cap = window_tables(wl)
    wcr = (win, winR, cap) + count_tables(win, winR, wl.n_layer) + value_bounds(wl, win)

    fit = {k: torch.empty(P, dtype=torch.int64, device=dev) for k in ("w", "phase")}
    log(f"workload {wl.name}: P={P} M={M} N={wl.n_layer} k_max={K}; warmup {args.warmup}")

    def labelled(n):
        """Genomes as cluster labels per device (the 16384-genome workload's GA)."""
        L0 = torch.from_numpy(wl.labels).to(dev)
        R0 = torch.from_numpy(wl.roles).to(dev)
        bufs = [(torch.empty_like(L0), torch.empty_like(R0)) for _ in range(2)]

        def step(g, cur):
            L, R = bufs[cur]
            e2.e2_eval_population(ctx, L, R, fp, with_rates=False, out=fit)
            e2.e2_ga_step(ctx, L, R, fit["w"], fit["phase"], wl.ga_params(g), out=bufs[1 - cur])

        def count(g, pop):
            L, R = pop
            sol = e2.e2_solve_partitions(ctx, L, R)
            sol0 = e2.e2_solve_partitions(ctx_free, L, R)
            f2 = e2.e2_eval_population(ctx, L, R, fp, with_rates=False)
            nxt = e2.e2_ga_step(ctx, L, R, f2["w"], f2["phase"], wl.ga_params(g))
            torch.cuda.synchronize()
            work = generation_work(wl, label_problems(L.cpu().numpy(), K), R.cpu().numpy(),
                                   e2.u64(sol["T"]), sol["master"].cpu().numpy(), wcr,
                                   e2.u64(sol0["T"]))
            return work, nxt

        return measure(torch, ctx, stream, bufs, (L0, R0), step, count, args.warmup, n)

    def two_chromosome(n):
        """Genomes as an ordering of the devices cut into replicas (App. A)."""
        op = workload.ordered_population(wl)
        log(f"two-chromosome genomes: P={P}, max replica {op.max_replica}")
        O0, S0, Q0 = (torch.from_numpy(x).to(dev) for x in (op.order, op.sizes, op.roles))
        bufs = [tuple(torch.empty_like(x) for x in (O0, S0, Q0)) for _ in range(2)]

        def step(g, cur):
            O, S, Q = bufs[cur]
            e2.e2_eval_population_ordered(ctx, O, S, Q, fp, with_rates=False, out=fit)
            e2.e2_ga_step_ordered(ctx, O, S, Q, fit["w"], fit["phase"], op.ga_params(wl, g),
                                  out=bufs[1 - cur])

        def count(g, pop):
            O, S, Q = pop
            sol = e2.e2_solve_partitions_ordered(ctx, O, S, Q)
            sol0 = e2.e2_solve_partitions_ordered(ctx_free, O, S, Q)
            f2 = e2.e2_eval_population_ordered(ctx, O, S, Q, fp, with_rates=False)
            nxt = e2.e2_ga_step_ordered(ctx, O, S, Q, f2["w"], f2["phase"], op.ga_params(wl, g))
            torch.cuda.synchronize()
            probs = ordered_problems(O.cpu().numpy(), S.cpu().numpy())
            work = generation_work(wl, probs, Q.cpu().numpy(), e2.u64(sol["T"]),
                                   sol["master"].cpu().numpy(), wcr, e2.u64(sol0["T"]))
            return work, nxt

        return measure(torch, ctx, stream, bufs, (O0, S0, Q0), step, count, args.warmup, n)

    def summary(t, n, genomes):
        return {
            "ms_per_step": t["elapsed"] * 1e3 / n,
            "fitness_evals_per_s": P * n / t["elapsed"],
            "kernel_candidates_per_s": (t["cand"] + t["cand32"]) / t["elapsed"],
            "dp_cells_per_step": t["cells"] / n,
            "j_candidates_per_step": (t["cand"] + t["cand32"]) / n,
            "j_candidates_u32_or_f64_keys_per_step": t["cand32"] / n,
            "roofline": roofline(t, n, profiled(wl.name, genomes)),
            "algorithm_1": algorithmic(t, n),
        }

    steps = {"labels": "one GA generation: e2_eval_population + e2_ga_step",
             "two_chromosome": "one GA generation: e2_eval_population_ordered + "
                               "e2_ga_step_ordered"}
    head = "two_chromosome" if args.genomes == "two_chromosome" else "labels"
    t = (two_chromosome if head == "two_chromosome" else labelled)(args.steps)
    result = {
        "metric": METRIC,
        "value": t["cells"] / t["elapsed"],
        "unit": "Algorithm-1-equivalent DP cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": wl.name, "devices": M, "layers": wl.n_layer,
                   "population": P, "clusters_per_genome": "32-48" if K == 48 else str(K),
                   "genomes": head, "step": steps[head]},
    }
    result.update(summary(t, args.steps, head))
    # the paper's two-chromosome genomes on the same problem instance and
    # population size
    if args.genomes == "both" and args.ordered_steps > 0:
        n = args.ordered_steps
        t2 = two_chromosome(n)
        result["two_chromosome"] = dict(step=steps["two_chromosome"], steps=n,
                                        dp_cells_per_s=t2["cells"] / t2["elapsed"],
                                        **summary(t2, n, "two_chromosome"))
    if args.genomes == "both" and args.search_steps > 0:
        result["role_search"] = role_search(torch, dev, args.search_steps, args.warmup)
        result["role_search_256_devices"] = role_search(torch, dev, args.search_steps,
                                                        args.warmup, "c5_256dev_126L_ga")
        result["ablations"] = ablations(torch, dev, args.search_steps, args.warmup)
    cfg_rows = {}
    if args.genomes == "both" and args.config_steps > 0:
        result["configs"] = {}
        for name in workload.NAMES[:4]:
            result["configs"][name], cfg_rows[name] = config_eval(torch, dev, name,
                                                                  args.config_steps, args.warmup)
    if args.cpu_seconds > 0 and head == "labels":
        L0 = torch.from_numpy(wl.labels).to(dev)
        R0 = torch.from_numpy(wl.roles).to(dev)
        sol = e2.e2_solve_partitions(ctx, L0, R0)
        fit0 = e2.e2_eval_population(ctx, L0, R0, fp)
        torch.cuda.synchronize()
        gpu0 = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
                    master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy(),
                    **{k: e2.u64(v) for k, v in fit0.items()})
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, gpu0, cfg_rows)
    print(json.dumps(result), flush=True)


SEARCH_WORKLOAD = "c3_64dev_80L"


def config_eval(torch, dev, name, steps, warmup):
    """One workload's whole population through e2_eval_population: time per
    call (wall clock around `steps` calls after `warmup`), the DP kernel's
    time from the library's events, fitness evaluations/s, and the
    Algorithm 1 cells and candidates of the population against the kernel's
    own candidates.  Returns that record and the GPU's rows of the
    population (T, Lambda, master, layers, w, phase, S_P, S_D)."""
    wl = workload.make(name)
    P, K = wl.population, wl.k_max
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    e2.e2_ctx_keep_scratch(ctx)
    ctx_free = e2.e2_ctx_create(head_free(wl.problem_arrays()))
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    fp = wl.fitness_params()
    out = e2.e2_eval_population(ctx, L, R, fp, with_rates=False)
    for _ in range(warmup):
        e2.e2_eval_population(ctx, L, R, fp, with_rates=False, out=out)
    torch.cuda.synchronize()
    e2.e2_ctx_dp_timing(ctx, steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        e2.e2_eval_population(ctx, L, R, fp, with_rates=False, out=out)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_dp, dp_ms = e2.e2_ctx_dp_elapsed(ctx)
    e2.e2_ctx_dp_timing(ctx, 0)
    sol = e2.e2_solve_partitions(ctx, L, R)
    sol0 = e2.e2_solve_partitions(ctx_free, L, R)
    fit = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    rows = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
                master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy(),
                **{k: e2.u64(v) for k, v in fit.items()})
    win, winR, cap = window_tables(wl)
    tabs = (win, winR, cap) + count_tables(win, winR, wl.n_layer) + value_bounds(wl, win)
    cells, cand, cand32, alg1 = generation_work(
        wl, label_problems(wl.labels, K), wl.roles, e2.u64(sol["T"]),
        sol["master"].cpu().numpy(), tabs, e2.u64(sol0["T"]))
    kern = cand + cand32
    dp_s = dp_ms / 1e3 / n_dp
    log(f"{name}: {elapsed * 1e3 / steps:.3f} ms per evaluation, DP kernel {dp_s * 1e3:.3f} ms")
    return {"devices": wl.n_dev, "layers": wl.n_layer, "population": P,
            "call": "e2_eval_population", "steps": steps,
            "ms_per_eval": elapsed * 1e3 / steps,
            "fitness_evals_per_s": P * steps / elapsed,
            "dp_cells_per_s": cells * steps / elapsed,
            "k_dp_avg_ms": dp_s * 1e3,
            "kernel_candidates_per_eval": kern,
            "kernel_candidates_per_s": kern * steps / elapsed,
            "alg1_candidates_per_eval": alg1,
            "frac": (cand * OPS_PER_CANDIDATE + cand32 * OPS_PER_CANDIDATE_NARROW) / dp_s
                    / INT_VALU_PEAK}, rows


def role_search(torch, dev, steps, warmup, name=None):
    """Time e2_search_roles (every cluster for prefill and each decode slot
    count, the QoS-feasible slot count, brute-force roles over the clusters
    with a decode rate) on a workload with its slot model (by default the
    1024-genome, 64-device one); count the Algorithm 1 cells of the feasible
    (cluster, role index) problems."""
    wl = workload.make(name or SEARCH_WORKLOAD)
    sm = workload.slot_model(wl)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    e2.e2_ctx_keep_scratch(ctx)
    L = torch.from_numpy(wl.labels).to(dev)
    fp = wl.fitness_params()
    out = e2.e2_search_roles(ctx, L, fp, wl.k_max, with_tables=True)
    for _ in range(warmup):
        e2.e2_search_roles(ctx, L, fp, wl.k_max, out=out)
    torch.cuda.synchronize()
    e2.e2_ctx_dp_timing(ctx, steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        e2.e2_search_roles(ctx, L, fp, wl.k_max, out=out)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_dp, dp_ms = e2.e2_ctx_dp_elapsed(ctx)
    e2.e2_ctx_dp_timing(ctx, 0)
    assert n_dp == steps, (n_dp, steps)
    T_all = e2.u64(out["T_all"])
    N = wl.n_layer
    cells = problems = 0
    for p, q, chain in label_problems(wl.labels, wl.k_max):
        m = len(chain)
        ok = int((T_all[p, q] != INF).sum())
        problems += ok
        cells += ok * m * (m * N - m * (m - 1) // 2)
    slots = out["slots"].cpu().numpy()
    # clusters with a decode rate (the ones the brute force enumerates)
    lam_max = 10**12 // wl.min_tps_milli if wl.min_tps_milli else INF
    free = ((T_all[:, :, 1:] != INF) & (e2.u64(out["Lambda_all"])[:, :, 1:] <= lam_max)).any(axis=2)
    free = free.sum(axis=1)
    log(f"role search on {wl.name}: {elapsed * 1e3 / steps:.3f} ms per call, DP kernel "
        f"{dp_ms / n_dp:.3f} ms; clusters with a decode rate: mean {free.mean():.2f}, "
        f"max {free.max()}")
    gen2 = ordered_search_generations(torch, dev, wl, sm, ctx, steps, warmup)
    klo, khi = workload.SPECS[wl.name]["K"]
    return {"workload": wl.name, "population": wl.population, "devices": wl.n_dev,
            "layers": N, "clusters_per_genome": f"{klo}-{khi}", "slot_model": sm,
            "call": "e2_search_roles", "steps": steps,
            "ms_per_call": elapsed * 1e3 / steps,
            "genomes_per_s": wl.population * steps / elapsed,
            "feasible_dp_problems_per_call": problems,
            "dp_cells_per_s": cells * steps / elapsed,
            "k_dp_avg_ms": dp_ms / n_dp,
            "decode_replicas_at_b_max": int((slots == sm["b_max"]).sum()),
            "clusters_with_a_decode_rate": {"mean": float(free.mean()), "max": int(free.max())},
            "genomes_not_searched": int((slots == 0xFF).all(axis=1).sum()),
            "two_chromosome_generation": gen2}


def ordered_search_generations(torch, dev, wl, sm, ctx, steps, warmup):
    """Algorithm 2's generation on the paper's two-chromosome genome (App. A):
    e2_search_roles_ordered (every replica for prefill and each decode slot
    count, the kept slot count, brute-force roles) scores the population,
    then e2_ga_step_ordered breeds the next one from those keys with the
    roles the search chose.  Timed over `steps` generations after `warmup`."""
    op = workload.ordered_population(wl)
    fp = wl.fitness_params()
    O0, S0 = (torch.from_numpy(x).to(dev) for x in (op.order, op.sizes))
    bufs = [(torch.empty_like(O0), torch.empty_like(S0), torch.empty((wl.population, wl.k_max),
                                                                     dtype=torch.uint8,
                                                                     device=dev))
            for _ in range(2)]
    res = e2.e2_search_roles_ordered(ctx, O0, S0, fp)

    def run(n):
        bufs[0][0].copy_(O0)
        bufs[0][1].copy_(S0)
        cur = 0
        for g in range(n):
            O, S, _ = bufs[cur]
            e2.e2_search_roles_ordered(ctx, O, S, fp, out=res)
            e2.e2_ga_step_ordered(ctx, O, S, res["roles"], res["w"], res["phase"],
                                  op.ga_params(wl, g), out=bufs[1 - cur])
            cur = 1 - cur
    run(warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log(f"two-chromosome search + GA on {wl.name}: {elapsed * 1e3 / steps:.3f} ms per generation")
    return {"genomes": "two_chromosome", "population": wl.population,
            "step": "e2_search_roles_ordered + e2_ga_step_ordered", "steps": steps,
            "ms_per_generation": elapsed * 1e3 / steps,
            "genomes_per_s": wl.population * steps / elapsed}


def _timed(torch, fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def _key_stats(w_a, ph_a, w_b, ph_b):
    """Genomes where the first method's (w, phase) is strictly better, equal,
    or worse than the second's."""
    a = list(zip(w_a.tolist(), ph_a.tolist()))
    b = list(zip(w_b.tolist(), ph_b.tolist()))
    return {"better": sum(x < y for x, y in zip(a, b)), "equal": sum(x == y for x, y in zip(a, b)),
            "worse": sum(x > y for x, y in zip(a, b))}


def ablations(torch, dev, steps, warmup):
    """The two ablations of Sec. 4.2 on the 1024-genome workload: the
    finishing-time objective against Algorithm 1's bottleneck (same genomes,
    roles and fitness), and the adapted-SplitWise role rule against the
    brute-force role search (same slot model and DP results)."""
    wl = workload.make(SEARCH_WORKLOAD)
    fp = wl.fitness_params()
    np_tok = wl.prompt_tokens()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    e2.e2_ctx_keep_scratch(ctx)
    bn = e2.e2_eval_population(ctx, L, R, fp, with_rates=False)
    ft = e2.e2_eval_population(ctx, L, R, fp, with_rates=False, objective="finish_time")
    ms_bn = _timed(torch, lambda: e2.e2_eval_population(ctx, L, R, fp, with_rates=False, out=bn),
                   steps, warmup)
    ms_ft = _timed(torch, lambda: e2.e2_eval_population(ctx, L, R, fp, with_rates=False, out=ft,
                                                       objective="finish_time"), steps, warmup)
    idle = e2.e2_solve_partitions(ctx, L, R, objective="idle")
    bnp = e2.e2_solve_partitions(ctx, L, R)
    ms_idle = _timed(torch, lambda: e2.e2_eval_population(ctx, L, R, fp, with_rates=False,
                                                         objective="idle"), steps, warmup)
    sm = workload.slot_model(wl)
    sctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    e2.e2_ctx_keep_scratch(sctx)
    se = e2.e2_search_roles(sctx, L, fp, wl.k_max)
    sw = e2.e2_search_roles(sctx, L, fp, wl.k_max, splitwise_np_tokens=np_tok)
    ms_sw = _timed(torch, lambda: e2.e2_search_roles(sctx, L, fp, wl.k_max, out=sw,
                                                    splitwise_np_tokens=np_tok),
                   steps, warmup)
    torch.cuda.synchronize()
    log(f"ablations on {wl.name}: eval {ms_bn:.3f} ms, finishing-time eval {ms_ft:.3f} ms, "
        f"SplitWise roles {ms_sw:.3f} ms, idle-device eval {ms_idle:.3f} ms")
    Ti, Tb = e2.u64(idle["T"]), e2.u64(bnp["T"])
    fin = Tb != INF
    return {"workload": wl.name, "population": wl.population, "steps": steps,
            "finish_time": {"call": "e2_eval_population_ft", "ms_per_call": ms_ft,
                            "bottleneck_ms_per_call": ms_bn,
                            "bottleneck_vs_finish_time": _key_stats(
                                e2.u64(bn["w"]), e2.u64(bn["phase"]), e2.u64(ft["w"]),
                                e2.u64(ft["phase"]))},
            "idle_devices": {"call": "e2_eval_population_idle", "ms_per_call": ms_idle,
                             "clusters_feasible": int((Ti != INF).sum()),
                             "clusters_feasible_algorithm_1": int(fin.sum()),
                             "clusters_lower_T": int((Ti[fin] < Tb[fin]).sum())},
            "splitwise": {"call": "e2_assign_roles_splitwise", "ms_per_call": ms_sw,
                          "search_vs_splitwise": _key_stats(
                              e2.u64(se["w"]), e2.u64(se["phase"]), e2.u64(sw["w"]),
                              e2.u64(sw["phase"]))}}


def measure(torch, ctx, stream, bufs, init, step, count, warmup, steps):
    """Time `steps` generations (after `warmup` untimed ones) from the
    initial population `init`, ping-ponging between the two buffer sets;
    then replay the same generations outside the timed region and count
    their work.  The library records HIP events around its DP kernel on the
    call's stream, one pair per evaluation."""
    def reset():
        for dst, src in zip(bufs[0], init):
            dst.copy_(src)
        torch.cuda.synchronize()

    def run(n):
        cur = 0
        for g in range(n):
            step(g, cur)
            cur = 1 - cur

    reset()
    run(warmup)
    torch.cuda.synchronize()
    reset()
    # the timed region holds the generations and the library's event pair
    # around each DP launch, nothing else (an event record costs the stream
    # a few microseconds)
    e2.e2_ctx_dp_timing(ctx, steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_dp, dp_ms = e2.e2_ctx_dp_elapsed(ctx)
    e2.e2_ctx_dp_timing(ctx, 0)
    assert n_dp == steps, (n_dp, steps)
    log(f"timed {steps} steps: {elapsed * 1e3:.2f} ms, {elapsed * 1e3 / steps:.3f} ms per "
        f"generation; DP kernel {dp_ms / n_dp:.3f} ms avg")
    cells = cand = cand32 = alg1 = 0
    pop = tuple(x.clone() for x in init)
    for g in range(steps):
        (c1, c2, c3, c4), pop = count(g, pop)
        cells += c1
        cand += c2
        cand32 += c3
        alg1 += c4
    return dict(elapsed=elapsed, dp_s=dp_ms / 1e3, step_ms=elapsed * 1e3 / steps, cells=cells,
                cand=cand, cand32=cand32, alg1=alg1)


def roofline(t, steps, prof):
    """The DP kernel against the int32 VALU peak.  frac counts the j-candidates
    the kernel itself evaluates (3 ops each on u32 or fp64 keys, 8 on u64
    keys) per second of its launches.  From the committed rocprofv3 profile
    of the same workload and sources (when there is one): HBM traffic, the
    VALU issue fraction (every issued wave instruction as 64 lane-ops), the
    share of those lane-ops that are candidate ops, VALUBusy, VALU lane
    utilisation, SALUBusy, LDS activity and LDS bank conflicts."""
    ops = t["cand"] * OPS_PER_CANDIDATE + t["cand32"] * OPS_PER_CANDIDATE_NARROW
    achieved = ops / t["dp_s"]
    out = {"bound": "alu", "kernel": "k_dp",
           "achieved": achieved / 1e12, "peak": INT_VALU_PEAK / 1e12,
           "unit": "TOP/s (int32 VALU)", "frac": achieved / INT_VALU_PEAK,
           "frac_counts": "j-candidates the kernel evaluates (banded decomposition), "
                          "3 VALU ops each",
           "traffic": prof.get("k_dp_hbm_bytes_per_launch") if prof else None,
           "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, "
                           "copy-calibrated)",
           "avg_launch_ms": t["dp_s"] * 1e3 / steps,
           "generation_ms": t["step_ms"]}
    if prof and prof.get("sq_insts_valu_per_launch"):
        us = prof["k_dp_avg_us"]
        valu_lane_ops = prof["sq_insts_valu_per_launch"] * 64
        out["profile"] = {
            "valu_issue_frac": valu_lane_ops / (us * 1e-6 * INT_VALU_PEAK),
            "candidate_share_of_valu_lane_ops": (ops / steps) / valu_lane_ops,
            "valu_busy_pct": prof.get("valu_busy_pct"),
            "valu_utilization_pct": prof.get("valu_utilization_pct"),
            "salu_busy_pct": prof.get("salu_busy_pct"),
            "lds_active_pct": prof.get("lds_active_pct"),
            "lds_bank_conflict_pct": prof.get("lds_bank_conflict_pct"),
            "wait_any_share_of_wave_cycles": prof.get("wait_any_share"),
            "hbm_read_bytes_per_launch": prof.get("k_dp_hbm_read_bytes"),
            "hbm_write_bytes_per_launch": prof.get("k_dp_hbm_write_bytes"),
            "k_dp_avg_us_profiled": us,
            "source": prof.get("summary")}
    return out


def algorithmic(t, steps):
    """Algorithm 1's own work next to the kernel's: its memory-feasible
    j-candidates (one full table per master) per step, their rate at 3 ops
    each over the kernel's time as a fraction of the peak (above 1 means the
    decomposition skips more work than the hardware could do), and the
    reduction factor."""
    kern = t["cand"] + t["cand32"]
    return {"alg1_candidates_per_step": t["alg1"] / steps,
            "kernel_candidates_per_step": kern / steps,
            "algorithmic_reduction": t["alg1"] / kern if kern else None,
            "alg1_equivalent_frac_of_peak":
                t["alg1"] * OPS_PER_CANDIDATE_NARROW / t["dp_s"] / INT_VALU_PEAK}


LIB_SOURCES = ("e2_internal.h", "e2_kernels.hip")  # the kernels and their launch configuration


def code_text(text: str) -> str:
    """C++ source without its comments and blank space: what the compiler
    sees, so that a comment edit keeps a profile current."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash() -> str:
    """Hash of the library sources that decide what the DP kernel does and
    how it is launched (their code, comments and layout aside); the host
    API's argument checks and allocations are not part of it."""
    import hashlib
    h = hashlib.sha256()
    for f in LIB_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_03770_amd", "csrc", f)) as fh:
            h.update(code_text(fh.read()).encode())
    return h.hexdigest()[:16]


def profiled(workload_name, genomes="labels"):
    """The committed rocprofv3 summary (profiles/k_dp_*.json) of this workload
    and genome kind, or None when none exists or the kernel sources have
    changed since it was taken."""
    import glob
    for f in sorted(glob.glob(os.path.join(ROOT, "profiles", "k_dp_*.json"))):
        with open(f) as fh:
            meta = json.load(fh)
        if (meta.get("workload") == workload_name and meta.get("genomes", "labels") == genomes
                and meta.get("sources_sha256_16") == source_hash()):
            meta["summary"] = os.path.relpath(f[:-5] + ".md", ROOT)
            return meta
    return None


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


def host_cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


CPU_CONFIG_GENOMES = 1024  # oracle sample per smaller workload (its first genomes)


def cpu_baseline(wl, seconds, gpu0=None, cfg_rows=None):
    """The oracle, as it is (single-threaded C, one host core), on the first S
    genomes of the generation-0 population, S sized from a short probe to
    take about `seconds`.  Its rows are then compared with the GPU's
    evaluation of the same genomes (gpu0: T, Lambda, master, layers, w,
    phase, S_P, S_D of generation 0).  With cfg_rows (the GPU's rows of the
    smaller workloads' populations), the oracle also evaluates the first
    CPU_CONFIG_GENOMES genomes of each, timed, and compares them row by row."""
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
    out = {"value": cells / dt, "unit": "Algorithm-1-equivalent DP cells/s", "cores": 1,
           "kind": "oracle",
           "sample": f"first {S} of {wl.population} genomes of generation 0 of the "
                     f"256-device workload, full evaluation (quantise, Algorithm 1 per "
                     f"cluster, Eq. 3-5), not the generation's GA step",
           "fitness_evals_per_s": S / dt, "seconds": dt,
           "host_cores": os.cpu_count(), "host_cpu_model": host_cpu_model()}
    if gpu0 is not None:
        keys = ("T", "Lambda", "master", "layers", "w", "phase", "s_p", "s_d")
        same = np.ones(S, dtype=bool)
        for k in keys:
            same &= np.asarray(gpu0[k][:S] == sol[k]).reshape(S, -1).all(axis=1)
        out["gpu_rows_equal"] = int(same.sum())
        out["gpu_rows_compared"] = S
    log(f"cpu oracle: {S} genomes in {dt:.2f} s"
        + (f"; {out['gpu_rows_equal']} of {S} equal the GPU's rows" if gpu0 is not None else ""))
    if cfg_rows:
        out["configs"] = {}
        for name, rows in cfg_rows.items():
            cw = workload.make(name)
            n = min(cw.population, CPU_CONFIG_GENOMES)
            t0 = time.perf_counter()
            ref = oracle.eval_population(cw.subset(np.arange(n)))
            cdt = time.perf_counter() - t0
            same = np.ones(n, dtype=bool)
            for k in ("T", "Lambda", "master", "layers", "w", "phase", "s_p", "s_d"):
                same &= np.asarray(rows[k][:n] == ref[k]).reshape(n, -1).all(axis=1)
            out["configs"][name] = {"genomes": n, "population": cw.population, "seconds": cdt,
                                    "ms_per_genome": cdt * 1e3 / n, "cores": 1,
                                    "gpu_rows_equal": int(same.sum()), "gpu_rows_compared": n}
            log(f"cpu oracle on {name}: {n} genomes in {cdt:.2f} s; {int(same.sum())} of {n} "
                f"equal the GPU's rows")
    return out


if __name__ == "__main__":
    main()
