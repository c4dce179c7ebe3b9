"""The bench's work accounting (host logic, no GPU).

bench.generation_work counts, with vectorised prefix tables, the useful
j-candidates the DP kernel evaluates, split by key width; the roofline's
`achieved` is built from it.  Here the same counts come from a direct walk
over every row, cell and window of the banded decomposition, and the key
width from a direct scan of every stage that fits memory.
"""
import dataclasses

import numpy as np
import pytest

import bench
import oracle
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

INF = bench.INF


def _windows(wl):
    """Smallest fitting start per stage end, by brute force over starts."""
    M, N = wl.n_dev, wl.n_layer
    b = [int(x) for x in wl.layer_bytes]
    win = np.full((2, M, N), 255, dtype=np.int64)
    winR = np.full((M, N), 255, dtype=np.int64)
    for d in range(M):
        mem = int(wl.mem_bytes[d])
        for f in range(2):
            extra = int(wl.head_bytes) if f else 0
            for i in range(N):
                for j in range(i + 1):
                    if sum(b[j:i + 1]) + extra <= mem:
                        win[f, d, i] = j
                        break
        for x in range(N):          # reversed blocks y..x = blocks N-1-x..N-1-y
            for y in range(x + 1):
                if sum(b[N - 1 - x:N - y]) <= mem:
                    winR[d, x] = y
                    break
    return win, winR


def _free_optima(orc, wl, labels=None, order=None, sizes=None, roles=None):
    """Optima without a master: the oracle on the same genomes with no head
    time and no head bytes."""
    wf = dataclasses.replace(wl, head_flops=np.zeros(2, dtype=np.uint64), head_bytes=0)
    if order is not None:
        return orc.eval_population_ordered(wf, order, sizes, roles)["T"]
    return orc.eval_population(wf)["T"]


def _direct(wl, problems, roles, T, master, T0):
    N = wl.n_layer
    win, winR = _windows(wl)
    t, h, tau = e2.e2_quantise(wl.problem_arrays())
    cap = np.zeros((2, wl.n_dev), dtype=np.int64)
    for f in range(2):
        for d in range(wl.n_dev):
            ok = win[f, d] != 255
            cap[f, d] = max((i - win[f, d, i] + 1 for i in range(N) if ok[i]), default=0)

    def stage_max(r, d):
        best = 0
        for f in range(2):
            for i in range(N):
                j = int(win[f, d, i])
                if j != 255:
                    best = max(best, int(t[r, d, j:i + 1].sum()) + (int(h[r, d]) if f else 0))
        return best

    def cnt(w, kmin, lo, hi):
        return sum(max(0, i - max(int(w[i]), kmin) + 1) for i in range(lo, hi + 1) if w[i] != 255)

    c64 = c32 = 0
    for p, q, ch in problems:
        m = len(ch)
        c0, cH = cap[0][ch], cap[1][ch]
        if not (m <= N and c0.sum() >= N and c0.min() >= 1 and cH.max() >= 1):
            continue
        r = int(roles[p, q] != 0)
        pre = np.r_[0, np.cumsum(c0)]
        tot = pre[m]
        flo = {k: max(k - 1, N - 1 - (tot - pre[k])) for k in range(1, m + 1)}
        fhi = {k: min(N - 1 - (m - k), pre[k] - 1) for k in range(1, m + 1)}
        pool = sum(max(0, fhi[k] - flo[k] + 1) for k in range(1, m))
        mu = int(np.nonzero(ch == master[p, q])[0][0]) + 1 if T[p, q] != INF else 0
        c = 0
        # every band total is at most (m - 1)(N - m + 1)
        assert pool <= (m - 1) * (N - m + 1)
        banded = m <= 64 and pool <= bench.pool_cells(N)
        if banded:
            for tt in range(2, m):                           # reversed rows
                kd = m + 1 - tt
                gl = max(kd - 1, N - (tot - pre[kd - 1]))
                gh = min(pre[kd - 1], N - (m - kd + 1))
                if gh >= gl:
                    c += cnt(winR[ch[kd - 1]], max(tt - 1, N - 1 - gh - c0[kd - 1] + 1),
                             N - 1 - gh, N - 1 - gl)
            if m >= 2:                                       # the full reversed table's last cell
                c += cnt(winR[ch[0]], max(m - 1, N - 1 - c0[0] + 1), N - 1, N - 1)
            # masters in ascending position with the forward row after each,
            # up to the first master whose optimum is the optimum without one
            t0 = int(T0[p, q])
            last = 0 if t0 == INF else (mu if int(T[p, q]) == t0 else m)
            # a stop in a paired pass (combine and forward row of one master
            # in one pass, bands of at most 32 cells): the forward row of the
            # stopping master is evaluated too, and the combine's row stands
            # for the chosen master's first row
            paired_stop = (last == mu and 2 <= mu <= m - 1 and
                           1 <= fhi[mu] - flo[mu] + 1 <= bench.PAIR_MAX_CELLS)
            for mm in range(1, last + 1):
                if mm >= 2 and cH[mm - 1] > 0:               # combine of master mm
                    c += cnt(win[1][ch[mm - 1]], max(mm - 1, flo[mm] - cH[mm - 1] + 1),
                             flo[mm], fhi[mm])
                if (2 <= mm < last or (paired_stop and mm == last)) and mm < m:  # forward row mm
                    c += cnt(win[0][ch[mm - 1]], max(mm - 1, flo[mm] - c0[mm - 1] + 1),
                             flo[mm], fhi[mm])
            if mu:                                           # chosen master's rows
                for k in range(max(mu + int(paired_stop), 2), m):
                    f = int(k == mu)
                    cp = cH[k - 1] if f else c0[k - 1]
                    c += cnt(win[f][ch[k - 1]], max(k - 1, flo[k] - cp + 1), flo[k], fhi[k])
                if m >= 2:
                    f = int(mu == m)
                    cp = cH[m - 1] if f else c0[m - 1]
                    c += cnt(win[f][ch[m - 1]], max(m - 1, N - cp), N - 1, N - 1)
        else:                                                # one table per master
            for mm in list(range(1, m + 1)) + ([mu] if mu else []):
                for k in range(2, m + 1):
                    c += cnt(win[int(k == mm)][ch[k - 1]], k - 1, k - 1, N - 1)
        links = [int(tau[r, ch[k - 1], ch[k]]) for k in range(1, m)]
        links = [x for x in links if x != INF]
        bound = max([stage_max(r, d) for d in ch] + links)
        bound_tot = max([int(t[r, d].sum(dtype=np.uint64)) + int(h[r, d]) for d in ch] + links)
        narrow = bound <= bench.U32_MAX_VALUE or bound_tot < bench.F64_LIMIT
        if banded and not narrow:      # the reference path: recount as full tables
            c = 0
            for mm in list(range(1, m + 1)) + ([mu] if mu else []):
                for k in range(2, m + 1):
                    c += cnt(win[int(k == mm)][ch[k - 1]], k - 1, k - 1, N - 1)
            banded = False
        if banded:
            c32 += c
        else:
            c64 += c
    return c64, c32


def _alg1_direct(wl, problems):
    """Memory-feasible split points of every cell of every master's table
    (rows 2..m, cells k-1..N-1, starts j >= k-1) over the problems that pass
    the pre-check (m <= N, every device holds a block, total capacity >= N,
    some device holds a block with the head)."""
    N = wl.n_layer
    b = np.concatenate([[0], np.cumsum([int(x) for x in wl.layer_bytes])])
    HB = int(wl.head_bytes)

    def cap(d, extra):
        best = 0
        for i in range(N):
            for j in range(i + 1):
                if b[i + 1] - b[j] + extra <= int(wl.mem_bytes[d]):
                    best = max(best, i - j + 1)
                    break
        return best
    c0 = {d: cap(d, 0) for d in range(wl.n_dev)}
    cH = {d: cap(d, HB) for d in range(wl.n_dev)}
    total = 0
    for _, _, chain in problems:
        m = len(chain)
        if not (m <= N and min(c0[d] for d in chain) >= 1 and
                sum(c0[d] for d in chain) >= N and max(cH[d] for d in chain) >= 1):
            continue
        for mu in range(1, m + 1):
            for k in range(2, m + 1):
                mem = int(wl.mem_bytes[chain[k - 1]])
                extra = HB if k == mu else 0
                for i in range(k - 1, N):
                    total += sum(1 for j in range(k - 1, i + 1) if b[i + 1] - b[j] + extra <= mem)
    return total


@pytest.mark.parametrize("name,P", [("c1_tiny_12dev_32L", 16), ("c2_32dev_48L", 24),
                                    ("c5_256dev_126L_ga", 6)])
def test_candidate_counts_match_a_direct_walk(orc, name, P):
    wl = workload.make(name, population=P)
    sol = oracle.eval_population(wl)
    T0 = _free_optima(orc, wl)
    win, winR, cap = bench.window_tables(wl)
    tabs = (win, winR, cap) + bench.count_tables(win, winR, wl.n_layer) + bench.value_bounds(wl, win)
    probs = bench.label_problems(wl.labels, wl.k_max)
    cells, c64, c32, alg1 = bench.generation_work(wl, probs, wl.roles, sol["T"], sol["master"],
                                                  tabs, T0)
    assert (c64, c32) == _direct(wl, probs, wl.roles, sol["T"], sol["master"], T0)
    assert c64 + c32 > 0
    assert c32 > 0                   # u32 / fp64 keys
    # Algorithm 1's own candidates (the direct walk), more than the kernel's
    assert alg1 == _alg1_direct(wl, probs)
    assert alg1 > c64 + c32
    # both ends of the master sweep occur: optima equal to T0 and above it
    fin = sol["T"] != INF
    assert (sol["T"][fin] == T0[fin]).any()


def test_reference_path_counts(orc):
    """Chains with more than 64 devices take one full table per master (u64 keys)."""
    wl = workload.random_small(3, M=70, N=80, P=1, k_max=1, mem_lo_layers=3, mem_hi_layers=30)
    sol = oracle.eval_population(wl)
    T0 = _free_optima(orc, wl)
    win, winR, cap = bench.window_tables(wl)
    tabs = (win, winR, cap) + bench.count_tables(win, winR, wl.n_layer) + bench.value_bounds(wl, win)
    probs = bench.label_problems(wl.labels, wl.k_max)
    _, c64, c32, _ = bench.generation_work(wl, probs, wl.roles, sol["T"], sol["master"], tabs, T0)
    assert (c64, c32) == _direct(wl, probs, wl.roles, sol["T"], sol["master"], T0)
    assert c64 > 0 and c32 == 0   # the reference path has u64 keys only


@pytest.mark.parametrize("name,P", [("c2_32dev_48L", 24), ("c5_256dev_126L_ga", 6)])
def test_candidate_counts_of_ordered_genomes(orc, name, P):
    """Two-chromosome genomes: the problems are the replicas' ordering runs
    (checked against the oracle's replica ranges) and the counts match the
    direct walk over those chains."""
    wl = workload.make(name, population=P)
    op = workload.ordered_population(wl)
    probs = bench.ordered_problems(op.order, op.sizes)
    want = []
    for p in range(P):
        for q in range(wl.k_max):
            lo, hi = orc.replica_range(op.sizes[p], q, wl.n_dev)
            if hi > lo:
                want.append((p, q, list(op.order[p, lo:hi])))
    assert [(p, q, list(c)) for p, q, c in probs] == want
    sol = oracle.eval_population_ordered(wl, op.order, op.sizes, op.roles)
    T0 = _free_optima(orc, wl, order=op.order, sizes=op.sizes, roles=op.roles)
    win, winR, cap = bench.window_tables(wl)
    tabs = (win, winR, cap) + bench.count_tables(win, winR, wl.n_layer) + bench.value_bounds(wl, win)
    cells, c64, c32, alg1 = bench.generation_work(wl, probs, op.roles, sol["T"], sol["master"],
                                                  tabs, T0)
    assert alg1 == _alg1_direct(wl, probs)
    assert (c64, c32) == _direct(wl, probs, op.roles, sol["T"], sol["master"], T0)
    assert c64 + c32 > 0 and cells > 0


def test_window_tables_match_brute_force():
    wl = workload.random_small(11, M=9, N=21, P=1, k_max=2, mem_lo_layers=1, mem_hi_layers=12)
    win, winR, _ = bench.window_tables(wl)
    w2, wR2 = _windows(wl)
    assert (win == w2).all() and (winR == wR2).all()


def test_source_hash_ignores_comments_and_layout():
    """The profile records are keyed by the code the compiler sees."""
    a = "int f(int x) { return x + 1; } // one\n/* two\n lines */ int g;"
    b = "int f(int x)  {\n  return x + 1;\n}\n\nint g;"
    assert bench.code_text(a) == bench.code_text(b)
    assert bench.code_text(a) != bench.code_text(a.replace("x + 1", "x + 2"))
    assert len(bench.source_hash()) == 16
