"""Pins for the oracle's idle-device relaxation (reading R2: a device may
hold no block and then sits out; links join consecutive participants; the
master always takes part, with its head).

Checked against exhaustive enumeration (brute.Chain.solve_idle_relaxed,
which never runs a recurrence), by re-evaluating the returned partition,
by the smallest optimal master, and against the invariants the relaxation
exists for: adding a device never worsens the optimum, the relaxed optimum
never exceeds Algorithm 1's, and chains longer than the model still fit.
"""
import numpy as np
import pytest

from oracle import brute
from paper_2606_03770_amd import workload

INF = brute.INF


def rand_idle_chain(rng, m, N):
    tk = rng.integers(1, 20, size=(m, N)).astype(np.uint64)
    hk = rng.integers(0, 15, size=m).astype(np.uint64)
    full = rng.integers(0, 25, size=(m, m)).astype(np.uint64)
    full = np.minimum(full, full.T)                 # symmetric links
    if rng.uniform() < 0.3:
        a, b = rng.choice(m, 2, replace=True)
        full[a, b] = full[b, a] = np.uint64(INF)
    np.fill_diagonal(full, 0)
    W = rng.integers(1, 5, size=N).astype(np.uint64)
    HB = int(rng.integers(0, 4))
    mem = rng.integers(2, 25, size=m).astype(np.uint64)
    return tk, hk, full, mem, W, HB


def _brute(tk, hk, full, mem, W, HB):
    m = len(tk)
    tl = np.array([0] + [full[k - 1, k] for k in range(1, m)], np.uint64)
    c = brute.Chain(tk, hk, tl, mem, W, HB)
    c.set_links(full)
    return c


def test_idle_matches_enumeration(orc):
    rng = np.random.default_rng(2718)
    feasible = 0
    for _ in range(400):
        m, N = int(rng.integers(1, 6)), int(rng.integers(1, 7))
        args = rand_idle_chain(rng, m, N)
        T, L, mu, sizes = orc.dp_idle(*args)
        c = _brute(*args)
        assert T == c.solve_idle_relaxed(), (m, N, args)
        if T == INF:
            assert mu == 0 and sizes == [0] * m
            continue
        feasible += 1
        # the returned partition is valid and optimal, its master the smallest optimal one
        assert sum(sizes) == N and min(sizes) >= 0
        assert c.idle_bottleneck(sizes, mu) == T
        assert all(c.solve_idle_relaxed(only_mu=u) > T for u in range(1, mu))
        # Lambda: the participants' stage times (+ head) and their links
        used = [k for k in range(m) if sizes[k] > 0 or k + 1 == mu]
        start = np.r_[0, np.cumsum(sizes)]
        lam = sum(int(args[0][k][start[k]:start[k + 1]].sum()) for k in used)
        lam += int(args[1][mu - 1])
        lam += sum(int(args[2][a, b]) for a, b in zip(used, used[1:]))
        assert L == lam
    assert feasible > 100


def test_more_devices_than_blocks(orc):
    """m > N: Algorithm 1 has no answer (R1), the relaxation seats N of them."""
    rng = np.random.default_rng(5)
    for _ in range(60):
        m, N = int(rng.integers(4, 8)), int(rng.integers(1, 4))
        tk, hk, full, mem, W, HB = rand_idle_chain(rng, m, N)
        mem[:] = 100
        full[full == INF] = 3
        T, L, mu, sizes = orc.dp_idle(tk, hk, full, mem, W, HB)
        assert T != INF and T == _brute(tk, hk, full, mem, W, HB).solve_idle_relaxed()
        assert sum(1 for k in range(m) if sizes[k] > 0) <= N
        tl = np.array([0] + [full[k - 1, k] for k in range(1, m)], np.uint64)
        assert orc.dp_pipe(tk, hk, tl, mem, W, HB)[0] == INF


def test_adding_a_device_never_worsens(orc):
    rng = np.random.default_rng(99)
    for _ in range(200):
        m, N = int(rng.integers(1, 6)), int(rng.integers(1, 8))
        tk, hk, full, mem, W, HB = rand_idle_chain(rng, m + 1, N)
        drop = int(rng.integers(0, m + 1))
        keep = [k for k in range(m + 1) if k != drop]
        small = orc.dp_idle(tk[keep], hk[keep], full[np.ix_(keep, keep)], mem[keep], W, HB)[0]
        big = orc.dp_idle(tk, hk, full, mem, W, HB)[0]
        assert big <= small


def test_relaxed_optimum_never_exceeds_algorithm_1(orc):
    rng = np.random.default_rng(12)
    for _ in range(200):
        m, N = int(rng.integers(1, 6)), int(rng.integers(1, 10))
        tk, hk, full, mem, W, HB = rand_idle_chain(rng, m, N)
        tl = np.array([0] + [full[k - 1, k] for k in range(1, m)], np.uint64)
        assert orc.dp_idle(tk, hk, full, mem, W, HB)[0] <= orc.dp_pipe(tk, hk, tl, mem, W, HB)[0]


def test_population_solve_idle_uses_each_clusters_chain(orc):
    wl = workload.random_small(33, M=10, N=6, P=5, k_max=2, mem_hi_layers=10, zero_bw_frac=0.1)
    got = orc.eval_population_idle(wl)
    t, h, tau = orc.quantise(**wl.problem_arrays())
    for p in range(wl.population):
        for q in range(wl.k_max):
            ch = np.nonzero(wl.labels[p] == q)[0]
            if len(ch) == 0:
                assert got["T"][p, q] == INF
                continue
            r = int(wl.roles[p, q] != 0)
            T, L, mu, sizes = orc.dp_idle(t[r][ch], h[r][ch], tau[r][np.ix_(ch, ch)],
                                          wl.mem_bytes[ch], wl.layer_bytes, wl.head_bytes)
            assert (int(got["T"][p, q]), int(got["Lambda"][p, q])) == (T, L)
            if T != INF:
                assert got["master"][p, q] == ch[mu - 1]
                assert list(got["layers"][p][ch]) == sizes
    fit = orc.fitness(got["T"], got["Lambda"], wl.roles, **wl.fitness_params())
    assert (fit["w"] == got["w"]).all()
