"""Pins for the oracle's population solve (cluster extraction + Algorithm 1
per replica + Eq. 3-5 per individual)."""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2606_03770_amd import workload

INF = oracle.INF


def test_population_solve_matches_brute_force_per_cluster(orc):
    """Every (individual, cluster) result equals enumeration on the chain of
    that cluster's devices in ascending id order."""
    for seed in range(4):
        wl = workload.random_small(100 + seed, M=9, N=7, P=6, k_max=3, mem_hi_layers=8,
                                   zero_bw_frac=0.1)
        t, h, tau = oracle.quantise(**wl.problem_arrays())
        sol = oracle.solve((t, h, tau), wl.mem_bytes, wl.layer_bytes, wl.head_bytes,
                           wl.labels, wl.roles, wl.k_max)
        for p in range(wl.population):
            for q in range(wl.k_max):
                chain = [d for d in range(wl.n_dev) if wl.labels[p, d] == q]
                if not chain:
                    assert sol["T"][p, q] == INF and sol["master"][p, q] == -1
                    continue
                r = int(wl.roles[p, q] != 0)
                tl = [0] + [int(tau[r, chain[k - 1], chain[k]]) for k in range(1, len(chain))]
                bT, bL, bmu, bs = brute.Chain(t[r, chain], h[r, chain], tl,
                                              wl.mem_bytes[chain], wl.layer_bytes,
                                              wl.head_bytes).solve()
                assert int(sol["T"][p, q]) == bT
                if bT == INF:
                    assert sol["master"][p, q] == -1 and int(sol["Lambda"][p, q]) == INF
                    assert all(sol["layers"][p, d] == 0 for d in chain)
                else:
                    assert int(sol["Lambda"][p, q]) == bL
                    assert sol["master"][p, q] == chain[bmu - 1]
                    assert [int(sol["layers"][p, d]) for d in chain] == list(bs)


def test_unassigned_labels_are_ignored(orc):
    wl = workload.random_small(7, M=8, N=6, P=4, k_max=2, mem_hi_layers=10)
    labels = wl.labels.copy()
    labels[:, 0] = 200  # device 0 belongs to no cluster
    labels[1, :] = 255
    t = oracle.quantise(**wl.problem_arrays())
    sol = oracle.solve(t, wl.mem_bytes, wl.layer_bytes, wl.head_bytes, labels, wl.roles, 2)
    assert (sol["layers"][:, 0] == 0).all()
    assert (sol["T"][1] == INF).all() and (sol["layers"][1] == 0).all()
    labels2 = labels.copy()
    labels2[:, 0] = 2  # another out-of-range id: same result
    sol2 = oracle.solve(t, wl.mem_bytes, wl.layer_bytes, wl.head_bytes, labels2, wl.roles, 2)
    for k in ("T", "Lambda", "master", "layers"):
        assert (sol[k] == sol2[k]).all()


@pytest.mark.parametrize("name", ["c1_tiny_12dev_32L", "c2_32dev_48L"])
def test_named_workload_structure(orc, name):
    """Feasible clusters place all N blocks, >= 1 per device, master in the
    chain, T <= Lambda; every individual's w is INF or derived from finite S."""
    wl = workload.make(name, population=16 if name != "c1_tiny_12dev_32L" else None)
    sol = oracle.eval_population(wl)
    n_feasible = 0
    for p in range(wl.population):
        for q in range(wl.k_max):
            chain = [d for d in range(wl.n_dev) if wl.labels[p, d] == q]
            if sol["T"][p, q] == INF:
                continue
            n_feasible += 1
            blocks = [int(sol["layers"][p, d]) for d in chain]
            assert sum(blocks) == wl.n_layer and min(blocks) >= 1
            assert int(sol["master"][p, q]) in chain
            assert int(sol["T"][p, q]) <= int(sol["Lambda"][p, q])
        if sol["w"][p] != INF:
            assert sol["s_p"][p] != INF and sol["s_d"][p] != INF
    assert n_feasible > 0


def test_a_head_never_lowers_the_optimum(orc):
    """A head only adds time to the master's stage and bytes to its memory
    test, so every cluster's optimum is at least its optimum with no head
    (zero head time and bytes, where every master ties), and the two are
    equal in a cluster exactly when some master reaches that bound.  Both
    cases occur here; brute force confirms the head-free optimum on small
    clusters."""
    big = 0
    for seed in range(3):
        wl = workload.random_small(600 + seed, M=40, N=60, P=30, k_max=5, mem_lo_layers=2,
                                   mem_hi_layers=20)
        wl = dataclasses.replace(wl, head_flops=np.array([4 * 10**11] * 2, np.uint64),
                                 head_bytes=2 * 10**8)
        free = dataclasses.replace(wl, head_flops=np.zeros(2, np.uint64), head_bytes=0)
        T = orc.eval_population(wl)["T"]
        T0 = orc.eval_population(free)["T"]
        assert (T >= T0).all()
        assert (T[T0 == INF] == INF).all()           # no partition at all
        fin = T != INF
        big += int((T[fin] > T0[fin]).sum())
        assert (T[fin] == T0[fin]).any()
    assert big > 0
    # the head-free optimum is the optimum over partitions without a master
    wl = workload.random_small(9, M=7, N=9, P=4, k_max=2, mem_lo_layers=1, mem_hi_layers=5)
    free = dataclasses.replace(wl, head_flops=np.zeros(2, np.uint64), head_bytes=0)
    T0 = orc.eval_population(free)["T"]
    t, h, tau = orc.quantise(**free.problem_arrays())
    for p in range(wl.population):
        for q in range(wl.k_max):
            ch = np.nonzero(wl.labels[p] == q)[0]
            if len(ch) == 0:
                continue
            r = int(wl.roles[p, q] != 0)
            tl = np.array([0] + [tau[r, ch[k - 1], ch[k]] for k in range(1, len(ch))], np.uint64)
            c = brute.Chain(t[r][ch], h[r][ch], tl, free.mem_bytes[ch], free.layer_bytes, 0)
            assert int(T0[p, q]) == c.solve()[0]
