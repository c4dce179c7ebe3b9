"""Pins for the oracle's population solve (cluster extraction + Algorithm 1
per replica + Eq. 3-5 per individual)."""
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
