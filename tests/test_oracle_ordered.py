"""Pins for the oracle's two-chromosome genomes (the paper's App. A gene).

Replica extraction is checked against the paper's own gene example and
against brute force on chains in ordering order; the ordering crossover
against hand-worked children and the properties the repair must restore;
grouping regrowth and whole generations against the invariants a valid
gene must satisfy and the mutation shares App. A states.
"""
import json
import os

import numpy as np
import pytest

from oracle import brute
from paper_2606_03770_amd import workload

INF = brute.INF
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_paper_gene_example(orc):
    """App. A: [(0,1,2,3,4,5), (3,1,2)] places nodes 0-2 in the first
    replica, node 3 in the second and nodes 4, 5 in the third."""
    ex = json.load(open(os.path.join(GOLDEN, "paper_values.json")))["two_chromosome_gene"]
    order = np.array(ex["ordering"], dtype=np.uint8)
    sizes = np.array(ex["grouping"] + [0, 0], dtype=np.uint16)   # k_max = 5
    got = []
    for r in range(len(sizes)):
        lo, hi = orc.replica_range(sizes, r, len(order))
        if hi > lo:
            got.append(sorted(int(x) for x in order[lo:hi]))
    assert got == ex["replicas"]


@pytest.mark.parametrize("a,b,c,child", [
    # worked by hand: prefix of a, then b's part with its repeats replaced
    # by b's first-part nodes missing from a's prefix, in b's order
    ((0, 1, 2, 3, 4, 5), (5, 4, 3, 2, 1, 0), 2, (0, 1, 3, 2, 5, 4)),
    ((0, 1, 2, 3, 4, 5), (5, 4, 3, 2, 1, 0), 5, (0, 1, 2, 3, 4, 5)),
    ((0, 1, 2, 3, 4, 5), (5, 4, 3, 2, 1, 0), 1, (0, 4, 3, 2, 1, 5)),
    ((3, 0, 4, 1, 2), (1, 2, 3, 4, 0), 2, (3, 0, 1, 4, 2)),
    ((2, 0, 1), (2, 0, 1), 1, (2, 0, 1)),
])
def test_order_crossover_worked_examples(orc, a, b, c, child):
    assert tuple(orc.order_crossover(a, b, c)) == child


def test_order_crossover_restores_a_permutation(orc):
    rng = np.random.default_rng(7)
    for _ in range(400):
        M = int(rng.integers(2, 60))
        a, b = rng.permutation(M), rng.permutation(M)
        c = int(rng.integers(1, M))
        ch = orc.order_crossover(a, b, c)
        assert sorted(ch) == list(range(M))                 # each node once
        assert (ch[:c] == a[:c]).all()                       # a's prefix kept
        keep = ~np.isin(b[c:], a[:c])
        assert (ch[c:][keep] == b[c:][keep]).all()           # b's new nodes kept in place
        # the filled holes hold b's first-part nodes missing from a's prefix, in b's order
        fill = [x for x in b[:c] if x not in set(a[:c])]
        assert list(ch[c:][~keep]) == fill


def test_regrow_invariants(orc):
    rng = np.random.default_rng(11)
    for it in range(300):
        M = int(rng.integers(1, 80))
        k_max = int(rng.integers(1, 20))
        mx = int(rng.integers(1, 12))
        sizes = np.zeros(k_max, np.uint16)
        # a valid grouping to start from
        left, r = M, 0
        while left > 0:
            s = left if r == k_max - 1 else min(left, int(rng.integers(1, 9)))
            sizes[r] = s
            left -= s
            r += 1
        roles = rng.integers(0, 2, size=k_max).astype(np.uint8) * (sizes > 0)
        R = int((sizes > 0).sum())
        pos = int(rng.integers(0, R + 1))
        s2, r2 = orc.regrow(sizes, roles, M, 5, it, 3, pos, mx)
        assert (s2[:pos] == sizes[:pos]).all() and (r2[:pos] == roles[:pos]).all()
        assert int(s2.sum()) == M
        n = int((s2 > 0).sum())
        assert (s2[:n] > 0).all() and (s2[n:] == 0).all() and (r2[n:] == 0).all()
        # regrown replicas are at most max_replica, except the last slot,
        # which takes whatever remains
        for q in range(pos, n):
            assert s2[q] <= mx or q == k_max - 1
        assert set(np.unique(r2)) <= {0, 1}


def _tables_and_chain(orc, wl, chain, r):
    t, h, tau = orc.quantise(**wl.problem_arrays())
    tk = t[r][list(chain)]
    hk = h[r][list(chain)]
    tl = np.array([0] + [tau[r, chain[k - 1], chain[k]] for k in range(1, len(chain))],
                  dtype=np.uint64)
    mk = wl.mem_bytes[list(chain)]
    return brute.Chain(tk, hk, tl, mk, wl.layer_bytes, wl.head_bytes)


def test_solve_ordered_matches_brute_force_in_ordering_order(orc):
    """Each replica is solved as a chain in ordering order, not id order."""
    rng = np.random.default_rng(3)
    n_feasible = 0
    for it in range(40):
        M, N, k_max = int(rng.integers(2, 7)), int(rng.integers(2, 8)), 3
        wl = workload.random_small(500 + it, M=M, N=N, P=2, k_max=k_max, mem_hi_layers=8)
        order = np.stack([rng.permutation(M) for _ in range(2)]).astype(np.uint8)
        sizes = np.zeros((2, k_max), np.uint16)
        for p in range(2):
            cut = sorted(rng.choice(np.arange(1, M), size=min(k_max, M) - 1, replace=False))
            sizes[p, :len(cut) + 1] = np.diff([0] + list(cut) + [M])
        roles = rng.integers(0, 2, size=(2, k_max)).astype(np.uint8)
        tables = orc.quantise(**wl.problem_arrays())
        sol = orc.solve_ordered(tables, wl.mem_bytes, wl.layer_bytes, wl.head_bytes, order,
                                sizes, roles)
        for p in range(2):
            for q in range(k_max):
                lo, hi = orc.replica_range(sizes[p], q, M)
                chain = [int(x) for x in order[p, lo:hi]]
                if not chain:
                    assert sol["T"][p, q] == INF and sol["master"][p, q] == -1
                    continue
                T, L, mu, sz = _tables_and_chain(orc, wl, chain, int(roles[p, q] != 0)).solve()
                assert sol["T"][p, q] == T and sol["Lambda"][p, q] == L
                if T == INF:
                    assert sol["master"][p, q] == -1
                    assert all(sol["layers"][p, d] == 0 for d in chain)
                    continue
                n_feasible += 1
                assert sol["master"][p, q] == chain[mu - 1]
                assert [int(sol["layers"][p, d]) for d in chain] == list(sz)
    assert n_feasible > 20


def test_solve_ordered_with_id_ordering_equals_labelled_clusters(orc):
    """An identity ordering cut into runs gives the same replicas as labels
    that mark the same runs (chains in ascending id either way)."""
    wl = workload.random_small(42, M=30, N=40, P=5, k_max=6, mem_hi_layers=30)
    rng = np.random.default_rng(42)
    order = np.tile(np.arange(30, dtype=np.uint8), (5, 1))
    sizes = np.zeros((5, 6), np.uint16)
    labels = np.zeros((5, 30), np.uint8)
    for p in range(5):
        cut = sorted(rng.choice(np.arange(1, 30), size=5, replace=False))
        sz = np.diff([0] + list(cut) + [30])
        sizes[p] = sz
        labels[p] = np.repeat(np.arange(6), sz)
    a = orc.eval_population_ordered(wl, order, sizes, wl.roles)
    b = orc.eval_population(wl, labels, wl.roles)
    for k in ("T", "Lambda", "master", "layers", "w", "phase"):
        assert (a[k] == b[k]).all(), k


def test_ga_step_ordered_invariants_and_mutation_shares(orc):
    """Elites copied; every child is a valid gene; about 30% of children
    mutate, split 20/50/15/15 between the four mutations of App. A."""
    wl = workload.make("c3_64dev_80L")
    op = workload.ordered_population(wl, population=1024)
    M, k_max = wl.n_dev, wl.k_max
    rng = np.random.default_rng(1)
    w = rng.integers(0, 1000, size=1024).astype(np.uint64)
    ph = rng.integers(0, 1000, size=1024).astype(np.uint64)
    params = op.ga_params(wl, 3)
    params["n_elite"] = 4
    oo, so, ro = orc.ga_step_ordered(op.order, op.sizes, op.roles, w, ph, **params)
    keys = sorted(range(1024), key=lambda i: (int(w[i]), int(ph[i]), i))[:4]
    for e, src in enumerate(keys):
        assert (oo[e] == op.order[src]).all() and (so[e] == op.sizes[src]).all()
        assert (ro[e] == op.roles[src]).all()
    for s in range(1024):
        assert sorted(oo[s]) == list(range(M))
        assert int(so[s].sum()) == M
        n = int((so[s] > 0).sum())
        assert (so[s][n:] == 0).all() and set(np.unique(ro[s])) <= {0, 1}
    # mutation shares, from the generator's draws on the mutation stream
    fired = kinds = 0
    counts = [0, 0, 0, 0]
    for s in range(4, 1024):
        u = orc.rng(params["seed"], 3, s, 142, 0)
        if (u >> 32) < params["mutation_thresh_u32"]:
            fired += 1
            lo = u & 0xFFFFFFFF
            counts[0 if lo < 0.2 * 2**32 else 1 if lo < 0.7 * 2**32 else
                   2 if lo < 0.85 * 2**32 else 3] += 1
    assert abs(fired / 1020 - 0.3) < 0.05
    assert abs(counts[0] / fired - 0.2) < 0.07 and abs(counts[1] / fired - 0.5) < 0.08
    assert abs(counts[2] / fired - 0.15) < 0.06 and abs(counts[3] / fired - 0.15) < 0.06


def test_ga_step_ordered_without_mutation_recombines_parents(orc):
    """With mutation off, each child's ordering has a parent's prefix and
    its grouping and roles are one parent's, unchanged."""
    wl = workload.make("c2_32dev_48L")
    op = workload.ordered_population(wl, population=256)
    rng = np.random.default_rng(2)
    w = rng.integers(0, 10, size=256).astype(np.uint64)      # many ties
    ph = rng.integers(0, 10, size=256).astype(np.uint64)
    params = op.ga_params(wl, 1)
    params["mutation_thresh_u32"] = 0
    oo, so, ro = orc.ga_step_ordered(op.order, op.sizes, op.roles, w, ph, **params)
    groupings = {(tuple(op.sizes[p]), tuple(op.roles[p])) for p in range(256)}
    prefixes = {tuple(op.order[p][:1]) for p in range(256)}
    for s in range(params["n_elite"], 256):
        assert (tuple(so[s]), tuple(ro[s])) in groupings
        assert tuple(oo[s][:1]) in prefixes


def test_solve_ordered_with_a_non_device_id(orc):
    """An id >= M makes its replica infeasible and leaves the other replicas
    as they were; the device it displaced, now in no replica, gets 0 layers."""
    wl = workload.random_small(8, M=12, N=30, P=1, k_max=3, mem_hi_layers=40)
    order = np.arange(12, dtype=np.uint8)[None]
    sizes = np.array([[4, 4, 4]], np.uint16)
    roles = np.zeros((1, 3), np.uint8)
    tables = orc.quantise(**wl.problem_arrays())
    args = (tables, wl.mem_bytes, wl.layer_bytes, wl.head_bytes)
    base = orc.solve_ordered(*args, order, sizes, roles)
    assert (base["T"] != INF).all()
    bad = order.copy()
    bad[0, 5] = 200                                       # replica 1 loses device 5
    got = orc.solve_ordered(*args, bad, sizes, roles)
    assert got["T"][0, 1] == INF and got["master"][0, 1] == -1
    for q in (0, 2):
        assert got["T"][0, q] == base["T"][0, q] and got["master"][0, q] == base["master"][0, q]
    assert (got["layers"][0, 4:8] == 0).all()
    assert (got["layers"][0, :4] == base["layers"][0, :4]).all()
    assert (got["layers"][0, 8:] == base["layers"][0, 8:]).all()
