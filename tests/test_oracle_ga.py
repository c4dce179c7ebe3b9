"""Pins for the oracle's GA step (Algorithm 2; App. A elite preservation) and
its counter-based generator (SplitMix64, Steele, Lea and Flood, OOPSLA 2014).

The operators themselves (tournament of 4, uniform crossover, per-gene
mutation) and the stream layout are definitions of this implementation:
parity for them holds between two independent implementations of the same
written definition ("parity unpinned" by the paper).  What is pinned here is
the generator's published output, determinism, elitism and the operators'
limiting cases.
"""
import json
import os

import numpy as np

import oracle
from paper_2606_03770_amd import workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = oracle.INF


def test_splitmix64_known_answers(orc):
    """The generator seeded with 0 produces the published first outputs."""
    g = json.load(open(os.path.join(GOLDEN, "paper_values.json")))["splitmix64_seed0"]
    gamma = 0x9E3779B97F4A7C15
    got = [oracle.splitmix_out((i * gamma) % (1 << 64)) for i in range(3)]
    assert got == [int(x, 16) for x in g["outputs_hex"]]


def test_rng_is_a_pure_function_and_uniform(orc):
    a = [oracle.rng(5, 3, s, 130, d) for s in range(40) for d in range(50)]
    b = [oracle.rng(5, 3, s, 130, d) for s in range(40) for d in range(50)]
    assert a == b
    assert len(set(a)) == len(a)
    top = np.array([x >> 60 for x in a])
    counts = np.bincount(top, minlength=16)
    chi2 = float(((counts - len(a) / 16) ** 2 / (len(a) / 16)).sum())
    assert chi2 < 50  # 15 dof; p ~ 1e-5 threshold
    assert oracle.rng(5, 3, 0, 130, 0) != oracle.rng(5, 4, 0, 130, 0)
    assert oracle.rng(5, 3, 0, 130, 0) != oracle.rng(6, 3, 0, 130, 0)


def _pop(seed=1, P=64, M=24, k_max=5):
    rng = np.random.default_rng(seed)
    labels = rng.integers(0, k_max, size=(P, M)).astype(np.uint8)
    roles = rng.integers(0, 2, size=(P, k_max)).astype(np.uint8)
    w = rng.integers(0, 10**9, size=P).astype(np.uint64)
    w[rng.uniform(size=P) < 0.2] = np.uint64(INF)
    w[rng.uniform(size=P) < 0.2] = 0
    phase = rng.integers(0, 10**9, size=P).astype(np.uint64)
    return labels, roles, w, phase


def _key_order(w, phase):
    return sorted(range(len(w)), key=lambda p: (int(w[p]), int(phase[p]), p))


def test_elites_are_the_best_in_key_order(orc):
    labels, roles, w, phase = _pop()
    for n_elite in (1, 3, 8):
        lo, ro = oracle.ga_step(labels, roles, w, phase, 5, 9, 0, 4, 1 << 31, 1 << 24, n_elite)
        order = _key_order(w, phase)
        for e in range(n_elite):
            assert (lo[e] == labels[order[e]]).all() and (ro[e] == roles[order[e]]).all()


def test_deterministic_and_generation_dependent(orc):
    labels, roles, w, phase = _pop()
    a = oracle.ga_step(labels, roles, w, phase, 5, 9, 3, 4, 1 << 31, 1 << 24, 1)
    b = oracle.ga_step(labels, roles, w, phase, 5, 9, 3, 4, 1 << 31, 1 << 24, 1)
    c = oracle.ga_step(labels, roles, w, phase, 5, 9, 4, 4, 1 << 31, 1 << 24, 1)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()
    assert not (a[0] == c[0]).all()


def test_identical_parents_without_mutation_copy(orc):
    labels, roles, w, phase = _pop()
    labels[:] = labels[0]
    roles[:] = roles[0]
    lo, ro = oracle.ga_step(labels, roles, w, phase, 5, 9, 0, 4, 1 << 31, 0, 2)
    assert (lo == labels[0]).all() and (ro == roles[0]).all()


def test_no_crossover_no_mutation_picks_tournament_winners(orc):
    """With crossover and mutation off every child copies one tournament
    winner; with 64 draws from 32 members the winner is nearly always one of
    the best few in key order."""
    labels, roles, w, phase = _pop(P=32)
    labels = np.arange(32, dtype=np.uint8)[:, None].repeat(24, axis=1)  # row p holds p
    roles = np.zeros((32, 40), np.uint8)
    lo, _ = oracle.ga_step(labels, roles, w, phase, 40, 2, 0, 64, 0, 0, 1)
    rank = {p: r for r, p in enumerate(_key_order(w, phase))}
    child_rank = [rank[int(lo[s, 0])] for s in range(1, 32)]
    assert all((lo[s] == lo[s, 0]).all() for s in range(32))
    assert np.mean(child_rank) < 3  # 64 draws from 32: the winner is almost always top-3


def test_labels_stay_in_range_and_mutation_redraws_uniformly(orc):
    labels, roles, w, phase = _pop(P=200, M=60, k_max=7)
    lo, ro = oracle.ga_step(labels, roles, w, phase, 7, 1, 0, 4, 1 << 31, (1 << 32) - 1, 1)
    assert lo.max() < 7 and set(np.unique(ro)) <= {0, 1}
    counts = np.bincount(lo[1:].ravel(), minlength=7)
    exp = lo[1:].size / 7
    assert float(((counts - exp) ** 2 / exp).sum()) < 40


def test_mutation_rate(orc):
    """Per-gene mutation at 1/256 changes about 1/256 * (1 - 1/k) of the genes."""
    labels, roles, w, phase = _pop(P=400, M=256, k_max=40)
    labels[:] = labels[0]
    roles[:] = roles[0]
    lo, ro = oracle.ga_step(labels, roles, w, phase, 40, 3, 0, 4, 1 << 31, 1 << 24, 1)
    frac = float((lo[1:] != labels[0]).mean())
    assert abs(frac - (1 / 256) * (39 / 40)) < 0.0015
    rfrac = float((ro[1:] != roles[0]).mean())
    assert abs(rfrac - 1 / 256) < 0.003


def test_ga_loop_best_never_rises_and_resume_is_exact(orc, tmp_path):
    """Elitism keeps the best (w, phase) monotone; a resume from a saved
    population reproduces the straight run bit for bit."""
    wl = workload.random_small(31, M=10, N=9, P=24, k_max=3, mem_hi_layers=12)
    wl.t_arrival_ns = 0

    def run(labels, roles, g0, g1):
        best = []
        for g in range(g0, g1):
            sol = oracle.eval_population(wl, labels, roles)
            k = min((int(a), int(b)) for a, b in zip(sol["w"], sol["phase"]))
            best.append(k)
            labels, roles = oracle.ga_step(labels, roles, sol["w"], sol["phase"], wl.k_max,
                                           11, g, 4, 1 << 31, 1 << 26, 1)
        return labels, roles, best

    la, ra, best = run(wl.labels, wl.roles, 0, 6)
    assert all(best[i + 1] <= best[i] for i in range(len(best) - 1))
    lb, rb, _ = run(wl.labels, wl.roles, 0, 3)
    np.savez(tmp_path / "ck.npz", labels=lb, roles=rb, generation=3)
    ck = np.load(tmp_path / "ck.npz")
    lc, rc, _ = run(ck["labels"], ck["roles"], int(ck["generation"]), 6)
    assert (lc == la).all() and (rc == ra).all()
