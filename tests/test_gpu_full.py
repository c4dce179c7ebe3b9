"""Whole-population parity on the two largest workloads.

Every genome, not a sample: the HIP path's T, Lambda, master, layers, w,
phase, S_P and S_D equal the oracle's bit for bit on all 16384 genomes of
the 256-device generation 0 and all 4096 genomes of the 128-device
workload, with both genome kinds.  The GA chain of the 256-device workload
(Algorithm 2; 50 generations of tournament 4, uniform crossover 0.5 and
mutation 1/256 for label genomes, the App. A operators for two-chromosome
genomes) runs on the GPU; every one of its 50 GA steps is compared in full
with the oracle's GA fed the same population and fitness keys, every
generation's evaluation is checked on 256 sampled genomes, and the last
generation's on every genome.  Algorithm 2's own generation (the role and
slot search, then the GA from the searched roles and keys) runs for 50
generations of both genome kinds, every GA step compared in full and each
generation's search on 96 sampled genomes.

The oracle runs over genome ranges in worker processes (oracle.pool), which
the GPU results never feed: the oracle sees the population only.
"""
import time

import numpy as np
import pytest

import oracle
from oracle import pool
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

pytestmark = pytest.mark.gpu
INF = (1 << 64) - 1
KEYS = pool.KEYS
GENERATIONS = 50
SAMPLE = 256


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    e2.lib()
    return torch, torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)


def _host(sol, fit):
    out = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
               master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy())
    for k in ("w", "phase", "s_p", "s_d"):
        out[k] = e2.u64(fit[k])
    return out


def _gpu_labels(torch_dev, ctx, wl, L, R):
    torch, _ = torch_dev
    sol = e2.e2_solve_partitions(ctx, L, R)
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    return _host(sol, fit)


def _gpu_ordered(torch_dev, ctx, wl, O, S, Q):
    torch, _ = torch_dev
    sol = e2.e2_solve_partitions_ordered(ctx, O, S, Q)
    fit = e2.e2_eval_population_ordered(ctx, O, S, Q, wl.fitness_params())
    torch.cuda.synchronize()
    return _host(sol, fit)


def _assert_equal(got, want, rows=None, tag=""):
    n = None
    for k in KEYS:
        g = got[k] if rows is None else got[k][rows]
        w = want[k]
        n = len(w)
        bad = np.argwhere(np.asarray(g != w).reshape(len(w), -1).any(axis=1)).ravel()
        assert bad.size == 0, f"{tag} {k}: {bad.size} of {len(w)} genomes differ, first {bad[:5]}"
    return n


def _every_genome(torch_dev, name, kind):
    torch, dev = torch_dev
    wl = workload.make(name)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    t0 = time.perf_counter()
    if kind == "labels":
        L = torch.from_numpy(wl.labels).to(dev)
        R = torch.from_numpy(wl.roles).to(dev)
        got = _gpu_labels(torch_dev, ctx, wl, L, R)
        _say(f"{name} {kind}: GPU done ({wl.population} genomes); oracle on "
             f"{pool.workers()} processes")
        want = pool.eval_population(wl)
    else:
        op = workload.ordered_population(wl)
        O, S, Q = (torch.from_numpy(x).to(dev) for x in (op.order, op.sizes, op.roles))
        got = _gpu_ordered(torch_dev, ctx, wl, O, S, Q)
        _say(f"{name} {kind}: GPU done ({wl.population} genomes); oracle on "
             f"{pool.workers()} processes")
        want = pool.eval_population_ordered(wl, op.order, op.sizes, op.roles)
    n = _assert_equal(got, want, tag=f"{name} {kind}")
    assert n == wl.population
    feasible = int((want["T"] != INF).sum())
    _say(f"{name} {kind}: {n} genomes, {feasible} feasible clusters equal "
         f"({time.perf_counter() - t0:.1f} s)")
    assert feasible > 0 and (want["w"] != INF).any()


@pytest.mark.parametrize("kind", ["labels", "two_chromosome"])
def test_every_genome_256_devices_generation_0(torch_dev, kind):
    _every_genome(torch_dev, "c5_256dev_126L_ga", kind)


@pytest.mark.parametrize("kind", ["labels", "two_chromosome"])
def test_every_genome_128_devices(torch_dev, kind):
    _every_genome(torch_dev, "c4_128dev_80L", kind)


def _chain(torch_dev, kind):
    """Run the GA chain on the GPU; return the populations g = 0..G (G + 1
    of them) and the GPU's fitness of g = 0..G-1."""
    torch, dev = torch_dev
    wl = workload.make("c5_256dev_126L_ga")
    assert wl.generations == GENERATIONS
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    pops, fits = [], []
    if kind == "labels":
        cur = (torch.from_numpy(wl.labels).to(dev), torch.from_numpy(wl.roles).to(dev))
        op = None
    else:
        op = workload.ordered_population(wl)
        cur = tuple(torch.from_numpy(x).to(dev) for x in (op.order, op.sizes, op.roles))
    for g in range(GENERATIONS):
        if kind == "labels":
            L, R = cur
            sol = e2.e2_solve_partitions(ctx, L, R)
            fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
            nxt = e2.e2_ga_step(ctx, L, R, fit["w"], fit["phase"], wl.ga_params(g))
        else:
            O, S, Q = cur
            sol = e2.e2_solve_partitions_ordered(ctx, O, S, Q)
            fit = e2.e2_eval_population_ordered(ctx, O, S, Q, wl.fitness_params())
            nxt = e2.e2_ga_step_ordered(ctx, O, S, Q, fit["w"], fit["phase"],
                                        op.ga_params(wl, g))
        torch.cuda.synchronize()
        pops.append(tuple(x.cpu().numpy() for x in cur))
        fits.append(_host(sol, fit))
        cur = nxt
    torch.cuda.synchronize()
    pops.append(tuple(x.cpu().numpy() for x in cur))
    return wl, op, pops, fits


@pytest.mark.parametrize("kind", ["labels", "two_chromosome"])
def test_fifty_generations_256_devices(torch_dev, kind):
    t0 = time.perf_counter()
    wl, op, pops, fits = _chain(torch_dev, kind)
    _say(f"{kind}: {GENERATIONS} GPU generations in {time.perf_counter() - t0:.1f} s")
    # every GA step in full: the oracle's GA fed generation g's population
    # and the GPU's keys gives generation g + 1
    for g in range(GENERATIONS):
        w, ph = fits[g]["w"], fits[g]["phase"]
        if kind == "labels":
            want = oracle.ga_step(*pops[g], w, ph, wl.k_max, **wl.ga_params(g))
        else:
            want = oracle.ga_step_ordered(*pops[g], w, ph, **op.ga_params(wl, g))
        for a, b, part in zip(pops[g + 1], want, ("first", "second", "third")):
            assert np.array_equal(a, b), f"{kind} GA step {g}: {part} chromosome differs"
    _say(f"{kind}: {GENERATIONS} GA steps equal the oracle's")
    # evaluation: 256 sampled genomes of every generation, then every
    # genome of the last one (the keys the last GA step read)
    rng = np.random.default_rng(2606)
    picks = [np.sort(rng.choice(wl.population, SAMPLE, replace=False))
             for _ in range(GENERATIONS - 1)]
    rows = np.concatenate(picks)
    gens = np.repeat(np.arange(GENERATIONS - 1), SAMPLE)
    if kind == "labels":
        L = np.stack([pops[g][0][p] for g, p in zip(gens, rows)])
        R = np.stack([pops[g][1][p] for g, p in zip(gens, rows)])
        want = pool.eval_population(wl, L, R)
    else:
        O, S, Q = (np.stack([pops[g][i][p] for g, p in zip(gens, rows)]) for i in range(3))
        want = pool.eval_population_ordered(wl, O, S, Q)
    got = {k: np.stack([fits[g][k][p] for g, p in zip(gens, rows)]) for k in KEYS}
    _assert_equal(got, want, tag=f"{kind} sampled generations 0..{GENERATIONS - 2}")
    _say(f"{kind}: {len(rows)} sampled evaluations over {GENERATIONS - 1} generations equal")
    last = GENERATIONS - 1
    if kind == "labels":
        want = pool.eval_population(wl, *pops[last])
    else:
        want = pool.eval_population_ordered(wl, *pops[last])
    _assert_equal(fits[last], want, tag=f"{kind} generation {last}")
    _say(f"{kind}: every genome of generation {last} equal "
         f"({time.perf_counter() - t0:.1f} s in all)")
    # the search moved: the best key of the last generation is no worse than
    # generation 0's (one elite is kept every step)
    k0 = min(zip(fits[0]["w"].tolist(), fits[0]["phase"].tolist()))
    k1 = min(zip(fits[last]["w"].tolist(), fits[last]["phase"].tolist()))
    assert k1 <= k0


SEARCH_GENERATIONS = 50
SEARCH_SAMPLE = 96


@pytest.mark.parametrize("kind", ["labels", "two_chromosome"])
def test_search_and_breed_fifty_generations_256_devices(torch_dev, kind):
    """Algorithm 2's generation as the paper runs it on the 256-device
    workload: the role and slot search scores every genome (a DP per cluster
    for prefill and each of 1..8 decode requests in flight, the kept slot
    count, brute-force roles), then the GA breeds from the searched roles and
    keys.  Fifty generations on the GPU; every GA step equals the oracle's GA
    fed the same population, searched roles and keys, and each generation's
    search equals the oracle's on 96 sampled genomes (every DP result, role,
    slot count and key)."""
    torch, dev = torch_dev
    t0 = time.perf_counter()
    wl = workload.make("c5_256dev_126L_ga")
    sm = workload.slot_model(wl)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    fp = wl.fitness_params()
    op = workload.ordered_population(wl)
    if kind == "labels":
        cur = [torch.from_numpy(x).to(dev) for x in (wl.labels, wl.roles)]
    else:
        cur = [torch.from_numpy(x).to(dev) for x in (op.order, op.sizes)]
    rng = np.random.default_rng(2607)
    pops, searched = [], []
    for g in range(SEARCH_GENERATIONS):
        if kind == "labels":
            res = e2.e2_search_roles(ctx, cur[0], fp, wl.k_max, with_tables=True)
            nxt = e2.e2_ga_step(ctx, cur[0], res["roles"], res["w"], res["phase"],
                                wl.ga_params(g))
        else:
            res = e2.e2_search_roles_ordered(ctx, cur[0], cur[1], fp, with_tables=True)
            nxt = e2.e2_ga_step_ordered(ctx, cur[0], cur[1], res["roles"], res["w"],
                                        res["phase"], op.ga_params(wl, g))
        torch.cuda.synchronize()
        pick = np.sort(rng.choice(wl.population, SEARCH_SAMPLE, replace=False))
        idx = torch.from_numpy(pick).to(dev)
        searched.append(dict(pick=pick, roles=res["roles"].cpu().numpy(),
                             w=e2.u64(res["w"]), phase=e2.u64(res["phase"]),
                             slots=res["slots"].index_select(0, idx).cpu().numpy(),
                             T_all=e2.u64(res["T_all"].index_select(0, idx)),
                             Lambda_all=e2.u64(res["Lambda_all"].index_select(0, idx))))
        pops.append([x.cpu().numpy() for x in cur])
        cur = list(nxt)
    pops.append([x.cpu().numpy() for x in cur])
    _say(f"{kind}: {SEARCH_GENERATIONS} search + GA generations on the GPU in "
         f"{time.perf_counter() - t0:.1f} s")
    for g in range(SEARCH_GENERATIONS):
        s = searched[g]
        if kind == "labels":
            want = oracle.ga_step(pops[g][0], s["roles"], s["w"], s["phase"], wl.k_max,
                                  **wl.ga_params(g))
        else:
            want = oracle.ga_step_ordered(pops[g][0], pops[g][1], s["roles"], s["w"],
                                          s["phase"], **op.ga_params(wl, g))
        for a, b in zip(pops[g + 1], want):
            assert np.array_equal(a, b), f"{kind} GA step {g}"
        p = s["pick"]
        if kind == "labels":
            ref = pool.search_roles(wl, sm, pops[g][0][p])
        else:
            ref = pool.search_roles_ordered(wl, sm, pops[g][0][p], pops[g][1][p])
        got = dict(T_all=s["T_all"], Lambda_all=s["Lambda_all"], roles=s["roles"][p],
                   slots=s["slots"], w=s["w"][p], phase=s["phase"][p])
        for k in pool.SEARCH_KEYS:
            bad = np.argwhere(np.asarray(got[k] != ref[k]).reshape(len(p), -1).any(axis=1))
            assert bad.size == 0, f"{kind} generation {g} {k}: {bad.size} genomes differ"
        _say(f"{kind}: generation {g} GA step and {len(p)} searched genomes equal")
    # the search improves on generation 0's best key (elites are kept)
    k0 = min(zip(searched[0]["w"].tolist(), searched[0]["phase"].tolist()))
    k1 = min(zip(searched[-1]["w"].tolist(), searched[-1]["phase"].tolist()))
    assert k1 <= k0
