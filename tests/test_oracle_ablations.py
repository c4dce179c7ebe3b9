"""Pins for the oracle's two ablations of Sec. 4.2.

The finishing-time (FT) objective: each replica's master and split points
minimise its end-to-end time (stage plus link times) instead of the
bottleneck.  Checked against exhaustive enumeration, a closed form for
identical devices (every partition ties), the order it must keep against the
bottleneck DP (no larger end-to-end time, no smaller bottleneck, the same
feasibility) and the single-device case.

The adapted-SplitWise role rule: the token ratio sets how many replicas
prefill, the strongest by prefill rate take it.  Checked against the count
and ranking it states, against the already pinned fixed-role fitness for
the roles it picks, and against the brute-force search, which it can never
beat.
"""
import numpy as np
import pytest

import oracle
from oracle import brute
from paper_2606_03770_amd import workload

INF = brute.INF


def rand_chain(rng, m, N):
    tk = rng.integers(1, 20, size=(m, N)).astype(np.uint64)
    hk = rng.integers(0, 15, size=m).astype(np.uint64)
    tl = rng.integers(0, 25, size=m).astype(np.uint64)
    if rng.uniform() < 0.1:
        tl[rng.integers(0, m)] = np.uint64(INF)
    tl[0] = 0
    W = rng.integers(1, 5, size=N).astype(np.uint64)
    HB = int(rng.integers(0, 4))
    mem = rng.integers(2, 25, size=m).astype(np.uint64)
    return tk, hk, tl, mem, W, HB


def test_ft_matches_enumeration(orc):
    rng = np.random.default_rng(31337)
    feasible = 0
    for _ in range(500):
        m, N = int(rng.integers(1, 5)), int(rng.integers(1, 9))
        args = rand_chain(rng, m, N)
        got = orc.dp_pipe_ft(*args)
        want = brute.Chain(*args).solve_sum()
        assert got == (want[0], want[1], want[2], list(want[3])), (m, N, args)
        feasible += got[0] != INF
    assert feasible > 150


def test_ft_orders_against_the_bottleneck_dp(orc):
    """The FT partition has the least end-to-end time, so it is no slower end
    to end and no faster at the bottleneck than Algorithm 1's; both are
    feasible exactly when some partition fits."""
    rng = np.random.default_rng(8)
    for _ in range(400):
        m, N = int(rng.integers(1, 7)), int(rng.integers(1, 16))
        args = rand_chain(rng, m, N)
        T_ft, L_ft, _, _ = orc.dp_pipe_ft(*args)
        T_bn, L_bn, _, _, _ = orc.dp_pipe(*args)
        assert (T_ft == INF) == (T_bn == INF)
        if T_bn != INF:
            assert L_ft <= L_bn and T_ft >= T_bn


def test_ft_head_adds_at_least_the_masters_head_time(orc):
    """The head's time is added once, to the master's stage, and its bytes
    only narrow that stage's window: the least end-to-end time with a head
    is at least the head-free one plus the chosen master's head time, with
    equality when the head-free optimum fits with the head on that device
    (here: ample memory)."""
    rng = np.random.default_rng(19)
    equal = 0
    for _ in range(300):
        m, N = int(rng.integers(1, 6)), int(rng.integers(1, 12))
        tk, hk, tl, mem, W, HB = rand_chain(rng, m, N)
        T, L, mu, _ = orc.dp_pipe_ft(tk, hk, tl, mem, W, HB)
        T0, L0, _, _ = orc.dp_pipe_ft(tk, np.zeros_like(hk), tl, mem, W, 0)
        assert L0 != INF or L == INF                  # no partition at all
        if L == INF:
            continue
        assert L >= L0 + int(hk[mu - 1]) >= L0 + int(hk.min())
        # with memory to spare the head-free partitions stay feasible
        roomy = np.full(m, 10**9, np.uint64)
        _, Lr, mur, _ = orc.dp_pipe_ft(tk, hk, tl, roomy, W, HB)
        _, L0r, _, _ = orc.dp_pipe_ft(tk, np.zeros_like(hk), tl, roomy, W, 0)
        assert Lr == L0r + int(hk.min()) and int(hk[mur - 1]) == int(hk.min())
        equal += L == L0 + int(hk[mu - 1])
    assert equal > 50


def test_ft_identical_devices_closed_form(orc):
    """Identical devices, free links, no head, ample memory: every partition
    takes N t end to end, so every master and split ties; the smallest-j rule
    gives devices 1..m-1 one block each and the last the rest."""
    for m, N, t in ((1, 5, 3), (3, 10, 2), (4, 4, 7), (5, 12, 1)):
        tk = np.full((m, N), t, np.uint64)
        hk = np.zeros(m, np.uint64)
        tl = np.zeros(m, np.uint64)
        mem = np.full(m, 10**6, np.uint64)
        W = np.ones(N, np.uint64)
        T, L, mu, sizes = orc.dp_pipe_ft(tk, hk, tl, mem, W, 0)
        assert (L, mu) == (N * t, 1)
        assert sizes == [1] * (m - 1) + [N - m + 1]
        assert T == (N - m + 1) * t


def test_ft_single_device_equals_the_bottleneck_dp(orc):
    rng = np.random.default_rng(3)
    for _ in range(50):
        args = rand_chain(rng, 1, int(rng.integers(1, 12)))
        T_ft, L_ft, mu_ft, s_ft = orc.dp_pipe_ft(*args)
        T_bn, L_bn, mu_bn, s_bn, _ = orc.dp_pipe(*args)
        assert (T_ft, L_ft, mu_ft, s_ft) == (T_bn, L_bn, mu_bn, list(s_bn))


def test_ft_population_scores_its_partitions_by_eq_3_5(orc):
    """eval_population_ft's fitness is the fixed-role fitness of its own
    (T, Lambda), and its per-cluster results equal dp_pipe_ft on the chain."""
    wl = workload.random_small(21, M=12, N=20, P=6, k_max=3, mem_hi_layers=15)
    got = orc.eval_population_ft(wl)
    fit = orc.fitness(got["T"], got["Lambda"], wl.roles, **wl.fitness_params())
    assert (fit["w"] == got["w"]).all() and (fit["phase"] == got["phase"]).all()
    t, h, tau = orc.quantise(**wl.problem_arrays())
    for p in range(wl.population):
        for q in range(wl.k_max):
            ch = np.nonzero(wl.labels[p] == q)[0]
            if len(ch) == 0:
                continue
            r = int(wl.roles[p, q] != 0)
            tl = np.array([0] + [tau[r, ch[k - 1], ch[k]] for k in range(1, len(ch))], np.uint64)
            T, L, mu, _ = orc.dp_pipe_ft(t[r][ch], h[r][ch], tl, wl.mem_bytes[ch],
                                         wl.layer_bytes, wl.head_bytes)
            assert (got["T"][p, q], got["Lambda"][p, q]) == (T, L)
            assert got["master"][p, q] == (ch[mu - 1] if T != INF else -1)


@pytest.mark.parametrize("seed", range(4))
def test_splitwise_count_ranking_and_fitness(orc, seed):
    wl = workload.random_small(60 + seed, M=14, N=18, P=8, k_max=5, mem_hi_layers=14)
    wl.min_tps_milli = 0
    sm = dict(b_max=1, beta_ppm=0, kv_bytes_per_block_slot=0)
    got = orc.search_roles(wl, sm, policy="splitwise")
    NP, ND = orc.np_tokens(wl), int(wl.nd_tokens)
    for p in range(wl.population):
        used = sorted({int(x) for x in wl.labels[p] if x < wl.k_max})
        R = len(used)
        n_p = sum(1 for q in used if got["roles"][p, q] == 0)
        if R >= 2:
            want = int(np.floor(R * NP / (NP + ND) + 0.5)) if NP + ND else (R + 1) // 2
            assert n_p == min(max(want, 1), R - 1)
        # prefill clusters have the best prefill times (ties to smaller q)
        T0 = got["T_all"][p, :, 0]
        rank = sorted(used, key=lambda q: (-(0 if T0[q] == INF else (1 << 50) // max(int(T0[q]), 1)), q))
        assert sorted(rank[:n_p]) == [q for q in used if got["roles"][p, q] == 0]
        # its fitness is the fixed-role fitness of the roles it picked
        ev = oracle.eval_population(wl.subset([p]), wl.labels[p:p + 1], got["roles"][p:p + 1])
        assert (int(ev["w"][0]), int(ev["phase"][0])) == (int(got["w"][p]), int(got["phase"][p]))


def test_search_never_loses_to_splitwise(orc):
    wl = workload.make("c2_32dev_48L")
    sm = workload.slot_model(wl, b_max=4)
    s = orc.search_roles(wl, sm)
    r = orc.search_roles(wl, sm, policy="splitwise")
    assert (s["T_all"] == r["T_all"]).all()
    better = 0
    for p in range(wl.population):
        ks, kr = (int(s["w"][p]), int(s["phase"][p])), (int(r["w"][p]), int(r["phase"][p]))
        assert ks <= kr
        better += ks < kr
    assert better > 0
