"""Pins for the oracle's dynamic program (Algorithm 1, Eq. 1-2 of the paper).

None of these re-run the oracle's recurrence: each checks it against brute
force enumeration, a closed form, a bound, an invariant or a value the paper
prints.
"""
import json
import os

import numpy as np
import pytest

from oracle import brute

INF = brute.INF
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_chain(rng, m, N, *, inf_link=0.1, head=True, big_mem=False):
    tk = rng.integers(1, 20, size=(m, N)).astype(np.uint64)
    hk = rng.integers(0, 15, size=m).astype(np.uint64) if head else np.zeros(m, np.uint64)
    tl = rng.integers(0, 25, size=m).astype(np.uint64)
    if rng.uniform() < inf_link:
        tl[rng.integers(0, m)] = np.uint64(INF)
    tl[0] = 0
    W = rng.integers(1, 5, size=N).astype(np.uint64)
    HB = int(rng.integers(0, 4)) if head else 0
    mem = (np.full(m, 10**6) if big_mem else rng.integers(2, 25, size=m)).astype(np.uint64)
    return tk, hk, tl, mem, W, HB


def test_brute_force_random(orc):
    """T, master, stage sizes and Lambda equal exhaustive enumeration (N <= 9, m <= 5)."""
    rng = np.random.default_rng(20260601)
    n_feasible = 0
    for _ in range(700):
        m = int(rng.integers(1, 6))
        N = int(rng.integers(1, 10))
        args = rand_chain(rng, m, N)
        T, L, mu, sizes, _ = orc.dp_pipe(*args)
        bT, bL, bmu, bsizes = brute.Chain(*args).solve()
        assert (T, L, mu, list(sizes)) == (bT, bL, bmu, list(bsizes)), (m, N, args)
        n_feasible += T != INF
    assert n_feasible > 200  # the draw must exercise feasible and infeasible chains


def test_brute_force_ties(orc):
    """Many equal costs: tie-breaks over j (smallest) and over the master (smallest)."""
    rng = np.random.default_rng(7)
    for _ in range(300):
        m = int(rng.integers(1, 5))
        N = int(rng.integers(1, 10))
        tk = rng.integers(1, 3, size=(m, N)).astype(np.uint64)
        hk = rng.integers(0, 2, size=m).astype(np.uint64)
        tl = rng.integers(0, 3, size=m).astype(np.uint64)
        tl[0] = 0
        W = np.ones(N, np.uint64)
        mem = rng.integers(1, N + 2, size=m).astype(np.uint64)
        HB = int(rng.integers(0, 2))
        a = orc.dp_pipe(tk, hk, tl, mem, W, HB)
        b = brute.Chain(tk, hk, tl, mem, W, HB).solve()
        assert (a[0], a[1], a[2], list(a[3])) == (b[0], b[1], b[2], list(b[3]))


def test_single_device_closed_form(orc):
    """m = 1: T = Lambda = sum of block times + head time, INF when it does not fit."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        N = int(rng.integers(1, 40))
        t = rng.integers(0, 10**9, size=(1, N)).astype(np.uint64)
        h = rng.integers(0, 10**9, size=1).astype(np.uint64)
        W = rng.integers(1, 100, size=N).astype(np.uint64)
        HB = int(rng.integers(0, 100))
        mem = np.array([int(rng.integers(0, 60 * N))], np.uint64)
        T, L, mu, sizes, _ = orc.dp_pipe(t, h, [0], mem, W, HB)
        if int(W.sum()) + HB <= int(mem[0]):
            want = int(t.sum()) + int(h[0])
            assert (T, L, mu, list(sizes)) == (want, want, 1, [N])
        else:
            assert (T, L, mu, list(sizes)) == (INF, INF, 0, [0])


@pytest.mark.parametrize("N,m", [(N, m) for N in range(1, 21) for m in range(1, 7) if m <= N])
def test_identical_devices_closed_form(orc, N, m):
    """Identical devices, no transfer cost, no head, ample memory:
    the best bottleneck is ceil(N / m) blocks' time, and every master ties (mu* = 1)."""
    t = 7
    tk = np.full((m, N), t, np.uint64)
    T, L, mu, sizes, _ = orc.dp_pipe(tk, np.zeros(m), np.zeros(m), np.full(m, 10**6),
                                     np.ones(N), 0)
    assert T == -(-N // m) * t
    assert mu == 1
    assert L == N * t
    assert sizes.sum() == N and sizes.min() >= 1 and sizes.max() * t == T


def test_hand_derived_backtrack():
    """N = 10 blocks on 3 identical devices: T = 4 blocks; the backtrack gives
    the last stage the most blocks among ties: (3, 3, 4).  Derivation: the last
    stage starts at the smallest j with 10 - j <= 4 and ceil(j / 2) <= 4, so
    j = 6; then 6 blocks on 2 devices have optimum 3, reached first at j = 3."""
    import oracle
    T, L, mu, sizes, _ = oracle.dp_pipe(np.ones((3, 10)), np.zeros(3), np.zeros(3),
                                        np.full(3, 100), np.ones(10), 0)
    assert (T, list(sizes)) == (4, [3, 3, 4])


def test_two_devices_closed_form(orc):
    """m = 2: T = min over master and split point of max(stage 1, stage 2, link)."""
    rng = np.random.default_rng(11)
    for _ in range(300):
        N = int(rng.integers(1, 30))
        tk = rng.integers(0, 100, size=(2, N)).astype(np.uint64)
        hk = rng.integers(0, 100, size=2).astype(np.uint64)
        tau = int(rng.integers(0, 300))
        W = rng.integers(1, 10, size=N)
        HB = int(rng.integers(0, 10))
        mem = rng.integers(1, 8 * N, size=2)
        best = INF
        for mu in (1, 2):
            for j in range(1, N):
                b1 = int(W[:j].sum()) + (HB if mu == 1 else 0)
                b2 = int(W[j:].sum()) + (HB if mu == 2 else 0)
                if b1 > mem[0] or b2 > mem[1]:
                    continue
                c1 = int(tk[0, :j].sum()) + (int(hk[0]) if mu == 1 else 0)
                c2 = int(tk[1, j:].sum()) + (int(hk[1]) if mu == 2 else 0)
                best = min(best, max(c1, c2, tau))
        T = orc.dp_pipe(tk, hk, [0, tau], mem, W, HB)[0]
        assert T == best


def test_more_devices_than_blocks_is_infeasible(orc):
    for m in range(2, 8):
        N = m - 1
        T, L, mu, sizes, ev = orc.dp_pipe(np.ones((m, N)), np.zeros(m), np.zeros(m),
                                          np.full(m, 100), np.ones(N), 0)
        assert (T, mu, ev) == (INF, 0, 0) and sizes.sum() == 0


def test_total_memory_too_small_is_infeasible(orc):
    rng = np.random.default_rng(5)
    for _ in range(100):
        m = int(rng.integers(1, 6))
        N = int(rng.integers(m, 20))
        W = rng.integers(5, 20, size=N)
        HB = int(rng.integers(0, 20))
        need = int(W.sum()) + HB
        mem = rng.multinomial(need - 1, np.ones(m) / m)  # sum = need - 1
        T = orc.dp_pipe(np.ones((m, N)), np.zeros(m), np.zeros(m), mem, W, HB)[0]
        assert T == INF


def test_lower_bounds(orc):
    """Every device holds >= 1 block and every chain link is used, so
    T >= max_k min_n t[k][n] and T >= max link time.  For identical blocks the
    integer fluid bound holds: sum_k floor((T - head_k) / t_k) >= N."""
    rng = np.random.default_rng(13)
    checked = 0
    for _ in range(400):
        m = int(rng.integers(1, 7))
        N = int(rng.integers(m, 25))
        tk, hk, tl, mem, W, HB = rand_chain(rng, m, N, inf_link=0.0, big_mem=True)
        T, L, mu, sizes, _ = orc.dp_pipe(tk, hk, tl, mem, W, HB)
        assert T != INF
        assert T >= max(int(tk[k].min()) for k in range(m))
        assert T >= int(tl[1:].max(initial=0))
        assert L >= T
        tu = rng.integers(1, 30, size=m)
        tk2 = np.repeat(tu[:, None], N, axis=1).astype(np.uint64)
        T2, _, mu2, _, _ = orc.dp_pipe(tk2, hk, tl, mem, W, HB)
        cap = sum((T2 - (int(hk[k]) if k + 1 == mu2 else 0)) // int(tu[k]) for k in range(m))
        assert cap >= N
        checked += 1
    assert checked == 400


def test_monotone_in_costs_and_memory(orc):
    """Lowering a block time, a head time or a link time, or raising a memory
    cap, never raises the optimum."""
    rng = np.random.default_rng(17)
    for _ in range(300):
        m = int(rng.integers(1, 6))
        N = int(rng.integers(1, 14))
        tk, hk, tl, mem, W, HB = rand_chain(rng, m, N)
        T = orc.dp_pipe(tk, hk, tl, mem, W, HB)[0]
        kind = rng.integers(0, 4)
        tk2, hk2, tl2, mem2 = tk.copy(), hk.copy(), tl.copy(), mem.copy()
        k = int(rng.integers(0, m))
        if kind == 0:
            n = int(rng.integers(0, N))
            tk2[k, n] = tk2[k, n] // 2
        elif kind == 1:
            hk2[k] = 0
        elif kind == 2 and m > 1:
            tl2[max(k, 1)] = 0
        else:
            mem2[k] = mem2[k] + 10
        assert orc.dp_pipe(tk2, hk2, tl2, mem2, W, HB)[0] <= T


def test_reversal_symmetry(orc):
    """Reversing the chain together with the block order (symmetric links)
    leaves the optimum unchanged."""
    rng = np.random.default_rng(19)
    for _ in range(300):
        m = int(rng.integers(1, 6))
        N = int(rng.integers(1, 14))
        tk, hk, tl, mem, W, HB = rand_chain(rng, m, N)
        T = orc.dp_pipe(tk, hk, tl, mem, W, HB)[0]
        tk_r = tk[::-1, ::-1].copy()
        tl_r = np.zeros(m, np.uint64)
        for k in range(1, m):  # link between reversed positions k-1, k = old link m-k
            tl_r[k] = tl[m - k]
        Tr = orc.dp_pipe(tk_r, hk[::-1].copy(), tl_r, mem[::-1].copy(), W[::-1].copy(), HB)[0]
        assert Tr == T


def test_candidate_count_matches_quadratic_complexity(orc):
    """With ample memory and finite links, the number of candidates the
    recurrence evaluates is m * sum_{k=2..m} sum_{i=k-1..N-1} (i - k + 2)
    (O(M^2 N^2), Sec. 3.2)."""
    for m in range(1, 7):
        for N in range(m, 30, 3):
            ev = orc.dp_pipe(np.ones((m, N)), np.zeros(m), np.zeros(m), np.full(m, 10**6),
                             np.ones(N), 0)[4]
            want = m * sum(i - k + 2 for k in range(2, m + 1) for i in range(k - 1, N))
            assert ev == want


def test_r1_adding_a_device_can_worsen(orc):
    """Under reading R1 (each device takes >= 1 block) adding a device can
    raise the optimum: 2 blocks, fast device A, slow device B."""
    one = orc.dp_pipe([[1, 1]], [0], [0], [100], [1, 1], 0)[0]
    two = orc.dp_pipe([[1, 1], [100, 100]], [0, 0], [0, 0], [100, 100], [1, 1], 0)[0]
    assert (one, two) == (2, 100)
    link = orc.dp_pipe([[1, 1], [1, 1]], [0, 0], [0, 50], [100, 100], [1, 1], 0)[0]
    assert link == 50


def test_idle_relaxation_never_worsens_with_more_devices():
    """Under the idle-device relaxation, adding a device never raises the
    optimum, and the relaxed optimum never exceeds the R1 optimum."""
    rng = np.random.default_rng(23)
    for _ in range(120):
        m = int(rng.integers(1, 4))
        N = int(rng.integers(1, 7))
        full = rng.integers(0, 25, size=(m + 1, m + 1))
        full = np.triu(full, 1) + np.triu(full, 1).T
        tk = rng.integers(1, 20, size=(m + 1, N))
        hk = rng.integers(0, 10, size=m + 1)
        mem = rng.integers(2, 30, size=m + 1)
        W = rng.integers(1, 5, size=N)
        HB = int(rng.integers(0, 4))

        def chain(idx):
            tl = [0] + [int(full[idx[k - 1], idx[k]]) for k in range(1, len(idx))]
            c = brute.Chain(tk[idx], hk[idx], tl, mem[idx], W, HB)
            c.set_links(full[np.ix_(idx, idx)])
            return c

        small = chain(list(range(m)))
        ins = int(rng.integers(0, m + 1))
        idx_big = list(range(m))
        idx_big.insert(ins, m)
        big = chain(idx_big)
        assert big.solve_idle_relaxed() <= small.solve_idle_relaxed()
        assert small.solve_idle_relaxed() <= small.solve()[0]


def test_printed_plans_hold_every_block_once():
    """Every replica printed in the paper's plan tables holds all N blocks,
    each device at least one block and exactly one master: the structure
    reading R1 gives to every feasible partition."""
    doc = json.load(open(os.path.join(GOLDEN, "printed_plans.json")))
    n_rep = 0
    for plan in doc["plans"]:
        for rep in plan["replicas"]:
            blocks = [d["gpu_blocks"] + d["cpu_blocks"] for d in rep["devices"]]
            assert sum(blocks) == plan["n_blocks"]
            assert min(blocks) >= 1
            assert sum(d["master"] for d in rep["devices"]) == 1
            n_rep += 1
    assert n_rep >= 300
