"""Pins for the oracle's decode-slot tables and role search (Algorithm 2's
inner loop: one DP per role and slot count, the highest feasible slot count
under the QoS floor, brute-force role assignment).

The slot tables are checked against the plain tables, the closed forms of
their beta and link terms and the paper's transfer-time example; the search
against the already pinned fixed-role path (every role vector through
oracle.eval_population), single-device clusters in closed form,
monotonicity in the slot count and a symmetric tie.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2606_03770_amd import workload

INF = (1 << 64) - 1


def _problem(wl):
    return wl.problem_arrays()


def test_slot_tables_extend_the_plain_tables(orc):
    wl = workload.random_small(4, M=9, N=13, P=1, k_max=2, zero_bw_frac=0.2)
    t0, h0, tau0 = orc.quantise(**_problem(wl))
    t, h, tau = orc.quantise_slots(_problem(wl), 6, 250_000)
    assert t.shape == (7, 9, 13) and h.shape == (7, 9) and tau.shape == (7, 9, 9)
    for r in (0, 1):
        assert (t[r] == t0[r]).all() and (h[r] == h0[r]).all() and (tau[r] == tau0[r]).all()
    # a further request adds beta of a lone request's time, rounded up
    for b in range(2, 7):
        assert (t[b] >= t[1]).all() and (t[b] >= t[b - 1]).all()
        step = t[b] - t[b - 1]
        assert (step == t[2] - t[1]).all()
        assert (4 * step >= t[1]).all() and (4 * (step - 1) < t[1]).all()   # ceil(t / 4)


def test_slot_tables_closed_forms(orc):
    wl = workload.random_small(5, M=6, N=7, P=1, k_max=2, zero_bw_frac=0.3)
    t, h, tau = orc.quantise_slots(_problem(wl), 5, 0)
    for b in range(1, 6):                       # beta = 0: batching is free
        assert (t[b] == t[1]).all() and (h[b] == h[1]).all()
    t, h, tau = orc.quantise_slots(_problem(wl), 5, 1_000_000)
    for b in range(1, 6):                       # beta = 1: b lone requests' time
        assert (t[b] == b * t[1]).all() and (h[b] == b * h[1]).all()
    dead = tau[1] == INF
    for b in range(1, 6):
        # a link carries b activations: ceil(b x) lies in [b ceil(x) - (b - 1), b ceil(x)]
        assert ((tau[b] == INF) == dead).all()
        fin = ~dead
        assert (tau[b][fin] <= b * tau[1][fin]).all()
        assert (tau[b][fin] + (b - 1) >= b * tau[1][fin]).all()


def test_link_time_of_b_activations_matches_the_paper_example(orc):
    """20 kB over 100 Mbps takes 1.6 ms (Sec. 4.1); b of them take 1.6 b ms."""
    wl = workload.random_small(6, M=2, N=3, P=1, k_max=1)
    pr = _problem(wl)
    pr["bw_Bps"] = np.full(4, 12_500_000, dtype=np.uint64)
    pr["congestion_ppm"] = np.full(4, 1_000_000, dtype=np.uint32)
    pr["act_bytes"] = np.array([20_000, 20_000], dtype=np.uint64)
    _, _, tau = orc.quantise_slots(pr, 8, 125_000)
    for b in range(1, 9):
        assert tau[b][0, 1] == 1_600_000 * b


def _fixed_role_optimum(wl, labels):
    """min over every role vector of the fixed-role fitness (eval_population),
    per genome, with the smallest decode bitmask among ties."""
    P, K = labels.shape[0], wl.k_max
    best = []
    for p in range(P):
        used = sorted({int(x) for x in labels[p] if x < K})
        cands = []
        for bits in itertools.product((0, 1), repeat=len(used)):
            roles = np.zeros((1, K), np.uint8)
            for q, b in zip(used, bits):
                roles[0, q] = b
            sol = oracle.eval_population(wl.subset([p]), labels[p:p + 1], roles)
            mask = sum(1 << q for q, b in zip(used, bits) if b)
            cands.append((int(sol["w"][0]), int(sol["phase"][0]), mask))
        best.append(min(cands))
    return best


@pytest.mark.parametrize("seed", range(6))
def test_one_slot_search_equals_enumeration_of_fixed_roles(orc, seed):
    """b_max = 1 and no KV bytes: the search's optimum is the best of the
    fixed-role fitness over every role vector."""
    wl = workload.random_small(40 + seed, M=10, N=16, P=6, k_max=4, mem_hi_layers=12,
                               zero_bw_frac=0.1)
    sm = dict(b_max=1, beta_ppm=300_000, kv_bytes_per_block_slot=0)
    got = orc.search_roles(wl, sm)
    want = _fixed_role_optimum(wl, wl.labels)
    for p in range(wl.population):
        mask = sum(1 << q for q in range(wl.k_max) if got["roles"][p, q])
        assert (int(got["w"][p]), int(got["phase"][p]), mask) == want[p]
    # prefill and one-slot decode DPs are the plain solve with all-prefill /
    # all-decode roles
    for r in (0, 1):
        roles = np.full((wl.population, wl.k_max), r, np.uint8)
        sol = oracle.eval_population(wl, wl.labels, roles)
        assert (got["T_all"][:, :, r] == sol["T"]).all()
        assert (got["Lambda_all"][:, :, r] == sol["Lambda"]).all()


@pytest.mark.parametrize("floor", ["none", "median"])
def test_single_device_clusters_in_closed_form(orc, floor):
    """One device per cluster: T_b = its block times + head time when its
    blocks, their b KV slots and the head fit, and the kept slot count is the
    largest b whose T_b (= Lambda_b) meets the QoS floor."""
    M = N_ = 8
    wl = workload.random_small(77, M=M, N=N_, P=1, k_max=M, mem_lo_layers=7, mem_hi_layers=14)
    wl.labels = np.arange(M, dtype=np.uint8)[None]
    kv = int(wl.layer_bytes.mean()) // 8
    sm = dict(b_max=9, beta_ppm=200_000, kv_bytes_per_block_slot=kv)
    t, h, _ = orc.quantise_slots(_problem(wl), 9, 200_000)
    wl.min_tps_milli = 0
    if floor == "median":
        # a floor that some slot counts meet and others miss
        T = orc.search_roles(wl, sm)["T_all"][0, :, 1:]
        wl.min_tps_milli = 10**12 // int(np.median(T[T != INF]))
    fp = wl.fitness_params()
    lam = 10**12 // fp["min_tps_milli"] if fp["min_tps_milli"] else INF
    got = orc.search_roles(wl, sm)
    W = int(wl.layer_bytes.sum())
    n_slots_seen = 0
    for d in range(M):
        for r in range(10):
            slots = 1 if r == 0 else r
            fits = W + N_ * kv * slots + int(wl.head_bytes) <= int(wl.mem_bytes[d])
            want = int(t[r, d].sum()) + int(h[r, d]) if fits else INF
            assert int(got["T_all"][0, d, r]) == want
            assert int(got["Lambda_all"][0, d, r]) == want
        ok = [b for b in range(1, 10) if got["T_all"][0, d, b] != INF and
              got["T_all"][0, d, b] <= lam]
        if got["roles"][0, d]:
            assert got["slots"][0, d] == (max(ok) if ok else 0)
            n_slots_seen += 1
        else:
            assert got["slots"][0, d] == 0
    assert n_slots_seen >= 1


def test_slot_count_never_lowers_the_optimum(orc):
    """More slots mean more time per block and link and more bytes per
    block, so T and feasibility can only get worse as b grows."""
    wl = workload.random_small(9, M=14, N=24, P=8, k_max=3, mem_hi_layers=20, zero_bw_frac=0.05)
    sm = workload.slot_model(wl, b_max=7)
    T = orc.search_roles(wl, sm)["T_all"]
    for b in range(2, 8):
        assert (T[:, :, b] >= T[:, :, b - 1]).all()
    assert (T[:, :, 1:] != INF).any()


def test_symmetric_clusters_tie_to_the_smallest_decode_set(orc):
    """Two identical single-device clusters: either one can decode; the tie
    goes to the assignment whose decode bitmask is smaller (cluster 0)."""
    wl = workload.random_small(12, M=2, N=6, P=1, k_max=2, layer_var=False, mem_hi_layers=30,
                               cong_full=True)
    wl.speed_flops[:] = wl.speed_flops[0]
    wl.mem_bytes[:] = wl.mem_bytes.max()
    wl.labels = np.array([[0, 1]], dtype=np.uint8)
    wl.min_tps_milli = 0
    sm = dict(b_max=3, beta_ppm=100_000, kv_bytes_per_block_slot=0)
    got = orc.search_roles(wl, sm)
    assert (got["T_all"][0, 0] == got["T_all"][0, 1]).all()
    assert list(got["roles"][0]) == [1, 0] and got["w"][0] != INF


def test_empty_clusters_are_left_out(orc):
    wl = workload.random_small(13, M=6, N=10, P=3, k_max=5, mem_hi_layers=30)
    wl.labels = np.array([[0, 0, 0, 2, 2, 2], [1, 1, 1, 1, 1, 1], [4, 4, 4, 9, 9, 9]],
                         dtype=np.uint8)
    got = orc.search_roles(wl, workload.slot_model(wl, b_max=4))
    for p, used in enumerate(({0, 2}, {1}, {4})):
        for q in range(5):
            if q not in used:
                assert (got["T_all"][p, q] == INF).all()
                assert got["roles"][p, q] == 0 and got["slots"][p, q] == 0
    # one cluster cannot cover both roles
    assert got["w"][1] == INF and got["phase"][1] == INF


def _every_role_vector_optimum(wl, got, p):
    """b_max = 1: the smallest (w, phase, decode bitmask) over every role
    vector of genome p's non-empty clusters, each scored by the pinned
    fixed-role fitness on the search's own prefill (index 0) and one-slot
    decode (index 1) DP results."""
    K = wl.k_max
    used = sorted({int(x) for x in wl.labels[p] if x < K})
    n = len(used)
    bits = ((np.arange(1 << n)[:, None] >> np.arange(n)[None, :]) & 1).astype(np.uint8)
    roles = np.zeros((1 << n, K), np.uint8)
    roles[:, used] = bits
    T = np.where(roles == 1, got["T_all"][p, :, 1], got["T_all"][p, :, 0])
    L = np.where(roles == 1, got["Lambda_all"][p, :, 1], got["Lambda_all"][p, :, 0])
    f = oracle.fitness(T, L, roles, **wl.fitness_params())
    mask = (roles.astype(np.int64) << np.arange(K, dtype=np.int64)[None, :]).sum(axis=1)
    i = np.lexsort((mask, f["phase"], f["w"]))[0]
    return int(f["w"][i]), int(f["phase"][i]), int(mask[i])


@pytest.mark.parametrize("K", [17, 18])
def test_search_past_sixteen_clusters_equals_every_role_vector(orc, K):
    """More than 16 non-empty clusters, some with a prefill rate but no
    decode rate (a QoS floor set at the median decode Lambda): the search,
    which enumerates only clusters with a decode rate, finds the optimum of
    all 2^K role vectors."""
    wl = workload.random_small(900 + K, M=3 * K, N=10, P=2, k_max=K, mem_lo_layers=3,
                               mem_hi_layers=14, zero_bw_frac=0.05)
    rng = np.random.default_rng(K)
    wl.labels = np.stack([rng.permutation(np.concatenate([np.arange(K), rng.integers(0, K, 2 * K)]))
                          for _ in range(2)]).astype(np.uint8)     # every cluster non-empty
    sm = dict(b_max=1, beta_ppm=0, kv_bytes_per_block_slot=0)
    wl.min_tps_milli = 0
    L1 = orc.search_roles(wl, sm)["Lambda_all"][:, :, 1]
    wl.min_tps_milli = max(1, 10**12 // int(np.median(L1[L1 != INF])))
    got = orc.search_roles(wl, sm)
    lam_max = 10**12 // wl.min_tps_milli
    prefill_only = (got["T_all"][:, :, 0] != INF) & (got["Lambda_all"][:, :, 1] > lam_max)
    assert prefill_only.sum() >= 2
    for p in range(wl.population):
        assert len({int(x) for x in wl.labels[p]}) == K
        mask = sum(1 << q for q in range(K) if got["roles"][p, q])
        assert (int(got["w"][p]), int(got["phase"][p]), mask) == \
            _every_role_vector_optimum(wl, got, p), p


def test_search_with_more_than_24_free_clusters_is_not_searched(orc):
    """Single-device clusters on devices that each hold the model, no QoS
    floor: every cluster has a decode rate.  24 of them are searched (2^24
    role sets); 25 are not: roles 0, slots 0xFF, w = phase = INF."""
    M = N_ = 25
    wl = workload.random_small(501, M=M, N=N_, P=2, k_max=M, mem_lo_layers=60,
                               mem_hi_layers=80, head=False)
    wl.min_tps_milli = 0
    sm = dict(b_max=2, beta_ppm=125_000, kv_bytes_per_block_slot=0)
    labels = np.tile(np.arange(M, dtype=np.uint8), (2, 1))
    labels[0, 7] = 3                                   # 24 clusters
    got = orc.search_roles(wl, sm, labels=labels)
    assert (got["T_all"][:, :, 1:] != INF).all(axis=2).sum(axis=1).tolist() == [24, 25]
    assert got["w"][0] != INF and got["roles"][0].sum() >= 1 and (got["slots"][0] <= 2).all()
    assert got["w"][1] == INF and got["phase"][1] == INF
    assert (got["roles"][1] == 0).all() and (got["slots"][1] == 0xFF).all()
