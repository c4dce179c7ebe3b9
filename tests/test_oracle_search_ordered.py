"""Pins for the oracle's role and slot search on two-chromosome genomes
(Algorithm 2's inner loop on the App. A gene).

Replicas are runs of the ordering chromosome, so an identity ordering cut
into runs must search exactly like label genomes that mark the same runs
(the label search is pinned in test_oracle_slots).  With one slot and no KV
bytes the search must equal the best of the already pinned fixed-role path
(oracle.eval_population_ordered) over every role vector, ties to the
smallest decode set.  A replica holding an id >= M has no DP result and no
rates, so it is prefill with slot 0.
"""
import numpy as np

import oracle
from paper_2606_03770_amd import workload

INF = (1 << 64) - 1
KEYS = ("T_all", "Lambda_all", "roles", "slots", "w", "phase")


def _runs(rng, M, K):
    """Replica sizes along an ordering: runs of 1..4, the last slots maybe
    empty, the grouping maybe short of M."""
    sizes = np.zeros(K, dtype=np.uint16)
    left = M - int(rng.integers(0, 3))
    for q in range(K):
        if left <= 0:
            break
        s = min(int(rng.integers(1, 5)), left)
        sizes[q] = s
        left -= s
    return sizes


def test_identity_ordering_searches_like_labels():
    rng = np.random.default_rng(31)
    for seed in range(8):
        M, N, K, P = int(rng.integers(3, 14)), int(rng.integers(3, 20)), int(rng.integers(2, 7)), 5
        wl = workload.random_small(seed, M=M, N=N, P=P, k_max=K, zero_bw_frac=0.1)
        sm = workload.slot_model(wl, b_max=int(rng.integers(1, 5)))
        order = np.tile(np.arange(M, dtype=np.uint8), (P, 1))
        sizes = np.stack([_runs(rng, M, K) for _ in range(P)])
        labels = np.full((P, M), 255, dtype=np.uint8)
        for p in range(P):
            off = 0
            for q in range(K):
                labels[p, off:off + int(sizes[p, q])] = q
                off += int(sizes[p, q])
        got = oracle.search_roles_ordered(wl, sm, order, sizes)
        want = oracle.search_roles(wl, sm, labels=labels)
        for k in KEYS:
            assert np.array_equal(got[k], want[k]), (seed, k)


def test_one_slot_search_is_the_best_fixed_role_vector():
    rng = np.random.default_rng(7)
    for seed in range(6):
        M, N, K, P = int(rng.integers(4, 12)), int(rng.integers(4, 16)), 5, 4
        wl = workload.random_small(100 + seed, M=M, N=N, P=P, k_max=K, zero_bw_frac=0.1)
        sm = dict(b_max=1, beta_ppm=0, kv_bytes_per_block_slot=0)
        order = np.stack([rng.permutation(M) for _ in range(P)]).astype(np.uint8)
        sizes = np.stack([_runs(rng, M, K) for _ in range(P)])
        got = oracle.search_roles_ordered(wl, sm, order, sizes)
        for p in range(P):
            best = None
            for mask in range(1 << K):      # increasing decode sets: the first best wins ties
                roles = np.array([[(mask >> q) & 1 for q in range(K)]], dtype=np.uint8)
                f = oracle.eval_population_ordered(wl, order[p:p + 1], sizes[p:p + 1], roles)
                key = (int(f["w"][0]), int(f["phase"][0]))
                if best is None or key < best[0]:
                    best = (key, mask)
            assert (int(got["w"][p]), int(got["phase"][p])) == best[0], (seed, p)
            nonempty = [q for q in range(K) if oracle.replica_range(sizes[p], q, M)[1] >
                        oracle.replica_range(sizes[p], q, M)[0]]
            mask = sum(int(got["roles"][p, q]) << q for q in range(K))
            # the search's decode set scores as well as the best one and, among
            # equal scores, every decode replica has a decode rate
            roles = np.array([[(mask >> q) & 1 for q in range(K)]], dtype=np.uint8)
            f = oracle.eval_population_ordered(wl, order[p:p + 1], sizes[p:p + 1], roles)
            assert (int(f["w"][0]), int(f["phase"][0])) == best[0]
            assert all(q in nonempty for q in range(K) if (mask >> q) & 1)


def test_replica_with_a_foreign_id_has_no_rates():
    wl = workload.random_small(9, M=8, N=10, P=1, k_max=3, mem_hi_layers=30)
    sm = workload.slot_model(wl, b_max=3)
    order = np.arange(8, dtype=np.uint8)[None, :].copy()
    order[0, 4] = 200                                  # not a device: replica 1 (4..5)
    sizes = np.array([[3, 3, 2]], dtype=np.uint16)
    got = oracle.search_roles_ordered(wl, sm, order, sizes)
    assert (got["T_all"][0, 1] == INF).all() and (got["Lambda_all"][0, 1] == INF).all()
    assert got["roles"][0, 1] == 0 and got["slots"][0, 1] == 0
    # the other replicas are searched as usual: the same as without replica 1's devices
    sizes2 = np.array([[3, 0, 2]], dtype=np.uint16)
    order2 = np.array([[0, 1, 2, 6, 7, 3, 4, 5]], dtype=np.uint8)
    ref = oracle.search_roles_ordered(wl, sm, order2, sizes2)
    for k in ("T_all", "Lambda_all"):
        assert np.array_equal(got[k][0, [0, 2]], ref[k][0, [0, 2]])
    assert got["w"][0] == ref["w"][0] and got["phase"][0] == ref["phase"][0]
