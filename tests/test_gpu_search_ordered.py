"""GPU parity for the role and slot search on two-chromosome genomes, and
Algorithm 2's generation on the paper's genome (App. A).

e2_search_roles_ordered solves every replica (its run of the ordering) for
prefill and for every decode slot count, keeps the largest slot count that is
feasible and meets the QoS floor, and brute-forces the role assignment; every
output equals the CPU oracle bit for bit.  One GPU generation then chains the
search into e2_ga_step_ordered: the bred genomes carry the roles the search
chose, with the search's (w, phase) as fitness keys.
"""
import numpy as np
import pytest

import oracle
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

pytestmark = pytest.mark.gpu
INF = (1 << 64) - 1
KEYS = ("T_all", "Lambda_all", "roles", "slots", "w", "phase")


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    e2.lib()
    return torch, torch.device("cuda:0")


def _gpu(torch_dev, ctx, wl, order, sizes):
    torch, dev = torch_dev
    O = torch.from_numpy(np.ascontiguousarray(order)).to(dev)
    S = torch.from_numpy(np.ascontiguousarray(sizes)).to(dev)
    out = e2.e2_search_roles_ordered(ctx, O, S, wl.fitness_params(), with_tables=True)
    torch.cuda.synchronize()
    return dict(T_all=e2.u64(out["T_all"]), Lambda_all=e2.u64(out["Lambda_all"]),
                roles=out["roles"].cpu().numpy(), slots=out["slots"].cpu().numpy(),
                w=e2.u64(out["w"]), phase=e2.u64(out["phase"]))


def _assert_equal(got, want, rows=None, tag=""):
    for k in KEYS:
        g = got[k] if rows is None else got[k][rows]
        w = want[k]
        bad = np.argwhere(np.asarray(g != w).reshape(len(w), -1).any(axis=1)).ravel()
        assert bad.size == 0, f"{tag} {k}: {bad.size} genomes differ, first {bad[:5]}"


def _random_genomes(rng, P, M, K):
    order = np.stack([rng.permutation(M) for _ in range(P)]).astype(np.uint8)
    sizes = np.zeros((P, K), dtype=np.uint16)
    for p in range(P):
        left = M + int(rng.integers(-2, 3))          # short of M or past it
        for q in range(K):
            if left <= 0:
                break
            if rng.uniform() < 0.15:
                continue                             # an empty slot
            s = min(int(rng.integers(1, 6)), left)
            sizes[p, q] = s
            left -= s
    bad = rng.uniform(size=order.shape) < 0.02       # ids that are not devices
    order[bad] = 250
    return order, sizes


def test_search_ordered_random_parity(torch_dev):
    rng = np.random.default_rng(4242)
    for it in range(40):
        M = int(rng.integers(1, 48))
        N = int(rng.integers(1, 90))
        P = int(rng.integers(1, 10))
        K = int(rng.integers(1, 17))
        kw = dict(mem_lo_layers=float(rng.uniform(0.5, 3)),
                  mem_hi_layers=float(rng.uniform(3, 60)),
                  zero_bw_frac=float(rng.choice([0.0, 0.1])), head=bool(rng.integers(0, 2)),
                  layer_var=bool(rng.integers(0, 2)))
        wl = workload.random_small(7000 + it, M=M, N=N, P=P, k_max=K, **kw)
        if rng.uniform() < 0.5:
            wl.min_tps_milli = 0
        kv = int(rng.choice([0, 1, 10**6, int(wl.layer_bytes.mean()) // 4]))
        sm = dict(b_max=int(rng.choice([1, 2, 4, 8, 15])),
                  beta_ppm=int(rng.choice([0, 125_000, 1_000_000])),
                  kv_bytes_per_block_slot=kv)
        order, sizes = _random_genomes(rng, P, M, K)
        print(f"ordered search {it}: M={M} N={N} P={P} k_max={K} {sm}", flush=True)
        ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
        _assert_equal(_gpu(torch_dev, ctx, wl, order, sizes),
                      oracle.search_roles_ordered(wl, sm, order, sizes), tag=f"it {it}")


def test_search_ordered_many_replica_slots(torch_dev):
    """17 to 96 replica slots: the search runs over the replicas with a
    decode rate only (at most 24; genomes with more are not searched)."""
    rng = np.random.default_rng(96)
    for it, K in enumerate((17, 24, 40, 96)):
        M = int(rng.integers(K, min(256, 2 * K) + 1))
        N = int(rng.integers(4, 16))
        wl = workload.random_small(9100 + it, M=M, N=N, P=4, k_max=K, mem_lo_layers=1,
                                   mem_hi_layers=float(2 * N))
        wl.min_tps_milli = 0
        sm = dict(b_max=4, beta_ppm=125_000, kv_bytes_per_block_slot=10**6)
        order, sizes = _random_genomes(rng, 4, M, K)
        print(f"ordered search k_max={K}: M={M} N={N}", flush=True)
        ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
        _assert_equal(_gpu(torch_dev, ctx, wl, order, sizes),
                      oracle.search_roles_ordered(wl, sm, order, sizes), tag=f"K {K}")


@pytest.mark.parametrize("name,rows", [("c1_tiny_12dev_32L", None), ("c2_32dev_48L", None),
                                       ("c3_64dev_80L", 160), ("c4_128dev_80L", 128),
                                       ("c5_256dev_126L_ga", 64)])
def test_search_ordered_named_workloads(torch_dev, name, rows):
    print(f"ordered search workload {name}", flush=True)
    wl = workload.make(name)
    op = workload.ordered_population(wl)
    sm = workload.slot_model(wl)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    got = _gpu(torch_dev, ctx, wl, op.order, op.sizes)
    if rows is None:
        _assert_equal(got, oracle.search_roles_ordered(wl, sm, op.order, op.sizes), tag=name)
        return
    pick = np.sort(np.random.default_rng(17).choice(wl.population, rows, replace=False))
    want = oracle.search_roles_ordered(wl, sm, op.order[pick], op.sizes[pick])
    _assert_equal(got, want, rows=pick, tag=name)
    assert (got["w"] != INF).any() and (got["slots"] > 0).any()


def test_search_then_breed_on_the_64_device_workload(torch_dev):
    """Algorithm 2's generation on the two-chromosome genome: the role and
    slot search scores every genome, then the App. A GA breeds from those
    keys with the roles the search chose.  Three generations; each bred
    population equals the oracle GA fed the same population, roles and keys,
    and sampled genomes' search results equal the oracle's."""
    torch, dev = torch_dev
    wl = workload.make("c3_64dev_80L")
    op = workload.ordered_population(wl)
    sm = workload.slot_model(wl)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    O = torch.from_numpy(op.order).to(dev)
    S = torch.from_numpy(op.sizes).to(dev)
    rng = np.random.default_rng(2)
    for g in range(3):
        print(f"generation {g}", flush=True)
        res = e2.e2_search_roles_ordered(ctx, O, S, wl.fitness_params())
        oo, so, qo = e2.e2_ga_step_ordered(ctx, O, S, res["roles"], res["w"], res["phase"],
                                           op.ga_params(wl, g))
        torch.cuda.synchronize()
        order, sizes = O.cpu().numpy(), S.cpu().numpy()
        roles = res["roles"].cpu().numpy()
        w, ph = e2.u64(res["w"]), e2.u64(res["phase"])
        pick = np.sort(rng.choice(wl.population, 48, replace=False))
        want = oracle.search_roles_ordered(wl, sm, order[pick], sizes[pick])
        for k, v in (("roles", roles), ("w", w), ("phase", ph)):
            assert np.array_equal(v[pick], want[k]), (g, k)
        eo, es, eq = oracle.ga_step_ordered(order, sizes, roles, w, ph, **op.ga_params(wl, g))
        assert np.array_equal(oo.cpu().numpy(), eo), g
        assert np.array_equal(so.cpu().numpy(), es), g
        assert np.array_equal(qo.cpu().numpy(), eq), g
        O, S = oo, so


def test_search_ordered_arguments(torch_dev):
    torch, dev = torch_dev
    wl = workload.random_small(3, M=6, N=8, P=2, k_max=17)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    order = torch.zeros((2, 6), dtype=torch.uint8, device=dev)
    sizes = torch.zeros((2, 256), dtype=torch.uint16, device=dev)
    with pytest.raises(e2.E2Error) as ei:                  # 256 replica slots: refused
        e2.e2_search_roles_ordered(ctx, order, sizes, wl.fitness_params())
    assert ei.value.code == e2.E2_EINVAL
    out = e2.e2_search_roles_ordered(ctx, order[:0], sizes[:0, :4], wl.fitness_params())
    torch.cuda.synchronize()
    assert out["w"].numel() == 0
