"""GPU parity for the role and slot search (Algorithm 2's inner loop).

e2_search_roles solves every cluster for prefill and for every decode slot
count, keeps the largest slot count that is feasible and meets the QoS
floor, and brute-forces the role assignment; every output (all DP results,
roles, slot counts, w, phase) equals the CPU oracle bit for bit.
"""
import ctypes
import dataclasses

import numpy as np
import pytest

import oracle
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

pytestmark = pytest.mark.gpu
INF = (1 << 64) - 1


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    e2.lib()
    return torch, torch.device("cuda:0")


def _gpu_search(torch_dev, wl, sm, labels=None, ctx=None):
    torch, dev = torch_dev
    labels = wl.labels if labels is None else labels
    ctx = ctx or e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    L = torch.from_numpy(np.ascontiguousarray(labels)).to(dev)
    out = e2.e2_search_roles(ctx, L, wl.fitness_params(), wl.k_max, with_tables=True)
    torch.cuda.synchronize()
    return dict(T_all=e2.u64(out["T_all"]), Lambda_all=e2.u64(out["Lambda_all"]),
                roles=out["roles"].cpu().numpy(), slots=out["slots"].cpu().numpy(),
                w=e2.u64(out["w"]), phase=e2.u64(out["phase"]))


def _assert_equal(got, want, rows=None, tag=""):
    for k in ("T_all", "Lambda_all", "roles", "slots", "w", "phase"):
        g = got[k] if rows is None else got[k][rows]
        w = want[k]
        bad = np.argwhere(np.asarray(g != w).reshape(len(w), -1).any(axis=1)).ravel()
        assert bad.size == 0, f"{tag} {k}: {bad.size} genomes differ, first {bad[:5]}"


def test_search_random_parity(torch_dev):
    """48 seeded instances: slot counts 1-15, beta 0 to 1, no / small / large
    KV bytes, QoS floors on and off, dead links, unassigned devices."""
    rng = np.random.default_rng(909)
    for it in range(48):
        M = int(rng.integers(1, 40))
        N = int(rng.integers(1, 90))
        P = int(rng.integers(1, 10))
        k_max = int(rng.integers(1, 9))
        kw = dict(mem_lo_layers=float(rng.uniform(0.5, 3)),
                  mem_hi_layers=float(rng.uniform(3, 60)),
                  zero_bw_frac=float(rng.choice([0.0, 0.1])), head=bool(rng.integers(0, 2)),
                  layer_var=bool(rng.integers(0, 2)))
        wl = workload.random_small(5000 + it, M=M, N=N, P=P, k_max=k_max, **kw)
        labels = wl.labels.copy()
        labels[rng.uniform(size=labels.shape) < 0.05] = 200
        if rng.uniform() < 0.5:
            wl.min_tps_milli = 0
        kv = int(rng.choice([0, 1, 10**6, int(wl.layer_bytes.mean()) // 4]))
        sm = dict(b_max=int(rng.choice([1, 2, 4, 8, 15])),
                  beta_ppm=int(rng.choice([0, 125_000, 1_000_000])),
                  kv_bytes_per_block_slot=kv)
        print(f"search {it}: M={M} N={N} P={P} k_max={k_max} {sm}", flush=True)
        _assert_equal(_gpu_search(torch_dev, wl, sm, labels),
                      oracle.search_roles(wl, sm, labels), tag=f"it {it}")


def test_search_sixteen_clusters(torch_dev):
    """k_max = 16 with roomy devices: up to 2^16 role sets per genome."""
    wl = workload.random_small(31, M=64, N=20, P=6, k_max=16, mem_lo_layers=6,
                               mem_hi_layers=30)
    wl.min_tps_milli = 0
    sm = dict(b_max=4, beta_ppm=125_000, kv_bytes_per_block_slot=10**6)
    want = oracle.search_roles(wl, sm)
    free = (want["T_all"][:, :, 1:] != INF).any(axis=2).sum(axis=1)
    assert free.max() >= 12
    _assert_equal(_gpu_search(torch_dev, wl, sm), want, tag="k16")


def test_search_maximum_sizes(torch_dev):
    """256 devices, 255 blocks, 16 clusters, 15 decode slot counts with KV
    bytes: 16 role indices per cluster and one memory class per index."""
    wl = workload.random_small(12, M=256, N=255, P=2, k_max=16, mem_lo_layers=10,
                               mem_hi_layers=40)
    wl.min_tps_milli = 0
    sm = dict(b_max=15, beta_ppm=125_000, kv_bytes_per_block_slot=int(wl.layer_bytes.mean()) // 16)
    want = oracle.search_roles(wl, sm)
    assert (want["T_all"] != INF).sum() > 100 and (want["slots"] > 1).any()
    _assert_equal(_gpu_search(torch_dev, wl, sm), want, tag="max")


def test_search_past_sixteen_clusters(torch_dev):
    """k_max from 17 to 255: only clusters with a decode rate are
    enumerated, up to 24 of them per genome (2^24 role sets); genomes with
    more are not searched (slots 0xFF, w = phase = INF), on both sides."""
    rng = np.random.default_rng(1717)
    free_seen = []
    for it, K in enumerate((17, 20, 24, 31, 48, 64, 100, 255)):
        M = int(min(256, max(K, int(rng.integers(K // 2, 2 * K)))))
        N = int(rng.integers(4, 20))
        wl = workload.random_small(8100 + it, M=M, N=N, P=4, k_max=K,
                                   mem_lo_layers=float(N * rng.uniform(0.1, 0.5)),
                                   mem_hi_layers=float(N * rng.uniform(0.7, 1.5)),
                                   zero_bw_frac=0.05)
        if it % 3:
            wl.min_tps_milli = 0
        sm = dict(b_max=int(rng.choice([1, 3, 8])), beta_ppm=125_000,
                  kv_bytes_per_block_slot=int(rng.choice([0, 10**6])))
        print(f"search k_max={K}: M={M} N={N} {sm}", flush=True)
        want = oracle.search_roles(wl, sm)
        lam = 10**12 // wl.min_tps_milli if wl.min_tps_milli else INF
        F = ((want["T_all"][:, :, 1:] != INF) & (want["Lambda_all"][:, :, 1:] <= lam)).any(axis=2)
        free_seen += F.sum(axis=1).tolist()
        _assert_equal(_gpu_search(torch_dev, wl, sm), want, tag=f"k_max {K}")
    assert max(free_seen) > 24 and any(17 <= f <= 24 for f in free_seen), free_seen


def test_search_free_cluster_bound(torch_dev):
    """25 single-device clusters that each hold the model: with one device
    moved to another cluster (24 free clusters) the genome is searched over
    2^24 role sets; with all 25 it is not."""
    M = 25
    wl = workload.random_small(501, M=M, N=M, P=2, k_max=M, mem_lo_layers=60,
                               mem_hi_layers=80, head=False)
    wl.min_tps_milli = 0
    sm = dict(b_max=2, beta_ppm=125_000, kv_bytes_per_block_slot=0)
    labels = np.tile(np.arange(M, dtype=np.uint8), (2, 1))
    labels[0, 7] = 3
    want = oracle.search_roles(wl, sm, labels=labels)
    assert want["w"][0] != INF and want["w"][1] == INF and (want["slots"][1] == 0xFF).all()
    _assert_equal(_gpu_search(torch_dev, wl, sm, labels=labels), want, tag="bound")


@pytest.mark.parametrize("name,rows", [("c1_tiny_12dev_32L", None), ("c2_32dev_48L", None),
                                       ("c3_64dev_80L", 192), ("c4_128dev_80L", 128),
                                       ("c5_256dev_126L_ga", 64)])
def test_search_named_workloads(torch_dev, name, rows):
    print(f"search workload {name}", flush=True)
    wl = workload.make(name)
    sm = workload.slot_model(wl)
    got = _gpu_search(torch_dev, wl, sm)
    if rows is None:
        _assert_equal(got, oracle.search_roles(wl, sm), tag=name)
        return
    pick = np.sort(np.random.default_rng(17).choice(wl.population, rows, replace=False))
    sub = wl.subset(pick)
    _assert_equal(got, oracle.search_roles(sub, sm), rows=pick, tag=name)
    assert (got["slots"] > 1).any()


def test_plain_context_searches_one_slot(torch_dev):
    """A context without a slot model searches roles with one decode slot
    and no KV bytes."""
    wl = workload.make("c2_32dev_48L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    got = _gpu_search(torch_dev, wl, None, ctx=ctx)
    want = oracle.search_roles(wl, dict(b_max=1, beta_ppm=0, kv_bytes_per_block_slot=0))
    _assert_equal(got, want, tag="plain ctx")


def test_fixed_roles_on_a_slot_context(torch_dev):
    """e2_solve_partitions on a slot context solves prefill clusters at role
    index 0 and decode clusters at index 1, each with one request's KV
    bytes."""
    torch, dev = torch_dev
    wl = workload.make("c2_32dev_48L")
    sm = workload.slot_model(wl, b_max=3)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), sm)
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    sol = e2.e2_solve_partitions(ctx, L, R)
    torch.cuda.synchronize()
    want = oracle.search_roles(wl, sm)
    idx = (wl.roles != 0).astype(np.int64)
    T = np.take_along_axis(want["T_all"], idx[:, :, None], axis=2)[:, :, 0]
    Lam = np.take_along_axis(want["Lambda_all"], idx[:, :, None], axis=2)[:, :, 0]
    assert (e2.u64(sol["T"]) == T).all() and (e2.u64(sol["Lambda"]) == Lam).all()


def test_search_empty_population_and_bad_arguments(torch_dev):
    torch, dev = torch_dev
    wl = workload.random_small(2, M=5, N=6, P=1, k_max=2)
    ctx = e2.e2_ctx_create_slots(wl.problem_arrays(), workload.slot_model(wl, b_max=2))
    L = torch.zeros((0, 5), dtype=torch.uint8, device=dev)
    out = e2.e2_search_roles(ctx, L, wl.fitness_params(), 2)
    torch.cuda.synchronize()
    assert out["w"].numel() == 0
    L = torch.zeros((1, 5), dtype=torch.uint8, device=dev)
    with pytest.raises(e2.E2Error):
        e2.e2_search_roles(ctx, L, wl.fitness_params(), 256)       # k_max past 255
    T = torch.empty((1, 2, 3), dtype=torch.int64, device=dev)
    fp = e2.e2_fitness_params(1, 1, 0)
    r = torch.empty((1, 2), dtype=torch.uint8, device=dev)
    w = torch.empty(1, dtype=torch.int64, device=dev)
    rc = e2.lib().e2_search_roles(ctx.handle, None, 1, 2, ctypes.c_void_p(L.data_ptr()),
                                  ctypes.byref(fp), ctypes.c_void_p(r.data_ptr()),
                                  ctypes.c_void_p(r.data_ptr()), ctypes.c_void_p(w.data_ptr()),
                                  ctypes.c_void_p(w.data_ptr()), ctypes.c_void_p(T.data_ptr()),
                                  None)
    assert rc == e2.E2_EINVAL                                    # T_all without Lambda_all
    bad = dict(b_max=16, beta_ppm=0, kv_bytes_per_block_slot=0)
    with pytest.raises(e2.E2Error):
        e2.e2_ctx_create_slots(wl.problem_arrays(), bad)


def _one_ns_clusters(seed, M, k_max):
    """Two-block models on devices fast enough that every block takes 1 ns:
    clusters of one or two devices reach T = 1, the largest rate (2^50), so
    a genome's rate sums pass 2^53, where doubles stop being exact."""
    wl = workload.random_small(seed, M=M, N=2, P=6, k_max=k_max, mem_lo_layers=3,
                               mem_hi_layers=6)
    wl = dataclasses.replace(wl, speed_flops=np.full(wl.n_dev, 10**15, np.uint64),
                             layer_flops=np.ones_like(wl.layer_flops),
                             head_flops=np.zeros(2, np.uint64), act_bytes=np.zeros(2, np.uint64))
    wl.min_tps_milli = 0
    return wl


def test_search_rate_sums_past_2_53(torch_dev):
    """The role search's rate divisions at their largest sums (16 clusters of
    rate up to 2^50)."""
    wl = _one_ns_clusters(78, 32, 16)
    sm = dict(b_max=1, beta_ppm=0, kv_bytes_per_block_slot=0)
    want = oracle.search_roles(wl, sm)
    t = want["T_all"][:, :, 0]
    sums = [sum((1 << 50) // int(x) for x in row if x != INF) for row in t]
    assert max(sums) > 1 << 53
    _assert_equal(_gpu_search(torch_dev, wl, sm), want, tag="rates")


def test_fitness_rate_sums_past_2_53(torch_dev):
    """The fixed-role fitness at rate sums past 2^54 (40 clusters)."""
    torch, dev = torch_dev
    wl = _one_ns_clusters(79, 80, 40)
    want = oracle.eval_population(wl)
    fin = want["T"][want["T"] != INF]
    assert (fin == 1).sum() > 60
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    for k in ("w", "phase", "s_p", "s_d"):
        assert (e2.u64(fit[k]) == want[k]).all(), k


def test_search_with_chains_past_64_devices(torch_dev):
    """The role and slot search (every role index of every cluster) on
    clusters of about 70-130 devices: the long-chain kernel in search mode."""
    wl = workload.random_small(4401, M=256, N=140, P=2, k_max=3, mem_lo_layers=2,
                               mem_hi_layers=8)
    wl.min_tps_milli = 0
    sm = dict(b_max=3, beta_ppm=125_000, kv_bytes_per_block_slot=10**6)
    print("search long chains", flush=True)
    want = oracle.search_roles(wl, sm)
    assert (want["T_all"] != INF).any()
    _assert_equal(_gpu_search(torch_dev, wl, sm), want, tag="long search")
