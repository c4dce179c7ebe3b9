"""GPU parity for two-chromosome genomes (the paper's App. A gene).

The ordered entry points solve each replica's chain in ordering order and
breed with the ordering crossover, grouping inheritance and the four
mutations; every output equals the CPU oracle bit for bit (integer work).
Inputs are seeded synthetic genomes; the named workloads run at full
population and are checked on sampled individuals where the oracle would
take long.
"""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

pytestmark = pytest.mark.gpu
INF = (1 << 64) - 1
KEYS = ("T", "Lambda", "master", "layers", "w", "phase", "s_p", "s_d")


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    e2.lib()
    return torch, torch.device("cuda:0")


def _to_dev(torch_dev, *arrays):
    torch, dev = torch_dev
    return [torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in arrays]


def _gpu_eval(torch_dev, wl, order, sizes, roles, ctx=None):
    torch, _ = torch_dev
    ctx = ctx or e2.e2_ctx_create(wl.problem_arrays())
    O, S, R = _to_dev(torch_dev, order, sizes, roles)
    sol = e2.e2_solve_partitions_ordered(ctx, O, S, R)
    fit = e2.e2_eval_population_ordered(ctx, O, S, R, wl.fitness_params())
    torch.cuda.synchronize()
    out = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
               master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy())
    for k in ("w", "phase", "s_p", "s_d"):
        out[k] = e2.u64(fit[k])
    return out


def _assert_equal(got, want, rows=None, tag=""):
    for k in KEYS:
        g = got[k] if rows is None else got[k][rows]
        w = want[k]
        bad = np.argwhere(np.asarray(g != w).reshape(len(w), -1).any(axis=1)).ravel()
        assert bad.size == 0, f"{tag} {k}: {bad.size} rows differ, first {bad[:5]}"


def _random_genomes(rng, P, M, k_max, planted=False):
    """Permutations with random groupings: runs of random sizes, some empty
    replicas between them, groupings that stop short of M (devices outside
    every replica) or run past it (clipped); optionally an id >= M planted
    in some orderings."""
    order = np.stack([rng.permutation(M) for _ in range(P)]).astype(np.uint8)
    sizes = np.zeros((P, k_max), np.uint16)
    for p in range(P):
        left = M + int(rng.integers(-M // 3, M // 3 + 1))
        for r in range(k_max):
            if left <= 0:
                break
            if rng.uniform() < 0.1:
                continue                      # an empty replica
            s = int(rng.integers(1, max(2, 2 * M // k_max + 2)))
            sizes[p, r] = min(s, left) if rng.uniform() < 0.9 else s
            left -= s
    roles = rng.integers(0, 2, size=(P, k_max)).astype(np.uint8)
    roles[rng.uniform(size=roles.shape) < 0.1] = 7      # any nonzero role is decode
    if planted and M < 256:
        for p in range(0, P, 3):
            order[p, int(rng.integers(0, M))] = int(rng.integers(M, 256))
    return order, sizes, roles


def test_ordered_random_parity(torch_dev):
    """80 seeded instances across sizes, memory regimes and link failures."""
    rng = np.random.default_rng(4242)
    for it in range(80):
        M = int(rng.integers(1, 90))
        N = int(rng.integers(1, 130))
        P = int(rng.integers(1, 12))
        k_max = int(rng.choice([1, 2, 3, 5, 9, 17, 64]))
        kw = dict(mem_lo_layers=float(rng.uniform(0.5, 3)),
                  mem_hi_layers=float(rng.uniform(3, 80)),
                  zero_bw_frac=float(rng.choice([0.0, 0.05, 0.3])),
                  head=bool(rng.integers(0, 2)), layer_var=bool(rng.integers(0, 2)))
        wl = workload.random_small(3000 + it, M=M, N=N, P=P, k_max=k_max, **kw)
        order, sizes, roles = _random_genomes(rng, P, M, k_max, planted=bool(it % 4 == 1))
        print(f"ordered {it}: M={M} N={N} P={P} k_max={k_max} {kw}", flush=True)
        _assert_equal(_gpu_eval(torch_dev, wl, order, sizes, roles),
                      oracle.eval_population_ordered(wl, order, sizes, roles), tag=f"it {it}")


def test_ordered_maximum_sizes(torch_dev):
    """M = 256, N = 255: single-device replicas (k_max = 255) and long chains
    (four replicas of ~64 devices)."""
    rng = np.random.default_rng(8)
    for k_max, P in ((255, 2), (4, 2)):
        print(f"ordered max sizes k_max={k_max}", flush=True)
        wl = workload.random_small(77 + k_max, M=256, N=255, P=P, k_max=k_max,
                                   mem_lo_layers=2, mem_hi_layers=25)
        order = np.stack([rng.permutation(256) for _ in range(P)]).astype(np.uint8)
        sizes = np.zeros((P, k_max), np.uint16)
        sizes[:, :] = 256 // k_max
        sizes[:, -1] += 256 - sizes[0].sum()
        _assert_equal(_gpu_eval(torch_dev, wl, order, sizes, wl.roles),
                      oracle.eval_population_ordered(wl, order, sizes, wl.roles),
                      tag=f"max k={k_max}")


def test_identity_ordering_matches_labelled_clusters(torch_dev):
    """The identity ordering cut into runs equals labels marking the same
    runs, through both GPU entry points."""
    wl = workload.make("c3_64dev_80L")
    P, M, k_max = wl.population, wl.n_dev, wl.k_max
    rng = np.random.default_rng(5)
    order = np.tile(np.arange(M, dtype=np.uint8), (P, 1))
    sizes = np.zeros((P, k_max), np.uint16)
    labels = np.zeros((P, M), np.uint8)
    for p in range(P):
        K = int(rng.integers(1, min(k_max, M) + 1))
        cuts = np.sort(rng.choice(np.arange(1, M), size=K - 1, replace=False))
        sz = np.diff(np.r_[0, cuts, M])
        sizes[p, :K] = sz
        labels[p] = np.repeat(np.arange(K), sz)
    got = _gpu_eval(torch_dev, wl, order, sizes, wl.roles)
    torch, _ = torch_dev
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L, R = _to_dev(torch_dev, labels, wl.roles)
    sol = e2.e2_solve_partitions(ctx, L, R)
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    assert (e2.u64(sol["T"]) == got["T"]).all() and (e2.u64(fit["w"]) == got["w"]).all()
    assert (sol["layers"].cpu().numpy() == got["layers"]).all()
    pick = np.arange(0, P, 17)
    want = oracle.eval_population_ordered(wl, order[pick], sizes[pick], wl.roles[pick])
    _assert_equal(got, want, rows=pick, tag="identity")


@pytest.mark.parametrize("name,rows", [
    ("c1_tiny_12dev_32L", None), ("c2_32dev_48L", None), ("c3_64dev_80L", None),
    ("c4_128dev_80L", 768), ("c5_256dev_126L_ga", 160)])
def test_ordered_named_workloads(torch_dev, name, rows):
    print(f"ordered workload {name}", flush=True)
    wl = workload.make(name)
    op = workload.ordered_population(wl)
    got = _gpu_eval(torch_dev, wl, op.order, op.sizes, op.roles)
    if rows is None:
        pick = np.arange(wl.population)
    else:
        rng = np.random.default_rng(31)
        pick = np.sort(np.r_[np.arange(4), rng.choice(np.arange(4, wl.population), rows - 4,
                                                       replace=False)])
    sub = op.subset(pick)
    want = oracle.eval_population_ordered(wl, sub.order, sub.sizes, sub.roles)
    _assert_equal(got, want, rows=None if rows is None else pick, tag=name)
    assert (got["T"] != INF).any()


def _gpu_ga(torch_dev, wl, order, sizes, roles, w, phase, params, ctx=None):
    torch, _ = torch_dev
    ctx = ctx or e2.e2_ctx_create(wl.problem_arrays())
    O, S, R = _to_dev(torch_dev, order, sizes, roles)
    W, PH = _to_dev(torch_dev, np.asarray(w, np.uint64).view(np.int64),
                    np.asarray(phase, np.uint64).view(np.int64))
    oo, so, ro = e2.e2_ga_step_ordered(ctx, O, S, R, W, PH, params)
    torch.cuda.synchronize()
    return oo.cpu().numpy(), so.cpu().numpy(), ro.cpu().numpy()


@pytest.mark.parametrize("M,k_max,n_elite,tk,mut,mx", [
    (37, 11, 1, 4, 1 << 30, 6),            # the paper's 30%-ish mutation rate
    (37, 11, 0, 1, 0xFFFFFFFF, 3),         # every child mutates: all four kinds
    (64, 64, 7, 9, 0xFFFFFFFF, 1),         # single-device regrowth
    (200, 5, 256, 4, 0xFFFFFFFF, 256),     # regrowth capped by the last slot
    (1, 1, 2, 2, 0xFFFFFFFF, 4),           # one device
    (2, 3, 0, 64, 0xFFFFFFFF, 2),
    (256, 255, 3, 4, 0xFFFFFFFF, 9),       # every ordering position in use
])
def test_ga_step_ordered_parity(torch_dev, M, k_max, n_elite, tk, mut, mx):
    print(f"ga ordered M={M} k_max={k_max} n_elite={n_elite} tk={tk}", flush=True)
    rng = np.random.default_rng(M * 7 + k_max)
    P = 300
    wl = workload.random_small(6, M=M, N=8, P=P, k_max=k_max)
    order, sizes, roles = _random_genomes(rng, P, M, k_max)
    w = rng.integers(0, 50, size=P).astype(np.uint64)        # many ties in w
    w[rng.uniform(size=P) < 0.2] = np.uint64(INF)
    ph = rng.integers(0, 5, size=P).astype(np.uint64)
    params = dict(seed=99 + M, generation=17, tournament_k=tk, mutation_thresh_u32=mut,
                  n_elite=n_elite, max_replica=mx)
    got = _gpu_ga(torch_dev, wl, order, sizes, roles, w, ph, params)
    want = oracle.ga_step_ordered(order, sizes, roles, w, ph, **params)
    for g_, w_, k in zip(got, want, ("order", "sizes", "roles")):
        bad = np.argwhere((g_ != w_).any(axis=1)).ravel()
        assert bad.size == 0, f"{k}: {bad.size} slots differ, first {bad[:5]}"


def test_ga_ordered_loop_on_the_16384_genome_workload(torch_dev):
    """Three generations of eval + GA on two-chromosome genomes: each GA
    output equals the oracle's GA fed the GPU's population and fitness, and
    sampled individuals' fitness equals the oracle's."""
    torch, _ = torch_dev
    wl = workload.make("c5_256dev_126L_ga")
    op = workload.ordered_population(wl)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    O, S, R = _to_dev(torch_dev, op.order, op.sizes, op.roles)
    rng = np.random.default_rng(6)
    for g in range(3):
        print(f"ordered generation {g}", flush=True)
        fit = e2.e2_eval_population_ordered(ctx, O, S, R, wl.fitness_params())
        oo, so, ro = e2.e2_ga_step_ordered(ctx, O, S, R, fit["w"], fit["phase"],
                                           op.ga_params(wl, g))
        torch.cuda.synchronize()
        order, sizes, roles = O.cpu().numpy(), S.cpu().numpy(), R.cpu().numpy()
        w, ph = e2.u64(fit["w"]), e2.u64(fit["phase"])
        pick = np.sort(rng.choice(wl.population, 10, replace=False))
        want = oracle.eval_population_ordered(wl, order[pick], sizes[pick], roles[pick])
        assert (w[pick] == want["w"]).all() and (ph[pick] == want["phase"]).all()
        eo, es, er = oracle.ga_step_ordered(order, sizes, roles, w, ph, **op.ga_params(wl, g))
        assert (oo.cpu().numpy() == eo).all() and (so.cpu().numpy() == es).all()
        assert (ro.cpu().numpy() == er).all()
        O, S, R = oo, so, ro


def test_ordered_empty_population_and_bad_arguments(torch_dev):
    torch, dev = torch_dev
    wl = workload.random_small(1, M=4, N=4, P=1, k_max=2)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    O = torch.zeros((0, 4), dtype=torch.uint8, device=dev)
    S = torch.zeros((0, 2), dtype=torch.uint16, device=dev)
    R = torch.zeros((0, 2), dtype=torch.uint8, device=dev)
    out = e2.e2_solve_partitions_ordered(ctx, O, S, R)
    fit = e2.e2_eval_population_ordered(ctx, O, S, R, wl.fitness_params())
    torch.cuda.synchronize()
    assert out["T"].numel() == 0 and fit["w"].numel() == 0
    # argument checks happen on the host, before any launch
    O, S, R = _to_dev(torch_dev, np.array([[0, 1, 2, 3]], np.uint8),
                      np.array([[2, 2]], np.uint16), np.array([[0, 1]], np.uint8))
    W = torch.zeros(1, dtype=torch.int64, device=dev)
    params = dict(seed=1, generation=0, tournament_k=2, mutation_thresh_u32=0, n_elite=0,
                  max_replica=0)
    with pytest.raises(e2.E2Error):
        e2.e2_ga_step_ordered(ctx, O, S, R, W, W, params)
    params["max_replica"] = 2
    with pytest.raises(e2.E2Error):        # outputs overlapping the inputs
        e2.e2_ga_step_ordered(ctx, O, S, R, W, W, params, out=(O, S.clone(), R.clone()))
    with pytest.raises(e2.E2Error) as ei:  # roles_out inside the fitness keys
        e2.e2_ga_step_ordered(ctx, O, S, R, W, W, params,
                              out=(O.clone(), S.clone(), W.view(torch.uint8)[:2].view(1, 2)))
    assert ei.value.code == e2.E2_EINVAL
    rc = e2.lib().e2_solve_partitions_ordered(ctx.handle, None, 1, 2, None, ctypes.c_void_p(
        S.data_ptr()), ctypes.c_void_p(R.data_ptr()), None, None, None, None)
    assert rc == e2.E2_EINVAL


def test_ordered_replicas_past_64_devices(torch_dev):
    """Replicas of 70 to 150 devices along the ordering (the long-chain
    kernel) equal the oracle."""
    M, N = 256, 160
    wl = workload.random_small(2901, M=M, N=N, P=2, k_max=3, mem_lo_layers=2, mem_hi_layers=6)
    rng = np.random.default_rng(29)
    order = np.stack([rng.permutation(M) for _ in range(2)]).astype(np.uint8)
    sizes = np.array([[70, 150, 36], [100, 90, 66]], dtype=np.uint16)
    roles = np.array([[0, 1, 0], [1, 0, 1]], dtype=np.uint8)
    print("ordered long replicas", flush=True)
    want = oracle.eval_population_ordered(wl, order, sizes, roles)
    assert (want["T"] != INF).any()
    _assert_equal(_gpu_eval(torch_dev, wl, order, sizes, roles), want, tag="long replicas")
