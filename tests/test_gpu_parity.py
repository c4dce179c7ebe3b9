"""GPU parity: every output of the HIP path equals the CPU oracle bit for bit.

All integer work, so the bar is exact equality on T, Lambda, master, layers
(Algorithm 1 per cluster), w, phase, S_P, S_D (Eq. 3-5) and the bred
genomes (GA step).  Inputs are seeded synthetic workloads; the named ones are
run at their full population in the same launch configuration the bench
uses, and checked on sampled individuals where the oracle would take long.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import pool
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


def _gpu_all(torch_dev, wl, labels=None, roles=None, ctx=None):
    torch, dev = torch_dev
    labels = wl.labels if labels is None else labels
    roles = wl.roles if roles is None else roles
    ctx = ctx or e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(np.ascontiguousarray(labels)).to(dev)
    R = torch.from_numpy(np.ascontiguousarray(roles)).to(dev)
    sol = e2.e2_solve_partitions(ctx, L, R)
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    out = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
               master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy())
    for k in ("w", "phase", "s_p", "s_d"):
        out[k] = e2.u64(fit[k])
    return out


def _oracle_all(wl, labels=None, roles=None):
    return oracle.eval_population(wl, labels, roles)


def _assert_equal(got, want, rows=None, tag=""):
    for k in ("T", "Lambda", "master", "layers", "w", "phase", "s_p", "s_d"):
        g = got[k] if rows is None else got[k][rows]
        w = want[k]
        bad = np.argwhere(np.asarray(g != w).reshape(len(w), -1).any(axis=1)).ravel()
        assert bad.size == 0, f"{tag} {k}: {bad.size} rows differ, first {bad[:5]}"


def _small_cases():
    cases = []
    rng = np.random.default_rng(2026)
    for seed in range(24):
        M = int(rng.integers(1, 48))
        N = int(rng.integers(1, 70))
        P = int(rng.integers(1, 24))
        k_max = int(rng.integers(1, 9))
        kw = dict(mem_hi_layers=float(rng.uniform(3, 60)), zero_bw_frac=0.1,
                  head=bool(seed % 3), layer_var=bool(seed % 2))
        cases.append((seed, M, N, P, k_max, kw))
    return cases


@pytest.mark.parametrize("case", _small_cases(), ids=lambda c: f"s{c[0]}-M{c[1]}-N{c[2]}")
def test_random_small_parity(torch_dev, case):
    seed, M, N, P, k_max, kw = case
    print(f"case seed={seed} M={M} N={N} P={P} k_max={k_max}", flush=True)
    wl = workload.random_small(seed, M=M, N=N, P=P, k_max=k_max, **kw)
    labels = wl.labels.copy()
    rng = np.random.default_rng(seed)
    labels[rng.uniform(size=labels.shape) < 0.05] = 250  # some devices unassigned
    _assert_equal(_gpu_all(torch_dev, wl, labels), _oracle_all(wl, labels), tag=f"seed {seed}")


def test_random_sweep_parity(torch_dev):
    """120 more seeded instances across regimes: identical blocks (many ties),
    no head (every master ties), tight and loose memory, dead links, long
    chains (one cluster), many clusters."""
    rng = np.random.default_rng(77)
    for it in range(120):
        M = int(rng.integers(1, 80))
        N = int(rng.integers(1, 130))
        P = int(rng.integers(1, 6))
        k_max = int(rng.choice([1, 2, 3, 5, 9, 17]))
        kw = dict(mem_lo_layers=float(rng.uniform(0.5, 3)),
                  mem_hi_layers=float(rng.uniform(3, 80)),
                  zero_bw_frac=float(rng.choice([0.0, 0.05, 0.3])),
                  head=bool(rng.integers(0, 2)), layer_var=bool(rng.integers(0, 2)),
                  cong_full=bool(rng.integers(0, 2)))
        wl = workload.random_small(1000 + it, M=M, N=N, P=P, k_max=k_max, **kw)
        if not kw["layer_var"] and rng.uniform() < 0.5:
            wl.speed_flops[:] = wl.speed_flops[0]
        print(f"sweep {it}: M={M} N={N} P={P} k_max={k_max} {kw}", flush=True)
        _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag=f"sweep {it}")


def _scaled(seed, M, N, P, k_max, block_ns, head_ns, zero_blocks=0, **kw):
    """random_small with every device at 1e9 FLOP/s, so that a block takes
    exactly its FLOPs in ns: block times drawn from [block_ns / 2, block_ns],
    the head `head_ns`, `zero_blocks` blocks of 0 ns."""
    wl = workload.random_small(seed, M=M, N=N, P=P, k_max=k_max, **kw)
    rng = np.random.default_rng(seed + 1)
    wl.speed_flops[:] = 10**9
    lf = rng.integers(block_ns // 2, block_ns + 1, size=(2, N)).astype(np.uint64)
    if zero_blocks:
        lf[:, rng.choice(N, zero_blocks, replace=False)] = 0
    wl.layer_flops = lf
    wl.head_flops = np.array([head_ns, head_ns], dtype=np.uint64)
    return wl


@pytest.mark.parametrize("block_ns,head_ns,zeros", [
    (1 << 14, 1 << 12, 0),              # u32 keys, far from the limit
    (0xFFFFFE // 12, 0, 3),             # u32 keys near 2^24, blocks of 0 ns
    (0xFFFFFE // 6, 0xFFFFFE // 7, 0),  # around the u32 / fp64 switch
    ((1 << 45) // 30, 1 << 20, 2),      # fp64 keys near 2^53, blocks of 0 ns
    ((1 << 45) // 12, 1 << 40, 0),      # beyond the fp64 limit: u64 reference path
])
def test_key_width_boundaries(torch_dev, block_ns, head_ns, zeros):
    """Values around the limits of the u32 and fp64 key paths (each problem
    takes the narrowest exact width), including blocks that take 0 ns."""
    for seed in range(3):
        wl = _scaled(300 + seed, M=20, N=24, P=6, k_max=3, block_ns=block_ns, head_ns=head_ns,
                     zero_blocks=zeros, mem_lo_layers=2, mem_hi_layers=14, cong_full=True)
        print(f"block_ns={block_ns} head_ns={head_ns} seed={seed}", flush=True)
        _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag=f"{block_ns}/{seed}")


@pytest.mark.parametrize("seed", [600, 601, 602])
def test_master_sweep_stops_and_runs_through(torch_dev, seed):
    """The DP's master sweep stops at the first master whose optimum equals
    the optimum with no head.  A heavy head gives clusters where it stops at
    the first device, where it stops later, and where no master reaches that
    bound, so that every master is solved: the chosen one is then the first
    device (no previous row), the last (its combine came last), one row
    before the last (its previous forward row is still in LDS), or two or
    more rows before it (its previous forward row is copied back from the
    global pool).  All of them equal the oracle."""
    wl = workload.random_small(seed, M=40, N=60, P=30, k_max=5, mem_lo_layers=2,
                               mem_hi_layers=20)
    wl = dataclasses.replace(wl, head_flops=np.array([4 * 10**11] * 2, np.uint64),
                             head_bytes=2 * 10**8)
    want = _oracle_all(wl)
    got = _gpu_all(torch_dev, wl)
    _assert_equal(got, want, tag=f"sweep {seed}")
    free = dataclasses.replace(wl, head_flops=np.zeros(2, np.uint64), head_bytes=0)
    T0 = _gpu_all(torch_dev, free)["T"]
    assert (T0 == _oracle_all(free)["T"]).all()
    kinds = set()
    for p in range(wl.population):
        for q in range(wl.k_max):
            ch = np.nonzero(wl.labels[p] == q)[0]
            if len(ch) == 0 or want["T"][p, q] == INF:
                continue
            pos = int(np.nonzero(ch == want["master"][p, q])[0][0]) + 1
            m = len(ch)
            if want["T"][p, q] == T0[p, q]:
                kinds.add("stop at 1" if pos == 1 else "stop later")
            elif pos == 1:
                kinds.add("through, master 1")
            elif pos == m:
                kinds.add("through, master m")
            elif pos == m - 1:
                kinds.add("through, one row past")
            else:
                kinds.add("through, two or more rows past")
    assert kinds == {"stop at 1", "stop later", "through, master 1", "through, master m",
                     "through, one row past", "through, two or more rows past"}


def test_paired_pass_band_widths_and_single_cells(torch_dev):
    """The master sweep pairs a master's combine with the forward row after
    it when the band holds at most 32 cells, and a sweep that stops there
    keeps the combine's row as the chosen master's first row; wider bands
    take separate passes; the optimum without a master and the chosen
    table's last cell are single-cell reductions whose windows can exceed
    one wave.  Tight memory (22-40 layers per device over 140 blocks) gives
    stops at masters with bands on both sides of 32 cells, roomy memory
    (30-90 layers over 120 blocks) wider bands and first-device windows past
    64 blocks; every kind occurs and every output equals the oracle."""
    import bench
    kinds = set()
    for seed, N, lo, hi in [(700, 140, 22, 40), (701, 140, 22, 40), (702, 140, 22, 40),
                            (700, 120, 30, 90)]:
        wl = workload.random_small(seed, M=24, N=N, P=12, k_max=5, mem_lo_layers=lo,
                                   mem_hi_layers=hi)
        wl = dataclasses.replace(wl, head_flops=np.array([2 * 10**11] * 2, np.uint64),
                                 head_bytes=10**8)
        print(f"paired-pass case seed={seed} N={N} memory {lo}-{hi} layers", flush=True)
        want = _oracle_all(wl)
        _assert_equal(_gpu_all(torch_dev, wl), want, tag=f"paired {seed}")
        free = dataclasses.replace(wl, head_flops=np.zeros(2, np.uint64), head_bytes=0)
        T0 = _oracle_all(free)["T"]
        _, _, cap = bench.window_tables(wl)
        for p in range(wl.population):
            for q in range(wl.k_max):
                ch = np.nonzero(wl.labels[p] == q)[0]
                m = len(ch)
                if m == 0 or want["T"][p, q] == INF:
                    continue
                c0 = cap[0][ch]
                pre = np.concatenate([[0], np.cumsum(c0)])
                mu = int(np.nonzero(ch == want["master"][p, q])[0][0]) + 1
                lo_b = max(mu - 1, N - 1 - (pre[m] - pre[mu]))
                hi_b = min(N - 1 - (m - mu), pre[mu] - 1)
                n = hi_b - lo_b + 1
                if want["T"][p, q] == T0[p, q] and 2 <= mu <= m - 1:
                    kinds.add("paired stop" if n <= 32 else
                              "stop, band 33-64" if n <= 64 else "stop, band past 64")
                elif want["T"][p, q] == T0[p, q]:
                    kinds.add("stop at the first or last device")
                else:
                    kinds.add("through")
                if c0[0] > 64:
                    kinds.add("T0 window past 64")
    assert kinds == {"paired stop", "stop, band 33-64", "stop, band past 64",
                     "stop at the first or last device", "through", "T0 window past 64"}


def test_uniform_layers_many_ties(torch_dev):
    """Identical blocks and devices: every master and many split points tie."""
    wl = workload.random_small(5, M=30, N=40, P=12, k_max=3, layer_var=False,
                               mem_hi_layers=80, cong_full=True)
    wl.speed_flops[:] = wl.speed_flops[0]
    _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag="ties")


@pytest.mark.parametrize("M,N,P,head", [(40, 200, 3, True), (64, 255, 2, True),
                                         (30, 126, 4, False), (48, 100, 2, True)])
def test_long_bands_keep_split_points_in_global_memory(torch_dev, M, N, P, head):
    """One chain of up to 64 roomy devices: its forward bands total up to
    (m - 1)(N - m + 1) cells, beyond the LDS copy of the split points, and
    the banded path keeps them in the wave's global table."""
    import bench
    wl = workload.random_small(70 + M + N, M=M, N=N, P=P, k_max=1, mem_lo_layers=40,
                               mem_hi_layers=150, head=head)
    _, _, cap = bench.window_tables(wl)
    assert (M - 1) * (N - M + 1) > bench.LDS_TB_CELLS and cap[0].min() >= 1
    print(f"long bands M={M} N={N}", flush=True)
    _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag=f"long bands M{M} N{N}")


def test_large_chain_uses_global_split_table(torch_dev):
    """m * N above the LDS copy of the split-point table (70 x 100)."""
    wl = workload.random_small(8, M=70, N=100, P=2, k_max=1, mem_lo_layers=3,
                               mem_hi_layers=30)
    _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag="global tb")


def test_maximum_sizes(torch_dev):
    """M = 256 devices, N = 255 blocks, k_max = 255 (mostly single-device
    clusters) and k_max = 4 (chains of ~64 devices)."""
    for k_max, P in ((255, 3), (4, 2)):
        print(f"max sizes k_max={k_max}", flush=True)
        wl = workload.random_small(9 + k_max, M=256, N=255, P=P, k_max=k_max,
                                   mem_lo_layers=2, mem_hi_layers=25)
        _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag=f"max k={k_max}")


def test_degenerate_shapes(torch_dev):
    for (M, N, k_max) in ((1, 1, 1), (1, 7, 1), (5, 1, 5), (5, 1, 1), (3, 2, 1)):
        wl = workload.random_small(M * 100 + N, M=M, N=N, P=4, k_max=k_max, mem_hi_layers=20)
        _assert_equal(_gpu_all(torch_dev, wl), _oracle_all(wl), tag=f"M{M} N{N}")


def test_empty_population_is_a_no_op(torch_dev):
    torch, dev = torch_dev
    wl = workload.random_small(1, M=4, N=4, P=1, k_max=2)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.zeros((0, 4), dtype=torch.uint8, device=dev)
    R = torch.zeros((0, 2), dtype=torch.uint8, device=dev)
    out = e2.e2_solve_partitions(ctx, L, R)
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    assert out["T"].numel() == 0 and fit["w"].numel() == 0


@pytest.mark.parametrize("name,rows", [
    ("c1_tiny_12dev_32L", None), ("c2_32dev_48L", None), ("c3_64dev_80L", None),
    ("c4_128dev_80L", 384), ("c5_256dev_126L_ga", 48)])
def test_named_workloads(torch_dev, name, rows):
    """Full population on the GPU; the oracle checks all rows or a sample."""
    print(f"workload {name}", flush=True)
    wl = workload.make(name)
    got = _gpu_all(torch_dev, wl)
    if rows is None:
        _assert_equal(got, _oracle_all(wl), tag=name)
        return
    rng = np.random.default_rng(99)
    pick = np.sort(np.r_[np.arange(8), rng.choice(np.arange(8, wl.population), rows - 8,
                                                   replace=False)])
    sub = wl.subset(pick)
    _assert_equal(got, _oracle_all(sub), rows=pick, tag=name)
    # the feasible fraction must be meaningful for this workload
    assert (got["T"] != INF).any() and (got["w"] != INF).any()


def test_population_order_does_not_matter(torch_dev):
    wl = workload.make("c2_32dev_48L")
    a = _gpu_all(torch_dev, wl)
    perm = np.random.default_rng(3).permutation(wl.population)
    b = _gpu_all(torch_dev, wl, wl.labels[perm], wl.roles[perm])
    for k in a:
        assert (a[k][perm] == b[k]).all(), k


def _gpu_ga(torch_dev, wl, labels, roles, w, phase, gen):
    torch, dev = torch_dev
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(np.ascontiguousarray(labels)).to(dev)
    R = torch.from_numpy(np.ascontiguousarray(roles)).to(dev)
    W = torch.from_numpy(np.asarray(w, np.uint64).view(np.int64)).to(dev)
    PH = torch.from_numpy(np.asarray(phase, np.uint64).view(np.int64)).to(dev)
    lo, ro = e2.e2_ga_step(ctx, L, R, W, PH, wl.ga_params(gen))
    torch.cuda.synchronize()
    return lo.cpu().numpy(), ro.cpu().numpy()


@pytest.mark.parametrize("n_elite,tk", [(1, 4), (0, 1), (7, 9), (256, 4)])
def test_ga_step_parity_random(torch_dev, n_elite, tk):
    rng = np.random.default_rng(n_elite * 31 + tk)
    P, M, k_max = 300, 37, 11
    wl = workload.random_small(4, M=M, N=8, P=P, k_max=k_max)
    wl.n_elite, wl.tournament_k = n_elite, tk
    wl.mutation_thresh_u32 = 1 << 28
    w = rng.integers(0, 50, size=P).astype(np.uint64)  # many ties in w
    w[rng.uniform(size=P) < 0.2] = np.uint64(INF)
    ph = rng.integers(0, 5, size=P).astype(np.uint64)
    got = _gpu_ga(torch_dev, wl, wl.labels, wl.roles, w, ph, 17)
    want = oracle.ga_step(wl.labels, wl.roles, w, ph, k_max, **wl.ga_params(17))
    assert (got[0] == want[0]).all() and (got[1] == want[1]).all()


def test_ga_step_rejects_outputs_overlapping_any_input(torch_dev):
    """Argument checks on the host, before any launch: an output may not
    share bytes with the labels, roles or the fitness keys it reads."""
    torch, dev = torch_dev
    wl = workload.random_small(2, M=4, N=5, P=2, k_max=2)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    W = torch.zeros(2, dtype=torch.int64, device=dev)
    PH = torch.zeros(2, dtype=torch.int64, device=dev)
    ga = wl.ga_params(0)
    for key in (W, PH):
        alias = key.view(torch.uint8)[:4].view(2, 2)       # roles_out inside w or phase
        with pytest.raises(e2.E2Error) as ei:
            e2.e2_ga_step(ctx, L, R, W, PH, ga, out=(torch.empty_like(L), alias))
        assert ei.value.code == e2.E2_EINVAL
    with pytest.raises(e2.E2Error):
        e2.e2_ga_step(ctx, L, R, W, PH, ga, out=(L, torch.empty_like(R)))
    lo, ro = e2.e2_ga_step(ctx, L, R, W, PH, ga)
    torch.cuda.synchronize()
    assert lo.shape == L.shape and ro.shape == R.shape


def test_ga_loop_on_the_16384_genome_workload(torch_dev):
    """Three generations of eval + GA on the GPU; each generation's GA output
    equals the oracle's GA fed the GPU's population and fitness, and sampled
    individuals' fitness equals the oracle's."""
    torch, dev = torch_dev
    wl = workload.make("c5_256dev_126L_ga")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    rng = np.random.default_rng(5)
    for g in range(3):
        print(f"generation {g}", flush=True)
        fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
        lo, ro = e2.e2_ga_step(ctx, L, R, fit["w"], fit["phase"], wl.ga_params(g))
        torch.cuda.synchronize()
        labels, roles = L.cpu().numpy(), R.cpu().numpy()
        w, ph = e2.u64(fit["w"]), e2.u64(fit["phase"])
        pick = np.sort(rng.choice(wl.population, 12, replace=False))
        sub = wl.subset(pick)
        want = oracle.eval_population(sub, labels[pick], roles[pick])
        assert (w[pick] == want["w"]).all() and (ph[pick] == want["phase"]).all()
        el, er = oracle.ga_step(labels, roles, w, ph, wl.k_max, **wl.ga_params(g))
        assert (lo.cpu().numpy() == el).all() and (ro.cpu().numpy() == er).all()
        L, R = lo, ro


def test_dp_timing_records_each_launch(torch_dev):
    """The profiling hook records one event pair per solve/eval call, up to
    the requested number, and leaves results unchanged."""
    torch, dev = torch_dev
    wl = workload.make("c2_32dev_48L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    want = _gpu_all(torch_dev, wl, ctx=ctx)
    e2.e2_ctx_dp_timing(ctx, 2)
    got = _gpu_all(torch_dev, wl, ctx=ctx)          # solve + eval: two launches
    extra = _gpu_all(torch_dev, wl, ctx=ctx)        # beyond the limit: not recorded
    n, ms = e2.e2_ctx_dp_elapsed(ctx)
    assert n == 2 and ms > 0
    e2.e2_ctx_dp_timing(ctx, 0)
    assert e2.e2_ctx_dp_elapsed(ctx) == (0, 0.0)
    for k in want:
        assert (got[k] == want[k]).all() and (extra[k] == want[k]).all(), k


def test_injected_hip_failure_enqueues_nothing(torch_dev):
    """With a HIP failure injected, e2_eval_population returns E2_EHIP and
    leaves its outputs as they were; the next call runs normally."""
    torch, dev = torch_dev
    wl = workload.make("c2_32dev_48L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    out = {k: torch.full((wl.population,), 12345, dtype=torch.int64, device=dev)
           for k in ("w", "phase", "s_p", "s_d")}
    assert e2.e2_debug_inject_hip_error(1) == 0
    with pytest.raises(e2.E2Error) as ei:
        e2.e2_eval_population(ctx, L, R, wl.fitness_params(), out=out)
    assert ei.value.code == e2.E2_EHIP
    torch.cuda.synchronize()
    assert all((v == 12345).all().item() for v in out.values())
    assert e2.e2_debug_inject_hip_error(0) == 0
    e2.e2_eval_population(ctx, L, R, wl.fitness_params(), out=out)
    torch.cuda.synchronize()
    want = oracle.eval_population(wl)
    for k in out:
        assert np.array_equal(e2.u64(out[k]), want[k]), k


@pytest.mark.parametrize("kind", ["labels", "two_chromosome"])
def test_genome_ranges_merge_to_the_whole_population(torch_dev, kind):
    """The one-GPU part of sharding the evaluation by genome range: the
    16384-genome population evaluated as four contiguous ranges (separate
    calls on slices of the same device arrays, uneven sizes) concatenates
    to the single call's every output, bit for bit."""
    torch, dev = torch_dev
    wl = workload.make("c5_256dev_126L_ga")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    fp = wl.fitness_params()
    if kind == "labels":
        ins = [torch.from_numpy(x).to(dev) for x in (wl.labels, wl.roles)]
        solve, evaluate = e2.e2_solve_partitions, e2.e2_eval_population
    else:
        op = workload.ordered_population(wl)
        ins = [torch.from_numpy(x).to(dev) for x in (op.order, op.sizes, op.roles)]
        solve, evaluate = e2.e2_solve_partitions_ordered, e2.e2_eval_population_ordered

    def run(lo, hi):
        part = [x[lo:hi] for x in ins]
        sol = solve(ctx, *part)
        fit = evaluate(ctx, *part, fp)
        torch.cuda.synchronize()
        out = dict(T=e2.u64(sol["T"]), Lambda=e2.u64(sol["Lambda"]),
                   master=sol["master"].cpu().numpy(), layers=sol["layers"].cpu().numpy())
        out.update({k: e2.u64(fit[k]) for k in ("w", "phase", "s_p", "s_d")})
        return out

    whole = run(0, wl.population)
    cuts = [0, 1000, 5096, 12001, wl.population]
    parts = [run(a, b) for a, b in zip(cuts[:-1], cuts[1:])]
    for k in whole:
        assert np.array_equal(np.concatenate([p[k] for p in parts]), whole[k]), k


@pytest.mark.parametrize("M,N,k_max,P", [(65, 80, 1, 2), (130, 200, 2, 2), (200, 255, 1, 1),
                                         (255, 255, 1, 1), (256, 126, 3, 2)])
def test_chains_past_64_devices(torch_dev, M, N, k_max, P):
    """Chains of 65 to 255 devices take the long-chain kernel (the banded
    path with four positions per lane) and equal the oracle on every
    output; roomy devices so that they are feasible."""
    print(f"long chains M={M} N={N} k_max={k_max}", flush=True)
    wl = workload.random_small(1300 + M + N, M=M, N=N, P=P, k_max=k_max,
                               mem_lo_layers=max(1.0, 3.0 * N / M), mem_hi_layers=max(4.0, 8.0 * N / M),
                               zero_bw_frac=0.0)
    want = _oracle_all(wl)
    chains = [int((wl.labels[p] == q).sum()) for p in range(P) for q in range(k_max)]
    assert max(chains) > 64 and (want["T"] != INF).any(), (chains, want["T"])
    _assert_equal(_gpu_all(torch_dev, wl), want, tag=f"long M{M} N{N}")


def test_long_chain_among_many_cluster_ids_takes_the_reference_path(torch_dev):
    """With fewer than 16 devices per cluster id on average the long-chain
    kernel is not launched; a 70-device chain then takes k_dp's reference
    path, with the same results."""
    M, N, k_max = 100, 90, 7
    wl = workload.random_small(1777, M=M, N=N, P=2, k_max=k_max, mem_lo_layers=2,
                               mem_hi_layers=10)
    rng = np.random.default_rng(17)
    labels = rng.integers(1, k_max, size=(2, M)).astype(np.uint8)
    for p in range(2):
        labels[p, rng.choice(M, 70, replace=False)] = 0          # one 70-device chain
    want = _oracle_all(wl, labels=labels)
    assert (want["T"][:, 0] != INF).any()
    _assert_equal(_gpu_all(torch_dev, wl, labels=labels), want, tag="reference long")


@pytest.mark.parametrize("keep", [False, True])
def test_one_context_on_two_streams_at_once(torch_dev, keep):
    """A context's tables are immutable after creation and every call's
    scratch belongs to its stream, so two streams may evaluate different
    populations with one context at the same time; each result equals the
    same call made alone."""
    torch, dev = torch_dev
    wl = workload.make("c4_128dev_80L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    if keep:
        e2.e2_ctx_keep_scratch(ctx)
    fp = wl.fitness_params()
    halves = [np.arange(0, 2048), np.arange(2048, 4096)]
    ins = [(torch.from_numpy(np.ascontiguousarray(wl.labels[h])).to(dev),
            torch.from_numpy(np.ascontiguousarray(wl.roles[h])).to(dev)) for h in halves]
    alone = []
    for L, R in ins:
        out = e2.e2_eval_population(ctx, L, R, fp)
        torch.cuda.synchronize()
        alone.append({k: e2.u64(v).copy() for k, v in out.items()})
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    torch.cuda.synchronize()
    for rep in range(3):
        outs = []
        for (L, R), st in zip(ins, streams):
            with torch.cuda.stream(st):
                outs.append(e2.e2_eval_population(ctx, L, R, fp))
        torch.cuda.synchronize()
        for a, b in zip(outs, alone):
            for k in b:
                assert np.array_equal(e2.u64(a[k]), b[k]), (rep, k)


def test_scratch_kept_per_stream_across_sizes_and_streams(torch_dev):
    """e2_ctx_keep_scratch: the context keeps one scratch buffer per stream
    for its first 16 streams and grows it when a call needs more; later
    streams allocate per call.  Calls of three sizes on the null stream and
    18 side streams, launched back to back and in two rounds (the second
    reuses every kept buffer, grown or not), with GA steps between the
    evaluations on one stream, each equal the oracle's rows; turning the
    setting off releases the buffers, and calls then allocate per call."""
    torch, dev = torch_dev
    wl = workload.make("c3_64dev_80L")
    want = pool.eval_population(wl)
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    e2.e2_ctx_keep_scratch(ctx)
    e2.e2_ctx_keep_scratch(ctx)          # a second call keeps the same cache
    fp = wl.fitness_params()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    streams = [torch.cuda.default_stream()] + [torch.cuda.Stream() for _ in range(18)]
    sizes = (64, wl.population, 300)
    torch.cuda.synchronize()
    for rnd in range(2):
        outs = []
        for i, st in enumerate(streams):
            n = sizes[(i + rnd) % 3]
            lo = (97 * i) % (wl.population - n + 1)
            with torch.cuda.stream(st):
                outs.append((lo, n, e2.e2_eval_population(ctx, L[lo:lo + n], R[lo:lo + n], fp)))
        torch.cuda.synchronize()
        for i, (lo, n, out) in enumerate(outs):
            for k in ("w", "phase", "s_p", "s_d"):
                assert np.array_equal(e2.u64(out[k]), want[k][lo:lo + n]), (rnd, i, k)
    # a GA step (small scratch) between two evaluations on one stream
    st = streams[3]
    with torch.cuda.stream(st):
        f = e2.e2_eval_population(ctx, L, R, fp)
        L2, R2 = e2.e2_ga_step(ctx, L, R, f["w"], f["phase"], wl.ga_params(0))
        f2 = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    bred = oracle.ga_step(wl.labels, wl.roles, e2.u64(f["w"]), e2.u64(f["phase"]), wl.k_max,
                          **wl.ga_params(0))
    assert np.array_equal(L2.cpu().numpy(), bred[0]) and np.array_equal(R2.cpu().numpy(), bred[1])
    for k in ("w", "phase"):
        assert np.array_equal(e2.u64(f2[k]), want[k]), k
    e2.e2_ctx_keep_scratch(ctx, False)   # waits, releases, back to per-call scratch
    out = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    assert np.array_equal(e2.u64(out["w"]), want["w"])
    ctx.close()


def test_per_thread_default_stream_from_two_host_threads_with_kept_scratch(torch_dev):
    """hipStreamPerThread is one handle that names each host thread's own
    stream, so a context never keeps scratch behind it: two threads that
    evaluate through it at once, with the setting on, each get the
    single-threaded result on every call."""
    import threading
    import types
    torch, dev = torch_dev
    wl = workload.make("c3_64dev_80L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    e2.e2_ctx_keep_scratch(ctx)
    fp = wl.fitness_params()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    want = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    want = {k: e2.u64(v).copy() for k, v in want.items()}
    per_thread = types.SimpleNamespace(cuda_stream=2)   # hipStreamPerThread
    halves = np.array_split(np.arange(wl.population), 2)
    results, errors = [[] for _ in halves], []

    def work(i):
        try:
            lo, hi = int(halves[i][0]), int(halves[i][-1]) + 1
            outs = [e2.e2_eval_population(ctx, L[lo:hi], R[lo:hi], fp, stream=per_thread)
                    for _ in range(6)]
            torch.cuda.synchronize()
            results[i] = [{k: e2.u64(v).copy() for k, v in o.items()} for o in outs]
        except Exception as exc:  # reported below, in the main thread
            errors.append(repr(exc))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i, rows in enumerate(halves):
        for rep, out in enumerate(results[i]):
            for k in want:
                assert np.array_equal(out[k], want[k][rows]), (i, rep, k)


@pytest.mark.parametrize("keep", [False, True])
def test_one_context_from_four_host_threads(torch_dev, keep):
    """A context may serve several host threads at once: four threads, each
    on its own stream, evaluate their quarter of a population through one
    context (the binding releases the interpreter lock inside the library
    calls); every result equals the single-threaded evaluation."""
    import threading
    torch, dev = torch_dev
    wl = workload.make("c3_64dev_80L")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    if keep:
        e2.e2_ctx_keep_scratch(ctx)
    fp = wl.fitness_params()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    want = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    want = {k: e2.u64(v).copy() for k, v in want.items()}
    quarters = np.array_split(np.arange(wl.population), 4)
    results, errors = [None] * 4, []

    def work(i):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                rows = quarters[i]
                for _ in range(5):
                    out = e2.e2_eval_population(ctx, L[rows[0]:rows[-1] + 1],
                                                R[rows[0]:rows[-1] + 1], fp)
                st.synchronize()
            results[i] = {k: e2.u64(v).copy() for k, v in out.items()}
        except Exception as exc:  # reported below, in the main thread
            errors.append(repr(exc))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for k in want:
        assert np.array_equal(np.concatenate([r[k] for r in results]), want[k]), k
