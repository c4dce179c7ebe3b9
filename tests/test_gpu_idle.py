"""GPU parity for the idle-device relaxation (e2_solve_partitions_idle,
e2_eval_population_idle): T, Lambda, master, layers and the fitness equal
the CPU oracle bit for bit, including clusters with more devices than
blocks, and the relaxation's invariant holds on the GPU's own results.
"""
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


def _gpu_idle(torch_dev, wl, labels=None, ctx=None):
    torch, dev = torch_dev
    labels = wl.labels if labels is None else labels
    ctx = ctx or e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(np.ascontiguousarray(labels)).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    sol = e2.e2_solve_partitions(ctx, L, R, objective="idle")
    fit = e2.e2_eval_population(ctx, L, R, wl.fitness_params(), objective="idle")
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


def test_idle_random_parity(torch_dev):
    """40 instances; a third have fewer blocks than a cluster's devices."""
    rng = np.random.default_rng(6161)
    for it in range(40):
        M = int(rng.integers(1, 40))
        N = int(rng.integers(1, 6)) if it % 3 == 0 else int(rng.integers(1, 80))
        P = int(rng.integers(1, 8))
        k_max = int(rng.integers(1, 6))
        kw = dict(mem_lo_layers=float(rng.uniform(0.5, 3)),
                  mem_hi_layers=float(rng.uniform(3, 60)),
                  zero_bw_frac=float(rng.choice([0.0, 0.1, 0.3])),
                  head=bool(rng.integers(0, 2)), layer_var=bool(rng.integers(0, 2)))
        wl = workload.random_small(9000 + it, M=M, N=N, P=P, k_max=k_max, **kw)
        labels = wl.labels.copy()
        labels[rng.uniform(size=labels.shape) < 0.05] = 230
        print(f"idle {it}: M={M} N={N} P={P} k_max={k_max} {kw}", flush=True)
        _assert_equal(_gpu_idle(torch_dev, wl, labels), oracle.eval_population_idle(wl, labels),
                      tag=f"idle {it}")


def test_idle_maximum_sizes(torch_dev):
    """256 devices, 255 blocks, four chains of 53-73 devices (links of chain
    positions beyond 64 take the kernel's fallback path)."""
    wl = workload.random_small(9, M=256, N=255, P=1, k_max=4, mem_lo_layers=2, mem_hi_layers=25)
    got = _gpu_idle(torch_dev, wl)
    _assert_equal(got, oracle.eval_population_idle(wl), tag="idle max")
    assert (got["T"] != INF).all()


@pytest.mark.parametrize("name,rows", [("c1_tiny_12dev_32L", None), ("c2_32dev_48L", None),
                                       ("c3_64dev_80L", 256)])
def test_idle_named_workloads(torch_dev, name, rows):
    print(f"idle workload {name}", flush=True)
    wl = workload.make(name)
    got = _gpu_idle(torch_dev, wl)
    if rows is None:
        _assert_equal(got, oracle.eval_population_idle(wl), tag=name)
    else:
        pick = np.sort(np.random.default_rng(29).choice(wl.population, rows, replace=False))
        _assert_equal(got, oracle.eval_population_idle(wl.subset(pick)), rows=pick, tag=name)
    # never above Algorithm 1's optimum on the same clusters
    bn = oracle.eval_population(wl)
    assert (got["T"] <= bn["T"]).all()


def test_idle_adding_a_device_never_worsens(torch_dev):
    """Move one unassigned device into each cluster in turn: the GPU's
    relaxed optimum of that cluster never rises."""
    wl = workload.random_small(515, M=20, N=30, P=1, k_max=3, mem_hi_layers=12)
    base = wl.labels.copy()
    base[0, :4] = 200                           # four devices outside every cluster
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    before = _gpu_idle(torch_dev, wl, base, ctx)["T"][0]
    for d in range(4):
        for q in range(3):
            lab = base.copy()
            lab[0, d] = q
            after = _gpu_idle(torch_dev, wl, lab, ctx)["T"][0]
            assert after[q] <= before[q]
