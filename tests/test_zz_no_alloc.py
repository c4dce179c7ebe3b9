"""e2_eval_population_noalloc, the entry point for callers that cannot
allocate: through the C ABI, its results equal e2_eval_population's bit for
bit, on consecutive calls that reuse the library's fixed scratch (the second
call smaller than the first, so stale contents of the scratch are present),
and inputs beyond the scratch are rejected before any launch."""
import numpy as np
import pytest

import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    e2.lib()
    return torch, torch.device("cuda:0")


def _both(torch_dev, ctx, wl, labels, roles):
    torch, dev = torch_dev
    L = torch.from_numpy(np.ascontiguousarray(labels)).to(dev)
    R = torch.from_numpy(np.ascontiguousarray(roles)).to(dev)
    fp = wl.fitness_params()
    want = e2.e2_eval_population(ctx, L, R, fp)
    torch.cuda.synchronize()
    want = {k: e2.u64(v) for k, v in want.items()}
    got = e2.e2_eval_population(ctx, L, R, fp, objective="noalloc")
    torch.cuda.synchronize()
    got = {k: e2.u64(v) for k, v in got.items()}
    return got, want


def _check(got, want, tag):
    for k in ("w", "phase", "s_p", "s_d"):
        bad = np.nonzero(got[k] != want[k])[0]
        assert bad.size == 0, f"{tag} {k}: {bad.size} genomes differ, first {bad[:5]}"


def test_noalloc_equals_eval_population_two_calls(torch_dev):
    # the 16384-genome, 256-device generation 0, then a smaller population
    # of the same context: the second call finds the first one's contents
    wl = workload.make("c5_256dev_126L_ga")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    print("noalloc: 16384 genomes", flush=True)
    got, want = _both(torch_dev, ctx, wl, wl.labels, wl.roles)
    _check(got, want, "16384 genomes")
    assert (want["w"] != (1 << 64) - 1).any()
    print("noalloc: 1000 genomes after it", flush=True)
    rows = np.arange(5000, 6000)
    got, want = _both(torch_dev, ctx, wl, wl.labels[rows], wl.roles[rows])
    _check(got, want, "1000 genomes")


def test_noalloc_small_instances_and_another_context(torch_dev):
    for seed, (M, N, P, K) in enumerate([(40, 60, 200, 9), (7, 5, 3, 4), (64, 200, 50, 3)]):
        print(f"noalloc: random_small seed={seed} M={M} N={N} P={P} k_max={K}", flush=True)
        wl = workload.random_small(seed, M=M, N=N, P=P, k_max=K, zero_bw_frac=0.1)
        ctx = e2.e2_ctx_create(wl.problem_arrays())
        got, want = _both(torch_dev, ctx, wl, wl.labels, wl.roles)
        _check(got, want, f"random_small {seed}")


def test_noalloc_rejects_inputs_beyond_its_scratch(torch_dev):
    # 16384 genomes x 255 cluster ids need 134 MB of list and T/Lambda alone
    torch, dev = torch_dev
    wl = workload.make("c5_256dev_126L_ga")
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.zeros((wl.population, 255), dtype=torch.uint8, device=dev)
    with pytest.raises(e2.E2Error) as ei:
        e2.e2_eval_population(ctx, L, R, wl.fitness_params(), objective="noalloc")
    assert ei.value.code == e2.E2_EINVAL
    # the normal entry point takes the same input
    out = e2.e2_eval_population(ctx, L, R, wl.fitness_params())
    torch.cuda.synchronize()
    assert out["w"].shape[0] == wl.population


def test_noalloc_replays_from_a_captured_graph(torch_dev):
    """The allocation-free evaluation captured in a HIP graph (torch's
    capture of the current stream): each replay, after a different
    population is copied into the captured input buffers and with eager
    library calls and synchronisations between replays, equals the eager
    e2_eval_population on that population."""
    torch, dev = torch_dev
    wl = workload.make("c3_64dev_80L")
    P = wl.population
    ctx = e2.e2_ctx_create(wl.problem_arrays())
    fp = wl.fitness_params()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    out = {k: torch.empty(P, dtype=torch.int64, device=dev) for k in ("w", "phase", "s_p", "s_d")}
    e2.e2_eval_population(ctx, L, R, fp, objective="noalloc", out=out)  # set-up outside capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        e2.e2_eval_population(ctx, L, R, fp, objective="noalloc", out=out)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    for it in range(4):
        perm = rng.permutation(P)
        L.copy_(torch.from_numpy(np.ascontiguousarray(wl.labels[perm])).to(dev))
        R.copy_(torch.from_numpy(np.ascontiguousarray(wl.roles[perm])).to(dev))
        torch.cuda.synchronize()
        print(f"graph replay {it}", flush=True)
        graph.replay()
        torch.cuda.synchronize()
        got = {k: e2.u64(v).copy() for k, v in out.items()}
        want = e2.e2_eval_population(ctx, L, R, fp)   # eager, allocating entry point
        torch.cuda.synchronize()
        _check(got, {k: e2.u64(v) for k, v in want.items()}, f"replay {it}")
