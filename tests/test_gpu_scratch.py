"""GPU: every entry point gives the same results with the context's kept
per-stream scratch (e2_ctx_keep_scratch) as with per-call scratch.

The per-call results are the ones the other GPU tests compare with the
oracle; here one context of each kind runs every call twice in a row with
the setting on (the second call reuses the buffer the first one grew), on
a side stream and the null stream, and each output must equal the same call
on a context without it.  All integer outputs: exact equality.
"""
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


def _host(out):
    if isinstance(out, dict):
        return {k: v.detach().cpu().numpy().copy() for k, v in out.items()}
    return [v.detach().cpu().numpy().copy() for v in out]


def _calls(torch, dev, wl):
    """(name, function of a (ctx, slot ctx) pair) for every entry point that
    takes scratch, on the workload's label and two-chromosome populations."""
    fp = wl.fitness_params()
    L = torch.from_numpy(wl.labels).to(dev)
    R = torch.from_numpy(wl.roles).to(dev)
    op = workload.ordered_population(wl)
    O, S, Q = (torch.from_numpy(x).to(dev) for x in (op.order, op.sizes, op.roles))
    rng = np.random.default_rng(5)
    W = torch.from_numpy(rng.integers(0, 1 << 40, size=wl.population).astype(np.int64)).to(dev)
    PH = torch.from_numpy(rng.integers(0, 1 << 40, size=wl.population).astype(np.int64)).to(dev)
    np_tok = wl.prompt_tokens()
    return [
        ("solve", lambda c, s: e2.e2_solve_partitions(c, L, R)),
        ("eval", lambda c, s: e2.e2_eval_population(c, L, R, fp)),
        ("solve_ft", lambda c, s: e2.e2_solve_partitions(c, L, R, objective="finish_time")),
        ("eval_ft", lambda c, s: e2.e2_eval_population(c, L, R, fp, objective="finish_time")),
        ("solve_idle", lambda c, s: e2.e2_solve_partitions(c, L, R, objective="idle")),
        ("eval_idle", lambda c, s: e2.e2_eval_population(c, L, R, fp, objective="idle")),
        ("ga", lambda c, s: e2.e2_ga_step(c, L, R, W, PH, wl.ga_params(3))),
        ("solve_ordered", lambda c, s: e2.e2_solve_partitions_ordered(c, O, S, Q)),
        ("eval_ordered", lambda c, s: e2.e2_eval_population_ordered(c, O, S, Q, fp)),
        ("ga_ordered", lambda c, s: e2.e2_ga_step_ordered(c, O, S, Q, W, PH, op.ga_params(wl, 3))),
        ("search", lambda c, s: e2.e2_search_roles(s, L, fp, wl.k_max, with_tables=True)),
        ("splitwise", lambda c, s: e2.e2_search_roles(s, L, fp, wl.k_max,
                                                      splitwise_np_tokens=np_tok)),
        ("search_ordered", lambda c, s: e2.e2_search_roles_ordered(s, O, S, fp, with_tables=True)),
    ]


@pytest.mark.parametrize("name", ["c2_32dev_48L", "c3_64dev_80L"])
def test_kept_scratch_equals_per_call_scratch_on_every_entry_point(torch_dev, name):
    torch, dev = torch_dev
    wl = workload.make(name)
    sm = workload.slot_model(wl)
    plain = (e2.e2_ctx_create(wl.problem_arrays()), e2.e2_ctx_create_slots(wl.problem_arrays(), sm))
    kept = (e2.e2_ctx_create(wl.problem_arrays()), e2.e2_ctx_create_slots(wl.problem_arrays(), sm))
    for c in kept:
        e2.e2_ctx_keep_scratch(c)
    calls = _calls(torch, dev, wl)
    want = {}
    for call, fn in calls:
        want[call] = _host(fn(*plain))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    for rnd, st in enumerate((side, torch.cuda.default_stream(), side)):
        with torch.cuda.stream(st):
            got = [(call, fn(*kept)) for call, fn in calls]
        torch.cuda.synchronize()
        for call, out in got:
            g, w = _host(out), want[call]
            if isinstance(w, dict):
                for k in w:
                    assert np.array_equal(g[k], w[k]), (rnd, call, k)
            else:
                for i, (a, b) in enumerate(zip(g, w)):
                    assert np.array_equal(a, b), (rnd, call, i)
    for c in plain + kept:
        c.close()
