"""oracle.pool: the oracle over genome ranges in worker processes equals one
call over the whole population (a genome's results depend on it alone)."""
import numpy as np

import oracle
from oracle import pool
from paper_2606_03770_amd import workload


def test_ranges_equal_one_call_labels():
    wl = workload.make("c2_32dev_48L")
    want = oracle.eval_population(wl)
    got = pool.eval_population(wl, n_workers=3, chunks_per_worker=3)
    for k in pool.KEYS:
        assert np.array_equal(got[k], want[k]), k
    # a population given explicitly (reordered) is evaluated as given
    perm = np.random.default_rng(1).permutation(wl.population)
    got = pool.eval_population(wl, wl.labels[perm], wl.roles[perm], n_workers=2)
    for k in pool.KEYS:
        assert np.array_equal(got[k], want[k][perm]), k


def test_ranges_equal_one_call_ordered():
    wl = workload.make("c2_32dev_48L")
    op = workload.ordered_population(wl)
    want = oracle.eval_population_ordered(wl, op.order, op.sizes, op.roles)
    got = pool.eval_population_ordered(wl, op.order, op.sizes, op.roles, n_workers=3)
    for k in pool.KEYS:
        assert np.array_equal(got[k], want[k]), k


def test_worker_count_is_bounded():
    assert 1 <= pool.workers() <= 16
    assert pool.workers(limit=1) == 1


def test_search_ranges_equal_one_call():
    wl = workload.make("c2_32dev_48L")
    sm = workload.slot_model(wl)
    want = oracle.search_roles(wl, sm)
    got = pool.search_roles(wl, sm, wl.labels, n_workers=3)
    for k in pool.SEARCH_KEYS:
        assert np.array_equal(got[k], want[k]), k
    op = workload.ordered_population(wl)
    want = oracle.search_roles_ordered(wl, sm, op.order, op.sizes)
    got = pool.search_roles_ordered(wl, sm, op.order, op.sizes, n_workers=2)
    for k in pool.SEARCH_KEYS:
        assert np.array_equal(got[k], want[k]), k
