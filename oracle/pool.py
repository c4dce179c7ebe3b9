"""The oracle over genome ranges in worker processes (test infrastructure).

The oracle is single-threaded by design.  Whole-population checks (every
genome of a 16384-genome generation) split the population into contiguous
genome ranges and run the same oracle calls on each range in its own
process; a genome's results depend on that genome alone, so the concatenated
ranges equal one call over the whole population.  Workers start with the
"spawn" method: they import numpy and the oracle only, never a GPU runtime.

Only tests/, the smoke test and the bench's CPU baseline use this module.
"""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np

KEYS = ("T", "Lambda", "master", "layers", "w", "phase", "s_p", "s_d")
SEARCH_KEYS = ("T_all", "Lambda_all", "roles", "slots", "w", "phase")


def workers(limit: int = 16) -> int:
    """Host cores this process may use, at most `limit`."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover - non-Linux hosts
        n = os.cpu_count() or 1
    return max(1, min(limit, n))


def _eval_labels(wl, labels, roles):
    import oracle
    out = oracle.eval_population(wl, labels, roles)
    return {k: out[k] for k in KEYS}


def _eval_ordered(wl, order, sizes, roles):
    import oracle
    out = oracle.eval_population_ordered(wl, order, sizes, roles)
    return {k: out[k] for k in KEYS}


def _search_labels(wl, slot_model, labels):
    import oracle
    out = oracle.search_roles(wl, slot_model, labels=labels)
    return {k: out[k] for k in SEARCH_KEYS}


def _search_ordered(wl, slot_model, order, sizes):
    import oracle
    out = oracle.search_roles_ordered(wl, slot_model, order, sizes)
    return {k: out[k] for k in SEARCH_KEYS}


def _split(P: int, parts: int):
    edges = np.linspace(0, P, parts + 1).round().astype(int)
    return [(int(a), int(b)) for a, b in zip(edges[:-1], edges[1:]) if b > a]


def _run(fn, arrays, P, n_workers, chunks_per_worker, args_of, keys=KEYS):
    n_workers = workers() if n_workers is None else max(1, int(n_workers))
    ranges = _split(P, n_workers * chunks_per_worker)
    if not ranges:
        return None
    if n_workers == 1 or len(ranges) == 1:
        parts = [fn(*args_of(a, b)) for a, b in ranges]
    else:
        ctx = mp.get_context("spawn")
        with cf.ProcessPoolExecutor(max_workers=n_workers, mp_context=ctx) as ex:
            futs = [ex.submit(fn, *args_of(a, b)) for a, b in ranges]
            parts = [f.result() for f in futs]
    return {k: np.concatenate([p[k] for p in parts], axis=0) for k in keys}


def eval_population(wl, labels=None, roles=None, n_workers=None, chunks_per_worker=2):
    """oracle.eval_population over the whole population (label genomes),
    one contiguous genome range per task."""
    labels = wl.labels if labels is None else np.ascontiguousarray(labels)
    roles = wl.roles if roles is None else np.ascontiguousarray(roles)
    base = wl.subset(np.arange(0))  # the problem instance without a population
    return _run(_eval_labels, None, labels.shape[0], n_workers, chunks_per_worker,
                lambda a, b: (base, labels[a:b], roles[a:b]))


def eval_population_ordered(wl, order, sizes, roles, n_workers=None, chunks_per_worker=2):
    """oracle.eval_population_ordered over the whole population
    (two-chromosome genomes), one contiguous genome range per task."""
    order, sizes, roles = (np.ascontiguousarray(x) for x in (order, sizes, roles))
    base = wl.subset(np.arange(0))
    return _run(_eval_ordered, None, order.shape[0], n_workers, chunks_per_worker,
                lambda a, b: (base, order[a:b], sizes[a:b], roles[a:b]))


def search_roles(wl, slot_model, labels, n_workers=None, chunks_per_worker=2):
    """oracle.search_roles (the role and slot search) over label genomes,
    one contiguous genome range per task."""
    labels = np.ascontiguousarray(labels)
    base = wl.subset(np.arange(0))
    return _run(_search_labels, None, labels.shape[0], n_workers, chunks_per_worker,
                lambda a, b: (base, slot_model, labels[a:b]), SEARCH_KEYS)


def search_roles_ordered(wl, slot_model, order, sizes, n_workers=None, chunks_per_worker=2):
    """oracle.search_roles_ordered over two-chromosome genomes, one contiguous
    genome range per task."""
    order, sizes = (np.ascontiguousarray(x) for x in (order, sizes))
    base = wl.subset(np.arange(0))
    return _run(_search_ordered, None, order.shape[0], n_workers, chunks_per_worker,
                lambda a, b: (base, slot_model, order[a:b], sizes[a:b]), SEARCH_KEYS)
