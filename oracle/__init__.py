"""CPU oracle for the E2LLM population-fitness path (arXiv 2606.03770).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the bench's CPU-baseline leg, never by the product package.  It wraps the
plain C implementation in oracle.c (built with gcc into liboracle.so) and
shares nothing with the HIP library.

Functions mirror the paper's pieces:
  quantise   -> integer cost tables (Sec. 3.2 definitions of ell and tau)
  dp_pipe    -> Algorithm 1 / Eq. 1-2 on one device chain
  solve      -> dp_pipe for every (individual, cluster) of a population
  fitness    -> Eq. 3-5 with the QoS floor (Sec. 3.3, Sec. 3.5, Algorithm 2)
  ga_step    -> one generation: elites, tournament, crossover, mutation
  rng        -> counter-based SplitMix64 hash used by ga_step
Two-chromosome genomes (App. A: an ordering chromosome and replica sizes):
  replica_range, solve_ordered, eval_population_ordered,
  order_crossover, regrow, ga_step_ordered
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
INF = (1 << 64) - 1

_lib: Optional[ctypes.CDLL] = None


def build() -> str:
    """Compile liboracle.so from oracle.c (always recompiles)."""
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                           "-o", tmp, SRC])
    os.replace(tmp, LIB)
    return LIB


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    i32, u32, u64 = ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64
    lib.oracle_quantise.argtypes = [i32, i32, P, P, P, P, P, P, P, P, P]
    lib.oracle_quantise.restype = i32
    lib.oracle_dp_pipe.argtypes = [i32, i32, P, P, P, P, P, u64, P, P, P, P, P]
    lib.oracle_dp_pipe.restype = i32
    lib.oracle_solve.argtypes = [i32, i32, P, P, P, P, P, u64, i32, i32, P, P, P, P, P, P, P]
    lib.oracle_solve.restype = i32
    lib.oracle_fitness.argtypes = [i32, i32, P, P, P, u64, u64, u64, P, P, P, P]
    lib.oracle_fitness.restype = i32
    lib.oracle_ga_step.argtypes = [i32, i32, i32, P, P, P, P, u64, u32, u32, u32, u32, u32, P, P]
    lib.oracle_ga_step.restype = i32
    lib.oracle_solve_ordered.argtypes = [i32, i32, P, P, P, P, P, u64, i32, i32, P, P, P, P, P,
                                         P, P]
    lib.oracle_solve_ordered.restype = i32
    lib.oracle_ga_step_ordered.argtypes = [i32, i32, i32, P, P, P, P, P, u64, u32, u32, u32, u32,
                                           u32, P, P, P]
    lib.oracle_ga_step_ordered.restype = i32
    lib.oracle_order_crossover.argtypes = [i32, P, P, i32, P]
    lib.oracle_order_crossover.restype = None
    lib.oracle_regrow.argtypes = [i32, i32, u64, u64, i32, i32, i32, P, P]
    lib.oracle_regrow.restype = None
    lib.oracle_replica_range.argtypes = [i32, i32, P, i32, ctypes.POINTER(i32),
                                         ctypes.POINTER(i32)]
    lib.oracle_replica_range.restype = i32
    lib.oracle_quantise_slots.argtypes = [i32, i32, P, P, P, P, P, P, i32, u32, P, P, P]
    lib.oracle_quantise_slots.restype = i32
    lib.oracle_search_roles.argtypes = [i32, i32, P, P, P, P, P, u64, u64, i32, i32, i32, P,
                                        u64, u64, u64, P, P, P, P, P, P]
    lib.oracle_search_roles.restype = i32
    lib.oracle_search_roles_ordered.argtypes = [i32, i32, P, P, P, P, P, u64, u64, i32, i32, i32,
                                                P, P, u64, u64, u64, P, P, P, P, P, P]
    lib.oracle_search_roles_ordered.restype = i32
    lib.oracle_assign_roles_splitwise.argtypes = [i32, i32, P, P, P, P, P, u64, u64, i32, i32,
                                                  i32, P, u64, u64, u64, u64, P, P, P, P, P, P]
    lib.oracle_assign_roles_splitwise.restype = i32
    lib.oracle_solve_obj.argtypes = [i32, i32, P, P, P, P, P, u64, i32, i32, i32, P, P, P, P, P,
                                     P, P]
    lib.oracle_solve_obj.restype = i32
    lib.oracle_dp_pipe_obj.argtypes = [i32, i32, P, P, P, P, P, u64, i32, P, P, P, P, P]
    lib.oracle_dp_pipe_obj.restype = i32
    lib.oracle_dp_idle.argtypes = [i32, i32, P, P, P, P, P, u64, P, P, P, P]
    lib.oracle_dp_idle.restype = i32
    lib.oracle_solve_idle.argtypes = [i32, i32, P, P, P, P, P, u64, i32, i32, P, P, P, P, P, P]
    lib.oracle_solve_idle.restype = i32
    lib.oracle_rng.argtypes = [u64, u64, u64, u64, u64]
    lib.oracle_rng.restype = u64
    lib.oracle_splitmix_out.argtypes = [u64]
    lib.oracle_splitmix_out.restype = u64
    _lib = lib
    return lib


def _p(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _u64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint64))


class OracleError(RuntimeError):
    pass


def quantise(n_dev, n_layer, speed_flops, bw_Bps, congestion_ppm, layer_flops, act_bytes,
             head_flops, **_ignored):
    """Return (t [2][M][N], h [2][M], tau [2][M][M]) as uint64 arrays."""
    lib = _load()
    M, N = int(n_dev), int(n_layer)
    speed = _u64(speed_flops)
    bw = _u64(bw_Bps)
    cong = np.ascontiguousarray(np.asarray(congestion_ppm, dtype=np.uint32))
    lf = _u64(layer_flops).reshape(2, N)
    act = _u64(act_bytes)
    hf = _u64(head_flops)
    t = np.zeros((2, M, N), dtype=np.uint64)
    h = np.zeros((2, M), dtype=np.uint64)
    tau = np.zeros((2, M, M), dtype=np.uint64)
    rc = lib.oracle_quantise(M, N, _p(speed), _p(bw), _p(cong), _p(lf), _p(act), _p(hf),
                             _p(t), _p(h), _p(tau))
    if rc != 0:
        raise OracleError(f"oracle_quantise failed: {rc}")
    return t, h, tau


def dp_pipe(tk, hk, tau_link, memk, W, HB):
    """Algorithm 1 on one chain.  Returns (T, Lambda, mu_star, sizes, evaluated)."""
    lib = _load()
    tk = _u64(tk)
    m, N = tk.shape
    hk, tl, mk, Wv = _u64(hk), _u64(tau_link), _u64(memk), _u64(W)
    assert hk.shape == (m,) and tl.shape == (m,) and mk.shape == (m,) and Wv.shape == (N,)
    T = ctypes.c_uint64()
    L = ctypes.c_uint64()
    mu = ctypes.c_int()
    ev = ctypes.c_uint64()
    sizes = np.zeros(max(m, 1), dtype=np.int32)
    rc = lib.oracle_dp_pipe(m, N, _p(tk), _p(hk), _p(tl), _p(mk), _p(Wv), int(HB),
                            ctypes.byref(T), ctypes.byref(L), ctypes.byref(mu), _p(sizes),
                            ctypes.byref(ev))
    if rc != 0:
        raise OracleError(f"oracle_dp_pipe failed: {rc}")
    return T.value, L.value, mu.value, sizes[:m].copy(), ev.value


def solve(tables, mem_bytes, layer_bytes, head_bytes, labels, roles, k_max):
    """All (individual, cluster) problems.  tables = quantise(...) output.

    Returns dict with T, Lambda [P][k_max] u64, master [P][k_max] i16,
    layers [P][M] u8 and evaluated (candidate count).
    """
    lib = _load()
    t, h, tau = tables
    M, N = t.shape[1], t.shape[2]
    labels = np.ascontiguousarray(labels, dtype=np.uint8)
    roles = np.ascontiguousarray(roles, dtype=np.uint8)
    P = labels.shape[0]
    if labels.shape != (P, M) or roles.shape != (P, int(k_max)):
        raise OracleError("labels must be [P][M] and roles [P][k_max]")
    T = np.zeros((P, k_max), dtype=np.uint64)
    L = np.zeros((P, k_max), dtype=np.uint64)
    master = np.zeros((P, k_max), dtype=np.int16)
    layers = np.zeros((P, M), dtype=np.uint8)
    ev = ctypes.c_uint64()
    rc = lib.oracle_solve(M, N, _p(t), _p(h), _p(tau), _p(_u64(mem_bytes)),
                          _p(_u64(layer_bytes)), int(head_bytes), P, int(k_max),
                          _p(labels), _p(roles), _p(T), _p(L), _p(master), _p(layers),
                          ctypes.byref(ev))
    if rc != 0:
        raise OracleError(f"oracle_solve failed: {rc}")
    return dict(T=T, Lambda=L, master=master, layers=layers, evaluated=ev.value)


def fitness(T, Lambda, roles, t_arrival_ns, nd_tokens, min_tps_milli):
    """Eq. 3-5 per individual.  Returns dict w, phase, s_p, s_d (u64 [P])."""
    lib = _load()
    T, L = _u64(T), _u64(Lambda)
    roles = np.ascontiguousarray(roles, dtype=np.uint8)
    P, k_max = T.shape
    if L.shape != T.shape or roles.shape != T.shape:
        raise OracleError("T, Lambda and roles must share the shape [P][k_max]")
    out = {k: np.zeros(P, dtype=np.uint64) for k in ("w", "phase", "s_p", "s_d")}
    rc = lib.oracle_fitness(P, k_max, _p(T), _p(L), _p(roles), int(t_arrival_ns),
                            int(nd_tokens), int(min_tps_milli), _p(out["w"]), _p(out["phase"]),
                            _p(out["s_p"]), _p(out["s_d"]))
    if rc != 0:
        raise OracleError(f"oracle_fitness failed: {rc}")
    return out


def eval_population(wl, labels=None, roles=None):
    """Quantise, solve and score a workload's population (or the given one)."""
    tables = quantise(**wl.problem_arrays())
    labels = wl.labels if labels is None else labels
    roles = wl.roles if roles is None else roles
    sol = solve(tables, wl.mem_bytes, wl.layer_bytes, wl.head_bytes, labels, roles, wl.k_max)
    fit = fitness(sol["T"], sol["Lambda"], roles, **wl.fitness_params())
    sol.update(fit)
    return sol


def ga_step(labels, roles, w, phase, k_max, seed, generation, tournament_k,
            crossover_thresh_u32, mutation_thresh_u32, n_elite):
    lib = _load()
    labels = np.ascontiguousarray(labels, dtype=np.uint8)
    roles = np.ascontiguousarray(roles, dtype=np.uint8)
    P, M = labels.shape
    if roles.shape != (P, int(k_max)):
        raise OracleError(f"roles shape {roles.shape} != {(P, int(k_max))}")
    w, phase = _u64(w), _u64(phase)
    if w.shape != (P,) or phase.shape != (P,):
        raise OracleError("w and phase must have shape [P]")
    lo = np.zeros_like(labels)
    ro = np.zeros_like(roles)
    rc = lib.oracle_ga_step(M, P, int(k_max), _p(labels), _p(roles), _p(w),
                            _p(phase), int(seed), int(generation), int(tournament_k),
                            int(crossover_thresh_u32), int(mutation_thresh_u32), int(n_elite),
                            _p(lo), _p(ro))
    if rc != 0:
        raise OracleError(f"oracle_ga_step failed: {rc}")
    return lo, ro


def rng(seed, g, s, stream, gene) -> int:
    return int(_load().oracle_rng(seed, g, s, stream, gene))


def splitmix_out(z) -> int:
    return int(_load().oracle_splitmix_out(z))


# --- two-chromosome genomes (App. A) -------------------------------------

def replica_range(sizes, r, M):
    """[lo, hi) of replica r on the ordering chromosome (clipped to M)."""
    sizes = np.ascontiguousarray(sizes, dtype=np.uint16)
    lo, hi = ctypes.c_int(), ctypes.c_int()
    rc = _load().oracle_replica_range(int(M), sizes.shape[0], _p(sizes), int(r), ctypes.byref(lo),
                                      ctypes.byref(hi))
    if rc != 0:
        raise OracleError(f"oracle_replica_range failed: {rc}")
    return lo.value, hi.value


def solve_ordered(tables, mem_bytes, layer_bytes, head_bytes, order, sizes, roles):
    """All (individual, replica) problems of two-chromosome genomes:
    order u8 [P][M], sizes u16 [P][k_max], roles u8 [P][k_max]."""
    lib = _load()
    t, h, tau = tables
    M, N = t.shape[1], t.shape[2]
    order = np.ascontiguousarray(order, dtype=np.uint8)
    sizes = np.ascontiguousarray(sizes, dtype=np.uint16)
    roles = np.ascontiguousarray(roles, dtype=np.uint8)
    P, k_max = sizes.shape
    if order.shape != (P, M) or roles.shape != (P, k_max):
        raise OracleError("order must be [P][M], sizes and roles [P][k_max]")
    T = np.zeros((P, k_max), dtype=np.uint64)
    L = np.zeros((P, k_max), dtype=np.uint64)
    master = np.zeros((P, k_max), dtype=np.int16)
    layers = np.zeros((P, M), dtype=np.uint8)
    rc = lib.oracle_solve_ordered(M, N, _p(t), _p(h), _p(tau), _p(_u64(mem_bytes)),
                                  _p(_u64(layer_bytes)), int(head_bytes), P, k_max, _p(order),
                                  _p(sizes), _p(roles), _p(T), _p(L), _p(master), _p(layers))
    if rc != 0:
        raise OracleError(f"oracle_solve_ordered failed: {rc}")
    return dict(T=T, Lambda=L, master=master, layers=layers)


def eval_population_ordered(wl, order, sizes, roles):
    """Quantise, solve and score a population of two-chromosome genomes."""
    tables = quantise(**wl.problem_arrays())
    sol = solve_ordered(tables, wl.mem_bytes, wl.layer_bytes, wl.head_bytes, order, sizes, roles)
    sol.update(fitness(sol["T"], sol["Lambda"], roles, **wl.fitness_params()))
    return sol


def order_crossover(a, b, c):
    """The child ordering of parents a, b cut at c, repaired (App. A)."""
    a = np.ascontiguousarray(a, dtype=np.uint8)
    b = np.ascontiguousarray(b, dtype=np.uint8)
    child = np.zeros_like(a)
    _load().oracle_order_crossover(a.shape[0], _p(a), _p(b), int(c), _p(child))
    return child


def regrow(sizes, roles, M, seed, g, s, pos, max_replica):
    """Regrow a grouping from replica pos (in place on copies, returned)."""
    sizes = np.array(sizes, dtype=np.uint16)
    roles = np.array(roles, dtype=np.uint8)
    _load().oracle_regrow(int(M), sizes.shape[0], int(seed), int(g), int(s), int(pos),
                          int(max_replica), _p(sizes), _p(roles))
    return sizes, roles


def ga_step_ordered(order, sizes, roles, w, phase, seed, generation, tournament_k,
                    mutation_thresh_u32, n_elite, max_replica):
    lib = _load()
    order = np.ascontiguousarray(order, dtype=np.uint8)
    sizes = np.ascontiguousarray(sizes, dtype=np.uint16)
    roles = np.ascontiguousarray(roles, dtype=np.uint8)
    P, M = order.shape
    k_max = sizes.shape[1]
    if sizes.shape != (P, k_max) or roles.shape != (P, k_max):
        raise OracleError("sizes and roles must be [P][k_max]")
    w, phase = _u64(w), _u64(phase)
    if w.shape != (P,) or phase.shape != (P,):
        raise OracleError("w and phase must have shape [P]")
    oo, so, ro = np.zeros_like(order), np.zeros_like(sizes), np.zeros_like(roles)
    rc = lib.oracle_ga_step_ordered(M, P, k_max, _p(order), _p(sizes), _p(roles), _p(w), _p(phase),
                                    int(seed), int(generation), int(tournament_k),
                                    int(mutation_thresh_u32), int(n_elite), int(max_replica),
                                    _p(oo), _p(so), _p(ro))
    if rc != 0:
        raise OracleError(f"oracle_ga_step_ordered failed: {rc}")
    return oo, so, ro


def quantise_slots(problem, b_max, beta_ppm):
    """Cost tables for role indices r = 0 (prefill) and r = b = 1..b_max
    (decode with b requests in flight): (t [R][M][N], h [R][M], tau [R][M][M])."""
    lib = _load()
    M, N = int(problem["n_dev"]), int(problem["n_layer"])
    R = int(b_max) + 1
    speed = _u64(problem["speed_flops"])
    bw = _u64(problem["bw_Bps"])
    cong = np.ascontiguousarray(np.asarray(problem["congestion_ppm"], dtype=np.uint32))
    lf = _u64(problem["layer_flops"]).reshape(2, N)
    act = _u64(problem["act_bytes"])
    hf = _u64(problem["head_flops"])
    t = np.zeros((max(R, 2), M, N), dtype=np.uint64)
    h = np.zeros((max(R, 2), M), dtype=np.uint64)
    tau = np.zeros((max(R, 2), M, M), dtype=np.uint64)
    rc = lib.oracle_quantise_slots(M, N, _p(speed), _p(bw), _p(cong), _p(lf), _p(act), _p(hf),
                                   int(b_max), int(beta_ppm), _p(t), _p(h), _p(tau))
    if rc != 0:
        raise OracleError(f"oracle_quantise_slots failed: {rc}")
    return t[:R], h[:R], tau[:R]


def np_tokens(wl):
    """Prompt tokens NP of a workload: the ratio of its prefill to its decode
    activation bytes (NP tokens against one)."""
    act = [int(x) for x in wl.act_bytes]
    return act[0] // max(act[1], 1)


def search_roles(wl, slot_model, labels=None, policy="search"):
    """Algorithm 2's inner loop for a population of label genomes: the DP for
    prefill and for every decode slot count, the highest feasible slot count
    under the QoS floor, and the best role assignment by brute force.
    slot_model: dict(b_max, beta_ppm, kv_bytes_per_block_slot).  Returns dict
    T_all, Lambda_all [P][k_max][b_max + 1], roles, slots [P][k_max], w, phase [P].
    policy "splitwise": the adapted-SplitWise rule in place of the brute force."""
    lib = _load()
    labels = np.ascontiguousarray(wl.labels if labels is None else labels, dtype=np.uint8)
    P, M = labels.shape
    K = int(wl.k_max)
    b_max = int(slot_model["b_max"])
    R = b_max + 1
    t, h, tau = quantise_slots(wl.problem_arrays(), b_max, slot_model["beta_ppm"])
    t, h, tau = (np.ascontiguousarray(x) for x in (t, h, tau))
    T = np.zeros((P, K, R), dtype=np.uint64)
    L = np.zeros((P, K, R), dtype=np.uint64)
    roles = np.zeros((P, K), dtype=np.uint8)
    slots = np.zeros((P, K), dtype=np.uint8)
    w = np.zeros(P, dtype=np.uint64)
    ph = np.zeros(P, dtype=np.uint64)
    fp = wl.fitness_params()
    common = (M, wl.n_layer, _p(t), _p(h), _p(tau), _p(_u64(wl.mem_bytes)),
              _p(_u64(wl.layer_bytes)), int(wl.head_bytes),
              int(slot_model["kv_bytes_per_block_slot"]), b_max, P, K, _p(labels),
              int(fp["t_arrival_ns"]), int(fp["nd_tokens"]), int(fp["min_tps_milli"]))
    outs = (_p(T), _p(L), _p(roles), _p(slots), _p(w), _p(ph))
    if policy == "search":
        rc = lib.oracle_search_roles(*common, *outs)
    elif policy == "splitwise":
        rc = lib.oracle_assign_roles_splitwise(*common, np_tokens(wl), *outs)
    else:
        raise OracleError(f"unknown policy {policy}")
    if rc != 0:
        raise OracleError(f"oracle role assignment ({policy}) failed: {rc}")
    return dict(T_all=T, Lambda_all=L, roles=roles, slots=slots, w=w, phase=ph)


def search_roles_ordered(wl, slot_model, order, sizes):
    """The role and slot search for two-chromosome genomes (App. A): replica
    q's chain is its run of the ordering.  Returns the same dict as
    search_roles, per replica slot."""
    lib = _load()
    order = np.ascontiguousarray(order, dtype=np.uint8)
    sizes = np.ascontiguousarray(sizes, dtype=np.uint16)
    P, M = order.shape
    K = sizes.shape[1]
    if sizes.shape != (P, K) or M != wl.n_dev:
        raise OracleError("order must be [P][M] and sizes [P][k_max]")
    b_max = int(slot_model["b_max"])
    R = b_max + 1
    t, h, tau = quantise_slots(wl.problem_arrays(), b_max, slot_model["beta_ppm"])
    t, h, tau = (np.ascontiguousarray(x) for x in (t, h, tau))
    T = np.zeros((P, K, R), dtype=np.uint64)
    L = np.zeros((P, K, R), dtype=np.uint64)
    roles = np.zeros((P, K), dtype=np.uint8)
    slots = np.zeros((P, K), dtype=np.uint8)
    w = np.zeros(P, dtype=np.uint64)
    ph = np.zeros(P, dtype=np.uint64)
    fp = wl.fitness_params()
    rc = lib.oracle_search_roles_ordered(
        M, wl.n_layer, _p(t), _p(h), _p(tau), _p(_u64(wl.mem_bytes)), _p(_u64(wl.layer_bytes)),
        int(wl.head_bytes), int(slot_model["kv_bytes_per_block_slot"]), b_max, P, K, _p(order),
        _p(sizes), int(fp["t_arrival_ns"]), int(fp["nd_tokens"]), int(fp["min_tps_milli"]),
        _p(T), _p(L), _p(roles), _p(slots), _p(w), _p(ph))
    if rc != 0:
        raise OracleError(f"oracle_search_roles_ordered failed: {rc}")
    return dict(T_all=T, Lambda_all=L, roles=roles, slots=slots, w=w, phase=ph)


def eval_population_ft(wl, labels=None, roles=None):
    """The finishing-time ablation: each cluster's master and split points
    minimise its end-to-end time (stage plus link times) instead of the
    bottleneck; T is that partition's bottleneck, Lambda its end-to-end
    time; fitness by Eq. 3-5 as usual."""
    lib = _load()
    t, h, tau = quantise(**wl.problem_arrays())
    labels = np.ascontiguousarray(wl.labels if labels is None else labels, dtype=np.uint8)
    roles = np.ascontiguousarray(wl.roles if roles is None else roles, dtype=np.uint8)
    P, M = labels.shape
    K = int(wl.k_max)
    T = np.zeros((P, K), dtype=np.uint64)
    L = np.zeros((P, K), dtype=np.uint64)
    master = np.zeros((P, K), dtype=np.int16)
    layers = np.zeros((P, M), dtype=np.uint8)
    ev = np.zeros(1, dtype=np.uint64)
    rc = lib.oracle_solve_obj(M, wl.n_layer, _p(t), _p(h), _p(tau), _p(_u64(wl.mem_bytes)),
                              _p(_u64(wl.layer_bytes)), int(wl.head_bytes), 1, P, K, _p(labels),
                              _p(roles), _p(T), _p(L), _p(master), _p(layers), _p(ev))
    if rc != 0:
        raise OracleError(f"oracle_solve_obj failed: {rc}")
    sol = dict(T=T, Lambda=L, master=master, layers=layers)
    sol.update(fitness(T, L, roles, **wl.fitness_params()))
    return sol


def dp_pipe_ft(tk, hk, tau_link, memk, W, HB):
    """The finishing-time DP on one chain: (T = bottleneck of the chosen
    partition, Lambda = its end-to-end time, mu_star, sizes)."""
    lib = _load()
    tk = _u64(tk)
    m, N = tk.shape
    sizes = np.zeros(m, dtype=np.int32)
    T = np.zeros(1, np.uint64)
    L = np.zeros(1, np.uint64)
    mu = np.zeros(1, np.int32)
    ev = np.zeros(1, np.uint64)
    rc = lib.oracle_dp_pipe_obj(m, N, _p(tk), _p(_u64(hk)), _p(_u64(tau_link)), _p(_u64(memk)),
                                _p(_u64(W)), int(HB), 1, _p(T), _p(L), _p(mu), _p(sizes), _p(ev))
    if rc != 0:
        raise OracleError(f"oracle_dp_pipe_obj failed: {rc}")
    return int(T[0]), int(L[0]), int(mu[0]), [int(x) for x in sizes]


def dp_idle(tk, hk, tau_full, memk, W, HB):
    """The idle-device relaxation on one chain: (T, Lambda, mu_star, sizes),
    sizes 0 for devices that sit out; tau_full[a][b] links chain positions."""
    lib = _load()
    tk = _u64(tk)
    m, N = tk.shape
    sizes = np.zeros(m, dtype=np.int32)
    T = np.zeros(1, np.uint64)
    L = np.zeros(1, np.uint64)
    mu = np.zeros(1, np.int32)
    rc = lib.oracle_dp_idle(m, N, _p(tk), _p(_u64(hk)), _p(_u64(tau_full).reshape(m, m)),
                            _p(_u64(memk)), _p(_u64(W)), int(HB), _p(T), _p(L), _p(mu), _p(sizes))
    if rc != 0:
        raise OracleError(f"oracle_dp_idle failed: {rc}")
    return int(T[0]), int(L[0]), int(mu[0]), [int(x) for x in sizes]


def eval_population_idle(wl, labels=None, roles=None):
    """Quantise, solve under the idle-device relaxation and score."""
    lib = _load()
    t, h, tau = quantise(**wl.problem_arrays())
    labels = np.ascontiguousarray(wl.labels if labels is None else labels, dtype=np.uint8)
    roles = np.ascontiguousarray(wl.roles if roles is None else roles, dtype=np.uint8)
    P, M = labels.shape
    K = int(wl.k_max)
    T = np.zeros((P, K), dtype=np.uint64)
    L = np.zeros((P, K), dtype=np.uint64)
    master = np.zeros((P, K), dtype=np.int16)
    layers = np.zeros((P, M), dtype=np.uint8)
    rc = lib.oracle_solve_idle(M, wl.n_layer, _p(t), _p(h), _p(tau), _p(_u64(wl.mem_bytes)),
                               _p(_u64(wl.layer_bytes)), int(wl.head_bytes), P, K, _p(labels),
                               _p(roles), _p(T), _p(L), _p(master), _p(layers))
    if rc != 0:
        raise OracleError(f"oracle_solve_idle failed: {rc}")
    sol = dict(T=T, Lambda=L, master=master, layers=layers)
    sol.update(fitness(T, L, roles, **wl.fitness_params()))
    return sol
