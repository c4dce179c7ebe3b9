"""Python binding of libe2.so, the MI355X population-fitness library.

Argument marshalling only: every step of the path runs in the HIP kernels
behind the C ABI of include/e2.h.  torch supplies device memory (CUDA
tensors on ROCm) and streams.  The wrappers keep the C names:

    e2_quantise(problem)                              host tables (t, h, tau)
    e2_ctx_create(problem) -> Context                 quantise + upload
    e2_solve_partitions(ctx, labels, roles)           Algorithm 1 per cluster
    e2_eval_population(ctx, labels, roles, fitness)   Eq. 3-5 per individual
    e2_ga_step(ctx, labels, roles, w, phase, ga)      one GA generation
    e2_solve_partitions_ordered(ctx, order, sizes, roles)          the same on
    e2_eval_population_ordered(ctx, order, sizes, roles, fitness)  two-chromosome
    e2_ga_step_ordered(ctx, order, sizes, roles, w, phase, ga)     genomes (App. A)
    e2_ctx_create_slots(problem, slot_model) -> Context   with decode slot counts
    e2_search_roles(ctx, labels, fitness)   role + slot search (Algorithm 2 inner loop)
    e2_search_roles_ordered(ctx, order, sizes, fitness)   the same on two-chromosome genomes
    e2_search_roles(..., splitwise_np_tokens=NP)     the ablations of Sec. 4.2:
    e2_solve_partitions(..., objective="finish_time")  adapted-SplitWise roles,
    e2_eval_population(..., objective="finish_time")   finishing-time objective
    e2_solve_partitions / e2_eval_population(..., objective="idle")  idle devices

`problem` is a dict with the fields of e2_problem (numpy arrays), as
returned by workload.Workload.problem_arrays().  64-bit unsigned outputs
come back as torch.int64 tensors holding the same bits; u64() views them as
numpy uint64.

If libe2.so has not been built, importing works but every call raises
E2Error: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libe2.so")

E2_OK, E2_EINVAL, E2_EOVERFLOW, E2_ENOMEM, E2_EHIP = 0, -1, -2, -3, -4
INF = (1 << 64) - 1

EXPORTED = ("e2_ctx_create", "e2_ctx_destroy", "e2_quantise", "e2_solve_partitions",
            "e2_eval_population", "e2_ga_step", "e2_solve_partitions_ordered",
            "e2_eval_population_ordered", "e2_ga_step_ordered", "e2_ctx_create_slots",
            "e2_search_roles", "e2_assign_roles_splitwise", "e2_solve_partitions_ft",
            "e2_eval_population_ft", "e2_solve_partitions_idle", "e2_eval_population_idle",
            "e2_ctx_dp_timing", "e2_ctx_dp_elapsed", "e2_strerror",
            "e2_eval_population_noalloc", "e2_search_roles_ordered",
            "e2_debug_inject_hip_error", "e2_ctx_keep_scratch")


class E2Error(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = lib().e2_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{where}: {msg} ({code})")


class e2_problem(ctypes.Structure):
    _fields_ = [("n_dev", ctypes.c_int32), ("n_layer", ctypes.c_int32),
                ("speed_flops", ctypes.c_void_p), ("mem_bytes", ctypes.c_void_p),
                ("bw_Bps", ctypes.c_void_p), ("congestion_ppm", ctypes.c_void_p),
                ("layer_flops", ctypes.c_void_p), ("layer_bytes", ctypes.c_void_p),
                ("act_bytes", ctypes.c_uint64 * 2), ("head_flops", ctypes.c_uint64 * 2),
                ("head_bytes", ctypes.c_uint64)]


class e2_fitness_params(ctypes.Structure):
    _fields_ = [("t_arrival_ns", ctypes.c_uint64), ("nd_tokens", ctypes.c_uint64),
                ("min_tps_milli", ctypes.c_uint64)]


class e2_ga_params(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("generation", ctypes.c_uint32),
                ("tournament_k", ctypes.c_uint32), ("crossover_thresh_u32", ctypes.c_uint32),
                ("mutation_thresh_u32", ctypes.c_uint32), ("n_elite", ctypes.c_uint32)]


class e2_ga2_params(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("generation", ctypes.c_uint32),
                ("tournament_k", ctypes.c_uint32), ("mutation_thresh_u32", ctypes.c_uint32),
                ("n_elite", ctypes.c_uint32), ("max_replica", ctypes.c_uint32)]


class e2_slot_model(ctypes.Structure):
    _fields_ = [("b_max", ctypes.c_int32), ("beta_ppm", ctypes.c_uint32),
                ("kv_bytes_per_block_slot", ctypes.c_uint64)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Load libe2.so; raises E2Error(-4) style RuntimeError if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2606_03770_amd.csrc.build")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    L.e2_strerror.argtypes = [ctypes.c_int]
    L.e2_strerror.restype = ctypes.c_char_p
    L.e2_quantise.argtypes = [ctypes.POINTER(e2_problem), vp, vp, vp]
    L.e2_quantise.restype = ctypes.c_int
    L.e2_ctx_create.argtypes = [ctypes.POINTER(e2_problem), ctypes.POINTER(vp)]
    L.e2_ctx_create.restype = ctypes.c_int
    L.e2_ctx_destroy.argtypes = [vp]
    L.e2_ctx_destroy.restype = ctypes.c_int
    L.e2_solve_partitions.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp, vp]
    L.e2_solve_partitions.restype = ctypes.c_int
    L.e2_eval_population.argtypes = [vp, vp, i32, i32, vp, vp, ctypes.POINTER(e2_fitness_params),
                                     vp, vp, vp, vp]
    L.e2_eval_population.restype = ctypes.c_int
    L.e2_eval_population_noalloc.argtypes = L.e2_eval_population.argtypes
    L.e2_eval_population_noalloc.restype = ctypes.c_int
    L.e2_ga_step.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, ctypes.POINTER(e2_ga_params),
                             vp, vp]
    L.e2_ga_step.restype = ctypes.c_int
    L.e2_solve_partitions_ordered.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    L.e2_solve_partitions_ordered.restype = ctypes.c_int
    L.e2_eval_population_ordered.argtypes = [vp, vp, i32, i32, vp, vp, vp,
                                             ctypes.POINTER(e2_fitness_params), vp, vp, vp, vp]
    L.e2_eval_population_ordered.restype = ctypes.c_int
    L.e2_ga_step_ordered.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp,
                                     ctypes.POINTER(e2_ga2_params), vp, vp, vp]
    L.e2_ga_step_ordered.restype = ctypes.c_int
    L.e2_ctx_create_slots.argtypes = [ctypes.POINTER(e2_problem), ctypes.POINTER(e2_slot_model),
                                      ctypes.POINTER(vp)]
    L.e2_ctx_create_slots.restype = ctypes.c_int
    L.e2_search_roles.argtypes = [vp, vp, i32, i32, vp, ctypes.POINTER(e2_fitness_params), vp, vp,
                                  vp, vp, vp, vp]
    L.e2_search_roles.restype = ctypes.c_int
    L.e2_search_roles_ordered.argtypes = [vp, vp, i32, i32, vp, vp,
                                          ctypes.POINTER(e2_fitness_params), vp, vp, vp, vp, vp,
                                          vp]
    L.e2_search_roles_ordered.restype = ctypes.c_int
    L.e2_assign_roles_splitwise.argtypes = [vp, vp, i32, i32, vp,
                                            ctypes.POINTER(e2_fitness_params), ctypes.c_uint32,
                                            vp, vp, vp, vp, vp, vp]
    L.e2_assign_roles_splitwise.restype = ctypes.c_int
    L.e2_solve_partitions_ft.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp, vp]
    L.e2_solve_partitions_ft.restype = ctypes.c_int
    L.e2_eval_population_ft.argtypes = [vp, vp, i32, i32, vp, vp,
                                        ctypes.POINTER(e2_fitness_params), vp, vp, vp, vp]
    L.e2_eval_population_ft.restype = ctypes.c_int
    L.e2_solve_partitions_idle.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp, vp]
    L.e2_solve_partitions_idle.restype = ctypes.c_int
    L.e2_eval_population_idle.argtypes = [vp, vp, i32, i32, vp, vp,
                                          ctypes.POINTER(e2_fitness_params), vp, vp, vp, vp]
    L.e2_eval_population_idle.restype = ctypes.c_int
    L.e2_debug_inject_hip_error.argtypes = [i32]
    L.e2_debug_inject_hip_error.restype = ctypes.c_int
    L.e2_ctx_keep_scratch.argtypes = [vp, i32]
    L.e2_ctx_keep_scratch.restype = ctypes.c_int
    L.e2_ctx_dp_timing.argtypes = [vp, i32]
    L.e2_ctx_dp_timing.restype = ctypes.c_int
    L.e2_ctx_dp_elapsed.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double)]
    L.e2_ctx_dp_elapsed.restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int, where: str):
    if rc != E2_OK:
        raise E2Error(rc, where)


def _np(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def _make_problem(problem: dict):
    """Build an e2_problem; returns (struct, keepalive arrays)."""
    M, N = int(problem["n_dev"]), int(problem["n_layer"])
    keep = dict(
        speed=_np(problem["speed_flops"], np.uint64), mem=_np(problem["mem_bytes"], np.uint64),
        bw=_np(problem["bw_Bps"], np.uint64), cong=_np(problem["congestion_ppm"], np.uint32),
        lf=_np(problem["layer_flops"], np.uint64).reshape(-1),
        lb=_np(problem["layer_bytes"], np.uint64))
    act = _np(problem["act_bytes"], np.uint64)
    hf = _np(problem["head_flops"], np.uint64)
    s = e2_problem(M, N, keep["speed"].ctypes.data, keep["mem"].ctypes.data,
                   keep["bw"].ctypes.data, keep["cong"].ctypes.data, keep["lf"].ctypes.data,
                   keep["lb"].ctypes.data, (ctypes.c_uint64 * 2)(int(act[0]), int(act[1])),
                   (ctypes.c_uint64 * 2)(int(hf[0]), int(hf[1])), int(problem["head_bytes"]))
    return s, keep


def e2_quantise(problem: dict):
    """Host-only quantisation: returns numpy (t [2][M][N], h [2][M], tau [2][M][M])."""
    s, keep = _make_problem(problem)
    M, N = s.n_dev, s.n_layer
    if not (1 <= M <= 256 and 1 <= N <= 255):
        _check(E2_EINVAL, "e2_quantise")
    t = np.zeros((2, M, N), np.uint64)
    h = np.zeros((2, M), np.uint64)
    tau = np.zeros((2, M, M), np.uint64)
    _check(lib().e2_quantise(ctypes.byref(s), t.ctypes.data, h.ctypes.data, tau.ctypes.data),
           "e2_quantise")
    return t, h, tau


class Context:
    """Owns one e2_ctx (device tables of one problem instance)."""

    def __init__(self, handle: int, n_dev: int, n_layer: int, b_max: int = 1):
        self.handle = handle
        self.n_dev = n_dev
        self.n_layer = n_layer
        self.b_max = b_max  # decode slot counts (1 without a slot model)

    def close(self):
        if self.handle:
            _check(lib().e2_ctx_destroy(self.handle), "e2_ctx_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def e2_ctx_create(problem: dict) -> Context:
    s, keep = _make_problem(problem)
    h = ctypes.c_void_p()
    _check(lib().e2_ctx_create(ctypes.byref(s), ctypes.byref(h)), "e2_ctx_create")
    return Context(h.value, s.n_dev, s.n_layer)


def e2_ctx_create_slots(problem: dict, slot_model: dict) -> Context:
    """A context with decode slot counts 1..b_max; slot_model has b_max,
    beta_ppm and kv_bytes_per_block_slot."""
    s, keep = _make_problem(problem)
    sm = e2_slot_model(int(slot_model["b_max"]), int(slot_model["beta_ppm"]),
                       int(slot_model["kv_bytes_per_block_slot"]))
    h = ctypes.c_void_p()
    _check(lib().e2_ctx_create_slots(ctypes.byref(s), ctypes.byref(sm), ctypes.byref(h)),
           "e2_ctx_create_slots")
    return Context(h.value, s.n_dev, s.n_layer, sm.b_max)


def e2_ctx_destroy(ctx: Context):
    ctx.close()


def e2_debug_inject_hip_error(calls: int) -> int:
    """The next `calls` library calls that reach a HIP runtime call fail with
    E2_EHIP there (0: off).  Returns the injected failures still pending
    before this call."""
    rc = lib().e2_debug_inject_hip_error(int(calls))
    if rc < 0:
        raise E2Error(rc, "e2_debug_inject_hip_error")
    return rc


def e2_ctx_keep_scratch(ctx: Context, enable: bool = True):
    """Keep each stream's call scratch in ctx between calls (True), or
    release it and allocate per call again (False)."""
    _check(lib().e2_ctx_keep_scratch(ctx.handle, int(bool(enable))), "e2_ctx_keep_scratch")


def e2_ctx_dp_timing(ctx: Context, max_launches: int):
    """Record HIP events around the DP kernel of the next `max_launches`
    solve/eval calls on ctx (0 stops recording)."""
    _check(lib().e2_ctx_dp_timing(ctx.handle, int(max_launches)), "e2_ctx_dp_timing")


def e2_ctx_dp_elapsed(ctx: Context):
    """(recorded DP launches, their summed duration in ms); waits for them."""
    n = ctypes.c_int32()
    ms = ctypes.c_double()
    _check(lib().e2_ctx_dp_elapsed(ctx.handle, ctypes.byref(n), ctypes.byref(ms)),
           "e2_ctx_dp_elapsed")
    return n.value, ms.value


def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: want {dtype} {tuple(shape)} contiguous, got "
                         f"{t.dtype} {tuple(t.shape)}")
    return t


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def e2_solve_partitions(ctx: Context, labels, roles, stream=None, out: Optional[dict] = None,
                        objective: str = "bottleneck"):
    """Returns dict T, Lambda (int64 bits of u64) [P][k_max], master int16 [P][k_max],
    layers uint8 [P][M].  objective "finish_time" calls e2_solve_partitions_ft, "idle"
    e2_solve_partitions_idle."""
    torch = _torch()
    P, M = labels.shape
    k_max = roles.shape[1]
    _dev(labels, torch.uint8, (P, ctx.n_dev), "labels")
    _dev(roles, torch.uint8, (P, k_max), "roles")
    dev = labels.device
    if out is None:
        out = dict(T=torch.empty((P, k_max), dtype=torch.int64, device=dev),
                   Lambda=torch.empty((P, k_max), dtype=torch.int64, device=dev),
                   master=torch.empty((P, k_max), dtype=torch.int16, device=dev),
                   layers=torch.empty((P, M), dtype=torch.uint8, device=dev))
    name = {"bottleneck": "e2_solve_partitions", "finish_time": "e2_solve_partitions_ft",
            "idle": "e2_solve_partitions_idle"}[objective]
    _check(getattr(lib(), name)(ctx.handle, _stream(stream), P, k_max, _ptr(labels),
                                _ptr(roles), _ptr(out["T"]), _ptr(out["Lambda"]),
                                _ptr(out["master"]), _ptr(out["layers"])), name)
    return out


def e2_eval_population(ctx: Context, labels, roles, fitness: dict, stream=None,
                       with_rates: bool = True, out: Optional[dict] = None,
                       objective: str = "bottleneck"):
    """Returns dict w, phase (and s_p, s_d) as int64 bits of u64, shape [P].
    objective "finish_time" calls e2_eval_population_ft, "idle" e2_eval_population_idle,
    "noalloc" e2_eval_population_noalloc (the library's fixed scratch instead of an
    allocation; outputs still come from `out` or torch)."""
    torch = _torch()
    P = labels.shape[0]
    k_max = roles.shape[1]
    _dev(labels, torch.uint8, (P, ctx.n_dev), "labels")
    _dev(roles, torch.uint8, (P, k_max), "roles")
    dev = labels.device
    if out is None:
        names = ("w", "phase", "s_p", "s_d") if with_rates else ("w", "phase")
        out = {k: torch.empty(P, dtype=torch.int64, device=dev) for k in names}
    fp = e2_fitness_params(int(fitness["t_arrival_ns"]), int(fitness["nd_tokens"]),
                           int(fitness["min_tps_milli"]))
    name = {"bottleneck": "e2_eval_population", "finish_time": "e2_eval_population_ft",
            "idle": "e2_eval_population_idle", "noalloc": "e2_eval_population_noalloc"}[objective]
    _check(getattr(lib(), name)(ctx.handle, _stream(stream), P, k_max, _ptr(labels),
                                _ptr(roles), ctypes.byref(fp), _ptr(out["w"]),
                                _ptr(out["phase"]), _ptr(out.get("s_p")),
                                _ptr(out.get("s_d"))), name)
    return out


def e2_ga_step(ctx: Context, labels_in, roles_in, w, phase, ga: dict, stream=None,
               out: Optional[tuple] = None):
    """Returns (labels_out uint8 [P][M], roles_out uint8 [P][k_max])."""
    torch = _torch()
    P = labels_in.shape[0]
    k_max = roles_in.shape[1]
    _dev(labels_in, torch.uint8, (P, ctx.n_dev), "labels_in")
    _dev(roles_in, torch.uint8, (P, k_max), "roles_in")
    _dev(w, torch.int64, (P,), "w")
    _dev(phase, torch.int64, (P,), "phase")
    if out is None:
        out = (torch.empty_like(labels_in), torch.empty_like(roles_in))
    gp = e2_ga_params(int(ga["seed"]), int(ga["generation"]), int(ga["tournament_k"]),
                      int(ga["crossover_thresh_u32"]), int(ga["mutation_thresh_u32"]),
                      int(ga["n_elite"]))
    _check(lib().e2_ga_step(ctx.handle, _stream(stream), P, k_max, _ptr(labels_in),
                            _ptr(roles_in), _ptr(w), _ptr(phase), ctypes.byref(gp),
                            _ptr(out[0]), _ptr(out[1])),
           "e2_ga_step")
    return out


def _ordered_args(ctx, order, sizes, roles):
    torch = _torch()
    P, k_max = sizes.shape
    _dev(order, torch.uint8, (P, ctx.n_dev), "order")
    _dev(sizes, torch.uint16, (P, k_max), "sizes")
    _dev(roles, torch.uint8, (P, k_max), "roles")
    return P, k_max


def e2_solve_partitions_ordered(ctx: Context, order, sizes, roles, stream=None,
                                out: Optional[dict] = None):
    """As e2_solve_partitions, for genomes order uint8 [P][M], sizes uint16
    [P][k_max], roles uint8 [P][k_max]; outputs per replica."""
    torch = _torch()
    P, k_max = _ordered_args(ctx, order, sizes, roles)
    dev = order.device
    if out is None:
        out = dict(T=torch.empty((P, k_max), dtype=torch.int64, device=dev),
                   Lambda=torch.empty((P, k_max), dtype=torch.int64, device=dev),
                   master=torch.empty((P, k_max), dtype=torch.int16, device=dev),
                   layers=torch.empty((P, ctx.n_dev), dtype=torch.uint8, device=dev))
    _check(lib().e2_solve_partitions_ordered(ctx.handle, _stream(stream), P, k_max, _ptr(order),
                                             _ptr(sizes), _ptr(roles), _ptr(out["T"]),
                                             _ptr(out["Lambda"]), _ptr(out["master"]),
                                             _ptr(out["layers"])),
           "e2_solve_partitions_ordered")
    return out


def e2_eval_population_ordered(ctx: Context, order, sizes, roles, fitness: dict, stream=None,
                               with_rates: bool = True, out: Optional[dict] = None):
    """As e2_eval_population, for two-chromosome genomes."""
    torch = _torch()
    P, k_max = _ordered_args(ctx, order, sizes, roles)
    if out is None:
        names = ("w", "phase", "s_p", "s_d") if with_rates else ("w", "phase")
        out = {k: torch.empty(P, dtype=torch.int64, device=order.device) for k in names}
    fp = e2_fitness_params(int(fitness["t_arrival_ns"]), int(fitness["nd_tokens"]),
                           int(fitness["min_tps_milli"]))
    _check(lib().e2_eval_population_ordered(ctx.handle, _stream(stream), P, k_max, _ptr(order),
                                            _ptr(sizes), _ptr(roles), ctypes.byref(fp),
                                            _ptr(out["w"]), _ptr(out["phase"]),
                                            _ptr(out.get("s_p")), _ptr(out.get("s_d"))),
           "e2_eval_population_ordered")
    return out


def e2_ga_step_ordered(ctx: Context, order_in, sizes_in, roles_in, w, phase, ga: dict,
                       stream=None, out: Optional[tuple] = None):
    """Returns (order_out uint8 [P][M], sizes_out uint16 [P][k_max],
    roles_out uint8 [P][k_max])."""
    torch = _torch()
    P, k_max = _ordered_args(ctx, order_in, sizes_in, roles_in)
    _dev(w, torch.int64, (P,), "w")
    _dev(phase, torch.int64, (P,), "phase")
    if out is None:
        out = (torch.empty_like(order_in), torch.empty_like(sizes_in), torch.empty_like(roles_in))
    gp = e2_ga2_params(int(ga["seed"]), int(ga["generation"]), int(ga["tournament_k"]),
                       int(ga["mutation_thresh_u32"]), int(ga["n_elite"]),
                       int(ga["max_replica"]))
    _check(lib().e2_ga_step_ordered(ctx.handle, _stream(stream), P, k_max, _ptr(order_in),
                                    _ptr(sizes_in), _ptr(roles_in), _ptr(w), _ptr(phase),
                                    ctypes.byref(gp), _ptr(out[0]), _ptr(out[1]),
                                    _ptr(out[2])),
           "e2_ga_step_ordered")
    return out


def e2_search_roles(ctx: Context, labels, fitness: dict, k_max: int, stream=None,
                    with_tables: bool = False, out: Optional[dict] = None,
                    splitwise_np_tokens: Optional[int] = None):
    """Role and slot search for label genomes.  Returns dict roles, slots
    (uint8 [P][k_max]), w, phase (int64 bits of u64 [P]) and, with_tables,
    T_all, Lambda_all (int64 bits of u64 [P][k_max][b_max + 1]).  With
    splitwise_np_tokens, e2_assign_roles_splitwise in place of the brute
    force."""
    torch = _torch()
    P = labels.shape[0]
    _dev(labels, torch.uint8, (P, ctx.n_dev), "labels")
    dev = labels.device
    R = ctx.b_max + 1
    if out is None:
        out = dict(roles=torch.empty((P, k_max), dtype=torch.uint8, device=dev),
                   slots=torch.empty((P, k_max), dtype=torch.uint8, device=dev),
                   w=torch.empty(P, dtype=torch.int64, device=dev),
                   phase=torch.empty(P, dtype=torch.int64, device=dev))
        if with_tables:
            out["T_all"] = torch.empty((P, k_max, R), dtype=torch.int64, device=dev)
            out["Lambda_all"] = torch.empty((P, k_max, R), dtype=torch.int64, device=dev)
    fp = e2_fitness_params(int(fitness["t_arrival_ns"]), int(fitness["nd_tokens"]),
                           int(fitness["min_tps_milli"]))
    outs = (_ptr(out["roles"]), _ptr(out["slots"]), _ptr(out["w"]), _ptr(out["phase"]),
            _ptr(out.get("T_all")), _ptr(out.get("Lambda_all")))
    if splitwise_np_tokens is None:
        _check(lib().e2_search_roles(ctx.handle, _stream(stream), P, int(k_max), _ptr(labels),
                                     ctypes.byref(fp), *outs), "e2_search_roles")
    else:
        _check(lib().e2_assign_roles_splitwise(ctx.handle, _stream(stream), P, int(k_max),
                                               _ptr(labels), ctypes.byref(fp),
                                               int(splitwise_np_tokens), *outs),
               "e2_assign_roles_splitwise")
    return out


def e2_search_roles_ordered(ctx: Context, order, sizes, fitness: dict, stream=None,
                            with_tables: bool = False, out: Optional[dict] = None):
    """Role and slot search for two-chromosome genomes (order uint8 [P][M],
    sizes uint16 [P][k_max]).  Returns the same dict as e2_search_roles, per
    replica slot."""
    torch = _torch()
    P, k_max = sizes.shape
    _dev(order, torch.uint8, (P, ctx.n_dev), "order")
    _dev(sizes, torch.uint16, (P, k_max), "sizes")
    dev = order.device
    R = ctx.b_max + 1
    if out is None:
        out = dict(roles=torch.empty((P, k_max), dtype=torch.uint8, device=dev),
                   slots=torch.empty((P, k_max), dtype=torch.uint8, device=dev),
                   w=torch.empty(P, dtype=torch.int64, device=dev),
                   phase=torch.empty(P, dtype=torch.int64, device=dev))
        if with_tables:
            out["T_all"] = torch.empty((P, k_max, R), dtype=torch.int64, device=dev)
            out["Lambda_all"] = torch.empty((P, k_max, R), dtype=torch.int64, device=dev)
    fp = e2_fitness_params(int(fitness["t_arrival_ns"]), int(fitness["nd_tokens"]),
                           int(fitness["min_tps_milli"]))
    _check(lib().e2_search_roles_ordered(ctx.handle, _stream(stream), P, int(k_max), _ptr(order),
                                         _ptr(sizes), ctypes.byref(fp), _ptr(out["roles"]),
                                         _ptr(out["slots"]), _ptr(out["w"]), _ptr(out["phase"]),
                                         _ptr(out.get("T_all")), _ptr(out.get("Lambda_all"))),
           "e2_search_roles_ordered")
    return out


def u64(t) -> np.ndarray:
    """View an int64 tensor holding u64 bits as a numpy uint64 array (host copy)."""
    return t.detach().cpu().numpy().view(np.uint64)
