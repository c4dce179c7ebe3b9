"""CPU tests of the C ABI: the library loads, exports what include/e2.h
declares, rejects bad arguments before touching the GPU, and its host-side
quantisation (integer cost tables) equals the oracle's bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2606_03770_amd as e2
from paper_2606_03770_amd import workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "e2.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(e2_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(e2.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = e2.lib()
    for name in declared_functions():
        assert hasattr(L, name), name


def test_strerror():
    L = e2.lib()
    assert L.e2_strerror(0) == b"ok"
    assert L.e2_strerror(-1) == b"invalid argument"
    assert L.e2_strerror(-2).startswith(b"quantised")
    assert L.e2_strerror(12345) == b"unknown error"


@pytest.mark.parametrize("name", workload.NAMES)
def test_quantise_matches_oracle_on_named_workloads(name):
    wl = workload.make(name, population=1)
    got = e2.e2_quantise(wl.problem_arrays())
    want = oracle.quantise(**wl.problem_arrays())
    for g, w in zip(got, want):
        assert g.dtype == np.uint64 and (g == w).all()


def test_quantise_matches_oracle_random():
    rng = np.random.default_rng(0)
    for seed in range(30):
        M = int(rng.integers(1, 40))
        N = int(rng.integers(1, 60))
        wl = workload.random_small(seed, M=M, N=N, P=1, k_max=2, zero_bw_frac=0.2)
        p = wl.problem_arrays()
        p["speed_flops"] = rng.integers(1, 1 << 63, size=M, dtype=np.uint64) >> \
            rng.integers(0, 63, size=M).astype(np.uint64)
        p["speed_flops"] = np.maximum(p["speed_flops"], 1).astype(np.uint64)
        p["layer_flops"] = rng.integers(0, 1 << 40, size=(2, N), dtype=np.uint64)
        p["bw_Bps"] = rng.integers(0, 1 << 62, size=M * M, dtype=np.uint64) >> \
            rng.integers(0, 62, size=M * M).astype(np.uint64)
        try:
            want = oracle.quantise(**p)
        except oracle.OracleError:
            with pytest.raises(e2.E2Error) as ei:
                e2.e2_quantise(p)
            assert ei.value.code == e2.E2_EOVERFLOW
            continue
        got = e2.e2_quantise(p)
        for g, w in zip(got, want):
            assert (g == w).all()


def _base_problem():
    return workload.random_small(1, M=4, N=5, P=1, k_max=2).problem_arrays()


@pytest.mark.parametrize("mutate,code", [
    (lambda p: p.update(n_dev=0), e2.E2_EINVAL),
    (lambda p: p.update(n_dev=257), e2.E2_EINVAL),
    (lambda p: p.update(n_layer=256), e2.E2_EINVAL),
    (lambda p: p["speed_flops"].__setitem__(2, 0), e2.E2_EINVAL),
    (lambda p: p["congestion_ppm"].__setitem__(3, 10**6 + 1), e2.E2_EINVAL),
    (lambda p: p["layer_bytes"].__setitem__(0, 1 << 48), e2.E2_EOVERFLOW),
    (lambda p: p.update(head_bytes=1 << 48), e2.E2_EOVERFLOW),
    (lambda p: p.update(layer_flops=np.full((2, 5), 10**19, np.uint64)), e2.E2_EOVERFLOW),
])
def test_quantise_and_ctx_create_reject_before_any_hip_call(mutate, code):
    p = _base_problem()
    p = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in p.items()}
    mutate(p)
    M, N = p["n_dev"], p["n_layer"]
    if 1 <= M <= 256 and 1 <= N <= 255:
        with pytest.raises(e2.E2Error) as ei:
            e2.e2_quantise(p)
        assert ei.value.code == code
    s, keep = e2._make_problem(p)
    h = ctypes.c_void_p()
    assert e2.lib().e2_ctx_create(ctypes.byref(s), ctypes.byref(h)) == code
    assert h.value is None


def test_entry_points_reject_bad_arguments_without_a_device():
    L = e2.lib()
    fp = e2.e2_fitness_params(0, 1, 0)
    gp = e2.e2_ga_params(0, 0, 4, 1 << 31, 1 << 24, 1)
    nul = ctypes.c_void_p(0)
    assert L.e2_ctx_destroy(nul) == e2.E2_EINVAL
    assert L.e2_solve_partitions(nul, nul, 1, 1, nul, nul, nul, nul, nul, nul) == e2.E2_EINVAL
    assert L.e2_eval_population(nul, nul, 1, 1, nul, nul, ctypes.byref(fp), nul, nul, nul,
                                nul) == e2.E2_EINVAL
    assert L.e2_ga_step(nul, nul, 1, 1, nul, nul, nul, nul, ctypes.byref(gp), nul,
                        nul) == e2.E2_EINVAL
    assert L.e2_ctx_create(None, ctypes.byref(ctypes.c_void_p())) == e2.E2_EINVAL
    assert L.e2_ctx_keep_scratch(nul, 1) == e2.E2_EINVAL
    assert L.e2_ctx_keep_scratch(nul, 0) == e2.E2_EINVAL


def test_library_loads_beside_torchs_hip_runtime():
    """The binding loads libe2.so into processes that have imported torch,
    whose bundled HIP runtime is then the one every HIP symbol binds to: the
    library may use no symbol (or symbol version) that runtime lacks."""
    import subprocess
    import sys
    code = ("import torch, ctypes, sys; ctypes.CDLL(sys.argv[1]); print('ok')")
    r = subprocess.run([sys.executable, "-c", code, e2.LIB_PATH], capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stderr[-2000:]


@pytest.mark.parametrize("sm,code", [
    (dict(b_max=0, beta_ppm=0, kv_bytes_per_block_slot=0), e2.E2_EINVAL),
    (dict(b_max=16, beta_ppm=0, kv_bytes_per_block_slot=0), e2.E2_EINVAL),
    (dict(b_max=2, beta_ppm=1000001, kv_bytes_per_block_slot=0), e2.E2_EINVAL),
    # one slot's bytes at the limit, and a value whose product with the slot
    # count would wrap 64 bits
    (dict(b_max=2, beta_ppm=0, kv_bytes_per_block_slot=1 << 48), e2.E2_EOVERFLOW),
    (dict(b_max=2, beta_ppm=0, kv_bytes_per_block_slot=(1 << 63) + 1), e2.E2_EOVERFLOW),
    # b_max slots push a block to 2^48
    (dict(b_max=15, beta_ppm=0, kv_bytes_per_block_slot=(1 << 48) // 15 + 1), e2.E2_EOVERFLOW),
])
def test_slot_context_rejects_before_any_hip_call(sm, code):
    s, keep = e2._make_problem(_base_problem())
    m = e2.e2_slot_model(sm["b_max"], sm["beta_ppm"], sm["kv_bytes_per_block_slot"])
    h = ctypes.c_void_p()
    assert e2.lib().e2_ctx_create_slots(ctypes.byref(s), ctypes.byref(m), ctypes.byref(h)) == code
    assert h.value is None


def test_injected_hip_failure_comes_after_the_argument_checks():
    """e2_debug_inject_hip_error: a call consumes an injected failure only
    once its arguments pass, and then returns E2_EHIP before any HIP call."""
    assert e2.e2_debug_inject_hip_error(0) >= 0
    wl = workload.random_small(1, M=5, N=6, P=1, k_max=2)
    good = wl.problem_arrays()
    bad = dict(good, speed_flops=np.zeros(5, dtype=np.uint64))     # a device of speed 0
    assert e2.e2_debug_inject_hip_error(2) == 0
    with pytest.raises(e2.E2Error) as ei:
        e2.e2_ctx_create(bad)
    assert ei.value.code == e2.E2_EINVAL
    assert e2.e2_debug_inject_hip_error(2) == 2                    # nothing consumed
    with pytest.raises(e2.E2Error) as ei:
        e2.e2_ctx_create(good)
    assert ei.value.code == e2.E2_EHIP
    assert e2.e2_debug_inject_hip_error(0) == 1                    # one consumed
    with pytest.raises(e2.E2Error) as ei:
        e2.e2_debug_inject_hip_error(-1)
    assert ei.value.code == e2.E2_EINVAL


def test_missing_library_raises_instead_of_falling_back(monkeypatch, tmp_path):
    """Without libe2.so every entry point fails loudly: the binding has no
    CPU path to fall back on."""
    import paper_2606_03770_amd as pkg
    monkeypatch.setattr(pkg, "_lib", None)
    monkeypatch.setattr(pkg, "LIB_PATH", str(tmp_path / "libe2.so"))
    with pytest.raises(RuntimeError, match="not built"):
        pkg.lib()
    with pytest.raises(RuntimeError, match="not built"):
        pkg.e2_ctx_create(workload.make("c1_tiny_12dev_32L").problem_arrays())
