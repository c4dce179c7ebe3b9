"""Pins for the oracle's integer cost tables (times in ns, bytes).

The paper defines the block time as the profiled compute time and the link
time as tau = A / B (Sec. 3.2, after Eq. 2) with a worked example in Sec. 4.1.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = oracle.INF


def _problem(M=3, N=4, **kw):
    d = dict(n_dev=M, n_layer=N, speed_flops=np.full(M, 10**12, np.uint64),
             bw_Bps=np.full(M * M, 10**9, np.uint64),
             congestion_ppm=np.full(M * M, 10**6, np.uint32),
             layer_flops=np.full((2, N), 10**12, np.uint64),
             act_bytes=np.array([10**6, 10**3], np.uint64),
             head_flops=np.array([0, 0], np.uint64))
    d.update(kw)
    return d


def test_paper_tau_example(orc):
    """20 kB over 100 Mbps takes 1.6 ms (Sec. 4.1)."""
    g = json.load(open(os.path.join(GOLDEN, "paper_values.json")))["tau_example"]
    Bps = g["link_bits_per_s"] // 8
    p = _problem(M=2, N=1, bw_Bps=np.full(4, Bps, np.uint64),
                 act_bytes=np.array([g["act_bytes"], g["act_bytes"]], np.uint64))
    t, h, tau = oracle.quantise(**p)
    assert int(tau[0, 0, 1]) == g["expected_tau_ns"] == int(tau[1, 1, 0])
    assert int(tau[0, 0, 0]) == 0


def test_ceil_and_floor_definitions(orc):
    """t = ceil(F * 1e9 / S): t * S >= F * 1e9 > (t - 1) * S; the effective
    bandwidth is floor(bw * c / 1e6) and tau = ceil(A * 1e9 / Beff)."""
    rng = np.random.default_rng(1)
    M, N = 7, 9
    speed = rng.integers(1, 10**13, size=M).astype(np.uint64)
    lf = rng.integers(0, 10**14, size=(2, N)).astype(np.uint64)
    bw = rng.integers(1, 10**10, size=M * M).astype(np.uint64)
    cong = rng.integers(0, 10**6 + 1, size=M * M).astype(np.uint32)
    act = rng.integers(0, 10**7, size=2).astype(np.uint64)
    hf = rng.integers(0, 10**13, size=2).astype(np.uint64)
    t, h, tau = oracle.quantise(M, N, speed, bw, cong, lf, act, hf)
    for r in range(2):
        for d in range(M):
            S = int(speed[d])
            for n in range(N):
                v, F = int(t[r, d, n]), int(lf[r, n])
                assert v * S >= F * 10**9 and (v == 0 or (v - 1) * S < F * 10**9)
            v, F = int(h[r, d]), int(hf[r])
            assert v * S >= F * 10**9 and (v == 0 or (v - 1) * S < F * 10**9)
            for e in range(M):
                if d == e:
                    assert int(tau[r, d, e]) == 0
                    continue
                prod = int(bw[d * M + e]) * int(cong[d * M + e])
                beff = prod // 10**6
                assert beff * 10**6 <= prod < (beff + 1) * 10**6
                if beff == 0:
                    assert int(tau[r, d, e]) == INF
                else:
                    v, A = int(tau[r, d, e]), int(act[r])
                    assert v * beff >= A * 10**9 and (v == 0 or (v - 1) * beff < A * 10**9)


def test_zero_bandwidth_is_infinite_link(orc):
    p = _problem(M=2, N=2, congestion_ppm=np.array([10**6, 0, 0, 10**6], np.uint32))
    t, h, tau = oracle.quantise(**p)
    assert int(tau[0, 0, 1]) == INF and int(tau[1, 1, 0]) == INF


@pytest.mark.parametrize("field,value", [
    ("layer_flops", np.full((2, 4), 10**19, np.uint64)),
    ("head_flops", np.array([10**19, 0], np.uint64)),
    ("act_bytes", np.array([10**18, 0], np.uint64)),
])
def test_overflow_is_an_error(orc, field, value):
    """A finite time at or above 2^48 ns is rejected."""
    p = _problem(**{field: value})
    with pytest.raises(oracle.OracleError):
        oracle.quantise(**p)


def test_limits_just_below_2_48(orc):
    lim = 1 << 48
    p = _problem(M=1, N=1, speed_flops=np.array([10**9], np.uint64),
                 layer_flops=np.array([[lim - 1], [0]], np.uint64))
    t, h, tau = oracle.quantise(**p)
    assert int(t[0, 0, 0]) == lim - 1
    p = _problem(M=1, N=1, speed_flops=np.array([10**9], np.uint64),
                 layer_flops=np.array([[lim], [0]], np.uint64))
    with pytest.raises(oracle.OracleError):
        oracle.quantise(**p)


def test_invalid_inputs(orc):
    with pytest.raises(oracle.OracleError):
        oracle.quantise(**_problem(speed_flops=np.array([1, 0, 1], np.uint64)))
    with pytest.raises(oracle.OracleError):
        oracle.quantise(**_problem(congestion_ppm=np.full(9, 10**6 + 1, np.uint32)))
