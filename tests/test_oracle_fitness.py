"""Pins for the oracle's fitness (Eq. 3-5, Sec. 3.3; QoS floor, Sec. 3.5)."""
import json
import os

import numpy as np

import oracle

INF = oracle.INF
SCALE = 1 << 50
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def fit(T, L, roles, ta, nd, tps):
    out = oracle.fitness(np.array([T], np.uint64), np.array([L], np.uint64),
                         np.array([roles], np.uint8), ta, nd, tps)
    return {k: int(v[0]) for k, v in out.items()}


def test_hand_computed_pair(orc):
    """One prefill replica with bottleneck 2^20 ns, one decode replica with
    2^21 ns, ND = 3, T_a = 0:  NP/PS = 2^20, ND/DS = 3 * 2^21 (Eq. 3),
    bottleneck = 3 * 2^21 (Eq. 4), w = 2^20 + 3 * 2^21 (Eq. 5)."""
    r = fit([1 << 20, 1 << 21], [0, 0], [0, 1], 0, 3, 0)
    assert r["s_p"] == 1 << 20 and r["s_d"] == 3 << 21
    assert r["phase"] == 3 << 21
    assert r["w"] == (1 << 20) + (3 << 21)


def test_rates_add_over_replicas(orc):
    """Prefill replicas at 2^20, 2^21 and 2^22 ns serve like one replica at
    1 / (2^-20 + 2^-21 + 2^-22) = 2^22 / 7 ns, rounded up (rates summed over
    replicas, Sec. 3.3); with T_a above the phase the wait is 0 (Eq. 5)."""
    r = fit([1 << 20, 1 << 21, 1 << 22, 1 << 23], [0] * 4, [0, 0, 0, 1], 1 << 30, 1, 0)
    assert r["s_p"] == -(-(1 << 22) // 7) and r["s_d"] == 1 << 23
    assert r["phase"] == 1 << 23 and r["w"] == 0


def test_no_wait_below_arrival_interval(orc):
    rng = np.random.default_rng(2)
    for _ in range(200):
        K = int(rng.integers(2, 8))
        T = rng.integers(1, 10**10, size=K)
        roles = np.r_[0, 1, rng.integers(0, 2, size=K - 2)]
        r = fit(T, np.zeros(K), roles, INF - 1, int(rng.integers(0, 8193)), 0)
        assert r["w"] == 0 and r["phase"] != INF


def test_wait_formula_when_overloaded(orc):
    """Eq. 4-5: w = NP/PS + (phase - T_a) once the phase exceeds T_a."""
    r = fit([1 << 30, 1 << 30], [0, 0], [0, 1], 10**8, 2, 0)
    assert r["s_p"] == 1 << 30 and r["s_d"] == 2 << 30
    assert r["w"] == (1 << 30) + (2 << 30) - 10**8


def test_qos_floor(orc):
    """A decode replica is kept only if 1 / Lambda >= Min_TPS = 7 tokens/s
    (Algorithm 2, Sec. 3.5): Lambda <= 142857142 ns."""
    g = json.load(open(os.path.join(GOLDEN, "paper_values.json")))["qos_floor"]
    lim = g["lambda_max_ns"]
    ok = fit([10**6, 10**6], [0, lim], [0, 1], 0, 1, g["min_tps_milli"])
    assert ok["w"] != INF
    bad = fit([1 << 20, 1 << 20], [0, lim + 1], [0, 1], 0, 1, g["min_tps_milli"])
    assert bad["w"] == INF and bad["s_d"] == INF and bad["s_p"] == 1 << 20
    # prefill replicas are never filtered by the floor
    pre = fit([10**6, 10**6], [lim + 1, 0], [0, 1], 0, 1, g["min_tps_milli"])
    assert pre["w"] != INF
    # a zero floor disables the filter
    off = fit([10**6, 10**6], [0, INF - 1], [0, 1], 0, 1, 0)
    assert off["w"] != INF


def test_missing_role_is_infeasible(orc):
    assert fit([5, 7], [0, 0], [0, 0], 0, 1, 0)["w"] == INF
    assert fit([5, 7], [0, 0], [1, 1], 0, 1, 0)["w"] == INF
    assert fit([INF, 7], [INF, 0], [0, 1], 0, 1, 0)["w"] == INF


def test_adding_a_replica_never_slows_its_phase(orc):
    rng = np.random.default_rng(4)
    for _ in range(300):
        K = int(rng.integers(2, 9))
        T = rng.integers(1, 10**11, size=K)
        roles = np.r_[0, 1, rng.integers(0, 2, size=K - 2)]
        nd = int(rng.integers(0, 8193))
        base = fit(T, np.zeros(K), roles, 0, nd, 0)
        extra_role = int(rng.integers(0, 2))
        more = fit(np.r_[T, rng.integers(1, 10**11)], np.zeros(K + 1),
                   np.r_[roles, extra_role], 0, nd, 0)
        key = "s_p" if extra_role == 0 else "s_d"
        assert more[key] <= base[key]
        other = "s_d" if extra_role == 0 else "s_p"
        assert more[other] == base[other]


def test_fixed_point_brackets_exact_rates(orc):
    """With rho = floor(2^50 / T) and S_P = ceil(2^50 / sum rho):
    1 / sum(1/T) <= S_P <= 2^50 / (2^50 * sum(1/T) - K) + 1 for K replicas."""
    from fractions import Fraction
    rng = np.random.default_rng(6)
    for _ in range(300):
        T = rng.integers(1, 10**11, size=int(rng.integers(1, 6)))
        K = len(T)
        r = fit(np.r_[T, 10**6], np.zeros(K + 1), np.r_[np.zeros(K), 1], 0, 1, 0)
        inv = sum(Fraction(1, int(x)) for x in T)
        assert 1 / inv <= r["s_p"] <= Fraction(SCALE) / (SCALE * inv - K) + 1
