"""Seeded synthetic workloads for the population-fitness path.

This module builds integer input arrays only.  It holds none of the method's
arithmetic (no quantisation, no partitioning, no fitness): both the HIP path
and the CPU oracle consume the arrays it returns, so it is the one piece the
two sides share.

The recipe follows the paper's setting (Sec. 3.1-3.3 and Sec. 4.1 of
E2LLM, arXiv 2606.03770): a pool of heterogeneous edge devices with a
per-device compute speed and memory cap, a link-bandwidth matrix scaled by a
congestion factor, and a decoder-only model whose transformer blocks all have
the same size.  Layer costs are the analytic 2*params*tokens FLOPs of one
block, the activation crossing a link is hidden*2 bytes per token, and the LM
head plus output layer (2*hidden*V parameters, V = 32000) sit on the master
device of each replica.

Five named workloads span 12 to 256 devices and 16 to 16384 genomes.  Each
genome gives every device a cluster label in [0, K) (K drawn per genome) and
every cluster a role bit (0 = prefill, 1 = decode).

All floating-point draws are converted to integers here, once: speeds to
FLOP/s, bandwidths to B/s, congestion to parts per million.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

GB = 10**9
VOCAB = 32000


@dataclasses.dataclass
class Workload:
    """One problem instance plus one population, all integer arrays."""

    name: str
    n_dev: int
    n_layer: int
    speed_flops: np.ndarray      # u64 [M]
    mem_bytes: np.ndarray        # u64 [M]
    bw_Bps: np.ndarray           # u64 [M*M]
    congestion_ppm: np.ndarray   # u32 [M*M]
    layer_flops: np.ndarray      # u64 [2][N]; row 0 prefill (whole prompt), row 1 decode (one token)
    layer_bytes: np.ndarray      # u64 [N]
    act_bytes: np.ndarray        # u64 [2]
    head_flops: np.ndarray       # u64 [2]
    head_bytes: int
    labels: np.ndarray           # u8 [P][M]
    roles: np.ndarray            # u8 [P][k_max]
    k_max: int
    # fitness parameters (Eq. 3-5): arrival interval, generated tokens, QoS floor
    t_arrival_ns: int
    nd_tokens: int
    min_tps_milli: int
    # GA parameters (only meaningful for the 16384-genome workload)
    ga_seed: int = 0
    generations: int = 0
    tournament_k: int = 4
    crossover_thresh_u32: int = 1 << 31
    mutation_thresh_u32: int = 1 << 24
    n_elite: int = 1

    @property
    def population(self) -> int:
        return int(self.labels.shape[0])

    def problem_arrays(self) -> dict:
        return dict(
            n_dev=self.n_dev, n_layer=self.n_layer,
            speed_flops=self.speed_flops, mem_bytes=self.mem_bytes,
            bw_Bps=self.bw_Bps, congestion_ppm=self.congestion_ppm,
            layer_flops=self.layer_flops, layer_bytes=self.layer_bytes,
            act_bytes=self.act_bytes, head_flops=self.head_flops,
            head_bytes=self.head_bytes)

    def fitness_params(self) -> dict:
        return dict(t_arrival_ns=self.t_arrival_ns, nd_tokens=self.nd_tokens,
                    min_tps_milli=self.min_tps_milli)

    def prompt_tokens(self) -> int:
        """Prompt length NP in tokens, as the activation sizes were built:
        the prefill activation carries NP tokens, the decode one a single
        token."""
        act = [int(x) for x in self.act_bytes]
        return act[0] // max(act[1], 1)

    def ga_params(self, generation: int = 0) -> dict:
        return dict(seed=self.ga_seed, generation=generation,
                    tournament_k=self.tournament_k,
                    crossover_thresh_u32=self.crossover_thresh_u32,
                    mutation_thresh_u32=self.mutation_thresh_u32,
                    n_elite=self.n_elite)

    def subset(self, rows) -> "Workload":
        """Same problem instance, population restricted to the given genome rows."""
        w = dataclasses.replace(self)
        w.labels = np.ascontiguousarray(self.labels[rows])
        w.roles = np.ascontiguousarray(self.roles[rows])
        return w


# name: (M, N, bytes per layer, hidden, prompt tokens, mem choices (GB),
#        bandwidth kind, population, K range, P(prefill), GA generations)
SPECS = {
    "c1_tiny_12dev_32L": dict(M=12, N=32, layer_params=0.2e9, hidden=4096, prompt=512,
                              mem_gb=(4, 8, 16), bw="uniform_light", P=16, K=(3, 3),
                              p_prefill=0.5, generations=0),
    "c2_32dev_48L": dict(M=32, N=48, layer_params=0.27e9, hidden=5120, prompt=1024,
                         mem_gb=(4, 8, 16), bw="uniform_light", P=256, K=(4, 6),
                         p_prefill=0.5, generations=0),
    "c3_64dev_80L": dict(M=64, N=80, layer_params=0.9e9, hidden=8192, prompt=1024,
                         mem_gb=(8, 16, 24, 32), bw="congested", P=1024, K=(8, 12),
                         p_prefill=0.5, generations=0),
    "c4_128dev_80L": dict(M=128, N=80, layer_params=0.9e9, hidden=8192, prompt="lognormal",
                          mem_gb=(8, 16, 24, 32), bw="congested", P=4096, K=(16, 24),
                          p_prefill=0.3, generations=0),
    "c5_256dev_126L_ga": dict(M=256, N=126, layer_params=1.6e9, hidden=16384, prompt=1024,
                              mem_gb=(8, 16, 24, 32), bw="congested", P=16384, K=(32, 48),
                              p_prefill=0.5, generations=50),
}
NAMES = list(SPECS)


def _sym(rng_vals: np.ndarray, M: int) -> np.ndarray:
    """Mirror the upper triangle of an [M, M] draw; the diagonal is left as drawn."""
    up = np.triu(rng_vals, 1)
    return up + up.T + np.diag(np.diag(rng_vals))


def make(name: str, seed: Optional[int] = None, population: Optional[int] = None,
         layer_types: int = 1, type_ratio: float = 1.0) -> Workload:
    """Build a named workload.

    seed defaults to the workload's index (0..4) in NAMES.  population
    overrides P (the genome draws are the first rows of the same stream only
    when P is unchanged; a different P redraws).  layer_types > 1 alternates
    block types whose FLOPs and bytes differ by type_ratio (the paper notes
    that sliding-window and full-attention blocks profile differently,
    Sec. 3.1); the named workloads use one block type.
    """
    spec = SPECS[name]
    if seed is None:
        seed = NAMES.index(name)
    rng = np.random.Generator(np.random.PCG64(seed))
    M, N = spec["M"], spec["N"]
    P = spec["P"] if population is None else int(population)

    # 1. speeds: 10 TFLOP/s x lognormal(0, 0.5)
    speed = np.rint(10e12 * np.exp(rng.normal(0.0, 0.5, size=M))).astype(np.uint64)
    speed = np.maximum(speed, 1).astype(np.uint64)
    # 2. memory caps
    mem = (rng.choice(np.array(spec["mem_gb"], dtype=np.uint64), size=M) * GB).astype(np.uint64)
    # 3-4. bandwidth and congestion, symmetric
    if spec["bw"] == "uniform_light":
        bw = _sym(rng.uniform(0.1, 1.0, size=(M, M)), M)
        cong = _sym(rng.uniform(0.3, 1.0, size=(M, M)), M)
    else:
        bw = _sym(rng.uniform(0.05, 2.0, size=(M, M)), M)
        cong = _sym(np.where(rng.uniform(size=(M, M)) < 0.2, 0.1, 1.0), M)
    bw_Bps = np.rint(bw * GB).astype(np.uint64).reshape(-1)
    cong_ppm = np.rint(cong * 1e6).astype(np.uint32).reshape(-1)
    # 5. prompt length
    if spec["prompt"] == "lognormal":
        lens = np.exp(rng.normal(math.log(1024.0) - 0.32, 0.8, size=1000))
        lens = np.clip(lens, 64, 8192)
        prompt = int(round(float(np.mean(np.rint(lens)))))
    else:
        prompt = int(spec["prompt"])
    # 6. population: K per genome, labels, roles
    klo, khi = spec["K"]
    K = rng.integers(klo, khi + 1, size=P)
    labels = (rng.uniform(size=(P, M)) * K[:, None]).astype(np.uint8)
    roles = (rng.uniform(size=(P, khi)) >= spec["p_prefill"]).astype(np.uint8)

    params = spec["layer_params"]
    hidden = spec["hidden"]
    ltype = np.arange(N) % max(layer_types, 1)
    scale = np.where(ltype == 0, 1.0, type_ratio)
    layer_bytes = np.rint(params * scale).astype(np.uint64)
    lf_prefill = np.rint(2.0 * params * scale * prompt).astype(np.uint64)
    lf_decode = np.rint(2.0 * params * scale).astype(np.uint64)
    head = 2 * hidden * VOCAB
    return Workload(
        name=name, n_dev=M, n_layer=N,
        speed_flops=speed, mem_bytes=mem, bw_Bps=bw_Bps, congestion_ppm=cong_ppm,
        layer_flops=np.stack([lf_prefill, lf_decode]).astype(np.uint64),
        layer_bytes=layer_bytes,
        act_bytes=np.array([hidden * 2 * prompt, hidden * 2], dtype=np.uint64),
        head_flops=np.array([head, head], dtype=np.uint64),
        head_bytes=int(head),
        labels=labels, roles=roles, k_max=int(khi),
        t_arrival_ns=100_000_000, nd_tokens=prompt, min_tps_milli=7000,
        ga_seed=int(seed), generations=int(spec["generations"]))


def random_small(seed: int, M: int, N: int, P: int, k_max: int, *,
                 mem_lo_layers: float = 1.0, mem_hi_layers: float = 40.0,
                 zero_bw_frac: float = 0.0, head: bool = True,
                 layer_var: bool = True, cong_full: bool = False) -> Workload:
    """A small random instance for parity and property tests.

    Costs are drawn so that ties, tight memory and infeasible clusters all
    occur: per-layer FLOPs vary by layer (layer_var), memory caps are drawn in
    units of the mean layer size, and a fraction of links can have zero
    effective bandwidth (an infinite transfer time).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    speed = rng.integers(1, 50, size=M).astype(np.uint64) * np.uint64(10**11)
    lb_mean = 10**8
    if layer_var:
        layer_bytes = rng.integers(lb_mean // 2, 2 * lb_mean, size=N).astype(np.uint64)
        lf = rng.integers(1, 8, size=(2, N)).astype(np.uint64) * np.uint64(10**11)
    else:
        layer_bytes = np.full(N, lb_mean, dtype=np.uint64)
        lf = np.full((2, N), 3 * 10**11, dtype=np.uint64)
    mem = (rng.uniform(mem_lo_layers, mem_hi_layers, size=M) * lb_mean).astype(np.uint64)
    bw = _sym(rng.integers(10**6, 10**9, size=(M, M)).astype(np.float64), M)
    if cong_full:
        cong = np.full((M, M), 1e6)
    else:
        cong = _sym(rng.integers(100_000, 1_000_001, size=(M, M)).astype(np.float64), M)
    if zero_bw_frac > 0:
        z = _sym((rng.uniform(size=(M, M)) < zero_bw_frac).astype(np.float64), M)
        bw = np.where(z > 0, 0.0, bw)
    head_f = int(rng.integers(0, 3)) * 10**11 if head else 0
    head_b = int(rng.integers(0, 2)) * lb_mean if head else 0
    labels = rng.integers(0, k_max, size=(P, M)).astype(np.uint8)
    roles = rng.integers(0, 2, size=(P, k_max)).astype(np.uint8)
    return Workload(
        name=f"random_small_{seed}", n_dev=M, n_layer=N,
        speed_flops=speed, mem_bytes=mem,
        bw_Bps=bw.astype(np.uint64).reshape(-1),
        congestion_ppm=cong.astype(np.uint32).reshape(-1),
        layer_flops=lf, layer_bytes=layer_bytes,
        act_bytes=np.array([int(rng.integers(10**6, 10**8)), int(rng.integers(10**3, 10**5))],
                           dtype=np.uint64),
        head_flops=np.array([head_f, head_f // 7], dtype=np.uint64),
        head_bytes=head_b, labels=labels, roles=roles, k_max=k_max,
        t_arrival_ns=int(rng.integers(0, 10**9)), nd_tokens=int(rng.integers(0, 2048)),
        min_tps_milli=int(rng.choice([0, 7000, 100000])),
        ga_seed=seed, generations=0)


@dataclasses.dataclass
class OrderedPopulation:
    """A population of two-chromosome genomes (the paper's App. A gene): an
    ordering chromosome order[P][M] (a permutation of the devices), a
    grouping chromosome sizes[P][k_max] (replica sizes in ordering order,
    summing to M, zeros after the last replica) and a role per replica."""
    order: np.ndarray   # u8 [P][M]
    sizes: np.ndarray   # u16 [P][k_max]
    roles: np.ndarray   # u8 [P][k_max]
    max_replica: int    # largest replica size the GA draws when it regrows a grouping
    mutation_thresh_u32: int = int(0.3 * 2**32)  # App. A: about 30% of genes mutate

    def ga_params(self, wl: Workload, generation: int = 0) -> dict:
        return dict(seed=wl.ga_seed, generation=generation, tournament_k=wl.tournament_k,
                    mutation_thresh_u32=self.mutation_thresh_u32, n_elite=wl.n_elite,
                    max_replica=self.max_replica)

    def subset(self, rows) -> "OrderedPopulation":
        return dataclasses.replace(self, order=np.ascontiguousarray(self.order[rows]),
                                   sizes=np.ascontiguousarray(self.sizes[rows]),
                                   roles=np.ascontiguousarray(self.roles[rows]))


def ordered_population(wl: Workload, seed: Optional[int] = None,
                       population: Optional[int] = None) -> OrderedPopulation:
    """Two-chromosome genomes for a named workload's problem instance.

    Each genome is generated the way the GA regenerates both chromosomes: a
    uniform random ordering, then replicas of 1 + floor(U * max_replica)
    devices (U uniform in [0, 1)) along it until the devices run out, the
    last of the k_max slots taking whatever remains; roles prefill with the
    workload's P(prefill).  max_replica, also the GA's regrowth bound, is
    twice M over the mean of the workload's K range, so a genome holds about
    that many replicas.
    """
    spec = SPECS[wl.name] if wl.name in SPECS else None
    klo, khi = spec["K"] if spec else (1, wl.k_max)
    p_prefill = spec["p_prefill"] if spec else 0.5
    if seed is None:
        seed = 1000 + wl.ga_seed
    rng = np.random.Generator(np.random.PCG64(seed))
    M = wl.n_dev
    P = wl.labels.shape[0] if population is None else int(population)
    khi = min(khi, M)
    klo = min(klo, khi)
    max_replica = max(1, min(256, int(round(2 * M / ((klo + khi) / 2)))))
    K = wl.k_max
    order = np.stack([rng.permutation(M) for _ in range(P)]).astype(np.uint8)
    draws = 1 + (rng.uniform(size=(P, K)) * max_replica).astype(np.int64)
    sizes = np.zeros((P, K), dtype=np.uint16)
    for p in range(P):
        left = M
        for r in range(K):
            if left == 0:
                break
            s = left if r == K - 1 else min(int(draws[p, r]), left)
            sizes[p, r] = s
            left -= s
    roles = ((rng.uniform(size=(P, K)) >= p_prefill) & (sizes > 0)).astype(np.uint8)
    return OrderedPopulation(order=order, sizes=sizes, roles=roles, max_replica=max_replica)


def slot_model(wl: Workload, b_max: int = 8, beta_ppm: int = 125_000) -> dict:
    """Decode-slot model of a workload for the role and slot search.

    A request in flight holds the K and V of its NP + ND tokens for each
    block it passes: 2 * (hidden * 2 bytes) * (NP + ND) bytes per block,
    with hidden * 2 = the decode activation bytes and NP their ratio to the
    prefill activation.  Each further request adds beta_ppm / 1e6 of a lone
    request's decode block and head time.  b_max = 8 follows the paper's
    example of a device whose memory holds four or, with a second pipeline
    stage, eight concurrent requests.
    """
    kv = 2 * int(wl.act_bytes[1]) * (wl.prompt_tokens() + int(wl.nd_tokens))
    return dict(b_max=int(b_max), beta_ppm=int(beta_ppm), kv_bytes_per_block_slot=kv)
