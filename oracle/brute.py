"""Brute-force enumeration for tiny partition problems (test infrastructure only).

This is the independent pin for the oracle's dynamic program: it never runs
the recurrence of Eq. 1.  It enumerates every master position and every
composition of the N blocks into m contiguous non-empty stages (reading R1),
scores each with the bottleneck of Sec. 3.2 (stage compute time, the master's
head time, link transfer times inside the max, memory-infeasible = INF), and
derives

  T        the minimum bottleneck over masters and compositions;
  mu_star  the smallest master position attaining T (R5);
  sizes    the stage sizes that the paper's backtrack recovers (R3, R4):
           walking from the last device, the last stage starts at the
           smallest j whose prefix optimum (found by enumeration) combined
           with this stage reproduces the current subproblem optimum;
  Lambda   the sum of stage times plus link times (Sec. 3.2).

It also enumerates the idle-device relaxation (devices may hold zero blocks
and drop out of the pipeline; the master always takes part), under which the
"adding a device never worsens the optimum" invariant holds.
"""
from __future__ import annotations

import itertools
from functools import lru_cache

INF = (1 << 64) - 1


def compositions(n: int, parts: int, min_part: int = 1):
    """All tuples of `parts` integers >= min_part summing to n."""
    if parts == 0:
        if n == 0:
            yield ()
        return
    if min_part == 1:
        for cuts in itertools.combinations(range(1, n), parts - 1):
            b = (0,) + cuts + (n,)
            yield tuple(b[i + 1] - b[i] for i in range(parts))
    else:
        for cuts in itertools.combinations_with_replacement(range(0, n + 1), parts - 1):
            b = (0,) + cuts + (n,)
            yield tuple(b[i + 1] - b[i] for i in range(parts))


class Chain:
    """One device chain with its per-block times, head times, links, memory."""

    def __init__(self, tk, hk, tau_link, memk, W, HB):
        self.tk = [[int(x) for x in row] for row in tk]
        self.hk = [int(x) for x in hk]
        self.tl = [int(x) for x in tau_link]
        self.mem = [int(x) for x in memk]
        self.W = [int(x) for x in W]
        self.HB = int(HB)
        self.m = len(self.tk)
        self.N = len(self.W)

    def stage_cost(self, k: int, j: int, i: int, master: bool) -> int:
        """Time of device k (0-based) running blocks j..i, or INF if it does not fit."""
        b = sum(self.W[j:i + 1]) + (self.HB if master else 0)
        if b > self.mem[k]:
            return INF
        return sum(self.tk[k][j:i + 1]) + (self.hk[k] if master else 0)

    def bottleneck(self, sizes, mu: int) -> int:
        """Max over stage times and link times; mu is 1-based."""
        v = 0
        start = 0
        for k, s in enumerate(sizes):
            c = self.stage_cost(k, start, start + s - 1, k + 1 == mu)
            if c == INF:
                return INF
            v = max(v, c)
            if k >= 1:
                v = max(v, self.tl[k])
            start += s
        return v

    def solve(self):
        m, N = self.m, self.N
        if m > N:
            return INF, INF, 0, [0] * m
        best, best_mu = INF, 0
        for mu in range(1, m + 1):
            t_mu = min((self.bottleneck(c, mu) for c in compositions(N, m)), default=INF)
            if t_mu < best:
                best, best_mu = t_mu, mu
        if best == INF:
            return INF, INF, 0, [0] * m
        sizes = self._backtrack(best_mu)
        lam = 0
        start = 0
        for k, s in enumerate(sizes):
            lam += sum(self.tk[k][start:start + s])
            if k + 1 == best_mu:
                lam += self.hk[k]
            if k >= 1:
                lam += self.tl[k]
            start += s
        return best, lam, best_mu, sizes

    def _backtrack(self, mu: int):
        @lru_cache(maxsize=None)
        def opt(i: int, k: int) -> int:
            """Best bottleneck of blocks 0..i on devices 1..k (enumeration)."""
            if i + 1 < k:
                return INF
            best = INF
            for c in compositions(i + 1, k):
                v = 0
                start = 0
                for kk, s in enumerate(c):
                    cc = self.stage_cost(kk, start, start + s - 1, kk + 1 == mu)
                    if cc == INF:
                        v = INF
                        break
                    v = max(v, cc)
                    if kk >= 1:
                        v = max(v, self.tl[kk])
                    start += s
                best = min(best, v)
            return best

        sizes = [0] * self.m
        i = self.N - 1
        for k in range(self.m, 1, -1):
            target = opt(i, k)
            chosen = None
            for j in range(0, i + 1):
                prev = opt(j - 1, k - 1) if j >= 1 else INF
                if prev == INF:
                    continue
                c = self.stage_cost(k - 1, j, i, k == mu)
                if c == INF:
                    continue
                if max(prev, c, self.tl[k - 1]) == target:
                    chosen = j
                    break
            assert chosen is not None
            sizes[k - 1] = i - chosen + 1
            i = chosen - 1
        sizes[0] = i + 1
        return sizes

    def end_to_end(self, sizes, mu: int) -> int:
        """Sum of stage times and link times (the finishing-time objective);
        INF if a stage does not fit or a link is dead."""
        v = 0
        start = 0
        for k, s in enumerate(sizes):
            c = self.stage_cost(k, start, start + s - 1, k + 1 == mu)
            if c == INF or (k >= 1 and self.tl[k] == INF):
                return INF
            v += c + (self.tl[k] if k >= 1 else 0)
            start += s
        return v

    def solve_sum(self):
        """The finishing-time variant by enumeration: the master and stages
        with the least end-to-end time (smallest master on ties, then the
        split points the backtrack's smallest-j rule recovers).  Returns
        (bottleneck of that partition, its end-to-end time, mu, sizes)."""
        m, N = self.m, self.N
        if m > N:
            return INF, INF, 0, [0] * m
        best, best_mu = INF, 0
        for mu in range(1, m + 1):
            s_mu = min((self.end_to_end(c, mu) for c in compositions(N, m)), default=INF)
            if s_mu < best:
                best, best_mu = s_mu, mu
        if best == INF:
            return INF, INF, 0, [0] * m
        mu = best_mu

        @lru_cache(maxsize=None)
        def opt(i: int, k: int) -> int:
            """Least end-to-end time of blocks 0..i on devices 1..k."""
            if i + 1 < k:
                return INF
            return min((self.end_to_end(c, mu) for c in compositions(i + 1, k)), default=INF)

        sizes = [0] * m
        i = N - 1
        for k in range(m, 1, -1):
            target = opt(i, k)
            chosen = None
            for j in range(0, i + 1):
                prev = opt(j - 1, k - 1) if j >= 1 else INF
                c = self.stage_cost(k - 1, j, i, k == mu)
                if prev == INF or c == INF or self.tl[k - 1] == INF:
                    continue
                if prev + c + self.tl[k - 1] == target:
                    chosen = j
                    break
            assert chosen is not None
            sizes[k - 1] = i - chosen + 1
            i = chosen - 1
        sizes[0] = i + 1
        return self.bottleneck(sizes, mu), best, mu, sizes

    def solve_idle_relaxed(self, only_mu=None) -> int:
        """Optimum when devices may hold zero blocks (they then leave the
        pipeline; links join consecutive participating devices).  The master
        always participates, with its head, even with zero blocks.  With
        only_mu, the optimum for that master position."""
        m, N = self.m, self.N
        best = INF
        for mu in range(1, m + 1):
            if only_mu is not None and mu != only_mu:
                continue
            for c in compositions(N, m, min_part=0):
                used = [k for k in range(m) if c[k] > 0 or k + 1 == mu]
                v = 0
                start = [0] * m
                s = 0
                for k in range(m):
                    start[k] = s
                    s += c[k]
                for idx, k in enumerate(used):
                    if c[k] > 0:
                        cc = self.stage_cost(k, start[k], start[k] + c[k] - 1, k + 1 == mu)
                    else:
                        cc = self.hk[k] if self.HB <= self.mem[k] else INF
                    if cc == INF:
                        v = INF
                        break
                    v = max(v, cc)
                    if idx >= 1:
                        a, b = used[idx - 1], k
                        v = max(v, self.link(a, b))
                best = min(best, v)
        return best

    def idle_bottleneck(self, sizes, mu: int) -> int:
        """Bottleneck of a relaxed partition: participants are the devices
        with blocks and the master (head only when it holds none)."""
        used = [k for k in range(self.m) if sizes[k] > 0 or k + 1 == mu]
        start = [0] * self.m
        s = 0
        for k in range(self.m):
            start[k] = s
            s += sizes[k]
        v = 0
        for idx, k in enumerate(used):
            if sizes[k] > 0:
                c = self.stage_cost(k, start[k], start[k] + sizes[k] - 1, k + 1 == mu)
            else:
                c = self.hk[k] if self.HB <= self.mem[k] else INF
            if c == INF:
                return INF
            v = max(v, c)
            if idx >= 1:
                lt = self.link(used[idx - 1], k)
                if lt == INF:
                    return INF
                v = max(v, lt)
        return v

    def link(self, a: int, b: int) -> int:
        """Link time between chain positions a < b.  Only adjacent positions
        carry a given time in tau_link; a non-adjacent pair uses the matrix
        supplied with set_links (idle-device relaxation only)."""
        if b == a + 1:
            return self.tl[b]
        return self.full_links[a][b]

    def set_links(self, full):
        self.full_links = [[int(x) for x in row] for row in full]
