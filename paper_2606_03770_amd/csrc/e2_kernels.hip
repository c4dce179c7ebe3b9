// HIP kernels (gfx950, wave64) of the population-fitness path.
//
//   k_init        zero the per-call counters (a fill kernel, no memset node)
//   k_extract     one workgroup per individual: cluster sizes, a necessary
//                 memory/size pre-check, the list of clusters that need the
//                 DP; writes INF results for the others
//   k_dp          persistent waves: each takes the next listed cluster,
//                 rebuilds its device chain from the genome, runs the
//                 bottleneck DP of Algorithm 1 / Eq. 1-2 for every master
//                 position, picks the best master, backtracks and writes
//                 T, Lambda, master and per-device block counts
//   k_fitness     Eq. 3-5 per individual with the QoS floor
//   k_elites      one workgroup: the n_elite best keys (w, phase, index)
//   k_breed       one wave per output slot: elite copy or tournament +
//                 uniform crossover + per-gene mutation
//
// DP encoding.  A candidate of row k (device c holds blocks j..i, devices
// 1..k-1 hold 0..j-1) is scored max(DP(j-1, k-1), tau(k-1, k), cost(j, i)).
// Values are < 2^56 and j < 256, so the score is packed as (value << 8) | j:
// one unsigned min over packed scores yields the smallest value and, among
// equal values, the smallest j (the tie rule of the recurrence).  The
// prefix term max(DP(j-1, k-1), tau) is packed once per j; the stage cost is
// pre-shifted prefix sums, (P[i+1] << 8) - ((P[j] << 8) - j) = (cost << 8) | j.
// The memory cap turns into a window j >= win[i] (block bytes are
// non-negative, so the fitting starts of a stage ending at i are a suffix).

#include "e2_internal.h"

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
    for (int off = 32; off >= 1; off >>= 1) v = umin64(v, __shfl_xor(v, off, kWave));
    return v;
}

__global__ void k_init(uint32_t *counters)
{
    if (threadIdx.x < 4) counters[threadIdx.x] = 0;
}

// ---------------------------------------------------------------------------
// Extraction and pre-check: one 256-thread workgroup per individual.
// A cluster goes to the DP list unless it is empty or provably infeasible:
//   more devices than blocks (every device must hold a block), a device that
//   cannot hold a single block, total single-stage capacity below N, or no
//   device able to hold a block plus the head (no possible master).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_extract(E2Tables tb, int P, int k_max,
                                                 const uint8_t *__restrict__ labels,
                                                 uint32_t *counters, uint32_t *list,
                                                 uint64_t *T, uint64_t *Lambda, int16_t *master,
                                                 uint8_t *layers)
{
    __shared__ uint32_t cnt[256], csum[256], cmin[256], hasH[256];
    __shared__ uint8_t listed[256];
    __shared__ uint32_t nlist, base;
    const int p = blockIdx.x;
    const int t = threadIdx.x;
    const int M = tb.M, N = tb.N;
    cnt[t] = 0;
    csum[t] = 0;
    cmin[t] = 0xFFFFFFFFu;
    hasH[t] = 0;
    if (t == 0) nlist = 0;
    __syncthreads();
    int lab = 256;
    if (t < M) {
        lab = labels[(size_t)p * M + t];
        if (lab < k_max) {
            atomicAdd(&cnt[lab], 1u);
            atomicAdd(&csum[lab], (uint32_t)tb.cap0[t]);
            atomicMin(&cmin[lab], (uint32_t)tb.cap0[t]);
            if (tb.capH[t]) atomicOr(&hasH[lab], 1u);
        }
    }
    __syncthreads();
    bool feas = false;
    uint32_t slot = 0;
    if (t < k_max) {
        const uint32_t m = cnt[t];
        feas = m >= 1 && m <= (uint32_t)N && csum[t] >= (uint32_t)N && cmin[t] >= 1 && hasH[t];
        if (feas) slot = atomicAdd(&nlist, 1u);
        listed[t] = feas;
    }
    __syncthreads();
    if (t == 0 && nlist) base = atomicAdd(&counters[0], nlist);
    __syncthreads();
    if (t < k_max) {
        const size_t o = (size_t)p * k_max + t;
        if (feas) {
            list[base + slot] = ((uint32_t)p << 8) | (uint32_t)t;
        } else {
            T[o] = E2_INF64;
            Lambda[o] = E2_INF64;
            if (master) master[o] = -1;
        }
    }
    if (layers && t < M && (lab >= k_max || !listed[lab])) layers[(size_t)p * M + t] = 0;
}

// ---------------------------------------------------------------------------
// Shared-memory layout of one DP wave.  Rows hold N+1 entries.
// ---------------------------------------------------------------------------
struct DpSmem {
    uint64_t *Pp;    // packed prefix term of the current row, by split point j
    uint64_t *S2;    // packed prefix sums of the current row's device
    uint64_t *Ga;    // backward row (ping)
    uint64_t *Gb;    // backward row (pong)
    uint64_t *pool;  // band-packed forward rows, pool_cells entries
    uint8_t *tbp;    // split points, same packing as pool
    int pool_cells;
};

__device__ __forceinline__ const uint64_t *pref_row(const E2Tables &tb, int r, int c)
{
    return tb.pref + ((size_t)r * tb.M + c) * (tb.N + 1);
}
__device__ __forceinline__ const uint8_t *win_row(const E2Tables &tb, int f, int c)
{
    return tb.win + ((size_t)f * tb.M + c) * tb.N;
}
__device__ __forceinline__ uint64_t link_tau(const E2Tables &tb, int r, int a, int b)
{
    return tb.tau[((size_t)r * tb.M + a) * tb.M + b];
}
__device__ __forceinline__ uint64_t pack_prev(uint64_t prev, uint64_t tau, int j)
{
    return (prev == E2_INF64 || tau == E2_INF64) ? E2_INF64
                                                  : ((umax64(prev, tau) << 8) | (uint64_t)j);
}

// Minimum packed score of cell i: min over j in [jlo, i] of max(Pp[j], cost(j, i)).
__device__ __forceinline__ uint64_t cell_min(const uint64_t *Pp, const uint64_t *S2, uint64_t si1,
                                             int jlo, int i)
{
    uint64_t best = E2_INF64;
    for (int j = jlo; j <= i; ++j) best = umin64(best, umax64(Pp[j], si1 - S2[j]));
    return best;
}

// ---------------------------------------------------------------------------
// Exact reference path: one full table per master position (Algorithm 1 as
// stated), used when a chain's band-packed rows do not fit the LDS pool.
// D, Pp, S2 are LDS rows; tbp (LDS or global) receives split points of rows
// 2..m.  Returns DP_mu(N-1, m).
// ---------------------------------------------------------------------------
__device__ uint64_t dp_table(const E2Tables &tb, int r, const uint8_t *chain, int m, int mu,
                             uint8_t *tbp, uint64_t *D, uint64_t *Pp, uint64_t *S2, int lane)
{
    const int N = tb.N;
    {
        const int c = chain[0];
        const int f = (mu == 1);
        const uint64_t *pr = pref_row(tb, r, c);
        const uint8_t *wr = win_row(tb, f, c);
        const uint64_t hadd = f ? tb.head[r * tb.M + c] : 0;
        for (int i = lane; i < N; i += kWave) D[i] = (wr[i] == 0) ? pr[i + 1] + hadd : E2_INF64;
    }
    __syncthreads();
    for (int k = 2; k <= m; ++k) {
        const int c = chain[k - 1];
        const int f = (mu == k);
        const uint64_t tau = link_tau(tb, r, chain[k - 2], c);
        const uint64_t *pr = pref_row(tb, r, c);
        const uint8_t *wr = win_row(tb, f, c);
        const uint64_t hadd = f ? tb.head[r * tb.M + c] : 0;
        for (int j = lane; j < N; j += kWave) {
            Pp[j] = pack_prev(j == 0 ? E2_INF64 : D[j - 1], tau, j);
            S2[j] = (pr[j] << 8) - (uint64_t)j;
        }
        __syncthreads();
        for (int i = lane; i < N; i += kWave) {
            uint64_t best = E2_INF64;
            int lo = wr[i];
            if (lo != (int)E2_NO_START && i >= k - 1)
                best = cell_min(Pp, S2, (pr[i + 1] + hadd) << 8, lo < k - 1 ? k - 1 : lo, i);
            D[i] = (best == E2_INF64) ? E2_INF64 : (best >> 8);
            if (tbp) tbp[(size_t)(k - 2) * N + i] = (uint8_t)(best & 0xFF);
        }
        __syncthreads();
    }
    return D[N - 1];
}

// ---------------------------------------------------------------------------
// Band-pruned forward/backward path.
//
// With cap0[k] the longest stage device k holds without the head and
// pre[k] = cap0[1] + ... + cap0[k], a cell (i, k) of any table can lie on a
// complete memory-feasible partition only if
//     max(k-1, N-1-(pre[m]-pre[k])) <= i <= min(N-1-(m-k), pre[k]-1)
// (its devices cover blocks 0..i, the remaining devices cover the rest).
// Every memory-feasible candidate of an in-band cell reads an in-band cell
// of the previous row or an infinite one, so computing only in-band cells
// (others INF) leaves every in-band value and split point exact.
//
//   F_k  forward rows without master, k = 1..m-1 (pool, with split points)
//   G_k  backward rows without master: blocks j..N-1 on devices k..m,
//        k = m..2, each device >= 1 block, links k..m included
//   T_mu = min_i max( min_j max(A(j), cost_mu(j, i) + head), B(i) )
//        A(j) = max(F_{mu-1}(j-1), tau(mu-1, mu))   (mu = 1: j = 0 only)
//        B(i) = max(tau(mu, mu+1), G_{mu+1}(i+1))   (mu = m: i = N-1 only)
//   which is the optimum of the table of Algorithm 1 for master mu.  The
//   smallest mu attaining min T_mu is the master; rows mu*..m of its table
//   (rows below mu* are F) give the split points for the back tracing.
// Returns false (nothing written) if the bands do not fit the pool.
// ---------------------------------------------------------------------------
struct Bands {
    uint8_t flo[256], fhi[256];  // forward band per row 1..m
    uint8_t glo[256], ghi[256];  // backward band per row 2..m
    uint16_t off[257];           // pool offset per forward row 1..m-1
    uint16_t pre[257];           // prefix sums of cap0 over the chain
    uint8_t cH[256];             // capH per chain position (1-based)
};

// Forward row k of the table for master mu (mu = 0: no master), cells in
// [lo, hi], from the previous row (pool row k-1 with band plo..phi) into
// pool row k (values + split points).  Row 1 uses Eq. 2 directly.
__device__ void fwd_row(const E2Tables &tb, const DpSmem &sm, const Bands &bd, int r,
                        const uint8_t *chain, int k, int mu, int lane, uint64_t *out,
                        uint8_t *out_tb)
{
    const int c = chain[k - 1];
    const int f = (mu == k);
    const int lo = bd.flo[k], hi = bd.fhi[k];
    const uint64_t *pr = pref_row(tb, r, c);
    const uint8_t *wr = win_row(tb, f, c);
    const uint64_t hadd = f ? tb.head[r * tb.M + c] : 0;
    if (k == 1) {
        for (int i = lo + lane; i <= hi; i += kWave)
            out[i - lo] = (wr[i] == 0) ? pr[i + 1] + hadd : E2_INF64;
        __syncthreads();
        return;
    }
    const int cap = f ? bd.cH[k] : (int)(bd.pre[k] - bd.pre[k - 1]);
    int jmin = lo - cap + 1;
    if (jmin < k - 1) jmin = k - 1;
    const uint64_t tau = link_tau(tb, r, chain[k - 2], c);
    const int plo = bd.flo[k - 1], phi = bd.fhi[k - 1];
    const uint64_t *prev = sm.pool + bd.off[k - 1];
    for (int j = jmin + lane; j <= hi; j += kWave) {
        const int pj = j - 1;
        sm.Pp[j] = pack_prev((pj >= plo && pj <= phi) ? prev[pj - plo] : E2_INF64, tau, j);
        sm.S2[j] = (pr[j] << 8) - (uint64_t)j;
    }
    __syncthreads();
    for (int i = lo + lane; i <= hi; i += kWave) {
        uint64_t best = E2_INF64;
        const int w = wr[i];
        if (w != (int)E2_NO_START)
            best = cell_min(sm.Pp, sm.S2, (pr[i + 1] + hadd) << 8, w < jmin ? jmin : w, i);
        out[i - lo] = (best == E2_INF64) ? E2_INF64 : (best >> 8);
        out_tb[i - lo] = (uint8_t)(best & 0xFF);
    }
    __syncthreads();
}

// Backward row k (k = m..2) into Gout (full length, INF outside the band).
__device__ void bwd_row(const E2Tables &tb, const DpSmem &sm, const Bands &bd, int r,
                        const uint8_t *chain, int k, int m, int lane, const uint64_t *Gin,
                        uint64_t *Gout)
{
    const int N = tb.N;
    const int c = chain[k - 1];
    const int lo = bd.glo[k], hi = bd.ghi[k];
    const uint64_t *pr = pref_row(tb, r, c);
    if (k == m) {
        const int w = win_row(tb, 0, c)[N - 1];
        for (int j = lane; j < N; j += kWave)
            Gout[j] = (j >= lo && j <= hi && w != (int)E2_NO_START && j >= w)
                          ? pr[N] - pr[j] : E2_INF64;
        __syncthreads();
        return;
    }
    const uint8_t *we = tb.wend + (size_t)c * N;
    const int imax = N - 1 - (m - k);
    const int cap = bd.pre[k] - bd.pre[k - 1];
    int ihi = hi + cap - 1;
    if (ihi > imax) ihi = imax;
    const uint64_t tau = link_tau(tb, r, c, chain[k]);
    // Pp <- Q(i) = max(G_{k+1}(i+1), tau(k, k+1)); S2 <- plain prefix sums
    for (int i = lo + lane; i <= ihi; i += kWave) {
        const uint64_t g = Gin[i + 1];
        sm.Pp[i] = (g == E2_INF64 || tau == E2_INF64) ? E2_INF64 : umax64(g, tau);
    }
    for (int i = lo + lane; i <= ihi + 1; i += kWave) sm.S2[i] = pr[i];
    __syncthreads();
    for (int j = lane; j < N; j += kWave) {
        uint64_t best = E2_INF64;
        if (j >= lo && j <= hi) {
            const int e = we[j];
            if (e != (int)E2_NO_START) {
                const int iend = e < imax ? e : imax;
                const uint64_t pj = sm.S2[j];
                for (int i = j; i <= iend; ++i)
                    best = umin64(best, umax64(sm.Pp[i], sm.S2[i + 1] - pj));
            }
        }
        Gout[j] = best;
    }
    __syncthreads();
}

// T_mu from F_{mu-1} (pool), the head on device mu, and G_{mu+1} (Gnext).
__device__ uint64_t combine(const E2Tables &tb, const DpSmem &sm, const Bands &bd, int r,
                            const uint8_t *chain, int mu, int m, int lane, const uint64_t *Gnext)
{
    const int N = tb.N;
    const int c = chain[mu - 1];
    const int lo = bd.flo[mu], hi = bd.fhi[mu];
    const int cap = bd.cH[mu];
    uint64_t lane_best = E2_INF64;
    if (cap > 0 && lo <= hi) {
        const uint64_t *pr = pref_row(tb, r, c);
        const uint8_t *wr = win_row(tb, 1, c);
        const uint64_t hadd = tb.head[r * tb.M + c];
        int jmin = lo - cap + 1;
        if (jmin < mu - 1) jmin = mu - 1;
        if (mu == 1) {
            for (int j = jmin + lane; j <= hi; j += kWave) {
                sm.Pp[j] = (j == 0) ? 0ull : E2_INF64;
                sm.S2[j] = (pr[j] << 8) - (uint64_t)j;
            }
        } else {
            const uint64_t tau = link_tau(tb, r, chain[mu - 2], c);
            const int plo = bd.flo[mu - 1], phi = bd.fhi[mu - 1];
            const uint64_t *prev = sm.pool + bd.off[mu - 1];
            for (int j = jmin + lane; j <= hi; j += kWave) {
                const int pj = j - 1;
                sm.Pp[j] = pack_prev((pj >= plo && pj <= phi) ? prev[pj - plo] : E2_INF64, tau, j);
                sm.S2[j] = (pr[j] << 8) - (uint64_t)j;
            }
        }
        __syncthreads();
        const uint64_t tnext = (mu < m) ? link_tau(tb, r, c, chain[mu]) : 0;
        for (int i = lo + lane; i <= hi; i += kWave) {
            uint64_t b;
            if (mu == m) b = (i == N - 1) ? 0 : E2_INF64;
            else {
                const uint64_t g = (i + 1 < N) ? Gnext[i + 1] : E2_INF64;
                b = (g == E2_INF64 || tnext == E2_INF64) ? E2_INF64 : umax64(g, tnext);
            }
            const int w = wr[i];
            if (b == E2_INF64 || w == (int)E2_NO_START) continue;
            const uint64_t best =
                cell_min(sm.Pp, sm.S2, (pr[i + 1] + hadd) << 8, w < jmin ? jmin : w, i);
            if (best != E2_INF64) lane_best = umin64(lane_best, umax64(best >> 8, b));
        }
    }
    __syncthreads();
    return wave_min_u64(lane_best);
}

__device__ bool dp_banded(const E2Tables &tb, const DpSmem &sm, Bands &bd, int r,
                          const uint8_t *chain, int m, int lane, uint64_t *T_out, int *mu_out,
                          uint8_t *start)
{
    const int N = tb.N;
    // capacities and bands (one lane; m steps)
    if (lane == 0) {
        bd.pre[0] = 0;
        for (int k = 1; k <= m; ++k) {
            bd.pre[k] = bd.pre[k - 1] + tb.cap0[chain[k - 1]];
            bd.cH[k] = tb.capH[chain[k - 1]];
        }
        const int tot = bd.pre[m];
        int off = 0;
        for (int k = 1; k <= m; ++k) {
            int lo = N - 1 - (tot - bd.pre[k]);
            if (lo < k - 1) lo = k - 1;
            int hi = bd.pre[k] - 1;
            if (hi > N - 1 - (m - k)) hi = N - 1 - (m - k);
            if (hi < lo) { lo = 1; hi = 0; }
            bd.flo[k] = (uint8_t)lo;
            bd.fhi[k] = (uint8_t)hi;
            bd.off[k] = (uint16_t)off;
            if (k < m) off += hi - lo + 1;
            if (k >= 2) {
                int gl = N - (tot - bd.pre[k - 1]);
                if (gl < k - 1) gl = k - 1;
                int gh = bd.pre[k - 1];
                if (gh > N - (m - k + 1)) gh = N - (m - k + 1);
                if (gh < gl) { gl = 1; gh = 0; }
                bd.glo[k] = (uint8_t)gl;
                bd.ghi[k] = (uint8_t)gh;
            }
        }
        bd.off[m] = (uint16_t)(off > 65535 ? 65535 : off);
    }
    __syncthreads();
    if ((int)bd.off[m] > sm.pool_cells) return false;

    // forward rows F_1..F_{m-1}
    for (int k = 1; k < m; ++k)
        fwd_row(tb, sm, bd, r, chain, k, 0, lane, sm.pool + bd.off[k], sm.tbp + bd.off[k]);

    // combines, interleaved with the backward rows
    uint64_t best = combine(tb, sm, bd, r, chain, m, m, lane, nullptr);
    int best_mu = best == E2_INF64 ? 0 : m;
    uint64_t *Gcur = sm.Ga, *Gnew = sm.Gb;
    for (int k = m; k >= 2; --k) {
        bwd_row(tb, sm, bd, r, chain, k, m, lane, Gcur, Gnew);
        uint64_t *t = Gcur;
        Gcur = Gnew;
        Gnew = t;
        const uint64_t v = combine(tb, sm, bd, r, chain, k - 1, m, lane, Gcur);
        if (v <= best && v != E2_INF64) {  // descending mu: ties go to the smaller mu
            best = v;
            best_mu = k - 1;
        }
    }
    *T_out = best;
    *mu_out = best_mu;
    if (best == E2_INF64) return true;

    // rows mu*..m-1 of the chosen master's table overwrite F in the pool
    for (int k = best_mu; k < m; ++k)
        fwd_row(tb, sm, bd, r, chain, k, best_mu, lane, sm.pool + bd.off[k], sm.tbp + bd.off[k]);
    // split point of the last stage: cell N-1 of row m
    if (m >= 2) {
        const int c = chain[m - 1];
        const int f = (best_mu == m);
        const uint64_t *pr = pref_row(tb, r, c);
        const int w = win_row(tb, f, c)[N - 1];
        const uint64_t tau = link_tau(tb, r, chain[m - 2], c);
        const int plo = bd.flo[m - 1], phi = bd.fhi[m - 1];
        const uint64_t *prev = sm.pool + bd.off[m - 1];
        const uint64_t si1 = (pr[N] + (f ? tb.head[r * tb.M + c] : 0)) << 8;
        // lanes over j, then the smallest j with the minimum packed score
        uint64_t lb = E2_INF64;
        for (int j = (w > m - 1 ? w : m - 1) + lane; j <= N - 1; j += kWave) {
            const int pj = j - 1;
            const uint64_t pp = pack_prev((pj >= plo && pj <= phi) ? prev[pj - plo] : E2_INF64,
                                          tau, j);
            lb = umin64(lb, umax64(pp, si1 - ((pr[j] << 8) - (uint64_t)j)));
        }
        const uint64_t key = wave_min_u64(lb);
        if (lane == 0) {
            int i = N - 1;
            int j = (int)(key & 0xFF);
            if (j > i) j = i;
            start[m - 1] = (uint8_t)j;
            i = j - 1;
            for (int k = m - 1; k >= 2; --k) {
                // path cells lie in their band; the clamp only keeps a
                // corrupted table from indexing outside its row
                const int ii = i < bd.flo[k] ? bd.flo[k] : (i > bd.fhi[k] ? bd.fhi[k] : i);
                j = sm.tbp[bd.off[k] + (ii - bd.flo[k])];
                if (j > i) j = i;
                start[k - 1] = (uint8_t)j;
                i = j - 1;
            }
        }
    }
    if (lane == 0) start[0] = 0;
    __syncthreads();
    return true;
}
// ---------------------------------------------------------------------------
// Persistent DP kernel: one wave per workgroup; waves take listed problems
// in list order through an atomic counter and exit when the list is
// exhausted.  Dynamic LDS: four rows of N+1 u64, then the forward-row pool
// (pool_cells u64) and its split-point bytes.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_dp(E2Tables tb, int k_max, int pool_cells,
                                           const uint8_t *__restrict__ labels,
                                           const uint8_t *__restrict__ roles,
                                           uint32_t *counters, const uint32_t *__restrict__ list,
                                           uint8_t *tb_global, uint64_t *T, uint64_t *Lambda,
                                           int16_t *master, uint8_t *layers)
{
    extern __shared__ uint64_t dyn[];
    __shared__ Bands bd;
    __shared__ uint8_t chain[256];
    __shared__ uint8_t start[256];
    __shared__ uint32_t job;
    const int lane = threadIdx.x;
    const int M = tb.M, N = tb.N;
    const int R = N + 1;
    DpSmem sm;
    sm.Pp = dyn;
    sm.S2 = dyn + R;
    sm.Ga = dyn + 2 * R;
    sm.Gb = dyn + 3 * R;
    sm.pool = dyn + 4 * R;
    sm.tbp = reinterpret_cast<uint8_t *>(sm.pool + pool_cells);
    sm.pool_cells = pool_cells;
    const uint32_t n_jobs = counters[0];

    for (;;) {
        if (lane == 0) job = atomicAdd(&counters[1], 1u);
        __syncthreads();
        const uint32_t idx = job;
        __syncthreads();
        if (idx >= n_jobs) break;
        const uint32_t code = list[idx];
        const int p = (int)(code >> 8);
        const int q = (int)(code & 0xFF);

        // chain = devices with label q in ascending id (wave ballot compaction)
        int m = 0;
        for (int base = 0; base < M; base += kWave) {
            const int d = base + lane;
            const bool in = d < M && labels[(size_t)p * M + d] == q;
            const uint64_t mask = __ballot(in);
            if (in) chain[m + __popcll(mask & ((1ull << lane) - 1))] = (uint8_t)d;
            m += __popcll(mask);
        }
        __syncthreads();
        const int r = roles[(size_t)p * k_max + q] != 0;
        const size_t o = (size_t)p * k_max + q;

        uint64_t best = E2_INF64;
        int best_mu = 0;
        if (!dp_banded(tb, sm, bd, r, chain, m, lane, &best, &best_mu, start)) {
            // exact reference path: a full table per master, then the chosen
            // master's table again with split points
            for (int mu = 1; mu <= m; ++mu) {
                const uint64_t v = dp_table(tb, r, chain, m, mu, nullptr, sm.Ga, sm.Pp, sm.S2, lane);
                if (v < best) {
                    best = v;
                    best_mu = mu;
                }
            }
            if (best != E2_INF64) {
                uint8_t *tbp = ((size_t)(m - 1) * N <= (size_t)pool_cells * 8)
                                   ? reinterpret_cast<uint8_t *>(sm.pool)
                                   : tb_global + (size_t)blockIdx.x * N * N;
                dp_table(tb, r, chain, m, best_mu, tbp, sm.Ga, sm.Pp, sm.S2, lane);
                __threadfence_block();
                __syncthreads();
                if (lane == 0) {
                    int i = N - 1;
                    for (int k = m; k >= 2; --k) {
                        int j = tbp[(size_t)(k - 2) * N + (i < 0 ? 0 : i)];
                        if (j > i) j = i < 0 ? 0 : i;
                        start[k - 1] = (uint8_t)j;
                        i = j - 1;
                    }
                    start[0] = 0;
                }
                __syncthreads();
            }
        }
        if (best == E2_INF64) {
            if (lane == 0) {
                T[o] = E2_INF64;
                Lambda[o] = E2_INF64;
                if (master) master[o] = -1;
            }
            if (layers)
                for (int k = lane; k < m; k += kWave) layers[(size_t)p * M + chain[k]] = 0;
            __syncthreads();
            continue;
        }
        // Lambda: stage times (+ head on the master) plus the chain's link times
        uint64_t part = 0;
        for (int k = lane; k < m; k += kWave) {
            const int c = chain[k];
            const int s0 = start[k] < N ? start[k] : N;
            int e = (k + 1 < m) ? start[k + 1] : N;
            if (e > N) e = N;
            if (e < s0) e = s0;
            const uint64_t *pr = pref_row(tb, r, c);
            part += pr[e] - pr[s0];
            if (k + 1 == best_mu) part += tb.head[r * M + c];
            if (k >= 1) part += link_tau(tb, r, chain[k - 1], c);
            if (layers) layers[(size_t)p * M + c] = (uint8_t)(e - s0);
        }
        const uint64_t lam = wave_sum_u64(part);
        if (lane == 0) {
            T[o] = best;
            Lambda[o] = lam;
            if (master) master[o] = (int16_t)chain[best_mu - 1];
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Fitness (Eq. 3-5): one thread per individual.
// ---------------------------------------------------------------------------
constexpr uint64_t kScale = 1ull << 50;

__global__ void k_fitness(int P, int k_max, const uint64_t *__restrict__ T,
                          const uint64_t *__restrict__ Lambda, const uint8_t *__restrict__ roles,
                          uint64_t t_arrival, uint64_t nd, uint64_t lambda_max, uint64_t *w,
                          uint64_t *phase, uint64_t *s_p, uint64_t *s_d)
{
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= P) return;
    uint64_t sp = 0, sd = 0;
    for (int q = 0; q < k_max; ++q) {
        const size_t o = (size_t)p * k_max + q;
        const uint64_t t = T[o];
        if (t == E2_INF64) continue;
        const bool dec = roles[o] != 0;
        if (dec && Lambda[o] > lambda_max) continue;
        const uint64_t rho = kScale / (t > 0 ? t : 1);
        if (dec) sd += rho;
        else sp += rho;
    }
    const uint64_t SP = sp ? (kScale + sp - 1) / sp : E2_INF64;
    const uint64_t SD = sd ? nd * ((kScale + sd - 1) / sd) : E2_INF64;
    if (s_p) s_p[p] = SP;
    if (s_d) s_d[p] = SD;
    if (SP == E2_INF64 || SD == E2_INF64) {
        w[p] = E2_INF64;
        phase[p] = E2_INF64;
        return;
    }
    const uint64_t ph = umax64(SP, SD);
    const uint64_t excess = ph > t_arrival ? ph - t_arrival : 0;
    phase[p] = ph;
    w[p] = excess ? SP + excess : 0;
}

// ---------------------------------------------------------------------------
// GA.  Counter-based generator: the SplitMix64 output function (Steele, Lea,
// Flood, OOPSLA 2014) keyed by (seed, generation, slot, stream, gene), each
// component folded in by xor followed by one output step.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t sm64(uint64_t x)
{
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

constexpr uint32_t kStSelA = 0, kStSelB = 64, kStXoLabel = 128, kStXoRole = 129,
                   kStMutLabel = 130, kStMutRole = 131;

__device__ __forceinline__ bool key_less(const uint64_t *w, const uint64_t *ph, uint32_t a,
                                         uint32_t b)
{
    if (w[a] != w[b]) return w[a] < w[b];
    if (ph[a] != ph[b]) return ph[a] < ph[b];
    return a < b;
}

// n_elite rounds of "smallest key strictly after the previous pick".
__global__ __launch_bounds__(1024) void k_elites(int P, uint32_t n_elite,
                                                 const uint64_t *__restrict__ w,
                                                 const uint64_t *__restrict__ ph,
                                                 uint32_t *elite)
{
    __shared__ uint32_t cand[1024];
    const int t = threadIdx.x;
    uint32_t last = 0xFFFFFFFFu;
    for (uint32_t e = 0; e < n_elite; ++e) {
        uint32_t pick = 0xFFFFFFFFu;
        for (int p = t; p < P; p += blockDim.x) {
            if (last != 0xFFFFFFFFu && !key_less(w, ph, last, (uint32_t)p)) continue;
            if (pick == 0xFFFFFFFFu || key_less(w, ph, (uint32_t)p, pick)) pick = (uint32_t)p;
        }
        cand[t] = pick;
        __syncthreads();
        for (int s = blockDim.x / 2; s >= 1; s >>= 1) {
            if (t < s) {
                const uint32_t a = cand[t], b = cand[t + s];
                if (b != 0xFFFFFFFFu && (a == 0xFFFFFFFFu || key_less(w, ph, b, a))) cand[t] = b;
            }
            __syncthreads();
        }
        last = cand[0];
        if (t == 0) elite[e] = last;
        __syncthreads();
    }
}

__global__ __launch_bounds__(64) void k_breed(int M, int P, int k_max,
                                              const uint8_t *__restrict__ labels_in,
                                              const uint8_t *__restrict__ roles_in,
                                              const uint64_t *__restrict__ w,
                                              const uint64_t *__restrict__ ph, uint64_t seed,
                                              uint32_t g, uint32_t tk, uint32_t xo, uint32_t mut,
                                              uint32_t n_elite, const uint32_t *__restrict__ elite,
                                              uint8_t *labels_out, uint8_t *roles_out)
{
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    uint8_t *lo = labels_out + (size_t)s * M;
    uint8_t *ro = roles_out + (size_t)s * k_max;
    if ((uint32_t)s < n_elite) {
        const uint32_t src = elite[s];
        for (int d = lane; d < M; d += kWave) lo[d] = labels_in[(size_t)src * M + d];
        for (int q = lane; q < k_max; q += kWave) ro[q] = roles_in[(size_t)src * k_max + q];
        return;
    }
    const uint64_t hs = sm64(sm64(seed ^ (uint64_t)g) ^ (uint64_t)s);  // (seed, g, s) prefix
    // lane 0 runs the tournament of parent a, lane 1 that of parent b
    uint32_t win = 0;
    if (lane < 2) {
        const uint32_t st0 = lane == 0 ? kStSelA : kStSelB;
        uint32_t best = 0xFFFFFFFFu;
        for (uint32_t t = 0; t < tk; ++t) {
            const uint64_t u = sm64(sm64(hs ^ (uint64_t)(st0 + t)) ^ 0ull);
            const uint32_t idx = (uint32_t)(((u >> 32) * (uint64_t)P) >> 32);
            if (best == 0xFFFFFFFFu || key_less(w, ph, idx, best)) best = idx;
        }
        win = best;
    }
    const uint32_t a = __shfl(win, 0, kWave);
    const uint32_t b = __shfl(win, 1, kWave);
    const uint64_t h_xl = sm64(hs ^ kStXoLabel), h_ml = sm64(hs ^ kStMutLabel);
    const uint64_t h_xr = sm64(hs ^ kStXoRole), h_mr = sm64(hs ^ kStMutRole);
    for (int d = lane; d < M; d += kWave) {
        const uint64_t u = sm64(h_xl ^ (uint64_t)d);
        uint8_t v = ((uint32_t)u < xo) ? labels_in[(size_t)b * M + d] : labels_in[(size_t)a * M + d];
        const uint64_t z = sm64(h_ml ^ (uint64_t)d);
        if ((uint32_t)(z >> 32) < mut) v = (uint8_t)(((uint64_t)(uint32_t)z * (uint64_t)k_max) >> 32);
        lo[d] = v;
    }
    for (int q = lane; q < k_max; q += kWave) {
        const uint64_t u = sm64(h_xr ^ (uint64_t)q);
        uint8_t v = ((uint32_t)u < xo) ? roles_in[(size_t)b * k_max + q] : roles_in[(size_t)a * k_max + q];
        v = v != 0;
        const uint64_t z = sm64(h_mr ^ (uint64_t)q);
        if ((uint32_t)(z >> 32) < mut) v ^= 1u;
        ro[q] = v;
    }
}

}  // namespace

int e2_dp_pool_cells(int N)
{
    (void)N;
    return 1024;
}

size_t e2_dp_lds_bytes(int N)
{
    return (size_t)4 * (N + 1) * 8 + (size_t)e2_dp_pool_cells(N) * 9;
}

int e2_dp_slots(int problems)
{
    const int cap = 256 * 16;  // 16 one-wave workgroups per CU on a 256-CU part
    return problems < cap ? (problems > 0 ? problems : 1) : cap;
}

hipError_t e2_launch_partitions(const E2Tables &t, hipStream_t s, int P, int k_max,
                                const uint8_t *labels, const uint8_t *roles, const E2Work &wk,
                                uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    k_init<<<1, 64, 0, s>>>(wk.counters);
    k_extract<<<P, 256, 0, s>>>(t, P, k_max, labels, wk.counters, wk.list, T, Lambda, master,
                                layers);
    const int pool = e2_dp_pool_cells(t.N);
    k_dp<<<wk.n_slots, 64, e2_dp_lds_bytes(t.N), s>>>(t, k_max, pool, labels, roles, wk.counters,
                                                      wk.list, wk.tb_global, T, Lambda, master,
                                                      layers);
    return hipGetLastError();
}

hipError_t e2_launch_fitness(hipStream_t s, int P, int k_max, const uint64_t *T,
                             const uint64_t *Lambda, const uint8_t *roles, uint64_t t_arrival,
                             uint64_t nd, uint64_t lambda_max, uint64_t *w, uint64_t *phase,
                             uint64_t *s_p, uint64_t *s_d)
{
    k_fitness<<<(P + 255) / 256, 256, 0, s>>>(P, k_max, T, Lambda, roles, t_arrival, nd,
                                              lambda_max, w, phase, s_p, s_d);
    return hipGetLastError();
}

hipError_t e2_launch_ga(hipStream_t s, int M, int P, int k_max, const uint8_t *labels_in,
                        const uint8_t *roles_in, const uint64_t *w, const uint64_t *phase,
                        uint64_t seed, uint32_t generation, uint32_t tournament_k,
                        uint32_t xo_thresh, uint32_t mut_thresh, uint32_t n_elite,
                        uint32_t *elite_scratch, uint8_t *labels_out, uint8_t *roles_out)
{
    if (n_elite > 0) k_elites<<<1, 1024, 0, s>>>(P, n_elite, w, phase, elite_scratch);
    k_breed<<<P, 64, 0, s>>>(M, P, k_max, labels_in, roles_in, w, phase, seed, generation,
                             tournament_k, xo_thresh, mut_thresh, n_elite, elite_scratch,
                             labels_out, roles_out);
    return hipGetLastError();
}
