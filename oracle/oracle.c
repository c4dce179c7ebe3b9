/*
 * CPU oracle for the E2LLM population-fitness path (arXiv 2606.03770).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the bench's CPU
 * baseline leg do.  It shares no code, header, table or helper with the HIP
 * library: it quantises its own inputs, runs its own dynamic program and its
 * own fitness and GA arithmetic.
 *
 * Style: plain, single-threaded, no SIMD, no blocking, no pruning beyond what
 * the paper's algorithm states.  Unsigned 64-bit integers throughout,
 * unsigned __int128 only where a product can exceed 64 bits.  INF is
 * 2^64 - 1.
 *
 * Paper anchors:
 *   quantisation     "profiled compute time" of a block and tau = A / B
 *                    (Sec. 3.2, definitions after Eq. 2); congestion scaling
 *                    of the bandwidth is part of the workload definition.
 *   dp_pipe          Algorithm 1 with Eq. 1 (k >= 2) and Eq. 2 (k = 1),
 *                    master enumeration, memory-infeasible candidates = INF,
 *                    argmin over the master, backtrack (Sec. 3.2).
 *   Lambda           end-to-end forward time, sum of stage times plus link
 *                    times (Sec. 3.2, the per-request TPOT paragraph).
 *   fitness          Eq. 3, Eq. 4, Eq. 5 with rates summed over replicas
 *                    (Sec. 3.3) and the QoS floor 1/Lambda >= Min_TPS
 *                    (Algorithm 2, Sec. 3.5).
 *   ga_step          elite preservation (Algorithm 2; App. A) with the
 *                    tournament / uniform-crossover / per-gene-mutation
 *                    operators of the 16384-genome workload.
 *
 * Readings where the paper is silent or its listing is inconsistent:
 *   R1  every device of a chain gets >= 1 contiguous block: DP(-1, k) = INF.
 *   R2  block indices are 0-based; DP(i, k) covers blocks 0..i.
 *   R3  TB(i, k) stores the start j of the last stage; the backtrack walks
 *       k = m..2 and the first device takes the remaining i + 1 blocks.
 *   R4  ties over j go to the smallest j (strict < in an ascending scan).
 *   R5  ties over the master go to the smallest chain position.
 *   R6  tau sits inside the max (compute and transfer overlap).
 *   R7  head time / bytes are charged to the master's stage.
 *   R8  memory: stage weight bytes (+ head bytes on the master) <= cap.
 *   R9  chain order is ascending device id within a cluster label.
 *   R10 ceil when quantising times, floor for the effective bandwidth.
 *   R11 fixed-point fitness with SCALE = 2^50 (see oracle_eval).
 *   R12 GA key (w, phase, index), smaller is better.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define INF UINT64_MAX
#define LIMIT48 ((uint64_t)1 << 48)
#define SCALE ((uint64_t)1 << 50)

enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_EOVERFLOW = -2, ORC_ENOMEM = -3 };

static uint64_t max2(uint64_t a, uint64_t b) { return a > b ? a : b; }

/* ceil(a * 1e9 / b) for b > 0, or INF when the result does not fit 64 bits */
static uint64_t ceil_ns(uint64_t a, uint64_t b)
{
    u128 num = (u128)a * 1000000000u;
    u128 q = (num + b - 1) / b;
    if (q >> 64) return INF;
    return (uint64_t)q;
}

/*
 * a0: integer cost tables.
 *   t[r][d][n] = ceil(layer_flops[r][n] * 1e9 / speed[d])   ns
 *   h[r][d]    = ceil(head_flops[r]     * 1e9 / speed[d])   ns
 *   Beff[d][e] = floor(bw[d][e] * cong[d][e] / 1e6)         B/s
 *   tau[r][d][e] = ceil(act[r] * 1e9 / Beff[d][e]), INF if Beff = 0; 0 on the diagonal
 * Any finite time >= 2^48 is an overflow error.
 */
int oracle_quantise(int M, int N, const uint64_t *speed, const uint64_t *bw,
                    const uint32_t *cong, const uint64_t *layer_flops /*[2][N]*/,
                    const uint64_t *act /*[2]*/, const uint64_t *head_flops /*[2]*/,
                    uint64_t *t /*[2][M][N]*/, uint64_t *h /*[2][M]*/,
                    uint64_t *tau /*[2][M][M]*/)
{
    if (M < 1 || M > 256 || N < 1 || N > 255) return ORC_EINVAL;
    for (int d = 0; d < M; d++)
        if (speed[d] == 0) return ORC_EINVAL;
    for (int i = 0; i < M * M; i++)
        if (cong[i] > 1000000u) return ORC_EINVAL;
    for (int r = 0; r < 2; r++) {
        for (int d = 0; d < M; d++) {
            for (int n = 0; n < N; n++) {
                uint64_t v = ceil_ns(layer_flops[r * N + n], speed[d]);
                if (v >= LIMIT48) return ORC_EOVERFLOW;
                t[((size_t)r * M + d) * N + n] = v;
            }
            uint64_t hv = ceil_ns(head_flops[r], speed[d]);
            if (hv >= LIMIT48) return ORC_EOVERFLOW;
            h[r * M + d] = hv;
        }
        for (int d = 0; d < M; d++) {
            for (int e = 0; e < M; e++) {
                uint64_t v;
                if (d == e) {
                    v = 0;
                } else {
                    uint64_t beff = (uint64_t)(((u128)bw[d * M + e] * cong[d * M + e]) / 1000000u);
                    if (beff == 0) {
                        v = INF;
                    } else {
                        v = ceil_ns(act[r], beff);
                        if (v >= LIMIT48) return ORC_EOVERFLOW;
                    }
                }
                tau[((size_t)r * M + d) * M + e] = v;
            }
        }
    }
    return ORC_OK;
}

/*
 * One DP table for a fixed master position mu (1-based), Eq. 1 and Eq. 2.
 * D and TB are [N][m+1] (column 0 unused).  pt is [m][N+1] prefix sums of the
 * chain devices' block times, pw is [N+1] prefix sums of block bytes, so
 * that the sum over blocks j..i is pt[i+1] - pt[j].  Returns the number of
 * candidates that reached the max/compare step.
 */
static uint64_t dp_table(int m, int N, int mu, const uint64_t *pt, const uint64_t *pw,
                         const uint64_t *hk, const uint64_t *tau_link, const uint64_t *memk,
                         uint64_t HB, uint64_t *D, int *TB)
{
    const int W = m + 1;
    uint64_t evaluated = 0;
    for (int i = 0; i < N; i++) {
        for (int k = 1; k <= m; k++) {
            const uint64_t *ptk = pt + (size_t)(k - 1) * (N + 1);
            const uint64_t head_t = (k == mu) ? hk[k - 1] : 0;
            const uint64_t head_b = (k == mu) ? HB : 0;
            D[i * W + k] = INF;
            TB[i * W + k] = -1;
            if (k == 1) {
                /* Eq. 2: the first device holds blocks 0..i */
                uint64_t bytes = pw[i + 1] - pw[0] + head_b;
                if (bytes <= memk[0])
                    D[i * W + 1] = ptk[i + 1] - ptk[0] + head_t;
                continue;
            }
            /* Eq. 1: device k holds blocks j..i, devices 1..k-1 hold 0..j-1 */
            for (int j = 0; j <= i; j++) {
                uint64_t prev = (j == 0) ? INF : D[(j - 1) * W + (k - 1)];
                if (prev == INF) continue;
                uint64_t bytes = pw[i + 1] - pw[j] + head_b;
                if (bytes > memk[k - 1]) continue;
                uint64_t cost = ptk[i + 1] - ptk[j] + head_t;
                uint64_t v = max2(max2(prev, cost), tau_link[k - 1]);
                evaluated++;
                if (v < D[i * W + k]) {
                    D[i * W + k] = v;
                    TB[i * W + k] = j;
                }
            }
        }
    }
    return evaluated;
}

/*
 * The finishing-time variant of one master's table (the FT ablation of
 * Sec. 4.2): Eq. 1 with the bottleneck max replaced by a sum, so that
 * DP(i, k) is the least end-to-end time of blocks 0..i on devices 1..k
 * (stage times plus link times); Eq. 2 and the memory test unchanged,
 * ties to the smallest j as R4.
 */
static uint64_t dp_table_sum(int m, int N, int mu, const uint64_t *pt, const uint64_t *pw,
                             const uint64_t *hk, const uint64_t *tau_link, const uint64_t *memk,
                             uint64_t HB, uint64_t *D, int *TB)
{
    const int W = m + 1;
    uint64_t evaluated = 0;
    for (int i = 0; i < N; i++) {
        for (int k = 1; k <= m; k++) {
            const uint64_t *ptk = pt + (size_t)(k - 1) * (N + 1);
            const uint64_t head_t = (k == mu) ? hk[k - 1] : 0;
            const uint64_t head_b = (k == mu) ? HB : 0;
            D[i * W + k] = INF;
            TB[i * W + k] = -1;
            if (k == 1) {
                uint64_t bytes = pw[i + 1] - pw[0] + head_b;
                if (bytes <= memk[0])
                    D[i * W + 1] = ptk[i + 1] - ptk[0] + head_t;
                continue;
            }
            if (tau_link[k - 1] == INF) continue;
            for (int j = 0; j <= i; j++) {
                uint64_t prev = (j == 0) ? INF : D[(j - 1) * W + (k - 1)];
                if (prev == INF) continue;
                uint64_t bytes = pw[i + 1] - pw[j] + head_b;
                if (bytes > memk[k - 1]) continue;
                uint64_t cost = ptk[i + 1] - ptk[j] + head_t;
                uint64_t v = prev + cost + tau_link[k - 1];
                evaluated++;
                if (v < D[i * W + k]) {
                    D[i * W + k] = v;
                    TB[i * W + k] = j;
                }
            }
        }
    }
    return evaluated;
}

/*
 * DP_Pipe for one chain of m devices (Algorithm 1).
 *   tk[m][N]   block times of the chain's devices, chain order
 *   hk[m]      head + output-layer time of each chain device if it is master
 *   tau_link[m] tau_link[k] = transfer time between chain positions k-1 and k
 *              (k >= 1); tau_link[0] is unused
 *   memk[m]    memory caps; W[N] block bytes; HB head bytes
 * Outputs: *T (INF if infeasible), *Lambda, *mu_star (1-based, 0 if
 * infeasible), sizes[m] (0 if infeasible), *evaluated (candidate count).
 */
static int dp_pipe_obj(int m, int N, const uint64_t *tk, const uint64_t *hk,
                       const uint64_t *tau_link, const uint64_t *memk, const uint64_t *W,
                       uint64_t HB, int objective, uint64_t *T, uint64_t *Lambda, int *mu_star,
                       int *sizes, uint64_t *evaluated);

int oracle_dp_pipe(int m, int N, const uint64_t *tk, const uint64_t *hk,
                   const uint64_t *tau_link, const uint64_t *memk, const uint64_t *W,
                   uint64_t HB, uint64_t *T, uint64_t *Lambda, int *mu_star, int *sizes,
                   uint64_t *evaluated)
{
    return dp_pipe_obj(m, N, tk, hk, tau_link, memk, W, HB, 0, T, Lambda, mu_star, sizes,
                       evaluated);
}

/*
 * objective 0: Algorithm 1 (least bottleneck).  objective 1: the
 * finishing-time variant (least end-to-end time, dp_table_sum); the master
 * and split points minimise that sum, *Lambda is the sum and *T the
 * bottleneck (max over stage times and link times, R6) of the chosen
 * partition.
 */
int oracle_dp_pipe_obj(int m, int N, const uint64_t *tk, const uint64_t *hk,
                       const uint64_t *tau_link, const uint64_t *memk, const uint64_t *W,
                       uint64_t HB, int objective, uint64_t *T, uint64_t *Lambda, int *mu_star,
                       int *sizes, uint64_t *evaluated)
{
    return dp_pipe_obj(m, N, tk, hk, tau_link, memk, W, HB, objective, T, Lambda, mu_star, sizes,
                       evaluated);
}

static int dp_pipe_obj(int m, int N, const uint64_t *tk, const uint64_t *hk,
                       const uint64_t *tau_link, const uint64_t *memk, const uint64_t *W,
                       uint64_t HB, int objective, uint64_t *T, uint64_t *Lambda, int *mu_star,
                       int *sizes, uint64_t *evaluated)
{
    *T = INF;
    *Lambda = INF;
    *mu_star = 0;
    *evaluated = 0;
    for (int k = 0; k < m; k++) sizes[k] = 0;
    if (m < 1 || N < 1) return ORC_EINVAL;
    if (m > N) return ORC_OK; /* R1: some device would hold no block */

    uint64_t *pt = malloc(sizeof(uint64_t) * (size_t)m * (N + 1));
    uint64_t *pw = malloc(sizeof(uint64_t) * (size_t)(N + 1));
    uint64_t *D = malloc(sizeof(uint64_t) * (size_t)N * (m + 1));
    int *TB = malloc(sizeof(int) * (size_t)N * (m + 1));
    int *TBbest = malloc(sizeof(int) * (size_t)N * (m + 1));
    if (!pt || !pw || !D || !TB || !TBbest) {
        free(pt); free(pw); free(D); free(TB); free(TBbest);
        return ORC_ENOMEM;
    }
    for (int k = 0; k < m; k++) {
        pt[(size_t)k * (N + 1)] = 0;
        for (int n = 0; n < N; n++)
            pt[(size_t)k * (N + 1) + n + 1] = pt[(size_t)k * (N + 1) + n] + tk[(size_t)k * N + n];
    }
    pw[0] = 0;
    for (int n = 0; n < N; n++) pw[n + 1] = pw[n] + W[n];

    /* outer loop over the master position; keep the smallest mu on ties (R5) */
    uint64_t best = INF;
    int best_mu = 0;
    for (int mu = 1; mu <= m; mu++) {
        *evaluated += objective ? dp_table_sum(m, N, mu, pt, pw, hk, tau_link, memk, HB, D, TB)
                                : dp_table(m, N, mu, pt, pw, hk, tau_link, memk, HB, D, TB);
        uint64_t Tmu = D[(N - 1) * (m + 1) + m];
        if (Tmu < best) {
            best = Tmu;
            best_mu = mu;
            memcpy(TBbest, TB, sizeof(int) * (size_t)N * (m + 1));
        }
    }
    if (best != INF) {
        /* backtrack (R3) */
        int i = N - 1;
        for (int k = m; k >= 2; k--) {
            int j = TBbest[i * (m + 1) + k];
            sizes[k - 1] = i - j + 1;
            i = j - 1;
        }
        sizes[0] = i + 1;
        /* Lambda: sum of stage times plus the chain's link times; the
         * bottleneck of the same partition (equal to best for objective 0) */
        uint64_t lam = 0, bott = 0;
        int start = 0;
        for (int k = 1; k <= m; k++) {
            int end = start + sizes[k - 1];
            uint64_t st = pt[(size_t)(k - 1) * (N + 1) + end] - pt[(size_t)(k - 1) * (N + 1) + start];
            if (k == best_mu) st += hk[k - 1];
            lam += st;
            bott = max2(bott, st);
            if (k >= 2) {
                lam += tau_link[k - 1];
                bott = max2(bott, tau_link[k - 1]);
            }
            start = end;
        }
        *T = objective ? bott : best;
        *Lambda = lam;
        *mu_star = best_mu;
    }
    free(pt); free(pw); free(D); free(TB); free(TBbest);
    return ORC_OK;
}

/*
 * Per-(individual, cluster) solve over a population.
 *   labels[P][M]  cluster id of each device; ids >= k_max mean "unassigned"
 *   roles[P][k_max] 0 = prefill, nonzero = decode
 * Outputs T, Lambda [P][k_max] (INF for an empty or infeasible cluster),
 * master [P][k_max] (device id, -1 if empty or infeasible), layers [P][M]
 * (blocks on each device, 0 for unassigned devices and infeasible clusters).
 * The chain of cluster q is its devices in ascending id (R9).
 */
int oracle_solve_obj(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                     const uint64_t *mem, const uint64_t *W, uint64_t HB, int objective,
                     int P, int k_max, const uint8_t *labels, const uint8_t *roles,
                     uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers,
                     uint64_t *evaluated_total);

int oracle_solve(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                 const uint64_t *mem, const uint64_t *W, uint64_t HB,
                 int P, int k_max, const uint8_t *labels, const uint8_t *roles,
                 uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers,
                 uint64_t *evaluated_total)
{
    return oracle_solve_obj(M, N, t, h, tau, mem, W, HB, 0, P, k_max, labels, roles, T, Lambda,
                            master, layers, evaluated_total);
}

/* oracle_solve with the DP objective of oracle_dp_pipe_obj */
int oracle_solve_obj(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                     const uint64_t *mem, const uint64_t *W, uint64_t HB, int objective,
                     int P, int k_max, const uint8_t *labels, const uint8_t *roles,
                     uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers,
                     uint64_t *evaluated_total)
{
    if (M < 1 || M > 256 || N < 1 || N > 255 || P < 0 || k_max < 1 || k_max > 255)
        return ORC_EINVAL;
    int chain[256];
    int sizes[256];
    uint64_t *tk = malloc(sizeof(uint64_t) * (size_t)M * N);
    uint64_t hk[256], tl[256], mk[256];
    if (!tk) return ORC_ENOMEM;
    uint64_t total = 0;
    for (int p = 0; p < P; p++) {
        for (int d = 0; d < M; d++) layers[(size_t)p * M + d] = 0;
        for (int q = 0; q < k_max; q++) {
            size_t o = (size_t)p * k_max + q;
            T[o] = INF;
            Lambda[o] = INF;
            master[o] = -1;
            int m = 0;
            for (int d = 0; d < M; d++)
                if (labels[(size_t)p * M + d] == q) chain[m++] = d;
            if (m == 0) continue;
            int r = roles[o] != 0;
            for (int k = 0; k < m; k++) {
                memcpy(tk + (size_t)k * N, t + ((size_t)r * M + chain[k]) * N, sizeof(uint64_t) * N);
                hk[k] = h[r * M + chain[k]];
                mk[k] = mem[chain[k]];
                tl[k] = (k == 0) ? 0 : tau[((size_t)r * M + chain[k - 1]) * M + chain[k]];
            }
            uint64_t Tv, Lv, ev;
            int mu;
            int rc = dp_pipe_obj(m, N, tk, hk, tl, mk, W, HB, objective, &Tv, &Lv, &mu, sizes, &ev);
            if (rc) { free(tk); return rc; }
            total += ev;
            if (Tv == INF) continue;
            T[o] = Tv;
            Lambda[o] = Lv;
            master[o] = (int16_t)chain[mu - 1];
            for (int k = 0; k < m; k++) layers[(size_t)p * M + chain[k]] = (uint8_t)sizes[k];
        }
    }
    free(tk);
    if (evaluated_total) *evaluated_total = total;
    return ORC_OK;
}

/*
 * Fitness of one individual from its clusters' (T, Lambda, role), Eq. 3-5.
 * Rates: a prefill replica serves NP tokens per T, so NP / PS = 1 / sum(1/T);
 * a decode replica with one KV slot emits one token per T, so
 * ND / DS = ND / sum(1/T).  In fixed point with SCALE = 2^50:
 *   rho_c = floor(SCALE / max(T_c, 1))
 *   S_P   = ceil(SCALE / sum_P rho),  S_D = ND * ceil(SCALE / sum_D rho)
 *   phase = max(S_P, S_D)                               (Eq. 3)
 *   excess = phase - T_a if phase > T_a else 0           (Eq. 4)
 *   w = S_P + excess if excess > 0 else 0                (Eq. 5)
 * Decode clusters whose Lambda exceeds floor(1e12 / min_tps_milli) ns fail
 * the QoS floor and are dropped (min_tps_milli = 0 disables the floor).
 * An individual with no usable prefill or no usable decode cluster gets
 * w = phase = INF.
 */
/* Eq. 3-5 from the summed fixed-point rates of the prefill and decode
 * replicas (0 = none usable) */
static void rates_fitness(uint64_t sum_p, uint64_t sum_d, uint64_t t_arrival, uint64_t nd,
                          uint64_t *w, uint64_t *phase, uint64_t *s_p, uint64_t *s_d)
{
    uint64_t SP = sum_p ? (SCALE + sum_p - 1) / sum_p : INF;
    uint64_t SD = sum_d ? nd * ((SCALE + sum_d - 1) / sum_d) : INF;
    *s_p = SP;
    *s_d = SD;
    if (SP == INF || SD == INF) {
        *w = INF;
        *phase = INF;
        return;
    }
    uint64_t ph = max2(SP, SD);
    uint64_t excess = ph > t_arrival ? ph - t_arrival : 0;
    *phase = ph;
    *w = excess > 0 ? SP + excess : 0;
}

static void fitness_one(int k_max, const uint64_t *T, const uint64_t *Lambda,
                        const uint8_t *roles, uint64_t t_arrival, uint64_t nd,
                        uint64_t min_tps_milli, uint64_t *w, uint64_t *phase,
                        uint64_t *s_p, uint64_t *s_d)
{
    uint64_t sum_p = 0, sum_d = 0;
    for (int q = 0; q < k_max; q++) {
        if (T[q] == INF) continue;
        int decode = roles[q] != 0;
        if (decode && min_tps_milli > 0 && Lambda[q] > 1000000000000ull / min_tps_milli)
            continue;
        uint64_t rho = SCALE / (T[q] > 0 ? T[q] : 1);
        if (decode) sum_d += rho;
        else sum_p += rho;
    }
    rates_fitness(sum_p, sum_d, t_arrival, nd, w, phase, s_p, s_d);
}

int oracle_fitness(int P, int k_max, const uint64_t *T, const uint64_t *Lambda,
                   const uint8_t *roles, uint64_t t_arrival, uint64_t nd, uint64_t min_tps_milli,
                   uint64_t *w, uint64_t *phase, uint64_t *s_p, uint64_t *s_d)
{
    if (P < 0 || k_max < 1 || k_max > 255 || nd > 8192) return ORC_EINVAL;
    for (int p = 0; p < P; p++)
        fitness_one(k_max, T + (size_t)p * k_max, Lambda + (size_t)p * k_max,
                    roles + (size_t)p * k_max, t_arrival, nd, min_tps_milli,
                    w + p, phase + p, s_p + p, s_d + p);
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* Counter-based random numbers: the SplitMix64 output function (Steele,   */
/* Lea and Flood, "Fast splittable pseudorandom number generators",        */
/* OOPSLA 2014) used as a keyed hash over (seed, generation, slot, stream, */
/* gene): h <- seed; for c in (g, s, stream, gene): h <- mix(h ^ c).       */
/* mix(z) = splitmix64 finaliser of (z + golden gamma).                     */
/* ---------------------------------------------------------------------- */
static uint64_t splitmix_out(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t oracle_rng(uint64_t seed, uint64_t g, uint64_t s, uint64_t stream, uint64_t gene)
{
    uint64_t x = seed;
    x = splitmix_out(x ^ g);
    x = splitmix_out(x ^ s);
    x = splitmix_out(x ^ stream);
    x = splitmix_out(x ^ gene);
    return x;
}

uint64_t oracle_splitmix_out(uint64_t z) { return splitmix_out(z); }

/* GA random streams */
#define ST_SEL_A 0u    /* + t, t < tournament_k: draws of the first parent  */
#define ST_SEL_B 64u   /* + t: draws of the second parent                   */
#define ST_XO_LABEL 128u
#define ST_XO_ROLE 129u
#define ST_MUT_LABEL 130u
#define ST_MUT_ROLE 131u

/* key order (w, phase, index): is individual a better (smaller) than b? */
static int key_less(const uint64_t *w, const uint64_t *ph, int a, int b)
{
    if (w[a] != w[b]) return w[a] < w[b];
    if (ph[a] != ph[b]) return ph[a] < ph[b];
    return a < b;
}

static int tournament(uint64_t seed, uint64_t g, int s, unsigned base, int k, int P,
                      const uint64_t *w, const uint64_t *ph)
{
    int best = -1;
    for (int t = 0; t < k; t++) {
        uint64_t u = oracle_rng(seed, g, (uint64_t)s, base + (unsigned)t, 0);
        int idx = (int)(((u >> 32) * (uint64_t)P) >> 32);
        if (best < 0 || key_less(w, ph, idx, best)) best = idx;
    }
    return best;
}

/*
 * One generation of the GA (Algorithm 2: elites; crossover; mutation).
 * Slots 0..n_elite-1 receive the n_elite best individuals in key order,
 * copied unchanged.  Every other slot s breeds a child:
 *   parents a, b: best of tournament_k uniform draws each (with replacement),
 *     index = floor(hi32(u) * P / 2^32)
 *   crossover, per label gene d: b[d] if lo32(u) < crossover_thresh else a[d];
 *     per role gene q likewise (roles are written as 0/1)
 *   mutation, per label gene: if hi32(u) < mutation_thresh the label is
 *     redrawn as floor(lo32(u) * k_max / 2^32); per role gene: the bit flips
 */
int oracle_ga_step(int M, int P, int k_max, const uint8_t *labels_in, const uint8_t *roles_in,
                   const uint64_t *w, const uint64_t *phase, uint64_t seed, uint32_t generation,
                   uint32_t tournament_k, uint32_t xo_thresh, uint32_t mut_thresh,
                   uint32_t n_elite, uint8_t *labels_out, uint8_t *roles_out)
{
    if (M < 1 || M > 256 || P < 1 || k_max < 1 || k_max > 255 || tournament_k < 1 ||
        tournament_k > 64 || (int)n_elite > P || n_elite > 256)
        return ORC_EINVAL;
    const uint64_t g = generation;
    /* elites: repeated selection of the next-best key (keys are distinct) */
    int last = -1;
    for (uint32_t e = 0; e < n_elite; e++) {
        int pick = -1;
        for (int p = 0; p < P; p++) {
            if (last >= 0 && !key_less(w, phase, last, p)) continue; /* only keys after last */
            if (pick < 0 || key_less(w, phase, p, pick)) pick = p;
        }
        memcpy(labels_out + (size_t)e * M, labels_in + (size_t)pick * M, (size_t)M);
        memcpy(roles_out + (size_t)e * k_max, roles_in + (size_t)pick * k_max, (size_t)k_max);
        last = pick;
    }
    for (int s = (int)n_elite; s < P; s++) {
        int a = tournament(seed, g, s, ST_SEL_A, (int)tournament_k, P, w, phase);
        int b = tournament(seed, g, s, ST_SEL_B, (int)tournament_k, P, w, phase);
        for (int d = 0; d < M; d++) {
            uint64_t u = oracle_rng(seed, g, (uint64_t)s, ST_XO_LABEL, (uint64_t)d);
            uint8_t v = ((uint32_t)u < xo_thresh) ? labels_in[(size_t)b * M + d]
                                                  : labels_in[(size_t)a * M + d];
            uint64_t z = oracle_rng(seed, g, (uint64_t)s, ST_MUT_LABEL, (uint64_t)d);
            if ((uint32_t)(z >> 32) < mut_thresh)
                v = (uint8_t)((((uint64_t)(uint32_t)z) * (uint64_t)k_max) >> 32);
            labels_out[(size_t)s * M + d] = v;
        }
        for (int q = 0; q < k_max; q++) {
            uint64_t u = oracle_rng(seed, g, (uint64_t)s, ST_XO_ROLE, (uint64_t)q);
            uint8_t v = ((uint32_t)u < xo_thresh) ? roles_in[(size_t)b * k_max + q]
                                                  : roles_in[(size_t)a * k_max + q];
            v = v != 0;
            uint64_t z = oracle_rng(seed, g, (uint64_t)s, ST_MUT_ROLE, (uint64_t)q);
            if ((uint32_t)(z >> 32) < mut_thresh) v ^= 1u;
            roles_out[(size_t)s * k_max + q] = v;
        }
    }
    return ORC_OK;
}

/* ====================================================================== */
/* Two-chromosome genomes (App. A): an ordering chromosome order[M] (a     */
/* permutation of the devices) and a grouping chromosome sizes[k_max]      */
/* (replica sizes).  Replica r holds the devices at ordering positions     */
/* off_r .. off_r + sizes[r] - 1, off_r = sizes[0] + ... + sizes[r-1],     */
/* clipped to M; its chain order is the ordering (Sec. 3.2 "node          */
/* ordering"; App. A gene example).  roles[k_max] belongs to the replicas. */
/* ====================================================================== */

/* replica r's ordering range [*lo, *hi), clipped to M */
static void replica_range(int M, int k_max, const uint16_t *sizes, int r, int *lo, int *hi)
{
    long off = 0;
    for (int q = 0; q < r && q < k_max; q++) off += sizes[q];
    long end = off + sizes[r];
    *lo = (int)(off < M ? off : M);
    *hi = (int)(end < M ? end : M);
}

int oracle_replica_range(int M, int k_max, const uint16_t *sizes, int r, int *lo, int *hi)
{
    if (M < 1 || M > 256 || k_max < 1 || k_max > 255 || r < 0 || r >= k_max) return ORC_EINVAL;
    replica_range(M, k_max, sizes, r, lo, hi);
    return ORC_OK;
}

/*
 * Per-(individual, replica) solve for two-chromosome genomes: as
 * oracle_solve, with replica r's chain = order[off_r .. off_r + m_r - 1].
 * Devices outside every replica get 0 layers; a replica holding an id
 * >= M (not a device) is infeasible.
 */
int oracle_solve_ordered(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                         const uint64_t *mem, const uint64_t *W, uint64_t HB, int P, int k_max,
                         const uint8_t *order, const uint16_t *sizes, const uint8_t *roles,
                         uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    if (M < 1 || M > 256 || N < 1 || N > 255 || P < 0 || k_max < 1 || k_max > 255)
        return ORC_EINVAL;
    int chain[256];
    int szs[256];
    uint64_t *tk = malloc(sizeof(uint64_t) * (size_t)M * N);
    uint64_t hk[256], tl[256], mk[256];
    if (!tk) return ORC_ENOMEM;
    for (int p = 0; p < P; p++) {
        for (int d = 0; d < M; d++) layers[(size_t)p * M + d] = 0;
        for (int q = 0; q < k_max; q++) {
            size_t o = (size_t)p * k_max + q;
            T[o] = INF;
            Lambda[o] = INF;
            master[o] = -1;
            int lo, hi;
            replica_range(M, k_max, sizes + (size_t)p * k_max, q, &lo, &hi);
            int m = hi - lo;
            if (m <= 0) continue;
            int valid = 1;
            for (int k = 0; k < m; k++) {
                chain[k] = order[(size_t)p * M + lo + k];
                if (chain[k] >= M) valid = 0;
            }
            if (!valid) continue;
            int r = roles[o] != 0;
            for (int k = 0; k < m; k++) {
                memcpy(tk + (size_t)k * N, t + ((size_t)r * M + chain[k]) * N, sizeof(uint64_t) * N);
                hk[k] = h[r * M + chain[k]];
                mk[k] = mem[chain[k]];
                tl[k] = (k == 0) ? 0 : tau[((size_t)r * M + chain[k - 1]) * M + chain[k]];
            }
            uint64_t Tv, Lv, ev;
            int mu;
            int rc = oracle_dp_pipe(m, N, tk, hk, tl, mk, W, HB, &Tv, &Lv, &mu, szs, &ev);
            if (rc) { free(tk); return rc; }
            if (Tv == INF) continue;
            T[o] = Tv;
            Lambda[o] = Lv;
            master[o] = (int16_t)chain[mu - 1];
            for (int k = 0; k < m; k++) layers[(size_t)p * M + chain[k]] = (uint8_t)szs[k];
        }
    }
    free(tk);
    return ORC_OK;
}

/* Two-chromosome GA streams */
#define ST_O_CUT 140u    /* crossover point of the ordering                 */
#define ST_O_GROUP 141u  /* which parent gives the grouping (and roles)     */
#define ST_O_MUT 142u    /* whether the child mutates, and which mutation   */
#define ST_O_SWAP 143u   /* the two ordering positions of a swap            */
#define ST_O_REGEN 144u  /* the replica from which the grouping regrows     */
#define ST_O_SIZE 145u   /* + nothing; gene = replica: its size and role    */
#define ST_O_PERM 146u   /* gene = step of the Fisher-Yates shuffle         */

/* mutation kinds, as fractions of 2^32 of a uniform u32 (App. A) */
#define MUT_SWAP_BELOW 858993459u    /* 0.20: exchange two ordering positions      */
#define MUT_REGROW_BELOW 3006477107u /* 0.70: regrow the grouping from a replica   */
#define MUT_ALLGROUP_BELOW 3650722201u /* 0.85: regrow the whole grouping; else both */

/*
 * Ordering crossover with repair (App. A): the child takes a[0..c) and
 * then b[c..M); a node of b's part that already occurs in a[0..c) leaves a
 * hole, and the holes are filled left to right with the nodes of b[0..c)
 * that are not in a[0..c), in b's order.  Every node then occurs once.
 */
void oracle_order_crossover(int M, const uint8_t *a, const uint8_t *b, int c, uint8_t *child)
{
    unsigned char used[256] = {0};
    for (int t = 0; t < c; t++) {
        child[t] = a[t];
        used[a[t]] = 1;
    }
    int fill[256], nf = 0;
    for (int t = 0; t < c; t++)
        if (!used[b[t]]) fill[nf++] = b[t];
    int k = 0;
    for (int t = c; t < M; t++) child[t] = used[b[t]] ? (uint8_t)fill[k++] : b[t];
}

/*
 * Regrow the grouping from replica pos: replicas 0..pos-1 keep their sizes
 * and roles; the remaining devices are cut into replicas of
 * 1 + floor(hi32(u) * max_replica / 2^32) devices (the last replica slot,
 * k_max - 1, takes whatever remains), each with role lo32(u) >= 2^31, u =
 * rng(seed, g, slot, ST_O_SIZE, replica); unused slots get size 0, role 0.
 */
static void regrow(int M, int k_max, uint64_t seed, uint64_t g, int s, int pos, int max_replica,
                   uint16_t *sizes, uint8_t *roles)
{
    long kept = 0;
    for (int r = 0; r < pos; r++) kept += sizes[r];
    long remaining = M - kept;
    if (remaining < 0) remaining = 0;
    int r = pos;
    while (remaining > 0 && r < k_max) {
        uint64_t u = oracle_rng(seed, g, (uint64_t)s, ST_O_SIZE, (uint64_t)r);
        long sz = 1 + (long)((((u >> 32)) * (uint64_t)max_replica) >> 32);
        if (r == k_max - 1 || sz > remaining) sz = remaining;
        sizes[r] = (uint16_t)sz;
        roles[r] = (uint32_t)u >= 0x80000000u;
        remaining -= sz;
        r++;
    }
    for (; r < k_max; r++) {
        sizes[r] = 0;
        roles[r] = 0;
    }
}

void oracle_regrow(int M, int k_max, uint64_t seed, uint64_t g, int s, int pos, int max_replica,
                   uint16_t *sizes, uint8_t *roles)
{
    regrow(M, k_max, seed, g, s, pos, max_replica, sizes, roles);
}

/* number of leading replicas that hold at least one device */
static int replica_count(int M, int k_max, const uint16_t *sizes)
{
    int n = 0;
    long off = 0;
    for (int r = 0; r < k_max; r++) {
        if (sizes[r] == 0 || off >= M) break;
        off += sizes[r];
        n++;
    }
    return n;
}

/*
 * One generation of the two-chromosome GA (Algorithm 2, App. A).
 * Slots 0..n_elite-1 receive the n_elite best individuals in key order,
 * unchanged.  Every other slot s:
 *   parents a, b: tournaments as in oracle_ga_step (streams 0.., 64..)
 *   ordering: crossover with repair at c = 1 + floor(lo32(u) * (M-1) / 2^32),
 *     u = rng(.., ST_O_CUT, 0) (the child copies a when M = 1)
 *   grouping and roles: from b if lo32(rng(.., ST_O_GROUP, 0)) < 2^31, else a
 *   mutation, u = rng(.., ST_O_MUT, 0): fires when hi32(u) < mutation_thresh;
 *     lo32(u) < 0.20 * 2^32: swap ordering positions floor(hi32(v) * M / 2^32)
 *       and floor(lo32(v) * M / 2^32), v = rng(.., ST_O_SWAP, 0);
 *     < 0.70: regrow the grouping from replica floor(hi32(rng(.., ST_O_REGEN,
 *       0)) * R / 2^32), R = replicas holding devices (0 if none);
 *     < 0.85: regrow the whole grouping;
 *     else: a new ordering (Fisher-Yates from the identity: for t = M-1..1
 *       swap t with floor(hi32(rng(.., ST_O_PERM, t)) * (t+1) / 2^32)) and a
 *       regrown grouping.
 *   roles are written as 0/1.
 */
int oracle_ga_step_ordered(int M, int P, int k_max, const uint8_t *order_in,
                           const uint16_t *sizes_in, const uint8_t *roles_in, const uint64_t *w,
                           const uint64_t *phase, uint64_t seed, uint32_t generation,
                           uint32_t tournament_k, uint32_t mut_thresh, uint32_t n_elite,
                           uint32_t max_replica, uint8_t *order_out, uint16_t *sizes_out,
                           uint8_t *roles_out)
{
    if (M < 1 || M > 256 || P < 1 || k_max < 1 || k_max > 255 || tournament_k < 1 ||
        tournament_k > 64 || (int)n_elite > P || n_elite > 256 || max_replica < 1 ||
        max_replica > 256)
        return ORC_EINVAL;
    const uint64_t g = generation;
    int last = -1;
    for (uint32_t e = 0; e < n_elite; e++) {
        int pick = -1;
        for (int p = 0; p < P; p++) {
            if (last >= 0 && !key_less(w, phase, last, p)) continue;
            if (pick < 0 || key_less(w, phase, p, pick)) pick = p;
        }
        memcpy(order_out + (size_t)e * M, order_in + (size_t)pick * M, (size_t)M);
        memcpy(sizes_out + (size_t)e * k_max, sizes_in + (size_t)pick * k_max,
               sizeof(uint16_t) * (size_t)k_max);
        memcpy(roles_out + (size_t)e * k_max, roles_in + (size_t)pick * k_max, (size_t)k_max);
        last = pick;
    }
    for (int s = (int)n_elite; s < P; s++) {
        int a = tournament(seed, g, s, ST_SEL_A, (int)tournament_k, P, w, phase);
        int b = tournament(seed, g, s, ST_SEL_B, (int)tournament_k, P, w, phase);
        uint8_t *ord = order_out + (size_t)s * M;
        uint16_t *sz = sizes_out + (size_t)s * k_max;
        uint8_t *ro = roles_out + (size_t)s * k_max;
        if (M >= 2) {
            uint64_t u = oracle_rng(seed, g, (uint64_t)s, ST_O_CUT, 0);
            int c = 1 + (int)((((uint64_t)(uint32_t)u) * (uint64_t)(M - 1)) >> 32);
            oracle_order_crossover(M, order_in + (size_t)a * M, order_in + (size_t)b * M, c, ord);
        } else {
            ord[0] = order_in[(size_t)a * M];
        }
        uint64_t ug = oracle_rng(seed, g, (uint64_t)s, ST_O_GROUP, 0);
        int src = ((uint32_t)ug < 0x80000000u) ? b : a;
        for (int r = 0; r < k_max; r++) {
            sz[r] = sizes_in[(size_t)src * k_max + r];
            ro[r] = roles_in[(size_t)src * k_max + r] != 0;
        }
        uint64_t um = oracle_rng(seed, g, (uint64_t)s, ST_O_MUT, 0);
        if ((uint32_t)(um >> 32) < mut_thresh) {
            uint32_t kind = (uint32_t)um;
            if (kind < MUT_SWAP_BELOW) {
                uint64_t v = oracle_rng(seed, g, (uint64_t)s, ST_O_SWAP, 0);
                int i = (int)(((v >> 32) * (uint64_t)M) >> 32);
                int j = (int)((((uint64_t)(uint32_t)v) * (uint64_t)M) >> 32);
                uint8_t x = ord[i];
                ord[i] = ord[j];
                ord[j] = x;
            } else if (kind < MUT_REGROW_BELOW) {
                int R = replica_count(M, k_max, sz);
                uint64_t v = oracle_rng(seed, g, (uint64_t)s, ST_O_REGEN, 0);
                int pos = (int)(((v >> 32) * (uint64_t)R) >> 32);
                regrow(M, k_max, seed, g, s, pos, (int)max_replica, sz, ro);
            } else {
                if (kind >= MUT_ALLGROUP_BELOW) {
                    for (int t = 0; t < M; t++) ord[t] = (uint8_t)t;
                    for (int t = M - 1; t >= 1; t--) {
                        uint64_t v = oracle_rng(seed, g, (uint64_t)s, ST_O_PERM, (uint64_t)t);
                        int j = (int)(((v >> 32) * (uint64_t)(t + 1)) >> 32);
                        uint8_t x = ord[t];
                        ord[t] = ord[j];
                        ord[j] = x;
                    }
                }
                regrow(M, k_max, seed, g, s, 0, (int)max_replica, sz, ro);
            }
        }
    }
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* Decode slots and role search (Algorithm 2's inner loop, Sec. 3.4).      */
/* ---------------------------------------------------------------------- */

/*
 * Cost tables for role indices r = 0..b_max: r = 0 is prefill, r = b is a
 * decode replica holding b requests in flight (b KV-cache slots).  The
 * paper profiles the decode block time per b without giving a model; this
 * build's synthetic one (parity unpinned by the paper):
 *   t[0], h[0], tau[0]   prefill tables, as oracle_quantise
 *   t[1], h[1], tau[1]   decode with one request, as oracle_quantise
 *   t[b][d][n] = t[1][d][n] + (b-1) * ceil(t[1][d][n] * beta_ppm / 1e6)
 *   h[b][d]    = h[1][d]    + (b-1) * ceil(h[1][d] * beta_ppm / 1e6)
 *   tau[b][d][e] = ceil(b * act[1] * 1e9 / Beff[d][e]) (INF if Beff = 0)
 * i.e. each further request costs beta of a lone request's block and head
 * time (decode is memory-bound), and a link carries b activations.
 */
int oracle_quantise_slots(int M, int N, const uint64_t *speed, const uint64_t *bw,
                          const uint32_t *cong, const uint64_t *layer_flops,
                          const uint64_t *act, const uint64_t *head_flops, int b_max,
                          uint32_t beta_ppm, uint64_t *t /*[R][M][N]*/, uint64_t *h /*[R][M]*/,
                          uint64_t *tau /*[R][M][M]*/)
{
    if (b_max < 1 || b_max > 15 || beta_ppm > 1000000u) return ORC_EINVAL;
    int rc = oracle_quantise(M, N, speed, bw, cong, layer_flops, act, head_flops, t, h, tau);
    if (rc) return rc;
    for (int b = 2; b <= b_max; b++) {
        for (int d = 0; d < M; d++) {
            for (int n = 0; n < N; n++) {
                uint64_t one = t[((size_t)1 * M + d) * N + n];
                uint64_t extra = (uint64_t)(((u128)one * beta_ppm + 999999u) / 1000000u);
                uint64_t v = one + (uint64_t)(b - 1) * extra;
                if (v >= LIMIT48) return ORC_EOVERFLOW;
                t[((size_t)b * M + d) * N + n] = v;
            }
            uint64_t one = h[M + d];
            uint64_t extra = (uint64_t)(((u128)one * beta_ppm + 999999u) / 1000000u);
            uint64_t hv = one + (uint64_t)(b - 1) * extra;
            if (hv >= LIMIT48) return ORC_EOVERFLOW;
            h[(size_t)b * M + d] = hv;
        }
        for (int d = 0; d < M; d++) {
            for (int e = 0; e < M; e++) {
                uint64_t v;
                if (d == e) {
                    v = 0;
                } else {
                    uint64_t beff = (uint64_t)(((u128)bw[d * M + e] * cong[d * M + e]) / 1000000u);
                    if (beff == 0) {
                        v = INF;
                    } else {
                        u128 num = (u128)act[1] * (uint64_t)b * 1000000000u;
                        u128 qv = (num + beff - 1) / beff;
                        if (qv >= LIMIT48) return ORC_EOVERFLOW;
                        v = (uint64_t)qv;
                    }
                }
                tau[((size_t)b * M + d) * M + e] = v;
            }
        }
    }
    return ORC_OK;
}

/*
 * The paper's inner loop for one population of label genomes (Algorithm 2;
 * Sec. 3.4, role assignment paragraph).  For every non-empty cluster q of
 * genome p (chain in ascending id):
 *   - DP_Pipe with the prefill tables (r = 0) and with the decode tables of
 *     each b = 1..b_max (r = b), block bytes W[n] + kv * slots(r), slots(0)
 *     = 1 (the request being prefilled), slots(b) = b;
 *     T_all, L_all [P][k_max][b_max + 1] receive T and Lambda (INF if empty
 *     or infeasible);
 *   - prefill rate rho_P = floor(SCALE / max(T_0, 1)), 0 if infeasible;
 *   - b* = the highest b whose DP is feasible and passes the QoS floor
 *     Lambda_b <= floor(1e12 / min_tps_milli) (no floor if 0); decode rate
 *     rho_D = floor(b* SCALE / max(T_b*, 1)), 0 if no b qualifies (b
 *     requests share the pipeline, which emits b tokens per T).
 * Then every assignment of a role to each non-empty cluster is scored by
 * Eq. 3-5 on the summed rates (rates_fitness), and the smallest (w, phase)
 * wins; ties go to the assignment whose decode set, as a bitmask over q, is
 * smallest.  roles_out[p][q] = 1 for decode, 0 for prefill and for empty
 * clusters; slots_out[p][q] = b* of a decode cluster (0 if none qualified),
 * 0 otherwise.
 *
 * Only the F "free" clusters, those with rho_D > 0, are enumerated (2^F
 * assignments); every other cluster is prefill.  This finds the same
 * winner as enumerating all non-empty clusters: w and phase never grow when
 * the prefill sum grows and the decode sum stays (S_P falls, so phase and
 * the excess fall, and w = S_P + excess or 0), so turning a cluster with
 * rho_D = 0 from decode to prefill gives a (w, phase) no larger and a
 * smaller decode bitmask.  A genome with more than ORC_MAX_FREE free
 * clusters is not searched: roles 0, every slots_out entry 0xFF and w =
 * phase = INF.
 */
static int assign_roles(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                        const uint64_t *mem, const uint64_t *W, uint64_t HB, uint64_t kv,
                        int b_max, int P, int k_max, const uint8_t *labels,
                        const uint8_t *order, const uint16_t *sizes_in, uint64_t t_arrival,
                        uint64_t nd, uint64_t min_tps_milli, int policy, uint64_t np_tokens,
                        uint64_t *T_all, uint64_t *L_all, uint8_t *roles_out, uint8_t *slots_out,
                        uint64_t *w, uint64_t *phase);

/* free clusters (a decode rate) a genome may have for the role search */
#define ORC_MAX_FREE 24

int oracle_search_roles(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                        const uint64_t *mem, const uint64_t *W, uint64_t HB, uint64_t kv,
                        int b_max, int P, int k_max, const uint8_t *labels, uint64_t t_arrival,
                        uint64_t nd, uint64_t min_tps_milli, uint64_t *T_all, uint64_t *L_all,
                        uint8_t *roles_out, uint8_t *slots_out, uint64_t *w, uint64_t *phase)
{
    return assign_roles(M, N, t, h, tau, mem, W, HB, kv, b_max, P, k_max, labels, NULL, NULL,
                        t_arrival, nd, min_tps_milli, 0, 0, T_all, L_all, roles_out, slots_out,
                        w, phase);
}

/*
 * The same search for two-chromosome genomes (App. A): replica q's chain is
 * its run of the ordering (replica_range); a replica holding an id >= M has
 * no DP result and no rates.
 */
int oracle_search_roles_ordered(int M, int N, const uint64_t *t, const uint64_t *h,
                                const uint64_t *tau, const uint64_t *mem, const uint64_t *W,
                                uint64_t HB, uint64_t kv, int b_max, int P, int k_max,
                                const uint8_t *order, const uint16_t *sizes, uint64_t t_arrival,
                                uint64_t nd, uint64_t min_tps_milli, uint64_t *T_all,
                                uint64_t *L_all, uint8_t *roles_out, uint8_t *slots_out,
                                uint64_t *w, uint64_t *phase)
{
    return assign_roles(M, N, t, h, tau, mem, W, HB, kv, b_max, P, k_max, NULL, order, sizes,
                        t_arrival, nd, min_tps_milli, 0, 0, T_all, L_all, roles_out, slots_out,
                        w, phase);
}

/*
 * The adapted-SplitWise role rule (the ablation of Sec. 4.2): the same
 * per-cluster DPs, prefill rates, kept slot counts and decode rates as
 * oracle_search_roles, but instead of the brute force the R' non-empty
 * clusters of a genome split by the token ratio: n_P = R'  NP / (NP + ND)
 * rounded half up and clamped to [1, R' - 1] (R' itself when R' <= 1; 1/2
 * of R' when NP + ND = 0), the n_P clusters with the highest prefill rate
 * (ties to the smaller q) take prefill and the rest decode.  k_max <= 255.
 */
int oracle_assign_roles_splitwise(int M, int N, const uint64_t *t, const uint64_t *h,
                                  const uint64_t *tau, const uint64_t *mem, const uint64_t *W,
                                  uint64_t HB, uint64_t kv, int b_max, int P, int k_max,
                                  const uint8_t *labels, uint64_t t_arrival, uint64_t nd,
                                  uint64_t min_tps_milli, uint64_t np_tokens, uint64_t *T_all,
                                  uint64_t *L_all, uint8_t *roles_out, uint8_t *slots_out,
                                  uint64_t *w, uint64_t *phase)
{
    return assign_roles(M, N, t, h, tau, mem, W, HB, kv, b_max, P, k_max, labels, NULL, NULL,
                        t_arrival, nd, min_tps_milli, 1, np_tokens, T_all, L_all, roles_out,
                        slots_out, w, phase);
}

static int assign_roles(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                        const uint64_t *mem, const uint64_t *W, uint64_t HB, uint64_t kv,
                        int b_max, int P, int k_max, const uint8_t *labels,
                        const uint8_t *order, const uint16_t *sizes_in, uint64_t t_arrival,
                        uint64_t nd, uint64_t min_tps_milli, int policy, uint64_t np_tokens,
                        uint64_t *T_all, uint64_t *L_all, uint8_t *roles_out, uint8_t *slots_out,
                        uint64_t *w, uint64_t *phase)
{
    if (M < 1 || M > 256 || N < 1 || N > 255 || P < 0 || k_max < 1 || k_max > 255 ||
        b_max < 1 || b_max > 15 || nd > 8192)
        return ORC_EINVAL;
    const int R = b_max + 1;
    int chain[256], sizes[256];
    uint64_t hk[256], tl[256], mk[256];
    uint64_t *tk = malloc(sizeof(uint64_t) * (size_t)M * N);
    uint64_t *Wr = malloc(sizeof(uint64_t) * (size_t)N);
    if (!tk || !Wr) { free(tk); free(Wr); return ORC_ENOMEM; }
    const uint64_t lam_max = min_tps_milli ? 1000000000000ull / min_tps_milli : INF;
    for (int p = 0; p < P; p++) {
        uint64_t rho_p[256], rho_d[256];
        int bstar[256], used[256], n_used = 0;
        for (int q = 0; q < k_max; q++) {
            /* the cluster's chain: the devices labelled q in ascending id,
             * or replica q's run of the ordering (an id >= M: infeasible) */
            int m = 0, valid = 1;
            if (labels) {
                for (int d = 0; d < M; d++)
                    if (labels[(size_t)p * M + d] == q) chain[m++] = d;
            } else {
                int lo, hi;
                replica_range(M, k_max, sizes_in + (size_t)p * k_max, q, &lo, &hi);
                for (int k = lo; k < hi; k++) {
                    chain[m] = order[(size_t)p * M + k];
                    if (chain[m] >= M) valid = 0;
                    m++;
                }
            }
            uint64_t *To = T_all + ((size_t)p * k_max + q) * R;
            uint64_t *Lo = L_all + ((size_t)p * k_max + q) * R;
            for (int r = 0; r < R; r++) To[r] = Lo[r] = INF;
            rho_p[q] = rho_d[q] = 0;
            bstar[q] = 0;
            if (m == 0) continue;
            used[n_used++] = q;
            if (!valid) continue;
            for (int r = 0; r < R; r++) {
                uint64_t slots = r == 0 ? 1 : (uint64_t)r;
                for (int n = 0; n < N; n++) Wr[n] = W[n] + kv * slots;
                for (int k = 0; k < m; k++) {
                    memcpy(tk + (size_t)k * N, t + ((size_t)r * M + chain[k]) * N,
                           sizeof(uint64_t) * N);
                    hk[k] = h[(size_t)r * M + chain[k]];
                    mk[k] = mem[chain[k]];
                    tl[k] = (k == 0) ? 0 : tau[((size_t)r * M + chain[k - 1]) * M + chain[k]];
                }
                uint64_t Tv, Lv, ev;
                int mu;
                int rc = oracle_dp_pipe(m, N, tk, hk, tl, mk, Wr, HB, &Tv, &Lv, &mu, sizes, &ev);
                if (rc) { free(tk); free(Wr); return rc; }
                To[r] = Tv;
                Lo[r] = Tv == INF ? INF : Lv;
            }
            if (To[0] != INF) rho_p[q] = SCALE / (To[0] > 0 ? To[0] : 1);
            for (int b = b_max; b >= 1; b--) {
                if (To[b] != INF && Lo[b] <= lam_max) {
                    bstar[q] = b;
                    rho_d[q] = ((uint64_t)b * SCALE) / (To[b] > 0 ? To[b] : 1);
                    break;
                }
            }
        }
        if (policy == 1) {
            /* prefill count from the token ratio, then the strongest
             * clusters by prefill rate take prefill */
            int n_p = n_used;
            if (n_used >= 2) {
                uint64_t tot = np_tokens + nd;
                n_p = tot ? (int)((2 * (uint64_t)n_used * np_tokens + tot) / (2 * tot))
                          : (n_used + 1) / 2;
                if (n_p < 1) n_p = 1;
                if (n_p > n_used - 1) n_p = n_used - 1;
            }
            uint8_t dec[256] = {0};
            for (int i = 0; i < n_used; i++) {
                int qi = used[i], rank = 0;
                for (int k = 0; k < n_used; k++) {
                    int qk = used[k];
                    if (rho_p[qk] > rho_p[qi] || (rho_p[qk] == rho_p[qi] && qk < qi)) rank++;
                }
                dec[qi] = rank >= n_p;
            }
            uint64_t sum_p = 0, sum_d = 0, sp, sd;
            for (int i = 0; i < n_used; i++) {
                int q = used[i];
                if (dec[q]) sum_d += rho_d[q];
                else sum_p += rho_p[q];
            }
            rates_fitness(sum_p, sum_d, t_arrival, nd, w + p, phase + p, &sp, &sd);
            for (int q = 0; q < k_max; q++) {
                roles_out[(size_t)p * k_max + q] = dec[q];
                slots_out[(size_t)p * k_max + q] = (uint8_t)(dec[q] ? bstar[q] : 0);
            }
            continue;
        }
        /* the free clusters in increasing q; the rest stay prefill */
        int fr[256], F = 0;
        for (int i = 0; i < n_used; i++)
            if (rho_d[used[i]] > 0) fr[F++] = used[i];
        if (F > ORC_MAX_FREE) {
            for (int q = 0; q < k_max; q++) {
                roles_out[(size_t)p * k_max + q] = 0;
                slots_out[(size_t)p * k_max + q] = 0xFF;
            }
            w[p] = phase[p] = INF;
            continue;
        }
        /* every role assignment of the free clusters: bit i of x makes fr[i]
         * decode; x increases with the decode bitmask over q, so the first
         * best x is the smallest bitmask among ties */
        uint64_t best_w = INF, best_ph = INF;
        uint32_t best_x = 0;
        int have = 0;
        uint64_t fixed_p = 0;
        for (int i = 0; i < n_used; i++)
            if (rho_d[used[i]] == 0) fixed_p += rho_p[used[i]];
        for (uint32_t x = 0; x < (1u << F); x++) {
            uint64_t sum_p = fixed_p, sum_d = 0;
            for (int j = 0; j < F; j++) {
                if ((x >> j) & 1u) sum_d += rho_d[fr[j]];
                else sum_p += rho_p[fr[j]];
            }
            uint64_t wv, pv, sp, sd;
            rates_fitness(sum_p, sum_d, t_arrival, nd, &wv, &pv, &sp, &sd);
            if (!have || wv < best_w || (wv == best_w && pv < best_ph)) {
                best_w = wv;
                best_ph = pv;
                best_x = x;
                have = 1;
            }
        }
        uint8_t dec[256] = {0};
        for (int j = 0; j < F; j++) dec[fr[j]] = (best_x >> j) & 1u;
        for (int q = 0; q < k_max; q++) {
            roles_out[(size_t)p * k_max + q] = dec[q];
            slots_out[(size_t)p * k_max + q] = (uint8_t)(dec[q] ? bstar[q] : 0);
        }
        w[p] = best_w;
        phase[p] = best_ph;
    }
    free(tk);
    free(Wr);
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* The idle-device relaxation (R2): devices may hold zero blocks.          */
/* ---------------------------------------------------------------------- */

/*
 * DP over a chain where a device may hold no block and then leaves the
 * pipeline; links join consecutive participating devices (tau_full gives
 * every ordered pair of chain positions); the master always participates,
 * with its head, and may hold no block (its stage is then the head alone).
 * For a master mu, with x = blocks placed so far (0..N):
 *   A_k(x)   = min over allowed predecessors k' (ascending, "none" first)
 *              of max(E_k'(x), tau(k', k)); "none" (k is the first
 *              participant) stands for E(0) = 0, E(x > 0) = INF, tau 0;
 *              allowed: k < mu and k = mu: none or 1..k-1; k > mu: mu..k-1
 *   E_k(x)   = min over j ascending in device k's window of
 *              max(A_k(j), cost_k(j, x-1)) (blocks j..x-1 on device k, the
 *              head on the master), then for k = mu the empty stage
 *              max(A_mu(x), head) when the head bytes fit (strict <, so a
 *              stage with blocks wins ties)
 *   T_mu     = min over k >= mu of E_k(N), the smallest k on ties
 * and mu* is the smallest master with the least T_mu.  Outputs as
 * oracle_dp_pipe: sizes[k] = 0 for devices that sit out, *Lambda = stage
 * times of the participants (+ head) + links between consecutive ones.
 */
int oracle_dp_idle(int m, int N, const uint64_t *tk, const uint64_t *hk, const uint64_t *tau_full,
                   const uint64_t *memk, const uint64_t *W, uint64_t HB, uint64_t *T,
                   uint64_t *Lambda, int *mu_star, int *sizes)
{
    *T = INF;
    *Lambda = INF;
    *mu_star = 0;
    for (int k = 0; k < m; k++) sizes[k] = 0;
    if (m < 1 || N < 1) return ORC_EINVAL;
    const int X = N + 1;
    uint64_t *pt = malloc(sizeof(uint64_t) * (size_t)m * X);
    uint64_t *pw = malloc(sizeof(uint64_t) * (size_t)X);
    uint64_t *E = malloc(sizeof(uint64_t) * (size_t)m * X);
    uint64_t *A = malloc(sizeof(uint64_t) * (size_t)m * X);
    int *Ek = malloc(sizeof(int) * (size_t)m * X);  /* predecessor of A_k(x): -1 none */
    int *Ej = malloc(sizeof(int) * (size_t)m * X);  /* stage start j, or x for an empty stage */
    if (!pt || !pw || !E || !A || !Ek || !Ej) {
        free(pt); free(pw); free(E); free(A); free(Ek); free(Ej);
        return ORC_ENOMEM;
    }
    for (int k = 0; k < m; k++) {
        pt[(size_t)k * X] = 0;
        for (int n = 0; n < N; n++) pt[(size_t)k * X + n + 1] = pt[(size_t)k * X + n] + tk[(size_t)k * N + n];
    }
    pw[0] = 0;
    for (int n = 0; n < N; n++) pw[n + 1] = pw[n] + W[n];

    uint64_t best = INF;
    int best_mu = 0, best_last = -1;
    for (int pass = 0; pass < 2; pass++) {
        /* pass 0 finds mu*; pass 1 rebuilds its tables for the back tracing */
        int mu_lo = pass ? best_mu : 1, mu_hi = pass ? best_mu : m;
        if (pass && best == INF) break;
        for (int mu = mu_lo; mu <= mu_hi; mu++) {
            for (int k = 1; k <= m; k++) {
                uint64_t *Ak = A + (size_t)(k - 1) * X;
                uint64_t *Erow = E + (size_t)(k - 1) * X;
                int *pk = Ek + (size_t)(k - 1) * X, *pj = Ej + (size_t)(k - 1) * X;
                const int none_ok = k <= mu;
                const int kp_lo = k > mu ? mu : 1;
                for (int x = 0; x <= N; x++) {
                    uint64_t a = INF;
                    int arg = -2;
                    if (none_ok && x == 0) {
                        a = 0;
                        arg = -1;
                    }
                    for (int kp = kp_lo; kp <= k - 1; kp++) {
                        uint64_t e = E[(size_t)(kp - 1) * X + x];
                        uint64_t tl = tau_full[(size_t)(kp - 1) * m + (k - 1)];
                        if (e == INF || tl == INF) continue;
                        uint64_t v = max2(e, tl);
                        if (v < a) {
                            a = v;
                            arg = kp;
                        }
                    }
                    Ak[x] = a;
                    pk[x] = arg;
                }
                const uint64_t *ptk = pt + (size_t)(k - 1) * X;
                const uint64_t head_t = (k == mu) ? hk[k - 1] : 0;
                const uint64_t head_b = (k == mu) ? HB : 0;
                for (int x = 0; x <= N; x++) {
                    uint64_t e = INF;
                    int jj = -1;
                    for (int j = 0; j < x; j++) {
                        if (Ak[j] == INF) continue;
                        if (pw[x] - pw[j] + head_b > memk[k - 1]) continue;
                        uint64_t v = max2(Ak[j], ptk[x] - ptk[j] + head_t);
                        if (v < e) {
                            e = v;
                            jj = j;
                        }
                    }
                    if (k == mu && Ak[x] != INF && HB <= memk[k - 1]) {
                        uint64_t v = max2(Ak[x], hk[k - 1]);
                        if (v < e) {
                            e = v;
                            jj = x;
                        }
                    }
                    Erow[x] = e;
                    pj[x] = jj;
                }
            }
            uint64_t tmu = INF;
            int last = -1;
            for (int k = mu; k <= m; k++) {
                uint64_t v = E[(size_t)(k - 1) * X + N];
                if (v < tmu) {
                    tmu = v;
                    last = k;
                }
            }
            if (!pass && tmu < best) {
                best = tmu;
                best_mu = mu;
            }
            if (pass) best_last = last;
        }
    }
    if (best != INF) {
        /* back tracing from (best_last, N) */
        int k = best_last, x = N;
        int prev_k = -1;
        uint64_t lam = 0;
        while (k >= 1) {
            int j = Ej[(size_t)(k - 1) * X + x];
            sizes[k - 1] = x - j;
            lam += pt[(size_t)(k - 1) * X + x] - pt[(size_t)(k - 1) * X + j];
            if (k == best_mu) lam += hk[k - 1];
            if (prev_k > 0) lam += tau_full[(size_t)(k - 1) * m + (prev_k - 1)];
            int kp = Ek[(size_t)(k - 1) * X + j];
            prev_k = k;
            k = kp;     /* -1: k was the first participant */
            x = j;
        }
        *T = best;
        *Lambda = lam;
        *mu_star = best_mu;
    }
    free(pt); free(pw); free(E); free(A); free(Ek); free(Ej);
    return ORC_OK;
}

/*
 * Population solve under the idle-device relaxation: as oracle_solve, with
 * links between any two chain devices from tau; m > N is allowed.
 */
int oracle_solve_idle(int M, int N, const uint64_t *t, const uint64_t *h, const uint64_t *tau,
                      const uint64_t *mem, const uint64_t *W, uint64_t HB, int P, int k_max,
                      const uint8_t *labels, const uint8_t *roles, uint64_t *T, uint64_t *Lambda,
                      int16_t *master, uint8_t *layers)
{
    if (M < 1 || M > 256 || N < 1 || N > 255 || P < 0 || k_max < 1 || k_max > 255)
        return ORC_EINVAL;
    int chain[256], sizes[256];
    uint64_t hk[256], mk[256];
    uint64_t *tk = malloc(sizeof(uint64_t) * (size_t)M * N);
    uint64_t *tf = malloc(sizeof(uint64_t) * (size_t)M * M);
    if (!tk || !tf) { free(tk); free(tf); return ORC_ENOMEM; }
    for (int p = 0; p < P; p++) {
        for (int d = 0; d < M; d++) layers[(size_t)p * M + d] = 0;
        for (int q = 0; q < k_max; q++) {
            size_t o = (size_t)p * k_max + q;
            T[o] = INF;
            Lambda[o] = INF;
            master[o] = -1;
            int m = 0;
            for (int d = 0; d < M; d++)
                if (labels[(size_t)p * M + d] == q) chain[m++] = d;
            if (m == 0) continue;
            int r = roles[o] != 0;
            for (int a = 0; a < m; a++) {
                memcpy(tk + (size_t)a * N, t + ((size_t)r * M + chain[a]) * N, sizeof(uint64_t) * N);
                hk[a] = h[r * M + chain[a]];
                mk[a] = mem[chain[a]];
                for (int b = 0; b < m; b++)
                    tf[(size_t)a * m + b] = a == b ? 0 : tau[((size_t)r * M + chain[a]) * M + chain[b]];
            }
            uint64_t Tv, Lv;
            int mu;
            int rc = oracle_dp_idle(m, N, tk, hk, tf, mk, W, HB, &Tv, &Lv, &mu, sizes);
            if (rc) { free(tk); free(tf); return rc; }
            if (Tv == INF) continue;
            T[o] = Tv;
            Lambda[o] = Lv;
            master[o] = (int16_t)chain[mu - 1];
            for (int a = 0; a < m; a++) layers[(size_t)p * M + chain[a]] = (uint8_t)sizes[a];
        }
    }
    free(tk);
    free(tf);
    return ORC_OK;
}
