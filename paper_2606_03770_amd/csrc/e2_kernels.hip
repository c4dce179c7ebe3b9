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
constexpr int kDpLdsTb = 4096;  // split-point table kept in LDS when m * N fits

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
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
// DP for one device chain and one master position mu (1-based).
// D, Pp, S2 are LDS rows of N entries; tbp (LDS or global, may be null)
// receives the split point of every cell of rows 2..m.
// Returns DP_mu(N-1, m).
// ---------------------------------------------------------------------------
__device__ uint64_t dp_table(const E2Tables &tb, int r, const uint8_t *chain, int m, int mu,
                             uint8_t *tbp, uint64_t *D, uint64_t *Pp, uint64_t *S2, int lane)
{
    const int M = tb.M, N = tb.N;
    {
        const int c = chain[0];
        const int f = (mu == 1);
        const uint64_t *pr = tb.pref + ((size_t)r * M + c) * (N + 1);
        const uint8_t *wr = tb.win + ((size_t)f * M + c) * N;
        const uint64_t hadd = f ? tb.head[r * M + c] : 0;
        for (int i = lane; i < N; i += kWave) D[i] = (wr[i] == 0) ? pr[i + 1] + hadd : E2_INF64;
    }
    __syncthreads();
    for (int k = 2; k <= m; ++k) {
        const int cp = chain[k - 2];
        const int c = chain[k - 1];
        const int f = (mu == k);
        const uint64_t tau = tb.tau[((size_t)r * M + cp) * M + c];
        const uint64_t *pr = tb.pref + ((size_t)r * M + c) * (N + 1);
        const uint8_t *wr = tb.win + ((size_t)f * M + c) * N;
        const uint64_t hadd = f ? tb.head[r * M + c] : 0;
        for (int j = lane; j < N; j += kWave) {
            const uint64_t prev = (j == 0) ? E2_INF64 : D[j - 1];
            Pp[j] = (prev == E2_INF64 || tau == E2_INF64) ? E2_INF64
                                                          : ((umax64(prev, tau) << 8) | (uint64_t)j);
            S2[j] = (pr[j] << 8) - (uint64_t)j;
        }
        __syncthreads();
        for (int i = lane; i < N; i += kWave) {
            uint64_t best = E2_INF64;
            int lo = wr[i];
            if (lo != (int)E2_NO_START && i >= k - 1) {
                if (lo < k - 1) lo = k - 1;
                const uint64_t si1 = (pr[i + 1] + hadd) << 8;
                for (int j = lo; j <= i; ++j) {
                    const uint64_t v = umax64(Pp[j], si1 - S2[j]);
                    best = umin64(best, v);
                }
            }
            D[i] = (best == E2_INF64) ? E2_INF64 : (best >> 8);
            if (tbp) tbp[(size_t)(k - 2) * N + i] = (uint8_t)(best & 0xFF);
        }
        __syncthreads();
    }
    return D[N - 1];
}

// ---------------------------------------------------------------------------
// Persistent DP kernel: one wave per workgroup; waves take listed problems
// in order through an atomic counter and exit when the list is exhausted.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_dp(E2Tables tb, int k_max,
                                           const uint8_t *__restrict__ labels,
                                           const uint8_t *__restrict__ roles,
                                           uint32_t *counters, const uint32_t *__restrict__ list,
                                           uint8_t *tb_global, uint64_t *T, uint64_t *Lambda,
                                           int16_t *master, uint8_t *layers)
{
    __shared__ uint64_t D[256], Pp[256], S2[256];
    __shared__ uint8_t chain[256];
    __shared__ uint8_t start[256];
    __shared__ uint8_t tb_lds[kDpLdsTb];
    __shared__ uint32_t job;
    const int lane = threadIdx.x;
    const int M = tb.M, N = tb.N;
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
        for (int mu = 1; mu <= m; ++mu) {
            const uint64_t v = dp_table(tb, r, chain, m, mu, nullptr, D, Pp, S2, lane);
            if (v < best) {
                best = v;
                best_mu = mu;
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
        uint8_t *tbp = (m * N <= kDpLdsTb) ? tb_lds : tb_global + (size_t)blockIdx.x * N * N;
        dp_table(tb, r, chain, m, best_mu, tbp, D, Pp, S2, lane);
        __threadfence_block();
        __syncthreads();
        if (lane == 0) {
            int i = N - 1;
            for (int k = m; k >= 2; --k) {
                const int j = tbp[(size_t)(k - 2) * N + i];
                start[k - 1] = (uint8_t)j;
                i = j - 1;
            }
            start[0] = 0;
        }
        __syncthreads();
        // Lambda: stage times (+ head on the master) plus the chain's link times
        uint64_t part = 0;
        for (int k = lane; k < m; k += kWave) {
            const int c = chain[k];
            const int s = start[k];
            const int e = (k + 1 < m) ? start[k + 1] : N;
            const uint64_t *pr = tb.pref + ((size_t)r * M + c) * (N + 1);
            part += pr[e] - pr[s];
            if (k + 1 == best_mu) part += tb.head[r * M + c];
            if (k >= 1) part += tb.tau[((size_t)r * M + chain[k - 1]) * M + c];
            if (layers) layers[(size_t)p * M + c] = (uint8_t)(e - s);
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
    k_dp<<<wk.n_slots, 64, 0, s>>>(t, k_max, labels, roles, wk.counters, wk.list, wk.tb_global,
                                   T, Lambda, master, layers);
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
