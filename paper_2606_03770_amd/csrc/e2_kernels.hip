// HIP kernels (gfx950, wave64) of the population-fitness path.
//
//   k_init        zero the per-call counters (a fill kernel, no memset node)
//   k_extract     one wave per individual: cluster sizes, a necessary
//                 memory/size pre-check, the list of clusters that need the
//                 DP (bucketed by chain length); INF results for the others
//   k_dp          persistent waves: each takes its share of the listed
//                 clusters, rebuilds a device chain from the genome, runs the
//                 bottleneck DP of Algorithm 1 / Eq. 1-2 over the master
//                 positions, picks the best master, backtracks and writes
//                 T, Lambda, master and per-device block counts
//   k_fitness     Eq. 3-5 per individual with the QoS floor (one wave per
//                 individual, lanes over clusters)
//   k_elites      one workgroup: the n_elite best keys (w, phase, index)
//   k_breed       one wave per output slot: elite copy or tournament +
//                 uniform crossover + per-gene mutation
//   k_breed_ordered  the same for two-chromosome genomes (App. A):
//                 ordering crossover with repair, one parent's grouping,
//                 four kinds of mutation
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

#include <atomic>

#include "../../include/e2.h"
#include "e2_internal.h"

namespace {

constexpr int kWave = 64;
// a pointer into LDS: reads and writes through it are ds_* instructions
// with 32-bit addresses instead of flat ones
template <typename T> using lds_t = __attribute__((address_space(3))) T;

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Wave-wide reductions: DPP permutations within each 16-lane row (quad
// swaps, half mirror, mirror), then the four row results read into scalars.
// The results are wave-uniform.
// CTRL is always a full permutation of each row (every lane reads a lane of
// its own row), so no lane keeps an old value and none is passed.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v)
{
    static_assert(CTRL == 0xb1 || CTRL == 0x4e || CTRL == 0x140 || CTRL == 0x141,
                  "a full permutation within each row");
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v)
{
    const int lo = dpp_i32<CTRL>((int)(uint32_t)v);
    const int hi = dpp_i32<CTRL>((int)(uint32_t)(v >> 32));
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
    v = umin64(v, dpp_u64<0xb1>(v));
    v = umin64(v, dpp_u64<0x4e>(v));
    v = umin64(v, dpp_u64<0x141>(v));
    v = umin64(v, dpp_u64<0x140>(v));
    return umin64(umin64(readlane_u64(v, 0), readlane_u64(v, 16)),
                  umin64(readlane_u64(v, 32), readlane_u64(v, 48)));
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
    v = umax64(v, dpp_u64<0xb1>(v));
    v = umax64(v, dpp_u64<0x4e>(v));
    v = umax64(v, dpp_u64<0x141>(v));
    v = umax64(v, dpp_u64<0x140>(v));
    return umax64(umax64(readlane_u64(v, 0), readlane_u64(v, 16)),
                  umax64(readlane_u64(v, 32), readlane_u64(v, 48)));
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
    v += dpp_u64<0xb1>(v);
    v += dpp_u64<0x4e>(v);
    v += dpp_u64<0x141>(v);
    v += dpp_u64<0x140>(v);
    return readlane_u64(v, 0) + readlane_u64(v, 16) + readlane_u64(v, 32) + readlane_u64(v, 48);
}

__global__ void k_init(uint32_t *counters)
{
    if (threadIdx.x < kCounters) counters[threadIdx.x * kCounterStride] = 0;
}

// ---------------------------------------------------------------------------
// Extraction and pre-check: one wave per genome, eg_of<SEARCH>() genomes per
// workgroup.
// A cluster goes to the DP list unless it is empty or provably infeasible:
//   more devices than blocks (every device must hold a block), a device that
//   cannot hold a single block, total single-stage capacity below N, or no
//   device able to hold a block plus the head (no possible master).
// Listed problems are bucketed by chain length into kClasses segments of the
// list (longest chains first), so the DP kernel schedules large problems
// early; each workgroup reserves its range of each segment with one atomic.
// Those atomics all meet on the segments' counters, so an evaluation's
// workgroup takes 16 genomes (1024 threads): half the reservations of 8 (a
// third less kernel time on the 16384-genome population).  The role
// search's instances hold about 80 VGPRs, so that one 1024-thread
// workgroup per CU would fit: they keep 8 genomes per workgroup.
// ---------------------------------------------------------------------------
template <bool SEARCH> constexpr int eg_of() { return SEARCH ? 8 : 16; }
constexpr int kDynTailShift = 2;  // the last 1/4 of the DP list is taken dynamically ...
constexpr uint32_t kDynTailMinPerWave = 16;  // ... with at least this many problems per wave
constexpr int kClasses = 4;  // chain-length classes: m >= 16, 12..15, 8..11, < 8
// longest chain whose per-position table fits one register per lane; longer
// chains of the bottleneck objective go to the list's last segment
constexpr int kMaxBandedChain = kWave;

__device__ __forceinline__ int size_class(int m)
{
    return m >= 16 ? 0 : (m >= 12 ? 1 : (m >= 8 ? 2 : 3));
}

// Replica of ordering position t of a two-chromosome genome: the largest r
// with offs[r] <= t (offs[r] = clipped start of replica r; empty replicas
// share their start with the next one), or 256 when t lies beyond every
// replica.
__device__ __forceinline__ int replica_at(const uint32_t *offs, int k_max, int t)
{
    if ((uint32_t)t >= offs[k_max]) return 256;
    int lo = 0, hi = k_max - 1;  // offs[lo] <= t < offs[hi + 1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (offs[mid] <= (uint32_t)t) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Memory class of a role index: one shared class, or one per role index.
__device__ __forceinline__ int mem_class(const E2Tables &tb, int r) { return tb.n_mem > 1 ? r : 0; }

// The tables with the memory windows and capacities of role index r.
__device__ __forceinline__ E2Tables mem_view(const E2Tables &tb, int r)
{
    E2Tables v = tb;
    const size_t c = (size_t)mem_class(tb, r);
    const size_t MN = (size_t)tb.M * tb.N;
    v.wtab += c * 6 * MN;
    v.cap0 += c * tb.M;
    v.capH += c * tb.M;
    return v;
}

// SEARCH = false: one problem per cluster, at role index (roles[q] != 0);
// SEARCH = true: one problem per cluster and role index (n_roles = R <= 16,
// P < 2^20), outputs [P][k_max][R] and list codes (p << 12) | (q << 4) | r.
// ORD: two-chromosome genomes (replicas are runs of the ordering), else
// label genomes.  One instance per genome kind and mode keeps the label
// path free of the ordering's LDS arrays and registers.
template <bool ORD, bool SEARCH>
__global__ __launch_bounds__(64 * eg_of<SEARCH>()) void k_extract(E2Tables tb, int P, int k_max,
                                                      E2Genomes gen, const uint8_t *roles,
                                                      int n_roles, int relaxed, int long_seg,
                                                      uint32_t *counters,
                                                      uint32_t *list, size_t seg_cap,
                                                      uint64_t *T, uint64_t *Lambda,
                                                      int16_t *master, uint8_t *layers)
{
    // per genome: (count << 16) + sum of cap0, min cap0, head-capable flag per
    // cluster, listed bitmask
    constexpr int kEG = eg_of<SEARCH>();
    __shared__ uint32_t packed[kEG][256];
    __shared__ uint32_t mincap[kEG][256];
    __shared__ uint32_t hflag[kEG][256];  // 1 when some device can hold a block and the head
    __shared__ uint32_t lmask[kEG][8];
    __shared__ uint32_t ncls[kEG][16][kListSegs];  // per genome, pass and list segment
    __shared__ uint32_t base[kEG][16][kListSegs];
    // two-chromosome genomes only: replica starts, cap0 | head bit per position
    __shared__ uint32_t offs[ORD ? kEG : 1][ORD ? 256 : 1];
    __shared__ uint16_t posc[ORD ? kEG : 1][ORD ? 256 : 1];
    __shared__ uint32_t bad[kEG][8];     // replicas holding a device id >= M
    const int g = threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    const int p = blockIdx.x * kEG + g;
    const int M = tb.M, N = tb.N;
    constexpr bool ordered = ORD;
    const int n_r = SEARCH ? n_roles : 0;
    if constexpr (ordered) if (p < P) {
        // offs[r] = min(M, sizes[0] + ... + sizes[r-1]), r = 0..k_max
        uint32_t carry = 0;
        for (int r0 = 0; r0 <= k_max; r0 += kWave) {
            const int r = r0 + lane;
            const uint32_t v = (r >= 1 && r <= k_max) ? gen.sizes[(size_t)p * k_max + r - 1] : 0;
            uint32_t x = v;
            for (int d = 1; d < kWave; d <<= 1) {
                const uint32_t y = __shfl_up(x, d, kWave);
                if (lane >= d) x += y;
            }
            if (r <= k_max) offs[g][r] = min(carry + x, (uint32_t)M);
            carry += __shfl(x, kWave - 1, kWave);
        }
    }
    if (lane < 8) bad[g][lane] = 0;
    __syncthreads();
    // labels: slot u of a lane is device x, in cluster labs[u]; ordered
    // genomes: ordering position x, holding device devs[u], in replica labs[u]
    int labs[4], devs[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int x = lane + 64 * u;
        labs[u] = 256;
        devs[u] = 0;
        if (p < P && x < M) {
            int lab, d = x;
            if constexpr (ordered) {
                d = gen.order[(size_t)p * M + x];
                lab = replica_at(offs[g], k_max, x);
                if (d >= M) {  // not a device: its replica cannot be solved
                    if (lab < k_max) atomicOr(&bad[g][lab >> 5], 1u << (lab & 31));
                    lab = 256;
                    d = 0;
                }
            } else {
                lab = gen.labels[(size_t)p * M + x];
            }
            labs[u] = lab < k_max ? lab : 256;
            devs[u] = d;
        }
    }
    // Every pass (one per role index) decides its clusters and counts them per
    // class; slot u keeps each pass's class + 1 (0: not listed) in 3 bits of
    // code[u].  The list ranges of all passes are then reserved with one
    // atomic per class per workgroup.
    const int passes = n_r > 0 ? n_r : 1;
    uint64_t code[4] = {0, 0, 0, 0};
    if (n_r > 0 && p < P) {
        // every role index of every cluster starts infeasible, in one
        // contiguous sweep of the genome's [k_max][R] block (the DP kernel,
        // which runs after this one, overwrites the listed problems)
        const size_t o0 = (size_t)p * k_max * n_r;
        for (int i = lane; i < k_max * n_r; i += kWave) {
            T[o0 + i] = E2_INF64;
            Lambda[o0 + i] = E2_INF64;
        }
    }
    for (int i = lane; i < 16 * kListSegs; i += kWave) ncls[g][i / kListSegs][i % kListSegs] = 0;
    for (int ri = 0; ri < passes; ++ri) {
        for (int q = lane; q < k_max; q += 64) {
            packed[g][q] = 0;
            mincap[g][q] = 0xFFFFFFFFu;
            hflag[g][q] = 0;
        }
        if (lane < 8) lmask[g][lane] = 0;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int lab = labs[u];
            if (lab < k_max) {
                // role index of this pass, or of the cluster
                const int r = n_r > 0 ? ri : (tb.n_mem > 1 ? roles[(size_t)p * k_max + lab] != 0 : 0);
                const int c = mem_class(tb, r);
                const uint32_t c0 = tb.cap0[(size_t)c * M + devs[u]];
                const uint32_t cH = tb.capH[(size_t)c * M + devs[u]];
                if constexpr (ordered) {
                    posc[g][lane + 64 * u] = (uint16_t)(c0 | (cH ? 0x100u : 0u));
                } else {
                    atomicAdd(&packed[g][lab], (1u << 16) | c0);
                    atomicMin(&mincap[g][lab], c0);
                    // a per-cluster flag: the atomics of one word meet only
                    // the devices of one cluster
                    if (cH) atomicOr(&hflag[g][lab], 1u);
                }
            }
        }
        __syncthreads();
        if constexpr (ordered) {
            // a replica is a run of ordering positions [offs[q], offs[q+1]):
            // one lane per replica sums its run, with no atomics (the lanes
            // of one run would all meet on its words).  Positions holding an
            // id >= M lie in replicas marked bad, which are not listed.
            for (int q = lane; p < P && q < k_max; q += kWave) {
                const int lo = (int)offs[g][q], hi = (int)offs[g][q + 1];
                uint32_t sum = 0, mn = 0xFFFFFFFFu, any = 0;
                for (int x = lo; x < hi; ++x) {
                    const uint32_t v = posc[g][x];
                    sum += v & 0xFFu;
                    mn = min(mn, v & 0xFFu);
                    any |= v >> 8;
                }
                packed[g][q] = ((uint32_t)(hi - lo) << 16) | sum;
                mincap[g][q] = mn;
                hflag[g][q] = any;
            }
            __syncthreads();
        }
        // decide per cluster; count listed problems per class (slots u with
        // no cluster id below k_max are skipped: the bound is uniform)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (64 * u >= k_max) break;
            const int q = lane + 64 * u;
            bool feas = false;
            int cls = 0;
            if (p < P && q < k_max) {
                const uint32_t pk = packed[g][q];
                const uint32_t m = pk >> 16, csum = pk & 0xFFFF;
                // the checks hold for chains whose every device takes a
                // block; with idle devices allowed, every non-empty cluster
                feas = m >= 1 && !((bad[g][q >> 5] >> (q & 31)) & 1u) &&
                       (relaxed || (m <= (uint32_t)N && csum >= (uint32_t)N &&
                                    mincap[g][q] >= 1 && hflag[g][q] != 0));
                cls = (long_seg && m > (uint32_t)kMaxBandedChain) ? kClasses : size_class((int)m);
                if (!feas && n_r == 0) {  // (every role index: filled above)
                    const size_t o = (size_t)p * k_max + q;
                    T[o] = E2_INF64;
                    Lambda[o] = E2_INF64;
                    if (master) master[o] = -1;
                }
            }
            code[u] |= (uint64_t)(feas ? cls + 1 : 0) << (3 * ri);
            const uint64_t fm = __ballot(feas);
            if (lane == 0 && fm) {
                // q = 64u + bit: listed bitmask words 2u and 2u + 1
                lmask[g][2 * u] = (uint32_t)fm;
                lmask[g][2 * u + 1] = (uint32_t)(fm >> 32);
            }
            for (int c = 0; c < kListSegs; ++c) {
                const uint64_t bm = __ballot(feas && cls == c);
                if (lane == 0) ncls[g][ri][c] += (uint32_t)__popcll(bm);
            }
        }
        __syncthreads();  // the next pass clears the per-cluster sums
    }
    // one atomic per class per workgroup; the ranges follow (genome, pass)
    if (threadIdx.x < kListSegs) {
        const int c = threadIdx.x;
        uint32_t tot = 0;
        for (int h = 0; h < kEG; ++h)
            for (int ri = 0; ri < passes; ++ri) tot += ncls[h][ri][c];
        uint32_t b0 = tot ? atomicAdd(&counters[c * kCounterStride], tot) : 0;
        for (int h = 0; h < kEG; ++h)
            for (int ri = 0; ri < passes; ++ri) {
                base[h][ri][c] = b0;
                b0 += ncls[h][ri][c];
            }
    }
    __syncthreads();
    for (int ri = 0; ri < passes; ++ri) {
        uint32_t run[kListSegs] = {0, 0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (64 * u >= k_max) break;
            const int q = lane + 64 * u;
            const uint32_t mc = (uint32_t)(code[u] >> (3 * ri)) & 7u;
            for (int c = 0; c < kListSegs; ++c) {
                const uint64_t bm = __ballot(mc == (uint32_t)(c + 1));
                if (mc == (uint32_t)(c + 1)) {
                    const uint32_t pos =
                        base[g][ri][c] + run[c] + (uint32_t)__popcll(bm & ((1ull << lane) - 1));
                    list[(size_t)c * seg_cap + pos] =
                        n_r > 0 ? ((uint32_t)p << 12) | ((uint32_t)q << 4) | (uint32_t)ri
                                : ((uint32_t)p << 8) | (uint32_t)q;
                }
                run[c] += (uint32_t)__popcll(bm);
            }
        }
    }
    // layers of devices the DP kernel will not write: those outside every
    // listed cluster; for ordered genomes every device (the DP kernel, which
    // runs after this one, writes the listed replicas' devices, and a device
    // missing from the ordering keeps 0)
    if (layers && p < P) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int x = lane + 64 * u;
            const int lab = labs[u];
            if (x < M && (ordered || lab >= k_max || !((lmask[g][lab >> 5] >> (lab & 31)) & 1u)))
                layers[(size_t)p * M + x] = 0;
        }
    }
}

// ---------------------------------------------------------------------------
// One forward DP row.  Stage device c holds blocks j..i after `kmin` devices
// that hold blocks 0..j-1:
//   out(i) = min_{j in [max(win(i), kmin), i]} max(prev(j-1), tau, cost(j, i) + head)
// as packed scores (value << 8 | j).  The backward rows of the decomposition
// are the same rows over reversed blocks (block N-1 first), so every row of
// every table goes through this code.
//
// Key width K.  Every finite value of a problem is at most the largest cost
// of a memory-fitting stage of its devices (with the head time where the
// stage carries the head) or its largest finite link time.  When that bound
// is below 2^24 - 1 the packed keys fit in 32 bits: rows, split-point pairs
// and pools hold u32 and a candidate costs one subtract, one max and one
// min; otherwise keys are u64 (values < 2^56).  Stage costs come from u64
// prefix sums; the 32-bit path keeps the low 32 bits of (P << 8), whose
// differences are exact because every visited stage cost is below 2^24.
//
// Lane mapping: S lanes per cell (S = 8 for at most 8 cells, 4 for at most
// 16, 2 for at most 32, else 1); lane o of a cell visits j = i - o - S t for
// t = 0, 1, ...
// With L = min(cap, hi - jmin + 1) an upper bound and Lm a lower bound of
// the cells' window lengths, the first floor(Lm / S) steps stay inside
// every window and run unclamped (four at a time); the remaining steps
// clamp j to the lane's window start (a repeated candidate leaves a minimum
// unchanged).  The S partial minima meet through DPP quad permutations.
// Split points keep (prefix term, shifted prefix sum) as one LDS pair.
//
// INF needs no branches: finite values are below the key's INF threshold
// divided by 256, so a packed key built from an INF prefix term or link is
// >= the threshold and loses every comparison with a finite key.
// ---------------------------------------------------------------------------
template <typename K> struct KeyT;
template <> struct KeyT<uint64_t> {
    static constexpr uint64_t inf = E2_INF64;
    static constexpr uint64_t inf_key = 0xFFFFFFFFFFFFFF00ull;
};
template <> struct KeyT<uint32_t> {
    static constexpr uint32_t inf = 0xFFFFFFFFu;
    static constexpr uint32_t inf_key = 0xFFFFFF00u;
};
// fp64 keys: value * 256 + j is an integer below 2^53, so sums, differences,
// max and min are exact; INF is +infinity
template <> struct KeyT<double> {
    static constexpr double inf = __builtin_huge_val();
    static constexpr double inf_key = __builtin_huge_val();
};
constexpr uint64_t kU32MaxValue = 0xFFFFFEull;         // largest finite value of the 32-bit path
constexpr uint64_t kF64Limit = 1ull << 45;             // every value of the fp64 path is below

// fp64 keys are never NaN, so the hardware max/min are used directly (the
// compiler's IEEE-mode fmax/fmin would first quiet every loaded operand)
__device__ __forceinline__ double vmax_f64(double a, double b)
{
    double r;
    asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ double vmin_f64(double a, double b)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
template <typename K> __device__ __forceinline__ K kmax(K a, K b)
{
    if constexpr (__is_same(K, double)) return vmax_f64(a, b);
    else return a > b ? a : b;
}
template <typename K> __device__ __forceinline__ K kmin(K a, K b)
{
    if constexpr (__is_same(K, double)) return vmin_f64(a, b);
    else return a < b ? a : b;
}
// v permuted within each 16-lane row, as an operand of a min.  For 32-bit
// keys the move carries the min's identity (all ones) as its old value, which
// lets the compiler fold it into the min (one DPP min instead of a DPP move
// and a min); the permutation is full, so no lane keeps the old value.
template <int CTRL, typename K> __device__ __forceinline__ K dppk(K v)
{
    if constexpr (__is_same(K, double))
        return __builtin_bit_cast(double, dpp_u64<CTRL>(__builtin_bit_cast(uint64_t, v)));
    else if constexpr (sizeof(K) == 8) return dpp_u64<CTRL>(v);
    else {
        static_assert(CTRL == 0xb1 || CTRL == 0x4e || CTRL == 0x140 || CTRL == 0x141,
                      "a full permutation within each row");
        return (K)(uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, CTRL, 0xf, 0xf, false);
    }
}
template <typename K> __device__ __forceinline__ K readlane_k(K v, int lane)
{
    if constexpr (__is_same(K, double))
        return __builtin_bit_cast(double, readlane_u64(__builtin_bit_cast(uint64_t, v), lane));
    else if constexpr (sizeof(K) == 8) return readlane_u64(v, lane);
    else return (K)(uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}
template <typename K> __device__ __forceinline__ K wave_min_k(K v)
{
    v = kmin(v, dppk<0xb1>(v));
    v = kmin(v, dppk<0x4e>(v));
    v = kmin(v, dppk<0x141>(v));
    v = kmin(v, dppk<0x140>(v));
    return kmin(kmin(readlane_k(v, 0), readlane_k(v, 16)),
                kmin(readlane_k(v, 32), readlane_k(v, 48)));
}
// a u64 time (INF allowed) as a key-width value
template <typename K> __device__ __forceinline__ K to_k(uint64_t v)
{
    return v == E2_INF64 ? KeyT<K>::inf : (K)v;
}
template <typename K> __device__ __forceinline__ uint64_t to_u64(K v)
{
    return v == KeyT<K>::inf ? E2_INF64 : (uint64_t)v;
}

template <typename K>
struct PS {
    K a;  // max(prev(j-1), tau) << 8 | j
    K s;  // (P[j] << 8) - j
};

// Wave-uniform description of a row (scalar registers).
template <typename K>
struct Row {
    const uint64_t *pr;    // prefix sums P[0..N] of the stage device
    const K *p8;           // P << 8 as a key (null for u64 keys, which shift pr)
    const uint8_t *wr;     // smallest stage start per stage end, E2_NO_START if none
    uint64_t hadd;         // head time when this device is the master, else 0
    K hadd8;               // hadd << 8 as a key
    K tau;                 // link from the previous device
    int lo, hi;            // cells of this row
    int kmin;              // devices before this one
    int cap;               // longest stage that fits the device
    int lmin;              // lower bound of window lengths over cells >= lo (0: none)
    const lds_t<K> *prev;  // previous row, band-packed over [plo, phi]; null: first device
    int plo, phi;
};

// Where a row's results go: stored values (+ split points), or, for a
// combine, a running per-lane minimum of (max(value(i), B(i)) << 8 | mu) with
// B(i) = max(tau_next, G(N-2-i)) from the band-packed reversed row G over
// [glo, ghi] (last_only: B = 0 at i = N-1, INF elsewhere).
template <typename K>
struct RowOut {
    lds_t<K> *vals;     // band-packed values, may be null in combine mode
    uint8_t *tbs;       // split points, or null
    bool combine;
    bool last_only;
    const lds_t<K> *G;
    int glo, ghi;
    K tau_next;
    int mu;
};

__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint64_t uni64(uint64_t x)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// a value every lane holds alike, moved to scalar registers
template <typename K> __device__ __forceinline__ K uni_k(K v)
{
    if constexpr (__is_same(K, uint32_t)) return (uint32_t)uni((int)v);
    else if constexpr (__is_same(K, double))
        return __builtin_bit_cast(double, uni64(__builtin_bit_cast(uint64_t, v)));
    else return uni64(v);
}

// *(p + off bytes) with a 32-bit unsigned byte offset from a wave-uniform
// base (the load then adds the offset to the scalar base itself)
template <typename T> __device__ __forceinline__ T at_byte(const T *p, uint32_t off)
{
    return *reinterpret_cast<const T *>(reinterpret_cast<const char *>(p) + off);
}

// Row starts of the per-device tables.  A prefix row block's byte offset
// fits in 32 bits (at most 16 x 256 blocks of 40 x 257 bytes); every part of
// a row comes from the one table base, so that the DP keeps one base live
// instead of a pointer per part.
__device__ __forceinline__ const uint8_t *prow_block(const E2Tables &tb, int r, int c)
{
    return tb.prow + (uint32_t)((r * tb.M + c) * kRowBlock * (tb.N + 1));
}
__device__ __forceinline__ const uint64_t *pref_row(const E2Tables &tb, int r, int c)
{
    return reinterpret_cast<const uint64_t *>(prow_block(tb, r, c));
}
__device__ __forceinline__ const uint64_t *prefR_row(const E2Tables &tb, int r, int c)
{
    return reinterpret_cast<const uint64_t *>(prow_block(tb, r, c) +
                                              (uint32_t)(kRowPrefR * (tb.N + 1)));
}
// P << 8 of the same rows as a key of type K (u32: modulo 2^32; fp64: exact
// for the problems that take fp64 keys)
template <typename K> __device__ __forceinline__ const K *pref8_row(const E2Tables &tb, int r, int c)
{
    constexpr int part = __is_same(K, double) ? kRowPref8d : kRowPref8u;
    return reinterpret_cast<const K *>(prow_block(tb, r, c) + (uint32_t)(part * (tb.N + 1)));
}
template <typename K> __device__ __forceinline__ const K *prefR8_row(const E2Tables &tb, int r, int c)
{
    constexpr int part = __is_same(K, double) ? kRowPrefR8d : kRowPrefR8u;
    return reinterpret_cast<const K *>(prow_block(tb, r, c) + (uint32_t)(part * (tb.N + 1)));
}
template <typename K> __device__ __forceinline__ K shift8(uint64_t v)
{
    if constexpr (__is_same(K, double)) return (double)v * 256.0;
    else return (K)(v << 8);
}
// P[x] << 8 of a row as a key
template <typename K> __device__ __forceinline__ K prefix8(const Row<K> &rw, uint32_t x)
{
    if constexpr (__is_same(K, uint64_t)) return rw.pr[x] << 8;
    else return at_byte(rw.p8, x * (uint32_t)sizeof(K));
}
// the memory-window tables of a view's class (wtab block: win, minwin,
// winR, minwinR)
__device__ __forceinline__ const uint8_t *win_row(const E2Tables &tb, int f, int c)
{
    return tb.wtab + (uint32_t)((f * tb.M + c) * tb.N);
}
__device__ __forceinline__ const uint8_t *winR_row(const E2Tables &tb, int c)
{
    return tb.wtab + (uint32_t)((4 * tb.M + c) * tb.N);
}
__device__ __forceinline__ int minwin_at(const E2Tables &tb, int f, int c, int x)
{
    return tb.wtab[(uint32_t)(((2 + f) * tb.M + c) * tb.N + x)];
}
__device__ __forceinline__ int minwinR_at(const E2Tables &tb, int c, int x)
{
    return tb.wtab[(uint32_t)((5 * tb.M + c) * tb.N + x)];
}
__device__ __forceinline__ uint64_t link_tau(const E2Tables &tb, int r, int a, int b)
{
    return tb.tau[((size_t)r * tb.M + a) * tb.M + b];
}
// same, for wave-uniform device ids (the result goes to scalar registers)
__device__ __forceinline__ uint64_t link_tau_u(const E2Tables &tb, int r, int a, int b)
{
    return uni64(link_tau(tb, r, a, b));
}
template <typename K> __device__ __forceinline__ K pack_prev(K prev, K tau, int j)
{
    if constexpr (__is_same(K, double)) return __builtin_fma(kmax(prev, tau), 256.0, (double)j);
    else return (kmax(prev, tau) << 8) | (K)j;
}
template <typename K> __device__ __forceinline__ K unpack_val(K key)
{
    if constexpr (__is_same(K, double))
        return key >= KeyT<K>::inf_key ? KeyT<K>::inf : __builtin_floor(key * (1.0 / 256.0));
    else return key >= KeyT<K>::inf_key ? KeyT<K>::inf : (key >> 8);
}
// low 8 bits of a finite key (the split point or master position it carries)
template <typename K> __device__ __forceinline__ int key_low8(K key)
{
    if constexpr (__is_same(K, double))
        return (int)(key - __builtin_floor(key * (1.0 / 256.0)) * 256.0);
    else return (int)(key & 0xFF);
}
// (v << 8) | x for a finite or infinite value v and x < 256
template <typename K> __device__ __forceinline__ K pack_low8(K v, int x)
{
    if constexpr (__is_same(K, double)) return __builtin_fma(v, 256.0, (double)x);
    else return (v << 8) | (K)x;
}
template <typename K> __device__ __forceinline__ K cand(const PS<K> &e, K si1)
{
    return kmax(e.a, (K)(si1 - e.s));
}
// v where keep holds, else INF, without a branch (all ones for integer keys,
// the bit pattern of +infinity for doubles)
template <typename K> __device__ __forceinline__ K inf_unless(K v, bool keep)
{
    if constexpr (__is_same(K, double))
        return __builtin_bit_cast(double, keep ? __builtin_bit_cast(uint64_t, v)
                                               : 0x7FF0000000000000ull);
    else return v | ((K)0 - (K)!keep);
}
template <typename K> __device__ __forceinline__ K combine_b(int i, int N, const RowOut<K> &ro)
{
    if (ro.last_only) return (i == N - 1) ? (K)0 : KeyT<K>::inf;
    // the load comes from a clamped index and the INF outside the band is
    // selected on the bit pattern, so that the load is not put under a branch
    const int x = N - 2 - i;
    const K g = ro.G[max(0, min(x - ro.glo, ro.ghi - ro.glo))];
    return kmax(inf_unless(g, x >= ro.glo && x <= ro.ghi), ro.tau_next);
}
template <typename K> __device__ __forceinline__ K combine_key(K v, K b, int mu)
{
    return pack_low8(kmax(v, b), mu);
}

// the entry at LDS byte address addr
template <typename K> __device__ __forceinline__ PS<K> ps_at(int addr)
{
    const lds_t<PS<K>> *p = (const lds_t<PS<K>> *)(uintptr_t)(uint32_t)addr;
    PS<K> e;
    e.a = p->a;
    e.s = p->s;
    return e;
}

template <int S, typename K>
__device__ __forceinline__ K scan_cell(const PS<K> *ps, int i, int jlo, int o, K si1, int t_safe,
                                       int t_all)
{
    K best = KeyT<K>::inf;
    int t = 0;
    const PS<K> *top = ps + (i - o);  // j at step t is top - S t
    for (; t + 4 <= t_safe; t += 4) {
        // all four entries are loaded before any is used (one wait per step)
        const PS<K> *q = top - S * (t + 3);
        const PS<K> e3 = q[3 * S], e2 = q[2 * S], e1 = q[S], e0 = q[0];
        best = kmin(kmin(best, cand(e3, si1)), cand(e2, si1));
        best = kmin(kmin(best, cand(e1, si1)), cand(e0, si1));
    }
    if (t + 2 <= t_safe) {  // a pair that every cell's window still holds
        const PS<K> *q = top - S * (t + 1);
        const PS<K> e1 = q[S], e0 = q[0];
        best = kmin(kmin(best, cand(e1, si1)), cand(e0, si1));
        t += 2;
    }
    // the rest two steps at a time, both entries loaded before use; indices
    // below the cell's window start read its first entry again (an odd last
    // step repeats a candidate, which leaves the minimum unchanged).  The
    // clamp works on LDS byte addresses (signed: the step's address may fall
    // below the array's start before it is clamped).
    const lds_t<PS<K>> *pl = (const lds_t<PS<K>> *)ps;
    const int a_lo = (int)(uint32_t)(uintptr_t)(pl + jlo);
    int a = (int)(uint32_t)(uintptr_t)pl + (i - o - S * t) * (int)sizeof(PS<K>);
    for (; t < t_all; t += 2) {
        const PS<K> e0 = ps_at<K>(max(a, a_lo));
        const PS<K> e1 = ps_at<K>(max(a - S * (int)sizeof(PS<K>), a_lo));
        best = kmin(kmin(best, cand(e0, si1)), cand(e1, si1));
        a -= 2 * S * (int)sizeof(PS<K>);
    }
    if (S >= 2) best = kmin(best, dppk<0xb1>(best));
    if (S >= 4) best = kmin(best, dppk<0x4e>(best));
    if (S >= 8) best = kmin(best, dppk<0x141>(best));  // row_half_mirror: the two quads
    return best;
}

// The previous row's value at block j-1, INF outside its band [plo, phi].
// Entry x = j-1-plo as an unsigned offset: outside [0, span] (x < 0 wraps
// above it) the entry is INF and the read goes to a clamped, in-range slot,
// so that the load is not put under a branch.  An empty previous band moves
// plo to -2 (plo_e), which puts every x above span = 0.
template <typename K>
__device__ __forceinline__ K prev_value(const Row<K> &rw, int j, int plo_e, uint32_t span)
{
    const uint32_t ux = (uint32_t)(j - 1 - plo_e);
    const uint32_t pxc = min(ux, span);
    const bool in = ux <= span;
    if constexpr (__is_same(K, double)) {
        // select on the bit pattern (INF = 0x7FF0000000000000)
        const uint64_t bits = reinterpret_cast<const lds_t<uint64_t> *>(rw.prev)[pxc];
        return __builtin_bit_cast(double, in ? bits : 0x7FF0000000000000ull);
    } else {  // all ones (INF) outside the previous band
        return inf_unless(rw.prev[pxc], in);
    }
}

// The staged pairs of a row for split points j = jmin..hi: a = max(prev(j-1),
// tau) << 8 | j and s = (P[j] << 8) - j, then the barrier before the scans.
template <typename K>
__device__ __forceinline__ void stage_pairs(const Row<K> &rw, PS<K> *ps, int lane, int jmin)
{
    // both loads of an entry go out before either is waited for
    const int pspan = rw.phi - rw.plo;
    const int plo_e = pspan < 0 ? -2 : rw.plo;
    const uint32_t span = pspan < 0 ? 0u : (uint32_t)pspan;
    // a uniform loop: lanes past the row repeat its last entry, writing the
    // same values to the same slot
    for (int j0 = jmin; j0 <= rw.hi; j0 += kWave) {
        const int j = min(j0 + lane, rw.hi);
        const K sj = prefix8(rw, (uint32_t)j);
        const K pv = prev_value(rw, j, plo_e, span);
        ps[j].a = pack_prev(pv, rw.tau, j);
        // (P[j] << 8) - j; fp64: exact, may be negative when blocks take 0 ns;
        // integers: modular, only differences are used
        ps[j].s = sj - (K)j;
    }
    __syncthreads();
}

template <int S, typename K>
__device__ __forceinline__ K row_pass_s(const Row<K> &rw, const RowOut<K> &ro, PS<K> *ps, int lane, int N)
{
    constexpr int CPP = kWave / S;  // cells per pass
    const int o = lane % S;
    const int cl = lane / S;
    const int jmin = max(rw.kmin, rw.lo - rw.cap + 1);
    // first pass's cell loads go out before the split points are built
    // (lanes past the row load its last cell, which they compute again)
    int w_nx;
    K p_nx;  // P[i+1] << 8
    K b_nx = 0;
    {
        const int i = min(rw.lo + cl, rw.hi);
        w_nx = rw.wr[i];
        p_nx = prefix8(rw, (uint32_t)(i + 1));
        if (ro.combine) b_nx = combine_b(i, N, ro);
    }
    stage_pairs(rw, ps, lane, jmin);
    const int L = min(rw.cap, rw.hi - jmin + 1);
    const int Lm = max(0, min(rw.lmin, rw.lo - jmin + 1));
    const int t_all = (L + S - 1) / S;
    const int t_safe = Lm / S;
    const int i_idle = jmin + (Lm > 0 ? Lm - 1 : 0);  // idle lanes: in-range reads
    K acc = KeyT<K>::inf;
    // Lanes past the row's last cell take that cell again: the S lanes of a
    // cell hold the same reduced key, so every lane stores its cell's result
    // (copies write the same value to the same slot) and no store is put
    // under a branch.
    for (int base = rw.lo; base <= rw.hi; base += CPP) {
        const int i = min(base + cl, rw.hi);
        const int w = w_nx;
        const K p1 = p_nx;
        const K b = b_nx;
        if (base + CPP <= rw.hi) {  // a next pass exists (uniform)
            const int in = min(base + CPP + cl, rw.hi);
            w_nx = rw.wr[in];
            p_nx = prefix8(rw, (uint32_t)(in + 1));
            if (ro.combine) b_nx = combine_b(in, N, ro);
        }
        const bool act = w != (int)E2_NO_START;
        const int ie = act ? i : i_idle;
        const int jlo = act ? max(w, jmin) : jmin;
        const K si1 = p1 + rw.hadd8;  // (P[i+1] + head) << 8
        const K best = scan_cell<S>(ps, ie, jlo, o, si1, t_safe, t_all);
        const K v = act ? unpack_val(best) : KeyT<K>::inf;
        if (!ro.combine) {
            ro.vals[i - rw.lo] = v;
            if (ro.tbs) ro.tbs[i - rw.lo] = (uint8_t)key_low8(best);
        } else {
            acc = kmin(acc, combine_key(v, b, ro.mu));
        }
    }
    __syncthreads();
    return acc;
}

// A master's combine (row mu of its table, rc) and the forward row F_mu
// without a master (rf) in one pass, one half-wave each: both rows run on
// device mu over the same band and read the same staged pairs of F_{mu-1}
// (the combine adds the head time and keeps the head-bytes window, whose
// stages are the shorter, so the forward row's staging range covers it).
// Rows of at most 32 cells (one pass per half, S2 lanes per cell).  Lanes
// 0-31 return the combine's keys as row_pass does (INF in lanes 32-63);
// lanes 32-63 leave their cell's value, split point and index in fv, fb and
// fi, which the caller stores once it knows that the sweep goes on (F_mu
// replaces F_{mu-1} in place).
template <int S2, typename K>
__device__ __forceinline__ K row_pass_pair_s(const Row<K> &rc, const Row<K> &rf,
                                             const RowOut<K> &ro, PS<K> *ps, int lane, int N,
                                             K &fv, int &fb, int &fi)
{
    const bool fwd = lane >= kWave / 2;
    const int l = lane % (kWave / 2);
    const int o = l % S2;
    const int cl = l / S2;
    const int jmin = max(rf.kmin, rf.lo - rf.cap + 1);
    // the cell loads go out before the pairs are staged
    const int i = min(rf.lo + cl, rf.hi);
    const int w = (fwd ? rf.wr : rc.wr)[i];
    const K p1 = prefix8(rf, (uint32_t)(i + 1));
    const K b = combine_b(i, N, ro);
    stage_pairs(rf, ps, lane, jmin);
    // uniform scan bounds: the longer stages' range, the shorter windows' bound
    const int L = min(rf.cap, rf.hi - jmin + 1);
    const int Lm = max(0, min(min(rf.lmin, rc.lmin), rf.lo - jmin + 1));
    const int t_all = (L + S2 - 1) / S2;
    const int t_safe = Lm / S2;
    const int i_idle = jmin + (Lm > 0 ? Lm - 1 : 0);
    const bool act = w != (int)E2_NO_START;
    const int ie = act ? i : i_idle;
    const int jlo = act ? max(w, jmin) : jmin;
    const K si1 = p1 + (fwd ? rf.hadd8 : rc.hadd8);
    const K best = scan_cell<S2>(ps, ie, jlo, o, si1, t_safe, t_all);
    const K v = act ? unpack_val(best) : KeyT<K>::inf;
    fv = v;
    fb = key_low8(best);
    fi = i - rf.lo;
    return fwd ? KeyT<K>::inf : combine_key(v, b, ro.mu);
}

template <typename K>
__device__ __forceinline__ K row_pass_pair(const Row<K> &rc, const Row<K> &rf, const RowOut<K> &ro,
                                           PS<K> *ps, int lane, int N, K &fv, int &fb, int &fi)
{
    const int n = rf.hi - rf.lo + 1;
    if (n <= 8) return row_pass_pair_s<4>(rc, rf, ro, ps, lane, N, fv, fb, fi);
    if (n <= 16) return row_pass_pair_s<2>(rc, rf, ro, ps, lane, N, fv, fb, fi);
    return row_pass_pair_s<1>(rc, rf, ro, ps, lane, N, fv, fb, fi);
}

// Cell N-1 of a row (lo = hi = N-1) without staging: one lane per split point
// j of its window, each candidate formed from the previous row and the prefix
// sums directly, then one wave minimum.  The same candidates and tie rule as
// row_pass on a one-cell row; returns the packed key (value << 8 | j), INF
// when no stage ending at block N-1 fits the device.
template <typename K>
__device__ __forceinline__ K single_cell_key(const Row<K> &rw, int lane, int N)
{
    const int i = N - 1;
    const int w = rw.wr[i];
    K best = KeyT<K>::inf;
    if (w != (int)E2_NO_START) {
        const int jlo = max(w, max(rw.kmin, rw.lo - rw.cap + 1));
        const K si1 = prefix8(rw, (uint32_t)(i + 1)) + rw.hadd8;
        const int pspan = rw.phi - rw.plo;
        const int plo_e = pspan < 0 ? -2 : rw.plo;
        const uint32_t span = pspan < 0 ? 0u : (uint32_t)pspan;
        for (int j0 = jlo; j0 <= i; j0 += kWave) {
            const int j = min(j0 + lane, i);  // lanes past the window repeat j = i
            PS<K> e;
            e.a = pack_prev(prev_value(rw, j, plo_e, span), rw.tau, j);
            e.s = prefix8(rw, (uint32_t)j) - (K)j;
            best = kmin(best, cand(e, si1));
        }
    }
    return wave_min_k(best);
}

// Store mode returns INF; combine mode returns the lane's running minimum of
// (max(value, B) << 8 | mu) (the caller reduces over the wave once).
template <typename K>
__device__ __forceinline__ K row_pass(const Row<K> &rw, const RowOut<K> &ro, PS<K> *ps, int lane, int N)
{
    if (rw.prev == nullptr) {  // first device: Eq. 2, no split point
        K acc = KeyT<K>::inf;
        for (int i0 = rw.lo; i0 <= rw.hi; i0 += kWave) {
            const int i = min(i0 + lane, rw.hi);  // copies of the last cell past the row
            const K v = inf_unless((K)(rw.pr[i + 1] + rw.hadd), rw.wr[i] == 0);
            if (!ro.combine) {
                ro.vals[i - rw.lo] = v;
            } else {
                acc = kmin(acc, combine_key(v, combine_b(i, N, ro), ro.mu));
            }
        }
        __syncthreads();
        return acc;
    }
    const int n = rw.hi - rw.lo + 1;
    if (n <= 0) {
        __syncthreads();
        return KeyT<K>::inf;
    }
    if (n <= 8) return row_pass_s<8>(rw, ro, ps, lane, N);
    if (n <= 16) return row_pass_s<4>(rw, ro, ps, lane, N);
    if (n <= 32) return row_pass_s<2>(rw, ro, ps, lane, N);
    return row_pass_s<1>(rw, ro, ps, lane, N);
}

template <typename K>
__device__ __forceinline__ RowOut<K> store_to(lds_t<K> *vals, uint8_t *tbs)
{
    RowOut<K> ro;
    ro.vals = vals;
    ro.tbs = tbs;
    ro.combine = false;
    ro.last_only = false;
    ro.G = nullptr;
    ro.glo = 1;
    ro.ghi = 0;
    ro.tau_next = 0;
    ro.mu = 0;
    return ro;
}

// ---------------------------------------------------------------------------
// Band-pruned decomposition of the master enumeration.
//
// With cap0[k] the longest stage device k holds without the head and
// pre[k] = cap0[1] + ... + cap0[k], a cell (i, k) can lie on a complete
// memory-feasible partition only if
//     max(k-1, N-1-(pre[m]-pre[k])) <= i <= min(N-1-(m-k), pre[k]-1).
// Every memory-feasible candidate of an in-band cell reads an in-band cell
// of the previous row or an infinite one, so computing only in-band cells
// (others INF) leaves every in-band value and split point exact.
//
//   F_k  forward rows without master, k = 1..m-1 (values kept for the
//        chosen master's first row, split points in LDS)
//   G_k  backward rows without master: blocks j..N-1 on devices k..m with
//        links k..m, computed as forward rows over reversed blocks
//   T_mu = min_i max( min_j max(F_{mu-1}(j-1), tau(mu-1, mu), cost_mu(j, i)
//                    + head_mu), tau(mu, mu+1), G_{mu+1}(i+1) )
//        (mu = 1: the stage starts at block 0; mu = m: it ends at N-1)
//   which is the optimum of the table of Algorithm 1 for master mu.  The
//   minimum of (T_mu << 8 | mu) gives the best T and the smallest master
//   attaining it; rows mu*..m of its table (rows below mu* are F) give the
//   split points for the back tracing.
//
// Schedule: all G rows first (kept in the wave's LDS backward-row pool), then the
// optimum T0 without any master (the full reversed table's last cell), then
// masters in ascending position, each combine followed by the forward row
// the next one reads.  Head time and head bytes only ever add, so
// T_mu >= T0 for every mu; the sweep stops at the first mu with
// min(T_1..T_mu) = T0, which is then the best T and the smallest master
// attaining it, and skips the forward rows and combines beyond it.
//
// The per-position data of a chain (device, capacities, links, head time,
// bands, pool offsets, window-length bounds) is loaded once, one position
// per lane (m <= 64; four per lane in the long-chain kernel), and each row
// reads its scalars with readlane.  Every row lives in LDS: forward rows in
// place in one buffer, backward rows in a pool (dp_banded).
// ---------------------------------------------------------------------------
// split-point bytes kept in LDS per wave; larger tables (the bands of long
// chains with roomy devices, or the reference path's full rows) go to the
// wave's region of the global split-point table
constexpr int kLdsTbCells = 2048;
// Dynamic LDS of k_dp: split-point pairs (16 N bytes), a row buffer, the
// backward-row pool's fixed part (a row) and the extra bytes below, a second
// row buffer and the split-point bytes.  The extra bytes lengthen the pool up
// to 6656 bytes in all; at 7424 the kernel measured a quarter slower (fewer
// resident waves).
constexpr int kDpLdsTarget = 6656;
__host__ __device__ constexpr int dp_lds_fixed(int N) { return 16 * N + 16 * (N + 1) + kLdsTbCells; }
__host__ __device__ constexpr int dp_lds_extra(int N)
{
    return dp_lds_fixed(N) < kDpLdsTarget ? ((kDpLdsTarget - dp_lds_fixed(N)) & ~7) : 0;
}

__device__ __forceinline__ int f8(uint32_t w, int sh) { return (int)((w >> sh) & 0xFFu); }

__device__ __forceinline__ int lane_i(int v, int k) { return __builtin_amdgcn_readlane(v, k); }
__device__ __forceinline__ uint32_t lane_w(uint32_t v, int k)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, k);
}
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int k) { return readlane_u64(v, k); }

// Per-position table of a chain: lane k-1 holds chain position k (1-based)
// as five packed words (fields < 256 except the pool offsets) and two u64
// times; a row reads its words with one readlane each and unpacks them in
// scalar registers.  Reversed row t's link (position m+1-t to m+2-t) is the
// forward link held by lane m+1-t.  The accessors take 0-based positions.
struct ChainRegs {
    uint32_t wa;    // dev | cap0 << 8 | capH << 16 | lmin0 << 24      (forward row k)
    uint32_t wb;    // flo | fhi << 8 | lmin1 << 16                    (forward row k)
    uint32_t wc;    // pool offset of row k | lminR << 16 | capR << 24 (reversed row t = k)
    uint32_t wd;    // devR | glo << 8 | ghi << 16                     (reversed row t = k)
    uint32_t we;    // offset of reversed row t = k in the backward-row pool
    uint64_t tau;   // link from position k-1 (k >= 2)
    uint64_t head;  // head time of the device
    int m;          // chain length (uniform)
    __device__ __forceinline__ uint32_t A(int k0) const { return lane_w(wa, k0); }
    __device__ __forceinline__ uint32_t B(int k0) const { return lane_w(wb, k0); }
    __device__ __forceinline__ uint32_t C(int k0) const { return lane_w(wc, k0); }
    __device__ __forceinline__ uint32_t D(int k0) const { return lane_w(wd, k0); }
    __device__ __forceinline__ uint32_t E(int k0) const { return lane_w(we, k0); }
    __device__ __forceinline__ uint64_t TAU(int k0) const { return lane_u64(tau, k0); }
    __device__ __forceinline__ uint64_t HEAD(int k0) const { return lane_u64(head, k0); }
};
// cap0 / capH are the longest stages without / with the head, [flo, fhi]
// the forward band, lmin0 / lmin1 its window-length bounds; reversed row
// t = k runs on device devR (position m+1-k) with cap0 capR over the band
// [glo, ghi] with window-length bound lminR.

// The same table for chains of up to kLongSets x 64 devices: position k0
// (0-based) sits in set k0 / 64 at lane k0 % 64.  Positions are uniform, so
// an accessor reads one lane of each set and keeps the one its set names.
constexpr int kLongSets = 4;
struct ChainRegsLong {
    ChainRegs s[kLongSets];  // the m field of each set is unused
    int m;
    template <typename F>
    __device__ __forceinline__ uint32_t pick(int k0, F f) const
    {
        const int set = k0 >> 6, l = k0 & 63;
        uint32_t v = lane_w(f(s[0]), l);
#pragma unroll
        for (int i = 1; i < kLongSets; ++i)
            if (set == i) v = lane_w(f(s[i]), l);
        return v;
    }
    template <typename F>
    __device__ __forceinline__ uint64_t pick64(int k0, F f) const
    {
        const int set = k0 >> 6, l = k0 & 63;
        uint64_t v = lane_u64(f(s[0]), l);
#pragma unroll
        for (int i = 1; i < kLongSets; ++i)
            if (set == i) v = lane_u64(f(s[i]), l);
        return v;
    }
    __device__ __forceinline__ uint32_t A(int k0) const { return pick(k0, [](const ChainRegs &c) { return c.wa; }); }
    __device__ __forceinline__ uint32_t B(int k0) const { return pick(k0, [](const ChainRegs &c) { return c.wb; }); }
    __device__ __forceinline__ uint32_t C(int k0) const { return pick(k0, [](const ChainRegs &c) { return c.wc; }); }
    __device__ __forceinline__ uint32_t D(int k0) const { return pick(k0, [](const ChainRegs &c) { return c.wd; }); }
    __device__ __forceinline__ uint32_t E(int k0) const { return pick(k0, [](const ChainRegs &c) { return c.we; }); }
    __device__ __forceinline__ uint64_t TAU(int k0) const { return pick64(k0, [](const ChainRegs &c) { return c.tau; }); }
    __device__ __forceinline__ uint64_t HEAD(int k0) const { return pick64(k0, [](const ChainRegs &c) { return c.head; }); }
};

// band of forward row k and its pool offset
template <class CR> __device__ __forceinline__ int band_lo(const CR &cr, int k) { return f8(cr.B(k - 1), 0); }
template <class CR> __device__ __forceinline__ int band_hi(const CR &cr, int k) { return f8(cr.B(k - 1), 8); }
template <class CR> __device__ __forceinline__ int pool_off(const CR &cr, int k)
{
    return (int)(cr.C(k - 1) & 0xFFFFu);
}
// band of reversed row t and its offset in the backward-row pool
template <class CR> __device__ __forceinline__ int rband_lo(const CR &cr, int t) { return f8(cr.D(t - 1), 8); }
template <class CR> __device__ __forceinline__ int rband_hi(const CR &cr, int t) { return f8(cr.D(t - 1), 16); }
template <class CR> __device__ __forceinline__ int gpool_off(const CR &cr, int t) { return (int)cr.E(t - 1); }

// Inclusive prefix sum over the wave with DPP moves only (no LDS round
// trips): prefixes of 4 lanes within each 16-lane row from the inputs, then
// of 8 and 16 lanes (row shifts by 4 and 8 on the upper banks), then the
// totals of rows 0 and 2 into rows 1 and 3 (broadcast of lane 15) and of
// rows 0-1 into rows 2 and 3 (broadcast of lane 31).  Disabled lanes and
// shifts across a row start contribute 0.
__device__ __forceinline__ int scan_incl_i32(int x, int lane)
{
    (void)lane;
    int s = x;
    s += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);  // row_shr:1
    s += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);  // row_shr:2
    s += __builtin_amdgcn_update_dpp(0, x, 0x113, 0xf, 0xf, true);  // row_shr:3
    s += __builtin_amdgcn_update_dpp(0, s, 0x114, 0xf, 0xe, true);  // row_shr:4, lanes 4-15
    s += __builtin_amdgcn_update_dpp(0, s, 0x118, 0xf, 0xc, true);  // row_shr:8, lanes 8-15
    s += __builtin_amdgcn_update_dpp(0, s, 0x142, 0xa, 0xf, false); // row_bcast:15, rows 1, 3
    s += __builtin_amdgcn_update_dpp(0, s, 0x143, 0xc, 0xf, false); // row_bcast:31, rows 2, 3
    return s;
}

struct DpSmem {
    void *ps;        // split-point pairs, N entries (LDS)
    lds_t<uint64_t> *Rw0;  // LDS row ping-pong, N+1 entries each
    lds_t<uint64_t> *Rw1;
    uint8_t *tbp;    // split points of the forward rows, band-packed (LDS)
    lds_t<char> *pool_end; // end of the backward-row pool (k_dp)
    int pool_cells;
};

// Row k (1-based) of the table for master mu (mu = 0: no master) as a
// forward row; prev / plo / phi are filled in by the caller.
template <typename K, class CR>
__device__ __forceinline__ Row<K> fwd_row_of(const E2Tables &tb, const CR &cr, int r, int k,
                                             int mu)
{
    const int f = (mu == k);
    const uint32_t wa = cr.A(k - 1), wb = cr.B(k - 1);
    const int c = f8(wa, 0);
    Row<K> rw;
    rw.pr = pref_row(tb, r, c);
    rw.p8 = pref8_row<K>(tb, r, c);
    rw.wr = win_row(tb, f, c);
    rw.hadd = f ? cr.HEAD(k - 1) : 0;
    rw.hadd8 = shift8<K>(rw.hadd);
    rw.tau = (k >= 2) ? to_k<K>(cr.TAU(k - 1)) : (K)0;
    rw.lo = f8(wb, 0);
    rw.hi = f8(wb, 8);
    rw.kmin = k - 1;
    rw.cap = f ? f8(wa, 16) : f8(wa, 8);
    rw.lmin = f ? f8(wb, 16) : f8(wa, 24);
    rw.prev = nullptr;
    rw.plo = 1;
    rw.phi = 0;
    return rw;
}

template <typename K>
__device__ __forceinline__ void set_prev(Row<K> &rw, const lds_t<K> *prev, int plo, int phi)
{
    rw.prev = prev;
    rw.plo = plo;
    rw.phi = phi;
}

// Reversed row t (1-based): the device at chain position m+1-t over the
// blocks in reverse order (block N-1 first), without a master; prev / plo /
// phi are filled in by the caller.  For t = m the caller also sets the cell
// range (the band fields of position 1 are not packed).
template <typename K, class CR>
__device__ __forceinline__ Row<K> rev_row_of(const E2Tables &tb, const CR &cr, int r, int t)
{
    const uint32_t wc = cr.C(t - 1), wd = cr.D(t - 1);
    const int c = f8(wd, 0);
    Row<K> g;
    g.pr = prefR_row(tb, r, c);
    g.p8 = prefR8_row<K>(tb, r, c);
    g.wr = winR_row(tb, c);
    g.hadd = 0;
    g.hadd8 = 0;
    g.tau = (t >= 2) ? to_k<K>(cr.TAU(cr.m + 1 - t)) : (K)0;  // link m+1-t -> m+2-t
    g.lo = f8(wd, 8);
    g.hi = f8(wd, 16);
    g.kmin = t - 1;
    g.cap = f8(wc, 24);
    g.lmin = f8(wc, 16);
    g.prev = nullptr;
    g.plo = 1;
    g.phi = 0;
    return g;
}

// every lane's v is at most lim (the answer is wave-uniform)
__device__ __forceinline__ bool wave_all_le(uint64_t v, uint64_t lim)
{
    return __ballot(v > lim) == 0;
}

// Per-position table of a chain and the largest finite value its DP can
// produce, as this lane's share (the bound is the maximum over the lanes:
// callers compare it with wave_all_le); false when the banded path cannot
// take the chain.
__device__ __forceinline__ bool chain_regs(const E2Tables &tb, const DpSmem &sm, int r,
                                           const uint8_t *chain, int m, int lane, ChainRegs &cr,
                                           uint64_t *bound, uint64_t *bound_tot, int *pool_cells)
{
    const int N = tb.N, M = tb.M;
    if (m > kMaxBandedChain) return false;
    const bool valid = lane < m;
    const int k1 = lane + 1;
    const int dev = valid ? chain[lane] : 0;
    const int cap0 = valid ? tb.cap0[dev] : 0;
    const int capH = valid ? tb.capH[dev] : 0;
    cr.head = valid ? tb.head[r * M + dev] : 0;
    cr.tau = (valid && lane >= 1) ? link_tau(tb, r, chain[lane - 1], dev) : 0;
    const uint64_t tf = cr.tau != E2_INF64 ? cr.tau : 0;
    *bound = umax64(valid ? tb.vmax[r * M + dev] : 0, tf);
    *bound_tot = umax64(valid ? tb.vtot[r * M + dev] : 0, tf);
    const int pre = scan_incl_i32(cap0, lane);
    const int tot = lane_i(pre, m - 1);
    int lo = max(k1 - 1, N - 1 - (tot - pre));
    int hi = min(N - 1 - (m - k1), pre - 1);
    if (hi < lo) { lo = 1; hi = 0; }
    const int size = (valid && k1 < m) ? hi - lo + 1 : 0;
    const int size_incl = scan_incl_i32(size, lane);
    const int off = size_incl - size;
    const int pool_need = lane_i(size_incl, kWave - 1);
    const int lmin0 = (valid && lo <= hi) ? minwin_at(tb, 0, dev, lo) : 0;
    const int lmin1 = (valid && lo <= hi) ? minwin_at(tb, 1, dev, lo) : 0;
    // reversed row t = k1 covers original position kk = m+1-t: blocks j..N-1
    // with max(kk-1, N-(tot-pre[kk-1])) <= j <= min(N-(m-kk+1), pre[kk-1]),
    // i.e. reversed cells x = N-1-j
    const int kk = m + 1 - k1;
    const int src = max(0, min(kWave - 1, kk - 1));
    const int devR = __shfl(dev, src, kWave);
    const int capR = __shfl(cap0, src, kWave);
    const int pre_km1 = (kk >= 2) ? __shfl(pre, max(0, kk - 2), kWave) : 0;
    cr.m = m;
    int glo = 1, ghi = 0, lminR = 0;
    {
        const bool vr = k1 < m;
        const int gl = max(kk - 1, N - (tot - pre_km1));
        const int gh = min(pre_km1, N - (m - kk + 1));
        if (vr && gh >= gl) {
            glo = N - 1 - gh;
            ghi = N - 1 - gl;
            lminR = minwinR_at(tb, devR, glo);
        }
    }
    cr.wa = (uint32_t)dev | (uint32_t)cap0 << 8 | (uint32_t)capH << 16 | (uint32_t)lmin0 << 24;
    cr.wb = (uint32_t)lo | (uint32_t)hi << 8 | (uint32_t)lmin1 << 16;
    cr.wc = ((uint32_t)off & 0xFFFFu) | (uint32_t)lminR << 16 | (uint32_t)capR << 24;
    cr.wd = (uint32_t)devR | (uint32_t)glo << 8 | (uint32_t)ghi << 16;
    // backward-row pool: reversed rows t = 1..m-1 band-packed in order (their
    // bands are the forward bands of positions m-1..1 moved by one block, so
    // they hold as many cells as the forward bands)
    const int gsize = ghi >= glo ? ghi - glo + 1 : 0;
    const int g_incl = scan_incl_i32(gsize, lane);
    cr.we = (uint32_t)(g_incl - gsize);
    const int gpool_need = lane_i(g_incl, kWave - 1);
    *pool_cells = pool_need;
    return pool_need <= sm.pool_cells && gpool_need <= sm.pool_cells;
}

// The per-position table of a chain of up to kLongSets x 64 devices (as
// chain_regs, position k0 = 64 i + lane in set i), with the prefix sums
// carried from set to set.  The banded path takes every such chain: its
// rows live in LDS, and split points beyond the LDS copy go to the wave's
// global table.
__device__ __forceinline__ void chain_regs_long(const E2Tables &tb, int r, const uint8_t *chain,
                                                int m, int lane, ChainRegsLong &cr,
                                                uint64_t *bound, uint64_t *bound_tot,
                                                int *pool_cells)
{
    const int N = tb.N, M = tb.M;
    cr.m = m;
    int dev[kLongSets], cap0[kLongSets], pre[kLongSets];
    uint64_t vb = 0, vt = 0;
    int carry = 0;
#pragma unroll
    for (int i = 0; i < kLongSets; ++i) {
        const int k0 = 64 * i + lane;
        const bool valid = k0 < m;
        dev[i] = valid ? chain[k0] : 0;
        cap0[i] = valid ? tb.cap0[dev[i]] : 0;
        ChainRegs &c = cr.s[i];
        c.m = m;
        c.head = valid ? tb.head[r * M + dev[i]] : 0;
        c.tau = (valid && k0 >= 1) ? link_tau(tb, r, chain[k0 - 1], dev[i]) : 0;
        const uint64_t tf = c.tau != E2_INF64 ? c.tau : 0;
        vb = umax64(vb, umax64(valid ? tb.vmax[r * M + dev[i]] : 0, tf));
        vt = umax64(vt, umax64(valid ? tb.vtot[r * M + dev[i]] : 0, tf));
        pre[i] = scan_incl_i32(cap0[i], lane) + carry;
        carry = lane_i(pre[i], kWave - 1);
    }
    *bound = vb;  // this lane's share, as in chain_regs
    *bound_tot = vt;
    auto at = [&](const int (&v)[kLongSets], int k0) {  // value of position k0, per lane
        const int l = k0 & 63, set = k0 >> 6;
        int x = 0;
#pragma unroll
        for (int i = 0; i < kLongSets; ++i) {
            const int y = __shfl(v[i], l, kWave);
            if (set == i) x = y;
        }
        return x;
    };
    int tot = 0;  // pre at the last position (a uniform set, selected without indexing)
#pragma unroll
    for (int i = 0; i < kLongSets; ++i) {
        const int v = lane_i(pre[i], (m - 1) & 63);
        if (((m - 1) >> 6) == i) tot = v;
    }
    int size_carry = 0, g_carry = 0;
#pragma unroll
    for (int i = 0; i < kLongSets; ++i) {
        ChainRegs &c = cr.s[i];
        const int k1 = 64 * i + lane + 1;
        const bool valid = k1 <= m;
        const int d = dev[i];
        const int capH = valid ? tb.capH[d] : 0;
        int lo = max(k1 - 1, N - 1 - (tot - pre[i]));
        int hi = min(N - 1 - (m - k1), pre[i] - 1);
        if (hi < lo) { lo = 1; hi = 0; }
        const int size = (valid && k1 < m) ? hi - lo + 1 : 0;
        const int size_incl = scan_incl_i32(size, lane) + size_carry;
        size_carry = lane_i(size_incl, kWave - 1);
        const int off = size_incl - size;
        const int lmin0 = (valid && lo <= hi) ? minwin_at(tb, 0, d, lo) : 0;
        const int lmin1 = (valid && lo <= hi) ? minwin_at(tb, 1, d, lo) : 0;
        // reversed row t = k1 covers original position kk = m+1-t
        const int kk = m + 1 - k1;
        const int src = max(0, min(kLongSets * 64 - 1, kk - 1));
        const int devR = at(dev, src);
        const int capR = at(cap0, src);
        const int pre_km1 = (kk >= 2) ? at(pre, max(0, kk - 2)) : 0;
        int glo = 1, ghi = 0, lminR = 0;
        {
            const bool vr = k1 < m;
            const int gl = max(kk - 1, N - (tot - pre_km1));
            const int gh = min(pre_km1, N - (m - kk + 1));
            if (vr && gh >= gl) {
                glo = N - 1 - gh;
                ghi = N - 1 - gl;
                lminR = minwinR_at(tb, devR, glo);
            }
        }
        c.wa = (uint32_t)d | (uint32_t)cap0[i] << 8 | (uint32_t)capH << 16 | (uint32_t)lmin0 << 24;
        c.wb = (uint32_t)lo | (uint32_t)hi << 8 | (uint32_t)lmin1 << 16;
        c.wc = ((uint32_t)off & 0xFFFFu) | (uint32_t)lminR << 16 | (uint32_t)capR << 24;
        c.wd = (uint32_t)devR | (uint32_t)glo << 8 | (uint32_t)ghi << 16;
        const int gsize = ghi >= glo ? ghi - glo + 1 : 0;
        const int g_incl = scan_incl_i32(gsize, lane) + g_carry;
        g_carry = lane_i(g_incl, kWave - 1);
        c.we = (uint32_t)(g_incl - gsize);
    }
    *pool_cells = size_carry;
}

// First backward row of the longest run of rows ending at row t_end that
// fits a backward-row pool of cap cells (rows band-packed in order).  Lane
// t-1 holds the pool offset of row t, so the cells of rows t..t_end are
// end(t_end) - offset(t), which falls as t grows.
__device__ __forceinline__ int g_window_lo(const ChainRegs &cr, int lane, int t_end, int cap)
{
    const int end = gpool_off(cr, t_end) + (rband_hi(cr, t_end) - rband_lo(cr, t_end) + 1);
    const bool fits = lane + 1 <= t_end && end - (int)cr.we <= cap;
    const uint64_t b = __ballot(fits);
    return b ? __builtin_ctzll(b) + 1 : t_end;
}
__device__ __forceinline__ int g_window_lo(const ChainRegsLong &cr, int lane, int t_end, int cap)
{
    const int end = gpool_off(cr, t_end) + (rband_hi(cr, t_end) - rband_lo(cr, t_end) + 1);
    int first = t_end;
#pragma unroll
    for (int i = kLongSets - 1; i >= 0; --i) {  // the lowest set with a fitting row wins
        const int t = 64 * i + lane + 1;
        const uint64_t b = __ballot(t <= t_end && end - (int)cr.s[i].we <= cap);
        if (b) first = 64 * i + __builtin_ctzll(b) + 1;
    }
    return first;
}

// Backward rows 1..t_end into the backward-row pool: rows from t_lo on at
// their band-packed offsets less that of t_lo, the rows before t_lo in place
// at the pool's start (a row reads its previous row completely before it
// writes: every row pass has a barrier between the two).
template <typename K, class CR>
__device__ __forceinline__ void g_rows(const E2Tables &tb, const CR &cr, int r, int t_end,
                                       int t_lo, lds_t<K> *gp, PS<K> *ps, int lane, int N)
{
    const int base = gpool_off(cr, t_lo);
    for (int t = 1; t <= t_end; ++t) {
        Row<K> g = rev_row_of<K>(tb, cr, r, t);
        if (t >= 2)
            set_prev(g, gp + (t - 1 >= t_lo ? gpool_off(cr, t - 1) - base : 0),
                     rband_lo(cr, t - 1), rband_hi(cr, t - 1));
        row_pass(g, store_to<K>(gp + (t >= t_lo ? gpool_off(cr, t) - base : 0), nullptr), ps,
                 lane, N);
    }
}

// The banded DP of one chain with keys of width K.  Returns the optimum as
// a u64 (INF if none) and its master position in *mu_out (0 if none); the
// stage starts go to start[].
//
// Every row lives in LDS.  Forward rows are computed in place in one row
// buffer.  Backward rows go to a pool (the LDS after the split-point pairs
// of this key width); the sweep reads them back in the reverse order, so
// the pool keeps the last rows that fit, and a combine whose backward row
// was not kept computes rows 1.. again, keeping the run that ends at the
// row it needs.  When the sweep runs through every master and the chosen
// one's previous forward row is no longer in the buffer, the forward rows
// up to it are computed again.
template <typename K, class CR>
__device__ __forceinline__ void dp_banded(const E2Tables &tb, const DpSmem &sm, const CR &cr, int r, int m,
                          int lane, uint64_t *T_out, int *mu_out, uint8_t *start, uint8_t *last_tb)
{
    const int N = tb.N;
    PS<K> *ps = static_cast<PS<K> *>(sm.ps);
    lds_t<K> *F = reinterpret_cast<lds_t<K> *>(sm.Rw0);  // forward rows, in place
    lds_t<char> *pool_c = (lds_t<char> *)sm.ps + (uint32_t)N * sizeof(PS<K>);
    lds_t<K> *gp = (lds_t<K> *)pool_c;
    const int gcap = (int)((sm.pool_end - pool_c) / (int)sizeof(K));
    // ---- backward rows G_1..G_{m-1}, the last ones that fit kept in the pool
    int g_lo = m >= 2 ? g_window_lo(cr, lane, m - 1, gcap) : 1;  // first kept row
    if (m >= 2) g_rows<K>(tb, cr, r, m - 1, g_lo, gp, ps, lane, N);
    // ---- the optimum without a master (no head time or bytes anywhere):
    // reversed row m at its last cell.  Every master's optimum is at least
    // this, and none exists when it is infinite.
    K tn = KeyT<K>::inf;
    if (m >= 2) {
        Row<K> g = rev_row_of<K>(tb, cr, r, m);
        set_prev(g, gp + (gpool_off(cr, m - 1) - gpool_off(cr, g_lo)), rband_lo(cr, m - 1),
                 rband_hi(cr, m - 1));
        g.lo = g.hi = N - 1;
        tn = unpack_val(single_cell_key(g, lane, N));
        if (tn == KeyT<K>::inf) {
            *T_out = E2_INF64;
            *mu_out = 0;
            return;
        }
    }

    // ---- masters in ascending position, each followed by the forward row
    // it leaves for the next (F_mu, in place, split points to tbp).  The
    // sweep stops at the first master whose optimum equals the optimum
    // without a master: no later master can do better (a head only adds time
    // and bytes), and ties go to the smaller master.
    K acc = KeyT<K>::inf;
    K key = KeyT<K>::inf;
    int f_last = 0;  // the forward row the buffer holds
    bool kept = false;  // the buffer holds row mu* of the chosen master's table
    for (int mu = 1; mu <= m; ++mu) {
        Row<K> rw = fwd_row_of<K>(tb, cr, r, mu, mu);
        if (rw.cap > 0) {
            if (mu >= 2) set_prev(rw, F, band_lo(cr, mu - 1), band_hi(cr, mu - 1));
            RowOut<K> ro = store_to<K>(nullptr, nullptr);
            ro.combine = true;
            ro.mu = mu;
            if (mu == m) {
                ro.last_only = true;  // the master's stage ends at block N-1
            } else {
                const int t = m - mu;  // backward row of devices mu+1..m
                if (t < g_lo) {        // not kept: rows 1..t again
                    g_lo = g_window_lo(cr, lane, t, gcap);
                    g_rows<K>(tb, cr, r, t, g_lo, gp, ps, lane, N);
                }
                ro.G = gp + (gpool_off(cr, t) - gpool_off(cr, g_lo));
                ro.glo = rband_lo(cr, t);
                ro.ghi = rband_hi(cr, t);
                ro.tau_next = to_k<K>(cr.TAU(mu));  // link mu -> mu+1
            }
            // with a previous row and a band of at most 32 cells, F_mu rides
            // along in the other half-wave and is stored only if the sweep
            // goes on
            const int n = rw.hi - rw.lo + 1;
            if (mu >= 2 && mu < m && n >= 1 && n <= kWave / 2) {
                Row<K> f = fwd_row_of<K>(tb, cr, r, mu, 0);
                set_prev(f, F, band_lo(cr, mu - 1), band_hi(cr, mu - 1));
                K fv;
                int fb, fi;
                acc = kmin(acc, row_pass_pair(rw, f, ro, ps, lane, N, fv, fb, fi));
                key = wave_min_k(acc);
                if (unpack_val(key) == tn) {
                    // mu is the chosen master (the first to reach T0), and the
                    // combine half holds row mu of its table: keep that row,
                    // values over F_{mu-1}, split points in tbp
                    if (lane < kWave / 2) {
                        F[fi] = fv;
                        sm.tbp[pool_off(cr, mu) + fi] = (uint8_t)fb;
                    }
                    __syncthreads();
                    kept = true;
                    break;
                }
                if (lane >= kWave / 2) {  // the S2 lanes of a cell store the same
                    F[fi] = fv;
                    sm.tbp[pool_off(cr, mu) + fi] = (uint8_t)fb;
                }
                __syncthreads();
                f_last = mu;
                continue;
            }
            acc = kmin(acc, row_pass(rw, ro, ps, lane, N));
            key = wave_min_k(acc);
            if (m >= 2 && unpack_val(key) == tn) break;
        }
        if (mu < m) {
            Row<K> f = fwd_row_of<K>(tb, cr, r, mu, 0);
            if (mu >= 2) set_prev(f, F, band_lo(cr, mu - 1), band_hi(cr, mu - 1));
            row_pass(f, store_to<K>(F, sm.tbp + pool_off(cr, mu)), ps, lane, N);
            f_last = mu;
        }
    }
    const K bestk = unpack_val(key);
    const int best_mu = bestk == KeyT<K>::inf ? 0 : key_low8(key);
    *T_out = to_u64(bestk);
    *mu_out = best_mu;
    if (bestk == KeyT<K>::inf) return;

    // ---- rows mu*..m-1 of the chosen master's table (split points overwrite
    // those of F), then cell N-1 of row m.  Their first row reads F_{mu*-1},
    // which the buffer holds unless the sweep went past it: then F_1..F_{mu*-1}
    // are computed again (their split points are in tbp already).  A sweep
    // that stopped in a paired pass has left row mu* itself in the buffer.
    if (!kept && best_mu >= 2 && f_last != best_mu - 1) {
        for (int k = 1; k < best_mu; ++k) {
            Row<K> f = fwd_row_of<K>(tb, cr, r, k, 0);
            if (k >= 2) set_prev(f, F, band_lo(cr, k - 1), band_hi(cr, k - 1));
            row_pass(f, store_to<K>(F, nullptr), ps, lane, N);
        }
    }
    for (int k = kept ? best_mu + 1 : best_mu; k < m; ++k) {
        Row<K> rw = fwd_row_of<K>(tb, cr, r, k, best_mu);
        if (k >= 2) set_prev(rw, F, band_lo(cr, k - 1), band_hi(cr, k - 1));
        row_pass(rw, store_to<K>(F, sm.tbp + pool_off(cr, k)), ps, lane, N);
    }
    if (m >= 2) {
        Row<K> rw = fwd_row_of<K>(tb, cr, r, m, best_mu);
        // row m-1 of the chosen table (F_{m-1} when mu* = m: the sweep's last row)
        set_prev(rw, F, band_lo(cr, m - 1), band_hi(cr, m - 1));
        rw.lo = rw.hi = N - 1;
        const K lk = single_cell_key(rw, lane, N);
        if (lane == 0) *last_tb = (uint8_t)key_low8(lk);
        // the split points may sit in global memory (long bands): complete
        // every lane's stores before lane 0 walks them
        __builtin_amdgcn_s_waitcnt(0);
        __threadfence_block();
        if (lane == 0) {
            int i = N - 1;
            int j = *last_tb;
            if (j > i) j = i;
            start[m - 1] = (uint8_t)j;
            i = j - 1;
            for (int k = m - 1; k >= 2; --k) {
                const int blo = band_lo(cr, k), bhi = band_hi(cr, k);
                // path cells lie in their band; the clamp only keeps a
                // corrupted table from indexing outside its row
                const int ii = i < blo ? blo : (i > bhi ? bhi : i);
                j = sm.tbp[pool_off(cr, k) + (ii - blo)];
                if (j > i) j = i;
                start[k - 1] = (uint8_t)j;
                i = j - 1;
            }
        }
    }
    if (lane == 0) start[0] = 0;
    __syncthreads();
}

// Reference path (chains whose bands exceed the pool): Algorithm 1's table
// for one master position, full rows k-1..N-1, ping-ponging the LDS row
// buffers; split points of rows 2..m go to tbp (row k at (k-2)*N) when tbp
// is not null.
__device__ __forceinline__ uint64_t dp_table(const E2Tables &tb, const DpSmem &sm, int r, const uint8_t *chain,
                             int m, int mu, uint8_t *tbp, int lane)
{
    const int N = tb.N;
    PS<uint64_t> *ps = static_cast<PS<uint64_t> *>(sm.ps);
    lds_t<uint64_t> *cur = sm.Rw0, *prv = sm.Rw1;
    for (int k = 1; k <= m; ++k) {
        const int c = uni(chain[k - 1]);
        const int f = (mu == k);
        Row<uint64_t> rw;
        rw.pr = pref_row(tb, r, c);
        rw.wr = win_row(tb, f, c);
        rw.hadd = f ? uni64(tb.head[r * tb.M + c]) : 0;
        rw.p8 = nullptr;
        rw.hadd8 = rw.hadd << 8;
        rw.lo = k - 1;
        rw.hi = N - 1;
        rw.kmin = k - 1;
        rw.cap = N;
        rw.lmin = uni(minwin_at(tb, f, c, rw.lo));
        if (k == 1) {
            rw.tau = 0;
            rw.prev = nullptr;
            rw.plo = 1;
            rw.phi = 0;
        } else {
            rw.tau = link_tau_u(tb, r, uni(chain[k - 2]), c);
            rw.prev = prv;
            rw.plo = k - 2;
            rw.phi = N - 1;
        }
        row_pass(rw,
                 store_to<uint64_t>(cur, (tbp && k >= 2) ? tbp + (size_t)(k - 2) * N + (k - 1)
                                                         : nullptr),
                 ps, lane, N);
        lds_t<uint64_t> *tmp = prv;
        prv = cur;
        cur = tmp;
    }
    return prv[(N - 1) - (m - 1)];
}

// The device chain of cluster q of genome p into chain[] (LDS); returns its
// length.  Labels: the devices with label q in ascending id (wave ballot
// compaction); two-chromosome genomes: replica q's run of the ordering.
__device__ __forceinline__ int build_chain(const E2Genomes &gen, int p, int q, int k_max, int M,
                                           int lane, uint8_t *chain)
{
    int m = 0;
    if (gen.labels) {
        // the genome's labels, device lane + 64 t in slot t, all loads issued
        // before the first is used (clamped indices: no branch around them)
        // (the lane index goes through an empty asm so that the offsets are
        // formed here, in 32 bits from the row's scalar base, instead of being
        // kept live across the job loop)
        constexpr int kSlots = (E2_MAX_DEV + kWave - 1) / kWave;
        const uint8_t *row = gen.labels + (size_t)p * M;
        int l = lane;
        asm volatile("" : "+v"(l));
        int lab[kSlots];
#pragma unroll
        for (int t = 0; t < kSlots; ++t) lab[t] = at_byte(row, (uint32_t)min(l + kWave * t, M - 1));
#pragma unroll
        for (int t = 0; t < kSlots; ++t) {
            if (kWave * t >= M) break;
            const int d = kWave * t + lane;
            const bool in = d < M && lab[t] == q;
            const uint64_t mask = __ballot(in);
            if (in) chain[m + __popcll(mask & ((1ull << lane) - 1))] = (uint8_t)d;
            m += __popcll(mask);
        }
    } else {
        uint64_t part = 0;
        for (int r = lane; r < q; r += kWave) part += gen.sizes[(size_t)p * k_max + r];
        const uint64_t off = wave_sum_u64(part);
        const int lo = (int)(off < (uint64_t)M ? off : (uint64_t)M);
        const uint64_t end = off + gen.sizes[(size_t)p * k_max + q];
        m = (int)(end < (uint64_t)M ? end : (uint64_t)M) - lo;
        for (int k = lane; k < m; k += kWave) chain[k] = gen.order[(size_t)p * M + lo + k];
    }
    return m;
}

// ---------------------------------------------------------------------------
// Persistent DP kernel: one wave per workgroup; wave w of W solves listed
// problems w, w + W, w + 2W, ... of the first part of the list (it runs
// longest chains first, so every wave gets a like mix), the rest from a
// shared counter when there are many problems per wave, and exits past the
// end of the list.  LDS: split-point pairs (N x 16 B), the backward-row pool,
// a row buffer and the split-point bytes of the forward rows (see k_dp).
// ---------------------------------------------------------------------------
template <bool L> struct CRSel { using T = ChainRegs; };
template <> struct CRSel<true> { using T = ChainRegsLong; };

template <bool LONG>
__device__ __forceinline__ void dp_jobs(const E2Tables &tb, int k_max, int pool_cells,
                                        const E2Genomes &gen, const uint8_t *__restrict__ roles,
                                        int n_r, uint32_t *counters,
                                        const uint32_t *__restrict__ list, size_t seg_cap,
                                        uint8_t *tb_global, uint64_t *T, uint64_t *Lambda,
                                        int16_t *master, uint8_t *layers, uint64_t *dyn,
                                        uint8_t *chain, uint8_t *start, uint8_t *last_tb_p)
{
    uint8_t &last_tb = *last_tb_p;
    const int lane = threadIdx.x;
    const int M = tb.M, N = tb.N;
    // LDS: split-point pairs, then the banded path's backward-row pool (the
    // pairs' unused half for 32-bit keys, a row buffer and the extra bytes),
    // a row buffer and the split-point bytes
    DpSmem sm;
    sm.ps = dyn;
    sm.Rw1 = (lds_t<uint64_t> *)(dyn + 2 * N);
    sm.pool_end = (lds_t<char> *)(dyn + 2 * N + (N + 1)) + dp_lds_extra(N);
    sm.Rw0 = (lds_t<uint64_t> *)sm.pool_end;
    sm.tbp = reinterpret_cast<uint8_t *>(dyn + 2 * N + 2 * (N + 1)) + dp_lds_extra(N);
    sm.pool_cells = pool_cells;
    static_assert(kClasses == 4, "job mapping below assumes four classes");
    const uint32_t n0 = LONG ? 0 : counters[0], n1 = LONG ? 0 : counters[kCounterStride],
                   n2 = LONG ? 0 : counters[2 * kCounterStride],
                   n3 = LONG ? 0 : counters[3 * kCounterStride];
    // the long-chain kernel takes segment kClasses alone, one job at a time
    const uint32_t n_jobs = LONG ? counters[kClasses * kCounterStride] : n0 + n1 + n2 + n3;
    const int job_ctr = (LONG ? kLongJobCounter : kJobCounter) * kCounterStride;

    // The list runs longest chains first.  Its first part is split statically
    // (wave w of W takes problems w, w + W, w + 2W, ...: every wave gets a
    // like mix, with no shared counter to contend for); with many problems
    // per wave, the short problems of the last part go to whichever wave is
    // free, from a shared counter, which evens out the waves' finishing
    // times.  (With few problems per wave the waves would all reach the
    // counter at once; the whole list is then split statically.)
    const bool dyn_tail = n_jobs >= kDynTailMinPerWave * gridDim.x;
    const uint32_t n_static =
        LONG ? 0u : (dyn_tail ? n_jobs - (n_jobs >> kDynTailShift) : n_jobs);
    auto take = [&](uint32_t done) -> uint32_t {
        if (done + gridDim.x < n_static) return done + gridDim.x;
        uint32_t v = 0;
        if (lane == 0) v = atomicAdd(&counters[job_ctr], 1u);
        return n_static + (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    };
    uint32_t first = blockIdx.x;
    if (first >= n_static) {
        uint32_t v = 0;
        if (lane == 0) v = atomicAdd(&counters[job_ctr], 1u);
        first = n_static + (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    }
    for (uint32_t job = first; job < n_jobs; job = take(job)) {
        uint32_t idx = job;
        // classes in order, longest chains first
        int cls = LONG ? kClasses : 0;
        if (!LONG) {
            if (idx >= n0) { idx -= n0; cls = 1;
                if (idx >= n1) { idx -= n1; cls = 2;
                    if (idx >= n2) { idx -= n2; cls = 3; } } }
        }
        const uint32_t code = list[(size_t)cls * seg_cap + idx];
        const int p = n_r > 0 ? (int)(code >> 12) : (int)(code >> 8);
        const int q = n_r > 0 ? (int)((code >> 4) & 0xFF) : (int)(code & 0xFF);

        const int m = build_chain(gen, p, q, k_max, M, lane, chain);
        __syncthreads();
        // role index: from the job (every role searched) or the genome's role
        const int r = n_r > 0 ? (int)(code & 0xF) : roles[(size_t)p * k_max + q] != 0;
        const size_t o = n_r > 0 ? ((size_t)p * k_max + q) * n_r + r : (size_t)p * k_max + q;
        const E2Tables tv = mem_view(tb, r);

        uint64_t best = E2_INF64;
        int best_mu = 0;
        typename CRSel<LONG>::T cr;
        uint64_t bound = E2_INF64, bound_tot = E2_INF64;
        int pool_need = 0;
        bool banded;
        if constexpr (LONG) {
            chain_regs_long(tv, r, chain, m, lane, cr, &bound, &bound_tot, &pool_need);
            banded = true;
        } else {
            banded = chain_regs(tv, sm, r, chain, m, lane, cr, &bound, &bound_tot, &pool_need);
        }
        // split points of bands beyond the LDS copy go to the global table
        DpSmem smb = sm;
        if (pool_need > kLdsTbCells) {
            smb.tbp = tb_global ? tb_global + (size_t)blockIdx.x * N * N : nullptr;
            banded = banded && tb_global != nullptr;
        }
        if (banded && wave_all_le(bound, kU32MaxValue))
            dp_banded<uint32_t>(tv, smb, cr, r, m, lane, &best, &best_mu, start, &last_tb);
        else if (banded && wave_all_le(bound_tot, kF64Limit - 1))
            dp_banded<double>(tv, smb, cr, r, m, lane, &best, &best_mu, start, &last_tb);
        else {
            // reference path: a full table per master, then the chosen
            // master's table again with split points
            for (int mu = 1; mu <= m; ++mu) {
                const uint64_t v = dp_table(tv, sm, r, chain, m, mu, nullptr, lane);
                if (v < best) {
                    best = v;
                    best_mu = mu;
                }
            }
            if (best != E2_INF64) {
                uint8_t *tbp = ((size_t)(m - 1) * N <= (size_t)kLdsTbCells)
                                   ? sm.tbp
                                   : tb_global + (size_t)blockIdx.x * N * N;
                dp_table(tv, sm, r, chain, m, best_mu, tbp, lane);
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
            const uint64_t *pr = pref_row(tv, r, c);
            part += pr[e] - pr[s0];
            if (k + 1 == best_mu) part += tv.head[r * M + c];
            if (k >= 1) part += link_tau(tv, r, chain[k - 1], c);
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

__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(5))) void k_dp(
    E2Tables tb, int k_max, int pool_cells, E2Genomes gen, const uint8_t *__restrict__ roles,
    int n_r, uint32_t *counters, const uint32_t *__restrict__ list, size_t seg_cap,
    uint8_t *tb_global, uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    extern __shared__ uint64_t dyn[];
    __shared__ uint8_t chain[256];
    __shared__ uint8_t start[256];
    __shared__ uint8_t last_tb;
    dp_jobs<false>(tb, k_max, pool_cells, gen, roles, n_r, counters, list, seg_cap, tb_global, T,
                   Lambda, master, layers, dyn, chain, start, &last_tb);
}

// Chains of more than 64 devices (the list's last segment): the same banded
// path with the per-position table four positions per lane.  A kernel of its
// own, so that its larger register table leaves k_dp's occupancy alone.
__global__ __launch_bounds__(64) void k_dp_long(
    E2Tables tb, int k_max, int pool_cells, E2Genomes gen, const uint8_t *__restrict__ roles,
    int n_r, uint32_t *counters, const uint32_t *__restrict__ list, size_t seg_cap,
    uint8_t *tb_global, uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    extern __shared__ uint64_t dyn[];
    __shared__ uint8_t chain[256];
    __shared__ uint8_t start[256];
    __shared__ uint8_t last_tb;
    dp_jobs<true>(tb, k_max, pool_cells, gen, roles, n_r, counters, list, seg_cap, tb_global, T,
                  Lambda, master, layers, dyn, chain, start, &last_tb);
}

// ---------------------------------------------------------------------------
// The finishing-time objective (the FT ablation): Eq. 1 with the bottleneck
// max replaced by a sum, so that a master's table holds the least
// end-to-end time (stage times plus link times) of blocks 0..i on devices
// 1..k; Eq. 2 and the memory windows unchanged.  One full table per master:
// lanes over cells i, each scanning its window of j in ascending order
// (strict <, so ties keep the smallest j); the two rows ping-pong in the
// wave's LDS; split points of rows 2..m go to tbp (row k at (k-2) N) when
// tbp is not null.  Values stay below 2^58 (at most 255 block times and 255
// link times, each below 2^48); INF terms are skipped.
// ---------------------------------------------------------------------------
__device__ uint64_t ft_table(const E2Tables &tb, const DpSmem &sm, int r, const uint8_t *chain,
                             int m, int mu, uint8_t *tbp, int lane)
{
    const int N = tb.N, M = tb.M;
    uint64_t *cur = (uint64_t *)sm.Rw0, *prv = (uint64_t *)sm.Rw1;
    for (int k = 1; k <= m; ++k) {
        const int c = uni(chain[k - 1]);
        const int f = (mu == k);
        const uint64_t *pr = pref_row(tb, r, c);
        const uint8_t *wr = win_row(tb, f, c);
        const uint64_t hadd = f ? uni64(tb.head[r * M + c]) : 0;
        const uint64_t tau = k >= 2 ? link_tau_u(tb, r, uni(chain[k - 2]), c) : 0;
        for (int i = lane; i < N; i += kWave) {
            uint64_t best = E2_INF64;
            int bj = 0;
            const int w = wr[i];
            if (i >= k - 1 && w != E2_NO_START) {
                const uint64_t end = pr[i + 1] + hadd;
                if (k == 1) {
                    if (w == 0) best = end - pr[0];
                } else if (tau != E2_INF64) {
                    for (int j = max(w, k - 1); j <= i; ++j) {
                        const uint64_t pv = prv[j - 1];
                        if (pv == E2_INF64) continue;
                        const uint64_t v = pv + tau + (end - pr[j]);
                        if (v < best) {
                            best = v;
                            bj = j;
                        }
                    }
                }
            }
            cur[i] = best;
            if (tbp && k >= 2) tbp[(size_t)(k - 2) * N + i] = (uint8_t)bj;
        }
        __threadfence_block();
        __syncthreads();
        uint64_t *tmp = prv;
        prv = cur;
        cur = tmp;
    }
    return prv[N - 1];
}

// One banded row of the finishing-time DP: cells i in [lo, hi],
//   out(i) = min over j in [max(win(i), kmin), i], ascending (the smallest j
//            on ties), of prev(j-1) + tau + P[i+1] - P[j] + hadd
// with prev band-packed over [plo, phi] (INF outside) or, for the first
// device, the stage 0..i alone.  Values to out[i - lo] (LDS or global),
// split points to tbs[i - lo] when tbs is not null.  The terms that depend
// on j alone, a(j) = prev(j-1) + (P[N] - P[j]) (INF when prev(j-1) is), are
// staged in LDS first (st, N entries), so that a candidate is one LDS read:
// a(j) + (P[i+1] + hadd + tau - P[N]) is the candidate exactly in modular
// u64 arithmetic.
__device__ __forceinline__ void ft_row_plain(const uint64_t *pr, const uint8_t *wr,
                                             uint64_t hadd, uint64_t tau, int lo, int hi,
                                             int kmin, const lds_t<uint64_t> *prev, int plo,
                                             int phi, lds_t<uint64_t> *out, uint8_t *tbs,
                                             lds_t<uint64_t> *st, int N, int lane)
{
    const uint64_t pN = pr[N];
    const bool linked = prev && tau != E2_INF64;
    if (linked) {
        for (int j = kmin + lane; j <= hi; j += kWave) {
            const int x = j - 1;
            uint64_t a = E2_INF64;
            if (x >= plo && x <= phi) {
                const uint64_t pv = prev[x - plo];
                if (pv != E2_INF64) a = pv + (pN - pr[j]);
            }
            st[j] = a;
        }
        __syncthreads();
    }
    for (int i = lo + lane; i <= hi; i += kWave) {
        uint64_t best = E2_INF64;
        int bj = 0;
        const int w = wr[i];
        if (w != E2_NO_START) {
            const uint64_t end = pr[i + 1] + hadd;
            if (!prev) {
                if (w == 0) best = end - pr[0];
            } else if (linked) {
                const uint64_t c = end + tau - pN;
                // four entries loaded before use, taken in ascending j with a
                // strict < (the smallest j keeps ties), without branches
                int j = max(w, kmin);
                for (; j + 3 <= i; j += 4) {
                    const uint64_t a0 = st[j], a1 = st[j + 1], a2 = st[j + 2], a3 = st[j + 3];
                    const uint64_t v0 = a0 + c, v1 = a1 + c, v2 = a2 + c, v3 = a3 + c;
                    const bool t0 = a0 != E2_INF64 && v0 < best;
                    best = t0 ? v0 : best;
                    bj = t0 ? j : bj;
                    const bool t1 = a1 != E2_INF64 && v1 < best;
                    best = t1 ? v1 : best;
                    bj = t1 ? j + 1 : bj;
                    const bool t2 = a2 != E2_INF64 && v2 < best;
                    best = t2 ? v2 : best;
                    bj = t2 ? j + 2 : bj;
                    const bool t3 = a3 != E2_INF64 && v3 < best;
                    best = t3 ? v3 : best;
                    bj = t3 ? j + 3 : bj;
                }
                for (; j <= i; ++j) {
                    const uint64_t a = st[j];
                    const uint64_t v = a + c;
                    const bool t = a != E2_INF64 && v < best;
                    best = t ? v : best;
                    bj = t ? j : bj;
                }
            }
        }
        out[i - lo] = best;
        if (tbs) tbs[i - lo] = (uint8_t)bj;
    }
    // rows live in LDS (the next row reads this one after the barrier); the
    // split points may be global and are waited for once, before the back
    // tracing
    __syncthreads();
}

// The same row with S lanes per cell.  A staged term is packed as a key
// (a(j) << 8) | j, so one unsigned min keeps the least a(j) and, among equal
// ones, the smallest j: the strict ascending scan above.  Lane o of a cell
// scans j = i - o, i - o - S, ... down to the window start; the S partial
// minima meet through DPP quad permutations (and a half-row mirror for
// S = 8).  Used when every a(j) of the problem is below 2^56.
template <int S>
__device__ __forceinline__ void ft_row_keyed_s(const uint64_t *pr, const uint8_t *wr,
                                               uint64_t hadd, uint64_t tau, int lo, int hi,
                                               int kmin, const lds_t<uint64_t> *prev, int plo,
                                               int phi, lds_t<uint64_t> *out, uint8_t *tbs,
                                               lds_t<uint64_t> *st, int N, int lane)
{
    constexpr int CPP = kWave / S;  // cells per pass
    const int o = lane % S;
    const int cl = lane / S;
    // the first pass's cell loads go out before the terms are staged
    int w_nx;
    uint64_t p_nx;  // P[i+1]
    {
        const int i = min(lo + cl, hi);
        w_nx = wr[i];
        p_nx = pr[i + 1];
    }
    const uint64_t pN = pr[N];
    for (int j = kmin + lane; j <= hi; j += kWave) {
        const int x = j - 1;
        uint64_t key = E2_INF64;
        if (x >= plo && x <= phi) {
            const uint64_t pv = prev[x - plo];
            if (pv != E2_INF64) key = ((pv + (pN - pr[j])) << 8) | (uint64_t)j;
        }
        st[j] = key;
    }
    __syncthreads();
    for (int base = lo; base <= hi; base += CPP) {
        const int i = min(base + cl, hi);  // lanes past the row repeat its last cell
        const int w = w_nx;
        const uint64_t p1 = p_nx;
        if (base + CPP <= hi) {  // the next pass's loads (uniform)
            const int in = min(base + CPP + cl, hi);
            w_nx = wr[in];
            p_nx = pr[in + 1];
        }
        uint64_t best = E2_INF64;
        if (w != E2_NO_START) {
            const int jlo = max(w, kmin);
            int j = i - o;
            for (; j - S >= jlo; j -= 2 * S) best = umin64(best, umin64(st[j], st[j - S]));
            if (j >= jlo) best = umin64(best, st[j]);
        }
        if (S >= 2) best = umin64(best, dpp_u64<0xb1>(best));
        if (S >= 4) best = umin64(best, dpp_u64<0x4e>(best));
        if (S >= 8) best = umin64(best, dpp_u64<0x141>(best));
        // the cell's value: a(j*) + P[i+1] + head + tau - P[N] (modular sums)
        const uint64_t v = best == E2_INF64 ? E2_INF64 : (best >> 8) + (p1 + hadd + tau - pN);
        out[i - lo] = v;
        if (tbs) tbs[i - lo] = (uint8_t)(best == E2_INF64 ? 0 : (best & 0xFF));
    }
    __syncthreads();
}

// One FT row: the keyed lane-split scan where it applies (a previous row, a
// finite link, keys that fit), else the one-lane-per-cell scan.
__device__ __forceinline__ void ft_row(const uint64_t *pr, const uint8_t *wr, uint64_t hadd,
                                       uint64_t tau, int lo, int hi, int kmin,
                                       const lds_t<uint64_t> *prev, int plo, int phi,
                                       lds_t<uint64_t> *out, uint8_t *tbs, lds_t<uint64_t> *st,
                                       int N, int lane, bool keyed)
{
    const int n = hi - lo + 1;
    if (!keyed || !prev || tau == E2_INF64 || n <= 0) {
        ft_row_plain(pr, wr, hadd, tau, lo, hi, kmin, prev, plo, phi, out, tbs, st, N, lane);
        return;
    }
    if (n <= 8)
        ft_row_keyed_s<8>(pr, wr, hadd, tau, lo, hi, kmin, prev, plo, phi, out, tbs, st, N, lane);
    else if (n <= 16)
        ft_row_keyed_s<4>(pr, wr, hadd, tau, lo, hi, kmin, prev, plo, phi, out, tbs, st, N, lane);
    else if (n <= 32)
        ft_row_keyed_s<2>(pr, wr, hadd, tau, lo, hi, kmin, prev, plo, phi, out, tbs, st, N, lane);
    else
        ft_row_keyed_s<1>(pr, wr, hadd, tau, lo, hi, kmin, prev, plo, phi, out, tbs, st, N, lane);
}

// Backward FT rows 1..t_end into the LDS backward-row pool, as g_rows does
// for Algorithm 1's rows: rows from t_lo on at their band-packed offsets less
// that of t_lo, the rows before it in place at the pool's start.
__device__ __forceinline__ void ft_g_rows(const E2Tables &tb, const ChainRegs &cr, int r, int m,
                                          int t_end, int t_lo, lds_t<uint64_t> *gp,
                                          lds_t<uint64_t> *st, int N, int lane, bool keyed)
{
    const int base = gpool_off(cr, t_lo);
    for (int t = 1; t <= t_end; ++t) {
        const uint32_t wd = cr.D(t - 1);
        const int c = f8(wd, 0);
        const uint64_t tau = t >= 2 ? cr.TAU(m + 1 - t) : 0;  // link m+1-t -> m+2-t
        ft_row(prefR_row(tb, r, c), winR_row(tb, c), 0, tau, f8(wd, 8), f8(wd, 16),
               t - 1, t >= 2 ? gp + (t - 1 >= t_lo ? gpool_off(cr, t - 1) - base : 0) : nullptr,
               t >= 2 ? rband_lo(cr, t - 1) : 1, t >= 2 ? rband_hi(cr, t - 1) : 0,
               gp + (t >= t_lo ? gpool_off(cr, t) - base : 0), nullptr, st, N, lane, keyed);
    }
}

// The finishing-time DP by the same banded decomposition and schedule as
// dp_banded: reversed rows G_t over the last t devices in the LDS
// backward-row pool (rows the sweep reaches that the pool did not keep are
// computed again), the head-free optimum T0 from the full reversed table's
// last cell, then masters in ascending position with
//   T_mu = min_i H_mu(i) + tau(mu, mu+1) + G_{m-mu}(N-2-i)
// (H_mu the master's forward row, head time and bytes, over F_{mu-1}), each
// followed by the forward row F_mu (no master), computed in place.  Since
// T_mu >= T0 + head(mu), the sweep stops once the best is at most T0 plus
// the least head time of the masters still ahead; the smallest mu with the
// least T_mu wins.  Rows mu*..m of its table are recomputed with split
// points (F_1..F_{mu*-1} first when the sweep went past them) and the back
// tracing fills start[].  Every in-band cell's value equals the full
// table's (bands depend on memory only), so the result is that of one full
// table per master.
__device__ void dp_ft_banded(const E2Tables &tb, const DpSmem &sm, const ChainRegs &cr, int r,
                             int m, int lane, uint64_t *T_out, int *mu_out, uint8_t *start,
                             bool keyed)
{
    const int N = tb.N, M = tb.M;
    lds_t<uint64_t> *st = (lds_t<uint64_t> *)sm.ps;  // ft_row's staged terms (N)
    lds_t<uint64_t> *gp = st + N;                     // backward-row pool
    const int gcap = (int)((sm.pool_end - (lds_t<char> *)gp) / 8);
    lds_t<uint64_t> *H = sm.Rw0;  // the master's row
    lds_t<uint64_t> *F = sm.Rw1;  // forward rows, in place
    // ---- backward rows G_1..G_{m-1}, the last ones that fit kept in the pool
    int g_lo = m >= 2 ? g_window_lo(cr, lane, m - 1, gcap) : 1;
    if (m >= 2) ft_g_rows(tb, cr, r, m, m - 1, g_lo, gp, st, N, lane, keyed);
    // ---- T0, the least end-to-end time with no head anywhere: reversed row
    // m at its last cell.  A master's optimum is at least T0 plus its head
    // time (the head time is added once, its bytes only narrow windows).
    uint64_t t0 = E2_INF64;
    if (m >= 2) {
        const int c = f8(cr.D(m - 1), 0);
        ft_row(prefR_row(tb, r, c), winR_row(tb, c), 0, cr.TAU(1), N - 1, N - 1,
               m - 1, gp + (gpool_off(cr, m - 1) - gpool_off(cr, g_lo)), rband_lo(cr, m - 1),
               rband_hi(cr, m - 1), H, nullptr, st, N, lane, keyed);
        t0 = uni64(H[0]);
        if (t0 == E2_INF64) {
            *T_out = E2_INF64;
            *mu_out = 0;
            return;
        }
    }
    // head time of each position able to take the head (INF otherwise)
    const uint64_t h_cap = (lane < m && f8(cr.wa, 16) != 0) ? cr.head : E2_INF64;

    // ---- masters in ascending position, each followed by F_mu (split points
    // kept for the rows below mu*).  The sweep stops once the best is at most
    // T0 plus the least head time of the masters still ahead: none of them
    // can do better, and ties go to the smaller master.
    uint64_t best = E2_INF64;
    int best_mu = 0;
    int f_last = 0;  // the forward row the buffer holds
    for (int mu = 1; mu <= m; ++mu) {
        const uint32_t wa = cr.A(mu - 1);
        const int c = f8(wa, 0);
        if (f8(wa, 16) != 0) {
            const int t = m - mu;  // backward row of devices mu+1..m
            if (mu < m && t < g_lo) {  // not kept: rows 1..t again
                g_lo = g_window_lo(cr, lane, t, gcap);
                ft_g_rows(tb, cr, r, m, t, g_lo, gp, st, N, lane, keyed);
            }
            const uint64_t tau = mu >= 2 ? cr.TAU(mu - 1) : 0;
            const int lo = band_lo(cr, mu), hi = mu == m ? N - 1 : band_hi(cr, mu);
            const int hlo = mu == m ? N - 1 : lo;
            ft_row(pref_row(tb, r, c), win_row(tb, 1, c), uni64(tb.head[r * M + c]), tau, hlo,
                   hi, mu - 1, mu >= 2 ? F : nullptr, mu >= 2 ? band_lo(cr, mu - 1) : 1,
                   mu >= 2 ? band_hi(cr, mu - 1) : 0, H, nullptr, st, N, lane, keyed);
            uint64_t tm = E2_INF64;
            if (mu == m) {
                tm = H[0];
            } else {
                const uint64_t tn = cr.TAU(mu);  // link mu -> mu+1
                const lds_t<uint64_t> *G = gp + (gpool_off(cr, t) - gpool_off(cr, g_lo));
                const int gl = rband_lo(cr, t), gh = rband_hi(cr, t);
                for (int i = hlo + lane; i <= hi; i += kWave) {
                    const uint64_t h = H[i - hlo];
                    const int x = N - 2 - i;
                    if (h == E2_INF64 || tn == E2_INF64 || x < gl || x > gh) continue;
                    const uint64_t g = G[x - gl];
                    if (g == E2_INF64) continue;
                    const uint64_t v = h + tn + g;
                    tm = v < tm ? v : tm;
                }
                tm = wave_min_u64(tm);
            }
            if (tm < best) {  // ascending positions: the smaller master keeps ties
                best = tm;
                best_mu = mu;
            }
            __syncthreads();
        }
        if (m >= 2 && best != E2_INF64) {
            const uint64_t ahead = wave_min_u64(lane >= mu ? h_cap : E2_INF64);
            if (ahead == E2_INF64 || best <= t0 + ahead) break;
        }
        if (mu < m) {
            const uint64_t tau = mu >= 2 ? cr.TAU(mu - 1) : 0;
            ft_row(pref_row(tb, r, c), win_row(tb, 0, c), 0, tau, band_lo(cr, mu), band_hi(cr, mu),
                   mu - 1, mu >= 2 ? F : nullptr, mu >= 2 ? band_lo(cr, mu - 1) : 1,
                   mu >= 2 ? band_hi(cr, mu - 1) : 0, F,
                   mu >= 2 ? sm.tbp + pool_off(cr, mu) : nullptr, st, N, lane, keyed);
            f_last = mu;
        }
    }
    *T_out = best;
    *mu_out = best_mu;
    if (best == E2_INF64) return;
    // ---- rows mu*..m of the chosen master's table with split points, in
    // place; their first row reads F_{mu*-1}, computed again when the sweep
    // went past it (its split points are in tbp already)
    uint8_t *tbp = sm.tbp;
    if (best_mu >= 2 && f_last != best_mu - 1) {
        for (int k = 1; k < best_mu; ++k) {
            const int c = f8(cr.A(k - 1), 0);
            ft_row(pref_row(tb, r, c), win_row(tb, 0, c), 0, k >= 2 ? cr.TAU(k - 1) : 0,
                   band_lo(cr, k), band_hi(cr, k), k - 1, k >= 2 ? F : nullptr,
                   k >= 2 ? band_lo(cr, k - 1) : 1, k >= 2 ? band_hi(cr, k - 1) : 0, F, nullptr,
                   st, N, lane, keyed);
        }
    }
    for (int k = best_mu; k <= m; ++k) {
        const uint32_t wa = cr.A(k - 1);
        const int c = f8(wa, 0);
        const int f = (k == best_mu);
        const uint64_t tau = k >= 2 ? cr.TAU(k - 1) : 0;
        const int lo = k == m ? N - 1 : band_lo(cr, k), hi = k == m ? N - 1 : band_hi(cr, k);
        uint8_t *tbs = k == m ? start + m : tbp + pool_off(cr, k);  // row m: one cell
        ft_row(pref_row(tb, r, c), win_row(tb, f, c), f ? uni64(tb.head[r * M + c]) : 0, tau, lo,
               hi, k - 1, k >= 2 ? F : nullptr, k >= 2 ? band_lo(cr, k - 1) : 1,
               k >= 2 ? band_hi(cr, k - 1) : 0, F, k >= 2 ? tbs : nullptr, st, N, lane, keyed);
    }
    // the split points may sit in global memory (long bands): complete every
    // lane's stores before lane 0 walks them
    __builtin_amdgcn_s_waitcnt(0);
    __threadfence_block();
    if (lane == 0) {
        int i = N - 1;
        int j = m >= 2 ? start[m] : 0;
        for (int k = m; k >= 2; --k) {
            if (k < m) {
                const int blo = band_lo(cr, k), bhi = band_hi(cr, k);
                const int ii = i < blo ? blo : (i > bhi ? bhi : i);
                j = tbp[pool_off(cr, k) + (ii - blo)];
            }
            if (j > i) j = i;
            start[k - 1] = (uint8_t)j;
            i = j - 1;
        }
        start[0] = 0;
    }
    __syncthreads();
}

__global__ __launch_bounds__(64) void k_dp_ft(E2Tables tb, int k_max, int pool_cells, E2Genomes gen,
                                              const uint8_t *__restrict__ roles,
                                              uint32_t *counters,
                                              const uint32_t *__restrict__ list, size_t seg_cap,
                                              uint8_t *tb_global, uint64_t *T,
                                              uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    extern __shared__ uint64_t dyn[];
    __shared__ uint8_t chain[256];
    __shared__ uint8_t start[256];
    __shared__ uint32_t job;
    const int lane = threadIdx.x;
    const int M = tb.M, N = tb.N;
    // LDS: the staged terms (N u64), the backward-row pool (N u64 and the
    // extra bytes), the master's row and the forward row, the split-point
    // bytes; the reference path uses the two rows as a ping-pong
    DpSmem sm;
    sm.ps = dyn;
    sm.pool_end = (lds_t<char> *)(dyn + 2 * N) + dp_lds_extra(N);
    sm.Rw0 = (lds_t<uint64_t> *)sm.pool_end;
    sm.Rw1 = sm.Rw0 + (N + 1);
    sm.tbp = reinterpret_cast<uint8_t *>(dyn + 2 * N + 2 * (N + 1)) + dp_lds_extra(N);
    sm.pool_cells = pool_cells;
    const uint32_t n0 = counters[0], n1 = counters[kCounterStride],
                   n2 = counters[2 * kCounterStride], n3 = counters[3 * kCounterStride];
    const uint32_t n_jobs = n0 + n1 + n2 + n3;
    // waves take the next listed problem from a shared counter: these grids
    // need not be resident at once, and their problems vary more in cost
    for (;;) {
        if (lane == 0) job = atomicAdd(&counters[kJobCounter * kCounterStride], 1u);
        __syncthreads();
        uint32_t idx = job;
        __syncthreads();
        if (idx >= n_jobs) break;
        int cls = 0;
        if (idx >= n0) { idx -= n0; cls = 1;
            if (idx >= n1) { idx -= n1; cls = 2;
                if (idx >= n2) { idx -= n2; cls = 3; } } }
        const uint32_t code = list[(size_t)cls * seg_cap + idx];
        const int p = (int)(code >> 8);
        const int q = (int)(code & 0xFF);
        const int m = build_chain(gen, p, q, k_max, M, lane, chain);
        __syncthreads();
        const int r = roles[(size_t)p * k_max + q] != 0;
        const size_t o = (size_t)p * k_max + q;
        const E2Tables tv = mem_view(tb, r);
        // least end-to-end time over masters, the smallest master on ties
        uint64_t best = E2_INF64;
        int best_mu = 0;
        ChainRegs cr;
        uint64_t bound, bound_tot;
        int pool_need = 0;
        bool banded = chain_regs(tv, sm, r, chain, m, lane, cr, &bound, &bound_tot, &pool_need);
        DpSmem smb = sm;
        if (pool_need > kLdsTbCells) {
            smb.tbp = tb_global ? tb_global + (size_t)blockIdx.x * N * N : nullptr;
            banded = banded && tb_global != nullptr;
        }
        if (banded) {
            // keyed rows when every staged term a(j) < 2^56: a(j) is at most the
            // chain's summed device totals and links plus one device's total
            const bool keyed =
                wave_all_le(bound_tot, (1ull << 56) / (uint64_t)(2 * m + 2) - 1);
            dp_ft_banded(tv, smb, cr, r, m, lane, &best, &best_mu, start, keyed);
        } else {
            for (int mu = 1; mu <= m; ++mu) {
                const uint64_t v = ft_table(tv, sm, r, chain, m, mu, nullptr, lane);
                if (v < best) {
                    best = v;
                    best_mu = mu;
                }
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
        if (!banded) {
            uint8_t *tbp = ((size_t)(m - 1) * N <= (size_t)kLdsTbCells)
                               ? sm.tbp
                               : tb_global + (size_t)blockIdx.x * N * N;
            ft_table(tv, sm, r, chain, m, best_mu, tbp, lane);
            __builtin_amdgcn_s_waitcnt(0);
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
        // the partition's end-to-end time and its bottleneck
        uint64_t part = 0, bott = 0;
        for (int k = lane; k < m; k += kWave) {
            const int c = chain[k];
            const int s0 = start[k] < N ? start[k] : N;
            int e = (k + 1 < m) ? start[k + 1] : N;
            if (e > N) e = N;
            if (e < s0) e = s0;
            const uint64_t *pr = pref_row(tv, r, c);
            uint64_t st = pr[e] - pr[s0];
            if (k + 1 == best_mu) st += tv.head[r * M + c];
            part += st;
            bott = umax64(bott, st);
            if (k >= 1) {
                const uint64_t tl = link_tau(tv, r, chain[k - 1], c);
                part += tl;
                bott = umax64(bott, tl);
            }
            if (layers) layers[(size_t)p * M + c] = (uint8_t)(e - s0);
        }
        const uint64_t lam = wave_sum_u64(part);
        const uint64_t bn = wave_max_u64(bott);
        if (lane == 0) {
            T[o] = bn;
            Lambda[o] = lam;
            if (master) master[o] = (int16_t)chain[best_mu - 1];
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// The idle-device relaxation: a device may hold no block and then sits out;
// links join consecutive participants (any pair of chain devices); the
// master always takes part, with its head, possibly with no block.  For a
// master mu and x = blocks placed so far:
//   A_k(x) = min over allowed predecessors k' (ascending; "none", meaning k
//            is the first participant, stands for 0 at x = 0) of
//            max(E_k'(x), tau(k', k)); k <= mu: none or 1..k-1, k > mu:
//            mu..k-1, so that every path past the master holds it
//   E_k(x) = min over j ascending in the window of max(A_k(j), cost(j..x-1))
//            then, for the master, the empty stage max(A_mu(x), head)
//   T_mu   = min over k >= mu of E_k(N), the smallest k on ties
// One wave per problem, lanes over x; A_k in LDS, the E rows (and, on the
// second pass for the best master, the predecessors and stage starts) in
// the wave's global region.
// ---------------------------------------------------------------------------
// The least T_mu of every master of the idle-device relaxation at once.
// F_k(x): the best bottleneck of x blocks on participants among devices
// 1..k ending with k (every participant holding blocks, no master); R_t(x):
// the same over reversed blocks for the last t devices (B_k'(y) =
// R_{m+1-k'}(N-y): blocks y..N-1 on participants from k' on, starting at
// k').  Then with
//   A_mu(x) = min(0 if x = 0, min_{k' < mu} max(F_k'(x), tau(k', mu)))
//   S_mu(y) = 0 if y = N, else min_{k'' > mu} max(tau(mu, k''), B_k''(y))
//   T_mu    = min over x <= y of max(A_mu(x), stage_mu(x..y-1) with the
//             head (the head alone when x = y), S_mu(y))
// which is the per-master table's optimum, exactly (the bottleneck splits
// at the master's stage); the smallest master with the least T_mu wins.
// O(m^2 N + m N W / 64) per problem instead of O(m^3 N + m^2 N W / 64).
__device__ void idle_masters(const E2Tables &tv, int r, const uint8_t *chain, int m, uint64_t *E,
                             uint64_t *B, uint64_t *A, uint64_t *S, uint64_t *P, int lane,
                             uint64_t *best_out, int *mu_out)
{
    // P (LDS, N+1 entries) holds the stage device's prefix sums, staged with
    // A, so that the candidate loops read no global memory
    const int N = tv.N, M = tv.M, X = N + 1;
    // forward rows F_k into E, reversed rows R_t into B
    for (int dir = 0; dir < 2; ++dir) {
        uint64_t *rows = dir ? B : E;
        for (int k = 1; k <= m; ++k) {
            // forward: device k; reversed: device m+1-k, links to the ones behind it
            const int pos = dir ? m - k : k - 1;
            const int c = uni(chain[pos]);
            const uint64_t *pr = dir ? prefR_row(tv, r, c) : pref_row(tv, r, c);
            // the links from the earlier rows' devices: row kp <= 64 from lane
            // kp-1, later rows (chains beyond 65 devices) load theirs
            uint64_t tlk = E2_INF64;
            if (lane < k - 1) {
                const int cp = chain[dir ? m - (lane + 1) : lane];
                // links run from the earlier chain position to the later one
                tlk = dir ? link_tau(tv, r, c, cp) : link_tau(tv, r, cp, c);
            }
            for (int x = lane; x <= N; x += kWave) {
                P[x] = pr[x];
                uint64_t a = x == 0 ? 0 : E2_INF64;
#pragma unroll 4
                for (int kp = 1; kp <= k - 1; ++kp) {
                    const uint64_t e = rows[(size_t)(kp - 1) * X + x];
                    uint64_t tl;
                    if (kp <= kWave) {
                        tl = readlane_u64(tlk, kp - 1);
                    } else {
                        const int cp = uni(chain[dir ? m - kp : kp - 1]);
                        tl = dir ? link_tau_u(tv, r, c, cp) : link_tau_u(tv, r, cp, c);
                    }
                    const uint64_t v = umax64(e, tl);  // INF when either is
                    a = v < a ? v : a;
                }
                A[x] = a;
            }
            __syncthreads();
            const uint8_t *wr = dir ? winR_row(tv, c) : win_row(tv, 0, c);
            for (int x = lane; x <= N; x += kWave) {
                uint64_t e = E2_INF64;
                if (x >= 1) {
                    const int w = wr[x - 1];
                    const uint64_t px = P[x];
                    // INF is the largest value, so an infeasible prefix needs
                    // no branch: the max is INF
                    if (w != E2_NO_START)
#pragma unroll 4
                        for (int j = w; j < x; ++j) {
                            const uint64_t v = umax64(A[j], px - P[j]);
                            e = v < e ? v : e;
                        }
                }
                rows[(size_t)(k - 1) * X + x] = e;
            }
            __builtin_amdgcn_s_waitcnt(0);
            __threadfence_block();
            __syncthreads();
        }
    }
    uint64_t best = E2_INF64;
    int best_mu = 0;
    for (int mu = 1; mu <= m; ++mu) {
        const int c = uni(chain[mu - 1]);
        const uint64_t *pr = pref_row(tv, r, c);
        // links into the master from position kp (lane kp-1, kp < mu) and out
        // of it to position kpp (lane kpp-1, kpp > mu); positions beyond 64
        // load theirs
        uint64_t tin = E2_INF64, tout = E2_INF64;
        if (lane < mu - 1) tin = link_tau(tv, r, chain[lane], c);
        if (lane >= mu && lane < m) tout = link_tau(tv, r, c, chain[lane]);
        for (int x = lane; x <= N; x += kWave) {
            P[x] = pr[x];
            uint64_t a = x == 0 ? 0 : E2_INF64;
#pragma unroll 4
            for (int kp = 1; kp < mu; ++kp) {
                const uint64_t e = E[(size_t)(kp - 1) * X + x];
                const uint64_t tl = kp <= kWave ? readlane_u64(tin, kp - 1)
                                                : link_tau_u(tv, r, uni(chain[kp - 1]), c);
                const uint64_t v = umax64(e, tl);
                a = v < a ? v : a;
            }
            A[x] = a;
            uint64_t sv = x == N ? 0 : E2_INF64;
#pragma unroll 4
            for (int kpp = mu + 1; kpp <= m; ++kpp) {
                // participants from kpp on: reversed row t = m + 1 - kpp at N - x
                const uint64_t e = B[(size_t)(m - kpp) * X + (N - x)];
                const uint64_t tl = kpp <= kWave ? readlane_u64(tout, kpp - 1)
                                                 : link_tau_u(tv, r, c, uni(chain[kpp - 1]));
                const uint64_t v = umax64(e, tl);
                sv = v < sv ? v : sv;
            }
            S[x] = sv;
        }
        __syncthreads();
        const uint8_t *wr = win_row(tv, 1, c);
        const uint64_t head = uni64(tv.head[r * M + c]);
        const bool empty_ok = tv.hfit[c];
        uint64_t tm = E2_INF64;
        for (int y = lane; y <= N; y += kWave) {
            const uint64_t sv = S[y];
            if (sv == E2_INF64) continue;
            if (y >= 1) {
                const int w = wr[y - 1];
                const uint64_t py = P[y] + head;
                if (w != E2_NO_START)
#pragma unroll 4
                    for (int x = w; x < y; ++x) {
                        const uint64_t v = umax64(umax64(A[x], py - P[x]), sv);
                        tm = v < tm ? v : tm;
                    }
            }
            if (empty_ok && A[y] != E2_INF64) {
                const uint64_t v = umax64(umax64(A[y], head), sv);
                tm = v < tm ? v : tm;
            }
        }
        tm = wave_min_u64(tm);
        if (tm < best) {
            best = tm;
            best_mu = mu;
        }
        __syncthreads();
    }
    *best_out = best;
    *mu_out = best_mu;
}

__global__ __launch_bounds__(64) void k_dp_idle(E2Tables tb, int k_max, E2Genomes gen,
                                                const uint8_t *__restrict__ roles,
                                                uint32_t *counters,
                                                const uint32_t *__restrict__ list, size_t seg_cap,
                                                uint8_t *idle, size_t idle_stride, uint64_t *T,
                                                uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    extern __shared__ uint64_t A[];  // [N+1], then S [N+1] and P [N+1]
    __shared__ uint8_t chain[256];
    __shared__ uint8_t sizes[256];
    __shared__ uint32_t job;
    const int lane = threadIdx.x;
    const int M = tb.M, N = tb.N, X = N + 1;
    uint64_t *S = A + X;
    uint64_t *P = S + X;
    uint64_t *E = reinterpret_cast<uint64_t *>(idle + (size_t)blockIdx.x * idle_stride);
    uint64_t *B = E + (size_t)M * X;
    uint16_t *Ek = reinterpret_cast<uint16_t *>(B + (size_t)M * X);
    uint8_t *Ej = reinterpret_cast<uint8_t *>(Ek + (size_t)M * X);
    const uint32_t n0 = counters[0], n1 = counters[kCounterStride],
                   n2 = counters[2 * kCounterStride], n3 = counters[3 * kCounterStride];
    const uint32_t n_jobs = n0 + n1 + n2 + n3;
    // waves take the next listed problem from a shared counter: these grids
    // need not be resident at once, and their problems vary more in cost
    for (;;) {
        if (lane == 0) job = atomicAdd(&counters[kJobCounter * kCounterStride], 1u);
        __syncthreads();
        uint32_t idx = job;
        __syncthreads();
        if (idx >= n_jobs) break;
        int cls = 0;
        if (idx >= n0) { idx -= n0; cls = 1;
            if (idx >= n1) { idx -= n1; cls = 2;
                if (idx >= n2) { idx -= n2; cls = 3; } } }
        const uint32_t code = list[(size_t)cls * seg_cap + idx];
        const int p = (int)(code >> 8);
        const int q = (int)(code & 0xFF);
        const int m = build_chain(gen, p, q, k_max, M, lane, chain);
        __syncthreads();
        const int r = roles[(size_t)p * k_max + q] != 0;
        const size_t o = (size_t)p * k_max + q;
        const E2Tables tv = mem_view(tb, r);
        uint64_t best = E2_INF64;
        int best_mu = 0, last = 0;
        idle_masters(tv, r, chain, m, E, B, A, S, P, lane, &best, &best_mu);
        for (int pass = 1; pass < 2; ++pass) {
            if (best == E2_INF64) break;
            const int mu_lo = best_mu, mu_hi = best_mu;
            for (int mu = mu_lo; mu <= mu_hi; ++mu) {
                for (int k = 1; k <= m; ++k) {
                    const int c = uni(chain[k - 1]);
                    const bool none_ok = k <= mu;
                    const int kp_lo = k > mu ? mu : 1;
                    const uint64_t *pr = pref_row(tv, r, c);
                    // links into position k from kp < k (lane kp-1; past 64 loaded)
                    const uint64_t tin = lane < k - 1 ? link_tau(tv, r, chain[lane], c) : E2_INF64;
                    for (int x = lane; x <= N; x += kWave) {
                        P[x] = pr[x];
                        uint64_t a = (none_ok && x == 0) ? 0 : E2_INF64;
                        int arg = 0;
#pragma unroll 4
                        for (int kp = kp_lo; kp <= k - 1; ++kp) {
                            const uint64_t e = E[(size_t)(kp - 1) * X + x];
                            const uint64_t tl = kp <= kWave ? readlane_u64(tin, kp - 1)
                                                            : link_tau_u(tv, r, uni(chain[kp - 1]), c);
                            const uint64_t v = umax64(e, tl);  // INF when either is
                            if (v < a) {
                                a = v;
                                arg = kp;
                            }
                        }
                        A[x] = a;
                        if (pass) Ek[(size_t)(k - 1) * X + x] = (uint16_t)arg;
                    }
                    __syncthreads();
                    const int f = (k == mu);
                    const uint8_t *wr = win_row(tv, f, c);
                    const uint64_t hadd = f ? uni64(tv.head[r * M + c]) : 0;
                    const bool empty_ok = f && tv.hfit[c];
                    for (int x = lane; x <= N; x += kWave) {
                        uint64_t e = E2_INF64;
                        int jj = 0;
                        if (x >= 1) {
                            const int w = wr[x - 1];
                            if (w != E2_NO_START) {
                                const uint64_t end = P[x] + hadd;
                                // an INF prefix gives an INF max, which never
                                // passes the strict test
#pragma unroll 4
                                for (int j = w; j < x; ++j) {
                                    const uint64_t v = umax64(A[j], end - P[j]);
                                    if (v < e) {
                                        e = v;
                                        jj = j;
                                    }
                                }
                            }
                        }
                        if (empty_ok && A[x] != E2_INF64) {
                            const uint64_t v = umax64(A[x], hadd);
                            if (v < e) {
                                e = v;
                                jj = x;
                            }
                        }
                        E[(size_t)(k - 1) * X + x] = e;
                        if (pass) Ej[(size_t)(k - 1) * X + x] = (uint8_t)jj;
                    }
                    __builtin_amdgcn_s_waitcnt(0);
                    __threadfence_block();
                    __syncthreads();
                }
                uint64_t tmu = E2_INF64;
                int lk = 0;
                for (int k = mu; k <= m; ++k) {
                    const uint64_t v = E[(size_t)(k - 1) * X + N];
                    if (v < tmu) {
                        tmu = v;
                        lk = k;
                    }
                }
                if (pass == 0 && tmu < best) {
                    best = tmu;
                    best_mu = mu;
                }
                if (pass == 1) last = lk;
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
        for (int k = lane; k < m; k += kWave) sizes[k] = 0;
        __syncthreads();
        if (lane == 0) {
            // back tracing from (last, N): participants in reverse order
            int k = last, x = N, next = 0;
            uint64_t lam = 0;
            while (k >= 1) {
                const int c = chain[k - 1];
                const int j = Ej[(size_t)(k - 1) * X + x];
                sizes[k - 1] = (uint8_t)(x - j);
                const uint64_t *pr = pref_row(tv, r, c);
                lam += pr[x] - pr[j];
                if (k == best_mu) lam += tv.head[r * M + c];
                if (next) lam += link_tau(tv, r, c, chain[next - 1]);
                next = k;
                k = Ek[(size_t)(k - 1) * X + j];
                x = j;
            }
            T[o] = best;
            Lambda[o] = lam;
            if (master) master[o] = (int16_t)chain[best_mu - 1];
        }
        __syncthreads();
        if (layers)
            for (int k = lane; k < m; k += kWave) layers[(size_t)p * M + chain[k]] = sizes[k];
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Fitness (Eq. 3-5): one thread per individual.
// ---------------------------------------------------------------------------
constexpr uint64_t kScale = 1ull << 50;

// Eq. 3-5 from the summed fixed-point rates of the prefill and the decode
// replicas (0 = none usable): S_P = ceil(SCALE / sum_P), S_D = ND *
// ceil(SCALE / sum_D), phase = max(S_P, S_D), w = S_P + (phase - T_a) when
// phase > T_a, else 0; INF without a usable replica of either role.
struct Fit {
    uint64_t w, phase, sp, sd;
};

// ceil(kScale / s) for 1 <= s < 2^58 (a sum of at most 255 rates of at most
// kScale each), without a 64-bit integer division: with n = kScale + s - 1
// the quotient n / s is below 2^51, so its double-precision estimate (three
// roundings of 2^-53 relative) is within 0.75 of it and the truncation is
// the exact floor or one off; the integer checks fix that (every product
// stays below n + 2s < 2^60).
__device__ __forceinline__ uint64_t ceil_scale_div(uint64_t s)
{
    const uint64_t n = kScale + s - 1;
    uint64_t q = (uint64_t)((double)n / (double)s);
    if (q * s > n) {
        q -= 1;
        if (q * s > n) q -= 1;
    } else if ((q + 1) * s <= n) {
        q += 1;
        if ((q + 1) * s <= n) q += 1;
    }
    return q;
}

__device__ __forceinline__ Fit fitness_of_rates(uint64_t sum_p, uint64_t sum_d, uint64_t t_arrival,
                                                uint64_t nd)
{
    Fit f;
    f.sp = sum_p ? ceil_scale_div(sum_p) : E2_INF64;
    f.sd = sum_d ? nd * ceil_scale_div(sum_d) : E2_INF64;
    if (f.sp == E2_INF64 || f.sd == E2_INF64) {
        f.w = f.phase = E2_INF64;
        return f;
    }
    f.phase = umax64(f.sp, f.sd);
    const uint64_t excess = f.phase > t_arrival ? f.phase - t_arrival : 0;
    f.w = excess ? f.sp + excess : 0;
    return f;
}

__global__ __launch_bounds__(256) void k_fitness(int P, int k_max, const uint64_t *__restrict__ T,
                                                 const uint64_t *__restrict__ Lambda,
                                                 const uint8_t *__restrict__ roles,
                                                 uint64_t t_arrival, uint64_t nd,
                                                 uint64_t lambda_max, uint64_t *w, uint64_t *phase,
                                                 uint64_t *s_p, uint64_t *s_d)
{
    // one wave per genome, lanes over clusters
    const int p = blockIdx.x * 4 + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (p >= P) return;
    uint64_t sp = 0, sd = 0;
    for (int q = lane; q < k_max; q += kWave) {
        const size_t o = (size_t)p * k_max + q;
        const uint64_t t = T[o];
        if (t == E2_INF64) continue;
        const bool dec = roles[o] != 0;
        if (dec && Lambda[o] > lambda_max) continue;
        const uint64_t rho = kScale / (t > 0 ? t : 1);
        if (dec) sd += rho;
        else sp += rho;
    }
    sp = wave_sum_u64(sp);
    sd = wave_sum_u64(sd);
    if (lane != 0) return;
    const Fit f = fitness_of_rates(sp, sd, t_arrival, nd);
    if (s_p) s_p[p] = f.sp;
    if (s_d) s_d[p] = f.sd;
    w[p] = f.w;
    phase[p] = f.phase;
}

// ---------------------------------------------------------------------------
// Role and slot search (Algorithm 2's inner loop and its brute-force role
// assignment, policy 0; the adapted-SplitWise rule, policy 1, below): one
// workgroup of four waves per genome.  Thread q < k_max turns cluster q's
// DP results into a prefill rate and, at the largest slot count b that is
// feasible and meets the QoS floor, a decode rate b * SCALE / T_b.  A
// cluster without a decode rate is prefill in every optimum: as decode it
// adds nothing to the decode sum and takes its prefill rate away, which
// never lowers w or phase (Eq. 3-5 fall as the prefill sum grows), and ties
// go to the smaller decode set.  So the workgroup enumerates the role sets
// of the F other ("free") clusters only: each thread fixes the low eight
// bits of the set and runs the high bits in Gray-code order, keeps its
// smallest (w, phase, set), and a reduction picks the overall smallest.  A
// genome with more than kMaxFree free clusters is not searched.
// ---------------------------------------------------------------------------
constexpr int kRolesThreads = 256;
constexpr int kRolesLowBits = 8;  // log2(kRolesThreads)
constexpr int kMaxFree = e2_search_max_free;

struct Best {
    uint64_t w, phase;
    uint32_t mask;
};

__device__ __forceinline__ bool best_less(const Best &a, const Best &b)
{
    if (a.w != b.w) return a.w < b.w;
    if (a.phase != b.phase) return a.phase < b.phase;
    return a.mask < b.mask;
}

__device__ __forceinline__ Best wave_min_best(Best best)
{
    for (int off = kWave / 2; off >= 1; off >>= 1) {
        Best o;
        o.w = __shfl_xor(best.w, off, kWave);
        o.phase = __shfl_xor(best.phase, off, kWave);
        o.mask = __shfl_xor(best.mask, off, kWave);
        if (best_less(o, best)) best = o;
    }
    return best;
}

__global__ __launch_bounds__(kRolesThreads) void k_roles(
    int P, int M, int k_max, int R, int policy, uint32_t np_tokens,
    const uint8_t *__restrict__ labels, const uint64_t *__restrict__ T_all,
    const uint64_t *__restrict__ L_all, uint64_t t_arrival, uint64_t nd, uint64_t lambda_max,
    uint8_t *roles_out, uint8_t *slots_out, uint64_t *w, uint64_t *phase)
{
    __shared__ uint64_t rho_p[256], rho_d[256];
    __shared__ uint32_t bstar[256];
    __shared__ uint32_t used[8];
    __shared__ uint64_t free_d[kMaxFree], free_p[kMaxFree];  // the free clusters' rates
    __shared__ uint8_t free_q[kMaxFree];                       // and ids, increasing
    __shared__ uint8_t dec[256];
    __shared__ int n_free;
    __shared__ uint64_t fixed_p;  // prefill rates of the clusters that are not free
    __shared__ Best wave_best[kRolesThreads / kWave];
    const int p = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wv = tid / kWave;
    if (tid < 8) used[tid] = 0;
    for (int q = tid; q < k_max; q += kRolesThreads) {
        const uint64_t *Tq = T_all + ((size_t)p * k_max + q) * R;
        const uint64_t *Lq = L_all + ((size_t)p * k_max + q) * R;
        const uint64_t t0 = Tq[0];
        rho_p[q] = t0 != E2_INF64 ? kScale / (t0 > 0 ? t0 : 1) : 0;
        uint32_t bs = 0;
        uint64_t rd = 0;
        for (int b = R - 1; b >= 1; --b) {
            const uint64_t tb = Tq[b];
            if (tb != E2_INF64 && Lq[b] <= lambda_max) {
                bs = (uint32_t)b;
                rd = ((uint64_t)b * kScale) / (tb > 0 ? tb : 1);
                break;
            }
        }
        rho_d[q] = rd;
        bstar[q] = bs;
        dec[q] = 0;
    }
    __syncthreads();
    if (policy == 1) {
        // adapted SplitWise: the token ratio sets the prefill count, the
        // highest prefill rates (ties to the smaller cluster id) take it
        for (int d = tid; d < M; d += kRolesThreads) {
            const int lab = labels[(size_t)p * M + d];
            if (lab < k_max) atomicOr(&used[lab >> 5], 1u << (lab & 31));
        }
        __syncthreads();
        if (wv != 0) return;
        int n_used = 0;
        for (int i = 0; i < 8; ++i) n_used += __popc(used[i]);
        int n_p = n_used;
        if (n_used >= 2) {
            const uint64_t tot = (uint64_t)np_tokens + nd;
            n_p = tot ? (int)((2 * (uint64_t)n_used * np_tokens + tot) / (2 * tot))
                      : (n_used + 1) / 2;
            n_p = n_p < 1 ? 1 : (n_p > n_used - 1 ? n_used - 1 : n_p);
        }
        uint64_t sp = 0, sd = 0;
        for (int q = lane; q < k_max; q += kWave) {
            uint32_t role = 0;
            if ((used[q >> 5] >> (q & 31)) & 1u) {
                int rank = 0;
                for (int k = 0; k < k_max; ++k) {
                    if (!((used[k >> 5] >> (k & 31)) & 1u)) continue;
                    rank += rho_p[k] > rho_p[q] || (rho_p[k] == rho_p[q] && k < q);
                }
                role = rank >= n_p;
                if (role) sd += rho_d[q];
                else sp += rho_p[q];
            }
            roles_out[(size_t)p * k_max + q] = (uint8_t)role;
            slots_out[(size_t)p * k_max + q] = (uint8_t)(role ? bstar[q] : 0);
        }
        sp = wave_sum_u64(sp);
        sd = wave_sum_u64(sd);
        if (lane == 0) {
            const Fit f = fitness_of_rates(sp, sd, t_arrival, nd);
            w[p] = f.w;
            phase[p] = f.phase;
        }
        return;
    }
    // brute force over the free clusters (a decode rate), listed in
    // increasing q by wave 0; the others are prefill
    if (wv == 0) {
        int F = 0;
        uint64_t fixed = 0;
        for (int base = 0; base < k_max; base += kWave) {
            const int q = base + lane;
            const bool in = q < k_max;
            const bool is_free = in && rho_d[q] != 0;
            const uint64_t bal = __ballot(is_free);
            if (is_free) {
                const int pos = F + (int)__popcll(bal & ((1ull << lane) - 1));
                if (pos < kMaxFree) {
                    free_q[pos] = (uint8_t)q;
                    free_d[pos] = rho_d[q];
                    free_p[pos] = rho_p[q];
                }
            } else if (in) {
                fixed += rho_p[q];
            }
            F += (int)__popcll(bal);
        }
        fixed = wave_sum_u64(fixed);
        if (lane == 0) {
            n_free = F;
            fixed_p = fixed;
        }
    }
    __syncthreads();
    const int F = n_free;
    if (F > kMaxFree) {  // not searched
        for (int q = tid; q < k_max; q += kRolesThreads) {
            roles_out[(size_t)p * k_max + q] = 0;
            slots_out[(size_t)p * k_max + q] = 0xFF;
        }
        if (tid == 0) w[p] = phase[p] = E2_INF64;
        return;
    }
    // A role set is x in [0, 2^F): bit i makes free cluster i decode.  x
    // orders sets as their decode bitmasks over q do (the free clusters are
    // listed in increasing q), so (w, phase, x) picks the same set as (w,
    // phase, mask), whatever order the sets are visited in.  Thread tid
    // holds the low bits of x; each Gray-code step of the high bits adds or
    // removes one cluster's rates.
    uint64_t p_all = fixed_p;  // every cluster prefill
    for (int i = 0; i < F; ++i) p_all += free_p[i];
    const int low = F < kRolesLowBits ? F : kRolesLowBits;
    Best best = {E2_INF64, E2_INF64, 0xFFFFFFFFu};
    if ((uint32_t)tid < (1u << low)) {
        uint64_t sd = 0, sxp = 0;  // decode and prefill rates of x's members
        for (int i = 0; i < low; ++i) {
            if ((tid >> i) & 1) {
                sd += free_d[i];
                sxp += free_p[i];
            }
        }
        uint32_t g = 0;  // high bits of x
        const uint32_t n_high = 1u << (F - low);
        for (uint32_t t = 0; t < n_high; ++t) {
            if (t) {
                const int bt = __builtin_ctz(t);
                const uint64_t d = free_d[bt + kRolesLowBits], pp = free_p[bt + kRolesLowBits];
                g ^= 1u << bt;
                if ((g >> bt) & 1u) {
                    sd += d;
                    sxp += pp;
                } else {
                    sd -= d;
                    sxp -= pp;
                }
            }
            const Fit f = fitness_of_rates(p_all - sxp, sd, t_arrival, nd);
            const Best c = {f.w, f.phase, (uint32_t)tid | (g << kRolesLowBits)};
            if (best_less(c, best)) best = c;
        }
    }
    best = wave_min_best(best);
    if (lane == 0) wave_best[wv] = best;
    __syncthreads();
    if (tid == 0) {
        for (int i = 1; i < kRolesThreads / kWave; ++i)
            if (best_less(wave_best[i], best)) best = wave_best[i];
        for (int i = 0; i < F; ++i)
            if ((best.mask >> i) & 1u) dec[free_q[i]] = 1;
        w[p] = best.w;
        phase[p] = best.phase;
    }
    __syncthreads();
    for (int q = tid; q < k_max; q += kRolesThreads) {
        roles_out[(size_t)p * k_max + q] = dec[q];
        slots_out[(size_t)p * k_max + q] = (uint8_t)(dec[q] ? bstar[q] : 0);
    }
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

// (w, phase, index) order of two keys held in registers
__device__ __forceinline__ bool kless(uint64_t wa, uint64_t pa, uint32_t ia, uint64_t wb,
                                      uint64_t pb, uint32_t ib)
{
    if (wa != wb) return wa < wb;
    if (pa != pb) return pa < pb;
    return ia < ib;
}

// The least key of the 32 lanes of each half-wave, in every lane of the half
// (xor shuffles that stay within the half).  The sentinel (all ones, index
// 0xFFFFFFFF) loses to every key of a genome.
__device__ __forceinline__ void half_wave_min_key(uint64_t &bw, uint64_t &bp, uint32_t &bi)
{
#pragma unroll
    for (int o = 16; o >= 1; o >>= 1) {
        const uint64_t ow = __shfl_xor(bw, o, kWave), op = __shfl_xor(bp, o, kWave);
        const uint32_t oi = __shfl_xor(bi, o, kWave);
        if (kless(ow, op, oi, bw, bp, bi)) {
            bw = ow;
            bp = op;
            bi = oi;
        }
    }
}

// Tournament selection of both parents: parent a takes the least key among
// its tk draws (draw t from stream kStSelA + t), parent b among its own
// (stream kStSelB + t).  Lanes 0-31 hold a's draws, lanes 32-63 b's (two per
// lane when tk > 32), so that every draw's key is loaded at once; the least
// key of a set does not depend on the order of its draws.
__device__ __forceinline__ void tournament_pair(const uint64_t *__restrict__ w,
                                                const uint64_t *__restrict__ ph, uint64_t hs,
                                                uint32_t P, uint32_t tk, int lane, uint32_t &a,
                                                uint32_t &b)
{
    const uint32_t st0 = lane < 32 ? kStSelA : kStSelB;
    uint64_t bw = ~0ull, bp = ~0ull;
    uint32_t bi = 0xFFFFFFFFu;
    for (uint32_t t = (uint32_t)(lane & 31); t < tk; t += 32) {
        const uint64_t u = sm64(sm64(hs ^ (uint64_t)(st0 + t)) ^ 0ull);
        const uint32_t idx = (uint32_t)(((u >> 32) * (uint64_t)P) >> 32);
        const uint64_t kw = w[idx], kp = ph[idx];
        if (kless(kw, kp, idx, bw, bp, bi)) {
            bw = kw;
            bp = kp;
            bi = idx;
        }
    }
    half_wave_min_key(bw, bp, bi);
    a = (uint32_t)__builtin_amdgcn_readlane((int)bi, 0);
    b = (uint32_t)__builtin_amdgcn_readlane((int)bi, 32);
}

// n_elite rounds of "smallest key strictly after the previous pick".  Each
// thread holds up to kEliteKeys keys in registers (populations of up to
// 16384 genomes; larger ones read theirs every round); a round reduces over
// each wave with shuffles and over the 16 waves through LDS.
constexpr int kEliteThreads = 1024, kEliteKeys = 16;
__global__ __launch_bounds__(kEliteThreads) void k_elites(int P, uint32_t n_elite,
                                                          const uint64_t *__restrict__ w,
                                                          const uint64_t *__restrict__ ph,
                                                          uint32_t *elite)
{
    constexpr int kWaves = kEliteThreads / kWave;
    __shared__ uint64_t rw[kWaves], rp[kWaves];
    __shared__ uint32_t ri[kWaves];
    const int t = threadIdx.x, lane = t % kWave, wv = t / kWave;
    const bool held = P <= kEliteThreads * kEliteKeys;
    uint64_t kw[kEliteKeys], kp[kEliteKeys];
    if (held) {
#pragma unroll
        for (int i = 0; i < kEliteKeys; ++i) {
            const int p = min(t + kEliteThreads * i, P - 1);  // in-range loads, no branch
            kw[i] = w[p];
            kp[i] = ph[p];
        }
    }
    bool have_last = false;  // no previous pick: every key qualifies
    uint64_t lw = 0, lp = 0;
    uint32_t li = 0;
    for (uint32_t e = 0; e < n_elite; ++e) {
        uint64_t bw = ~0ull, bp = ~0ull;
        uint32_t bi = 0xFFFFFFFFu;
        if (held) {
#pragma unroll
            for (int i = 0; i < kEliteKeys; ++i) {
                const uint32_t p = (uint32_t)(t + kEliteThreads * i);
                if (p < (uint32_t)P && (!have_last || kless(lw, lp, li, kw[i], kp[i], p)) &&
                    kless(kw[i], kp[i], p, bw, bp, bi)) {
                    bw = kw[i];
                    bp = kp[i];
                    bi = p;
                }
            }
        } else {
            for (int p = t; p < P; p += kEliteThreads) {
                const uint64_t xw = w[p], xp = ph[p];
                if ((!have_last || kless(lw, lp, li, xw, xp, (uint32_t)p)) &&
                    kless(xw, xp, (uint32_t)p, bw, bp, bi)) {
                    bw = xw;
                    bp = xp;
                    bi = (uint32_t)p;
                }
            }
        }
        half_wave_min_key(bw, bp, bi);
        {  // the two halves of the wave
            const uint64_t ow = __shfl_xor(bw, 32, kWave), op = __shfl_xor(bp, 32, kWave);
            const uint32_t oi = __shfl_xor(bi, 32, kWave);
            if (kless(ow, op, oi, bw, bp, bi)) {
                bw = ow;
                bp = op;
                bi = oi;
            }
        }
        if (lane == 0) {
            rw[wv] = bw;
            rp[wv] = bp;
            ri[wv] = bi;
        }
        __syncthreads();
        bw = rw[0];
        bp = rp[0];
        bi = ri[0];
        for (int j = 1; j < kWaves; ++j)
            if (kless(rw[j], rp[j], ri[j], bw, bp, bi)) {
                bw = rw[j];
                bp = rp[j];
                bi = ri[j];
            }
        __syncthreads();  // every thread has read the wave results
        if (t == 0) elite[e] = bi;
        have_last = bi != 0xFFFFFFFFu;
        lw = bw;
        lp = bp;
        li = bi;
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
    uint32_t a, b;
    tournament_pair(w, ph, hs, (uint32_t)P, tk, lane, a, b);
    const uint64_t h_xl = sm64(hs ^ kStXoLabel), h_ml = sm64(hs ^ kStMutLabel);
    const uint64_t h_xr = sm64(hs ^ kStXoRole), h_mr = sm64(hs ^ kStMutRole);
    // every gene's parent byte is loaded before any is used (gene lane + 64 t
    // in slot t; clamped indices past the row, whose results are not stored)
    constexpr int kSlots = (E2_MAX_DEV + kWave - 1) / kWave;
    uint8_t pl[kSlots], pr[kSlots];
#pragma unroll
    for (int t = 0; t < kSlots; ++t) {
        const int d = lane + kWave * t;
        const uint32_t src = (uint32_t)sm64(h_xl ^ (uint64_t)d) < xo ? b : a;
        pl[t] = labels_in[(size_t)src * M + min(d, M - 1)];
        const uint32_t srq = (uint32_t)sm64(h_xr ^ (uint64_t)d) < xo ? b : a;
        pr[t] = roles_in[(size_t)srq * k_max + min(d, k_max - 1)];
    }
#pragma unroll
    for (int t = 0; t < kSlots; ++t) {
        const int d = lane + kWave * t;
        if (d < M) {
            uint8_t v = pl[t];
            const uint64_t z = sm64(h_ml ^ (uint64_t)d);
            if ((uint32_t)(z >> 32) < mut) v = (uint8_t)(((uint64_t)(uint32_t)z * (uint64_t)k_max) >> 32);
            lo[d] = v;
        }
        if (d < k_max) {
            uint8_t v = pr[t] != 0;
            const uint64_t z = sm64(h_mr ^ (uint64_t)d);
            if ((uint32_t)(z >> 32) < mut) v ^= 1u;
            ro[d] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// Two-chromosome GA (App. A): an ordering chromosome (a permutation of the
// devices) and replica sizes, with a role per replica.  One wave per output
// slot: elite copy, or tournaments (as above), ordering crossover with
// repair, the grouping and roles of one parent, and with about 30%
// probability one of four mutations.
// ---------------------------------------------------------------------------
constexpr uint32_t kStOCut = 140, kStOGroup = 141, kStOMut = 142, kStOSwap = 143,
                   kStORegen = 144, kStOSize = 145, kStOPerm = 146;
// mutation kinds as fractions of 2^32: swap 0.20, regrow from a replica
// 0.50, regrow the whole grouping 0.15, new ordering and grouping 0.15
constexpr uint32_t kMutSwapBelow = 858993459u, kMutRegrowBelow = 3006477107u,
                   kMutAllGroupBelow = 3650722201u;

__device__ __forceinline__ uint64_t rng_at(uint64_t hs, uint32_t stream, uint64_t gene)
{
    return sm64(sm64(hs ^ (uint64_t)stream) ^ gene);
}

__global__ __launch_bounds__(64) void k_breed_ordered(
    int M, int P, int k_max, const uint8_t *__restrict__ order_in,
    const uint16_t *__restrict__ sizes_in, const uint8_t *__restrict__ roles_in,
    const uint64_t *__restrict__ w, const uint64_t *__restrict__ ph, uint64_t seed, uint32_t g,
    uint32_t tk, uint32_t mut, uint32_t n_elite, uint32_t max_replica,
    const uint32_t *__restrict__ elite, uint8_t *order_out, uint16_t *sizes_out,
    uint8_t *roles_out)
{
    __shared__ uint8_t child[256];
    __shared__ uint8_t fill[256];
    __shared__ uint32_t used[8];
    __shared__ uint16_t szs[256];
    __shared__ uint8_t rls[256];
    __shared__ uint64_t draw[256];  // size / role draws of a regrowth
    __shared__ uint8_t pj[256];     // swap partners of a new ordering
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    if ((uint32_t)s < n_elite) {
        const uint32_t src = elite[s];
        for (int t = lane; t < M; t += kWave)
            order_out[(size_t)s * M + t] = order_in[(size_t)src * M + t];
        for (int r = lane; r < k_max; r += kWave) {
            sizes_out[(size_t)s * k_max + r] = sizes_in[(size_t)src * k_max + r];
            roles_out[(size_t)s * k_max + r] = roles_in[(size_t)src * k_max + r];
        }
        return;
    }
    const uint64_t hs = sm64(sm64(seed ^ (uint64_t)g) ^ (uint64_t)s);  // (seed, g, s) prefix
    uint32_t a, b;
    tournament_pair(w, ph, hs, (uint32_t)P, tk, lane, a, b);
    const uint8_t *A = order_in + (size_t)a * M;
    const uint8_t *B = order_in + (size_t)b * M;
    const uint64_t lt = (1ull << lane) - 1;

    // ordering crossover at c: a's prefix, then b's positions; b's nodes
    // already in the prefix become holes, filled with b's prefix nodes that
    // are missing, in b's order (M = 1: the child copies a)
    if (lane < 8) used[lane] = 0;
    __syncthreads();
    int c = M;
    if (M >= 2) {
        const uint64_t u = rng_at(hs, kStOCut, 0);
        c = 1 + (int)((((uint64_t)(uint32_t)u) * (uint64_t)(M - 1)) >> 32);
    }
    for (int t = lane; t < c; t += kWave) {
        const uint32_t x = A[t];
        child[t] = (uint8_t)x;
        atomicOr(&used[x >> 5], 1u << (x & 31));
    }
    __syncthreads();
    uint32_t nfill = 0;
    for (int base = 0; base < c; base += kWave) {
        const int t = base + lane;
        bool f = false;
        uint32_t x = 0;
        if (t < c) {
            x = B[t];
            f = !((used[x >> 5] >> (x & 31)) & 1u);
        }
        const uint64_t mask = __ballot(f);
        if (f) fill[nfill + __popcll(mask & lt)] = (uint8_t)x;
        nfill += __popcll(mask);
    }
    __syncthreads();
    uint32_t nh = 0;
    for (int base = c; base < M; base += kWave) {
        const int t = base + lane;
        bool h = false;
        uint32_t x = 0;
        if (t < M) {
            x = B[t];
            h = (used[x >> 5] >> (x & 31)) & 1u;
        }
        const uint64_t mask = __ballot(h);
        if (t < M) {
            const uint32_t k = nh + __popcll(mask & lt);
            child[t] = h ? fill[k < nfill ? k : 0] : (uint8_t)x;
        }
        nh += __popcll(mask);
    }
    // grouping and roles of one parent
    const uint64_t ug = rng_at(hs, kStOGroup, 0);
    const uint32_t src = ((uint32_t)ug < 0x80000000u) ? b : a;
    for (int r = lane; r < k_max; r += kWave) {
        szs[r] = sizes_in[(size_t)src * k_max + r];
        rls[r] = roles_in[(size_t)src * k_max + r] != 0;
    }
    __syncthreads();
    const uint64_t um = rng_at(hs, kStOMut, 0);
    const bool mutate = (uint32_t)(um >> 32) < mut;
    const uint32_t kind = (uint32_t)um;
    if (mutate && kind >= kMutSwapBelow) {
        // the draws of the regrowth (and of a new ordering) are independent
        // counter-based values: all lanes compute them, lane 0 then runs the
        // sequential steps on them
        const uint64_t h_size = sm64(hs ^ (uint64_t)kStOSize);
        for (int r = lane; r < k_max; r += kWave) draw[r] = sm64(h_size ^ (uint64_t)r);
        if (kind >= kMutAllGroupBelow) {
            const uint64_t h_perm = sm64(hs ^ (uint64_t)kStOPerm);
            for (int t = lane; t < M; t += kWave) {
                const uint64_t v = sm64(h_perm ^ (uint64_t)t);
                pj[t] = (uint8_t)(((v >> 32) * (uint64_t)(t + 1)) >> 32);
            }
        }
        __syncthreads();
    }
    if (mutate && lane == 0) {
        if (kind < kMutSwapBelow) {
            const uint64_t v = rng_at(hs, kStOSwap, 0);
            const int i = (int)(((v >> 32) * (uint64_t)M) >> 32);
            const int j = (int)((((uint64_t)(uint32_t)v) * (uint64_t)M) >> 32);
            const uint8_t x = child[i];
            child[i] = child[j];
            child[j] = x;
        } else {
            int pos = 0;
            if (kind < kMutRegrowBelow) {
                // replicas that hold devices, then a uniform one among them
                int R = 0;
                long off = 0;
                for (int r = 0; r < k_max; ++r) {
                    if (szs[r] == 0 || off >= M) break;
                    off += szs[r];
                    ++R;
                }
                const uint64_t v = rng_at(hs, kStORegen, 0);
                pos = (int)(((v >> 32) * (uint64_t)R) >> 32);
            } else if (kind >= kMutAllGroupBelow) {
                // a new ordering: Fisher-Yates from the identity
                for (int t = 0; t < M; ++t) child[t] = (uint8_t)t;
                for (int t = M - 1; t >= 1; --t) {
                    const int j = pj[t];
                    const uint8_t x = child[t];
                    child[t] = child[j];
                    child[j] = x;
                }
            }
            // regrow the grouping from replica pos
            long remaining = M;
            for (int r = 0; r < pos; ++r) remaining -= szs[r];
            if (remaining < 0) remaining = 0;
            int r = pos;
            while (remaining > 0 && r < k_max) {
                const uint64_t u = draw[r];
                long sz = 1 + (long)(((u >> 32) * (uint64_t)max_replica) >> 32);
                if (r == k_max - 1 || sz > remaining) sz = remaining;
                szs[r] = (uint16_t)sz;
                rls[r] = (uint32_t)u >= 0x80000000u;
                remaining -= sz;
                ++r;
            }
            for (; r < k_max; ++r) {
                szs[r] = 0;
                rls[r] = 0;
            }
        }
    }
    __syncthreads();
    for (int t = lane; t < M; t += kWave) order_out[(size_t)s * M + t] = child[t];
    for (int r = lane; r < k_max; r += kWave) {
        sizes_out[(size_t)s * k_max + r] = szs[r];
        roles_out[(size_t)s * k_max + r] = rls[r];
    }
}

}  // namespace

int e2_dp_pool_cells(int N)
{
    // the forward bands of a chain of m devices hold at most
    // (m-1)(N-m+1) cells (band k lies in [k-1, N-1-(m-k)]); the pool takes
    // the largest such count over the chains the banded path accepts
    int best = 0;
    for (int m = 2; m <= kMaxBandedChain && m <= N; ++m) best = max(best, (m - 1) * (N - m + 1));
    return max(best, kLdsTbCells);
}

int e2_dp_idle_slots(int problems, int M, int N)
{
    // every wave holds 2 M x (N+1) rows in its own global region: as many
    // waves as 1 GiB of regions allows, at least 256 and at most 4096
    const size_t budget = (size_t)1 << 30;
    size_t cap = budget / e2_dp_idle_bytes(M, N);
    cap = cap < 256 ? 256 : (cap > 4096 ? 4096 : cap);
    return problems < (int)cap ? (problems > 0 ? problems : 1) : (int)cap;
}

size_t e2_dp_idle_bytes(int M, int N)
{
    // forward and reversed rows (u64), predecessors (u16), stage starts (u8)
    return ((size_t)M * (N + 1) * 19 + 255) & ~(size_t)255;
}

int e2_dp_lds_tb_cells(int N)
{
    (void)N;
    return kLdsTbCells;
}


size_t e2_dp_lds_bytes(int N) { return (size_t)dp_lds_fixed(N) + (size_t)dp_lds_extra(N); }

int e2_dp_slots(int N, int problems)
{
    // resident one-wave workgroups per CU for this LDS size (the occupancy
    // the compiled kernel reaches), times the CUs of the device; cached,
    // and threads that race here compute and store the same values
    static std::atomic<int> per_cu[256];
    static std::atomic<int> n_cu{0};
    if (N < 1 || N > 255) return 1;
    int cus = n_cu.load(std::memory_order_relaxed);
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                hipSuccess ||
            cus < 1) {
            (void)hipGetLastError();
            cus = 256;
        }
        n_cu.store(cus, std::memory_order_relaxed);
    }
    int nb = per_cu[N].load(std::memory_order_relaxed);
    if (nb == 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_dp, 64, e2_dp_lds_bytes(N)) !=
                hipSuccess ||
            nb < 1) {
            (void)hipGetLastError();
            nb = 20;
        }
        nb = nb > 32 ? 32 : nb;
        per_cu[N].store(nb, std::memory_order_relaxed);
    }
    const int cap = cus * nb;
    return problems < cap ? (problems > 0 ? problems : 1) : cap;
}

hipError_t e2_launch_partitions(const E2Tables &t, hipStream_t s, int P, int k_max,
                                const E2Genomes &gen, const uint8_t *roles, const E2Work &wk,
                                uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers,
                                int objective)
{
    // without roles, every role index of every cluster
    const int n_r = roles ? 0 : t.R;
    const size_t seg = (size_t)P * k_max * (n_r ? n_r : 1);
    k_init<<<1, 64, 0, s>>>(wk.counters);
    // Chains longer than the one-register table go to the long-chain kernel
    // when they are plausible: more devices than that, at least 16 per
    // cluster id on average.  Otherwise (no launch to pay for) the rare long
    // chain takes k_dp's reference path; the results are the same.
    const bool long_seg = objective == 0 && t.M > kMaxBandedChain && t.M >= 16 * k_max;
    const bool ord = gen.labels == nullptr;
    const auto extract = ord ? (n_r ? k_extract<true, true> : k_extract<true, false>)
                             : (n_r ? k_extract<false, true> : k_extract<false, false>);
    const int eg = n_r ? eg_of<true>() : eg_of<false>();
    extract<<<(P + eg - 1) / eg, 64 * eg, 0, s>>>(t, P, k_max, gen, roles, n_r, objective == 2,
                                                   long_seg, wk.counters, wk.list, seg, T,
                                                   Lambda, master, layers);
    const int pool = e2_dp_pool_cells(t.N);
    if (wk.ev_begin) (void)hipEventRecord(wk.ev_begin, s);
    if (objective == 2)
        k_dp_idle<<<wk.n_slots, 64, (size_t)(t.N + 1) * 24, s>>>(t, k_max, gen, roles, wk.counters,
                                                                wk.list, seg, wk.idle,
                                                                wk.idle_stride, T, Lambda,
                                                                master, layers);
    else if (objective == 1)
        k_dp_ft<<<wk.n_slots, 64, e2_dp_lds_bytes(t.N), s>>>(t, k_max, pool, gen, roles,
                                                          wk.counters, wk.list, seg, wk.tb_global,
                                                          T, Lambda, master, layers);
    else {
        k_dp<<<wk.n_slots, 64, e2_dp_lds_bytes(t.N), s>>>(t, k_max, pool, gen, roles, n_r,
                                                          wk.counters, wk.list, seg, wk.tb_global,
                                                          T, Lambda, master, layers);
        // the long chains, if any (each wave exits at once when there are none)
        if (long_seg)
            k_dp_long<<<wk.n_slots < 256 ? wk.n_slots : 256, 64, e2_dp_lds_bytes(t.N), s>>>(
                t, k_max, pool, gen, roles, n_r, wk.counters, wk.list, seg, wk.tb_global, T,
                Lambda, master, layers);
    }
    if (wk.ev_end) (void)hipEventRecord(wk.ev_end, s);
    return hipGetLastError();
}

hipError_t e2_launch_fitness(hipStream_t s, int P, int k_max, const uint64_t *T,
                             const uint64_t *Lambda, const uint8_t *roles, uint64_t t_arrival,
                             uint64_t nd, uint64_t lambda_max, uint64_t *w, uint64_t *phase,
                             uint64_t *s_p, uint64_t *s_d)
{
    k_fitness<<<(P + 3) / 4, 256, 0, s>>>(P, k_max, T, Lambda, roles, t_arrival, nd,
                                              lambda_max, w, phase, s_p, s_d);
    return hipGetLastError();
}

hipError_t e2_launch_roles(hipStream_t s, int P, int M, int k_max, int R, int policy,
                           uint32_t np_tokens, const uint8_t *labels, const uint64_t *T_all,
                           const uint64_t *L_all, uint64_t t_arrival, uint64_t nd,
                           uint64_t lambda_max, uint8_t *roles_out, uint8_t *slots_out,
                           uint64_t *w, uint64_t *phase)
{
    k_roles<<<P, kRolesThreads, 0, s>>>(P, M, k_max, R, policy, np_tokens, labels, T_all, L_all, t_arrival,
                             nd, lambda_max, roles_out, slots_out, w, phase);
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

hipError_t e2_launch_ga_ordered(hipStream_t s, int M, int P, int k_max, const uint8_t *order_in,
                                const uint16_t *sizes_in, const uint8_t *roles_in,
                                const uint64_t *w, const uint64_t *phase, uint64_t seed,
                                uint32_t generation, uint32_t tournament_k, uint32_t mut_thresh,
                                uint32_t n_elite, uint32_t max_replica, uint32_t *elite_scratch,
                                uint8_t *order_out, uint16_t *sizes_out, uint8_t *roles_out)
{
    if (n_elite > 0) k_elites<<<1, 1024, 0, s>>>(P, n_elite, w, phase, elite_scratch);
    k_breed_ordered<<<P, 64, 0, s>>>(M, P, k_max, order_in, sizes_in, roles_in, w, phase, seed,
                                     generation, tournament_k, mut_thresh, n_elite, max_replica,
                                     elite_scratch, order_out, sizes_out, roles_out);
    return hipGetLastError();
}
