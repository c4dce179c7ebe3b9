// Internal declarations shared by the host API (e2_api.hip) and the kernels
// (e2_kernels.hip) of libe2.so.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define E2_INF64 0xFFFFFFFFFFFFFFFFull
#define E2_NO_START 0xFFu  // window table: no stage ending at i fits

// Read-only device tables built once per context.  Role index r: 0 =
// prefill, b = 1..R-1 = decode with b requests in flight (R = 2 without a
// slot model).  Memory tables exist per memory class: one shared class
// (n_mem = 1, no KV bytes) or one per role index (n_mem = R, block bytes
// W[n] + kv * slots(r)); the [C] below is that class.
// Byte layout of a prefix row block (per role index r and device c, N+1
// entries in each part): the prefix sums of block times P (u64), the same
// over reversed blocks PR[x] = P[N] - P[N-x] (u64), P x 256 and PR x 256 as
// doubles (exact below 2^45, the only range the fp64 DP keys use), and
// P << 8 and PR << 8 modulo 2^32 (32-bit DP keys).  One block per (r, c), so
// that a row of the DP finds every part from one base and the row index.
constexpr int kRowPref = 0, kRowPrefR = 8, kRowPref8d = 16, kRowPrefR8d = 24, kRowPref8u = 32,
              kRowPrefR8u = 36, kRowBlock = 40;  // bytes per entry of N+1

struct E2Tables {
    const uint8_t *prow;   // [R][M] prefix row blocks of kRowBlock x (N+1) bytes (above)
    const uint64_t *head;  // [R][M] head + output-layer time per role and device
    const uint64_t *tau;   // [R][M][M] link time per role, INF for a dead link
    const uint8_t *wtab;   // [C] memory-window blocks of 6 M N bytes, each
                           //   [2][M][N] win: smallest stage start j so that blocks
                           //     j..i fit ([0]: no head bytes, [1]: with head bytes),
                           //     E2_NO_START if none;
                           //   [2][M][N] minwin: lower bound of window lengths
                           //     i - win(i) + 1 over cells i >= x (0 if unknown);
                           //   [M][N] winR: reversed-block window starts without the
                           //     head (smallest y so that reversed blocks y..x fit);
                           //   [M][N] minwinR: minwin of winR
    const uint8_t *cap0;   // [C][M] most blocks one stage can hold without the head
    const uint8_t *capH;   // [C][M] most blocks one stage can hold with the head
    const uint64_t *vmax;  // [R][M] largest cost of a fitting stage (+ head time when it
                           //   holds the head bytes) per role and device
    const uint64_t *vtot;  // [R][M] total time of all blocks + head time per role and device
    const uint8_t *hfit;   // [M] 1 when the head bytes alone fit the device
    int M;
    int N;
    int R;      // role indices
    int n_mem;  // memory classes: 1 or R
};

struct e2_ctx {
    int device;
    int M, N;
    int b_max;  // decode slot counts of the slot model (1 without one)
    uint64_t head_bytes;
    void *blob;  // one device allocation holding every table
    E2Tables tables;
    // DP launch timing (profiling): event pairs and how many are recorded
    hipEvent_t *dp_events;
    int dp_event_pairs;
    int dp_events_used;
    // device scratch kept per stream between calls (host API only)
    struct ScratchCache *scratch_cache;
};

// Per-call counters, each on a 256-byte line of its own so that the
// extraction's atomics on different counters do not serialise on one line.
constexpr int kCounters = 7;        // 0..4: problems listed per list segment, 5: next job,
constexpr int kCounterStride = 64;  // 6: next job of the long-chain kernel (u32 stride)
constexpr int kListSegs = 5;        // chain-length classes m >= 16, 12..15, 8..11, < 8, and
                                    // (bottleneck objective only) m > 64
constexpr int kJobCounter = 5;
constexpr int kLongJobCounter = 6;
constexpr size_t kCounterBytes = (size_t)kCounters * kCounterStride * 4;

// Scratch layout of one solve/eval call (device memory, stream-ordered).
struct E2Work {
    uint32_t *counters;  // [c * kCounterStride], one 256-byte line each (see kCounters)
    uint32_t *list;      // [kListSegs][P * k_max * n_r] problems needing the DP: (p << 8) | q, or
                         //   with every role index searched (p << 12) | (q << 4) | r
    uint8_t *tb_global;  // [n_slots][N][N] split-point table fallback, or null
    int n_slots;         // waves of the DP kernel
    uint8_t *idle;       // idle-device relaxation: per wave, rows E [M][N+1] u64, their
    size_t idle_stride;  //   predecessors [M][N+1] u16 and stage starts [M][N+1] u8
    hipEvent_t ev_begin; // recorded just before / after the DP kernel, or null
    hipEvent_t ev_end;
};

// Number of DP waves launched for at most `problems` problems of N blocks.
int e2_dp_slots(int N, int problems);
// Largest band total of a chain the one-register table takes, the LDS copy
// of the split points (bytes) and the DP kernels' dynamic LDS bytes.
int e2_dp_pool_cells(int N);
int e2_dp_lds_tb_cells(int N);
size_t e2_dp_lds_bytes(int N);
// Waves and per-wave bytes of the idle-device relaxation's DP kernel.
int e2_dp_idle_slots(int problems, int M, int N);
size_t e2_dp_idle_bytes(int M, int N);

// The genomes of a population: labels [P][M] (cluster id per device), or,
// when labels is null, two-chromosome genomes: an ordering order [P][M] and
// replica sizes [P][k_max].
struct E2Genomes {
    const uint8_t *labels;
    const uint8_t *order;
    const uint16_t *sizes;
};

// Enqueue cluster extraction + DP.  Outputs may be the caller's (solve) or
// scratch (eval; master/layers null).  With roles null, every cluster is
// solved for every role index (R <= 16, P < 2^20) and T, Lambda are
// [P][k_max][R]; master and layers must then be null.
// objective 1: the finishing-time variant (least end-to-end time per
// cluster; T reports that partition's bottleneck); objective 2: the
// idle-device relaxation (wk.idle must be set).  Both with roles only.
hipError_t e2_launch_partitions(const E2Tables &t, hipStream_t s, int P, int k_max,
                                const E2Genomes &gen, const uint8_t *roles, const E2Work &wk,
                                uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers,
                                int objective = 0);

// Clusters with a decode rate that a genome may have for the brute-force
// role search (2^24 role sets); a genome with more is not searched.
constexpr int e2_search_max_free = 24;

// Role assignment per genome from T, Lambda [P][k_max][R]: policy 0 the
// brute force over the clusters with a decode rate, policy 1 the
// adapted-SplitWise rule (labels give the non-empty clusters, np_tokens the
// prompt length).
hipError_t e2_launch_roles(hipStream_t s, int P, int M, int k_max, int R, int policy,
                           uint32_t np_tokens, const uint8_t *labels, const uint64_t *T_all,
                           const uint64_t *L_all, uint64_t t_arrival, uint64_t nd,
                           uint64_t lambda_max, uint8_t *roles_out, uint8_t *slots_out,
                           uint64_t *w, uint64_t *phase);

hipError_t e2_launch_fitness(hipStream_t s, int P, int k_max, const uint64_t *T,
                             const uint64_t *Lambda, const uint8_t *roles, uint64_t t_arrival,
                             uint64_t nd, uint64_t lambda_max, uint64_t *w, uint64_t *phase,
                             uint64_t *s_p, uint64_t *s_d);

hipError_t e2_launch_ga(hipStream_t s, int M, int P, int k_max, const uint8_t *labels_in,
                        const uint8_t *roles_in, const uint64_t *w, const uint64_t *phase,
                        uint64_t seed, uint32_t generation, uint32_t tournament_k,
                        uint32_t xo_thresh, uint32_t mut_thresh, uint32_t n_elite,
                        uint32_t *elite_scratch, uint8_t *labels_out, uint8_t *roles_out);

hipError_t e2_launch_ga_ordered(hipStream_t s, int M, int P, int k_max, const uint8_t *order_in,
                                const uint16_t *sizes_in, const uint8_t *roles_in,
                                const uint64_t *w, const uint64_t *phase, uint64_t seed,
                                uint32_t generation, uint32_t tournament_k, uint32_t mut_thresh,
                                uint32_t n_elite, uint32_t max_replica, uint32_t *elite_scratch,
                                uint8_t *order_out, uint16_t *sizes_out, uint8_t *roles_out);
