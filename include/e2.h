/*
 * e2.h - C ABI of the MI355X population-fitness library (libe2.so).
 *
 * The library evaluates whole populations of the deployment search of
 * E2LLM (arXiv 2606.03770): for every (individual, cluster) pair it runs
 * the paper's bottleneck-minimising layer partition (Algorithm 1, Eq. 1-2,
 * Sec. 3.2), reduces the clusters of each individual to the queueing
 * fitness of Eq. 3-5 (Sec. 3.3) under the QoS floor of Sec. 3.5, and
 * breeds the next generation (Algorithm 2, Sec. 3.4).  All arithmetic is
 * unsigned integer: times in nanoseconds, sizes in bytes.
 *
 * Conventions shared by every entry point:
 *   - Return value: 0 (E2_OK) or a negative E2_E* code; e2_strerror names it.
 *     Host-side argument checks run before anything is enqueued, so an
 *     error return means nothing was launched.
 *   - Device pointers ("device" below) are HIP device allocations owned by
 *     the caller (for example torch CUDA tensors).  They must stay valid
 *     until the work enqueued on `stream` has completed.  The library keeps
 *     no pointer after a call returns.
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *     Every compute call is asynchronous on that stream and never
 *     synchronises the device.  Calls that need temporary device memory
 *     take it stream-ordered from HIP's default memory pool
 *     (hipMallocAsync / hipFreeAsync on the same stream), per call, or
 *     from a buffer the context keeps per stream (e2_ctx_keep_scratch).
 *   - INF = UINT64_MAX marks "no feasible value" in every u64 output.
 *   - A context's tables are immutable after creation; besides them it
 *     holds only the profiling records of e2_ctx_dp_timing and, when
 *     e2_ctx_keep_scratch is on, per-stream scratch that its calls share
 *     under a lock.  One context may serve several streams and host threads
 *     at once.  It lives on the device that was
 *     current when it was created; calls must be made with that device
 *     current.
 */
#ifndef E2_H
#define E2_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define E2_OK 0
#define E2_EINVAL (-1)    /* null pointer, size out of range, bad parameter   */
#define E2_EOVERFLOW (-2) /* a quantised time would reach 2^48 ns             */
#define E2_ENOMEM (-3)    /* a device or host allocation failed               */
#define E2_EHIP (-4)      /* a HIP runtime call or kernel launch failed       */

#define E2_INF UINT64_MAX
#define E2_MAX_DEV 256    /* M: devices in the pool                          */
#define E2_MAX_LAYER 255  /* N: transformer blocks of the model              */
#define E2_MAX_CLUSTERS 255 /* k_max: cluster ids per genome                 */
#define E2_MAX_SLOTS 15     /* b_max: decode slot counts of a slot model      */
#define E2_MAX_SEARCH_FREE 24 /* clusters with a decode rate per searched genome */

/*
 * Problem instance: the inputs of Algorithm 1 and Algorithm 2 (Sec. 3.2,
 * Sec. 3.4).  All pointers are HOST pointers, read only during
 * e2_ctx_create / e2_quantise.
 *
 *   n_dev, n_layer   M in [1, 256] devices, N in [1, 255] blocks
 *   speed_flops[M]   device compute speed in FLOP/s, > 0
 *   mem_bytes[M]     memory available for weights on each device
 *   bw_Bps[M*M]      link bandwidth d -> e in B/s, row-major; diagonal unused
 *   congestion_ppm[M*M] bandwidth multiplier in parts per million, <= 1e6
 *   layer_flops[2*N] FLOPs of each block, row 0 for prefill (the whole
 *                    prompt), row 1 for decode (one token)
 *   layer_bytes[N]   weight bytes of each block, < 2^48
 *   act_bytes[2]     activation bytes one microbatch moves across a link
 *                    (prefill, decode)
 *   head_flops[2]    FLOPs of the LM head plus output layer, charged to the
 *                    master device of a replica (Sec. 3.1, Sec. 3.2)
 *   head_bytes       their weight bytes, counted on the master, < 2^48
 */
typedef struct e2_problem {
    int32_t n_dev;
    int32_t n_layer;
    const uint64_t *speed_flops;
    const uint64_t *mem_bytes;
    const uint64_t *bw_Bps;
    const uint32_t *congestion_ppm;
    const uint64_t *layer_flops;
    const uint64_t *layer_bytes;
    uint64_t act_bytes[2];
    uint64_t head_flops[2];
    uint64_t head_bytes;
} e2_problem;

/*
 * Fitness parameters (Eq. 3-5, Sec. 3.3; QoS floor, Sec. 3.5).
 *   t_arrival_ns   request inter-arrival time T_a
 *   nd_tokens      generated tokens per request ND, in [0, 8192]
 *   min_tps_milli  per-request decode floor Min_TPS in tokens/s * 1000;
 *                  0 disables the floor
 */
typedef struct e2_fitness_params {
    uint64_t t_arrival_ns;
    uint64_t nd_tokens;
    uint64_t min_tps_milli;
} e2_fitness_params;

/*
 * GA parameters (Algorithm 2).
 *   seed, generation      key of the counter-based generator
 *   tournament_k          draws per tournament, in [1, 64]
 *   crossover_thresh_u32  a gene comes from the second parent when a
 *                         uniform u32 draw is below it (2^31 = p 0.5)
 *   mutation_thresh_u32   a gene mutates when a uniform u32 draw is below
 *                         it (2^24 = rate 1/256)
 *   n_elite               best individuals copied unchanged, in [0, 256],
 *                         at most P
 */
typedef struct e2_ga_params {
    uint64_t seed;
    uint32_t generation;
    uint32_t tournament_k;
    uint32_t crossover_thresh_u32;
    uint32_t mutation_thresh_u32;
    uint32_t n_elite;
} e2_ga_params;

typedef struct e2_ctx e2_ctx;

/*
 * Validate and quantise a problem, upload the tables to the current device.
 * Quantisation (the profiled block time and tau = A / B of Sec. 3.2, after
 * Eq. 2), with exact 128-bit intermediates:
 *   t[r][d][n]  = ceil(layer_flops[r][n] * 1e9 / speed[d])       ns
 *   h[r][d]     = ceil(head_flops[r] * 1e9 / speed[d])           ns
 *   Beff[d][e]  = floor(bw[d][e] * congestion[d][e] / 1e6)       B/s
 *   tau[r][d][e]= ceil(act_bytes[r] * 1e9 / Beff[d][e]) ns, INF when Beff = 0
 * Returns E2_EINVAL for a bad size or pointer, a zero speed or congestion
 * above 1e6; E2_EOVERFLOW when a finite time reaches 2^48 ns or a byte
 * size reaches 2^48; E2_ENOMEM / E2_EHIP on allocation or copy failure.
 * On success *out owns device memory until e2_ctx_destroy.
 */
int e2_ctx_create(const e2_problem *prob, e2_ctx **out);

/*
 * Decode-slot model (Algorithm 2's b loop; Sec. 3.4).  A decode replica may
 * hold b = 1..b_max requests in flight, one KV-cache slot each.  The paper
 * profiles the decode block time for each b; this library models it:
 *   beta_ppm                 each further request adds ceil(beta * lone
 *                            time) to a block's and to the head's decode
 *                            time (beta = beta_ppm / 1e6, in [0, 1])
 *   kv_bytes_per_block_slot  KV-cache bytes one request keeps per block
 * and a link carries b activations: tau_b = ceil(b * act_bytes[1] * 1e9 /
 * Beff).  A stage's bytes become its blocks' weight bytes plus slots * kv
 * per block (+ head bytes on the master), slots = 1 for prefill (the
 * request being prefilled) and b for decode.
 */
typedef struct e2_slot_model {
    int32_t b_max;                    /* 1..E2_MAX_SLOTS */
    uint32_t beta_ppm;                /* 0..1000000 */
    uint64_t kv_bytes_per_block_slot; /* KV bytes per block per request */
} e2_slot_model;

/*
 * e2_ctx_create with a slot model: tables for role index 0 (prefill) and
 * b = 1..b_max (decode with b requests), each with its own memory windows
 * when kv_bytes_per_block_slot > 0.  e2_solve_partitions /
 * e2_eval_population on such a context use role index 0 or 1 (roles[] = 0
 * or nonzero), i.e. they count one request's KV bytes.  Errors as
 * e2_ctx_create, plus E2_EINVAL for a NULL or out-of-range model and
 * E2_EOVERFLOW when a block's bytes with b_max slots reach 2^48.
 */
int e2_ctx_create_slots(const e2_problem *prob, const e2_slot_model *sm, e2_ctx **out);

/* Free a context (E2_EINVAL for NULL).  Work using it must have completed.
 * When the context holds per-stream scratch it waits for the device
 * (hipDeviceSynchronize) before releasing it. */
int e2_ctx_destroy(e2_ctx *ctx);

/*
 * Per-stream scratch for serving loops: with enable = 1 the context keeps
 * the temporary device memory of its calls (counters, problem lists, the
 * per-cluster T and Lambda of an evaluation, the GA's elite list) in one
 * buffer per stream, for up to 16 streams told apart by handle, instead of
 * allocating and freeing it on the stream in every call.  A stream's buffer
 * is allocated on it (hipMallocAsync) by its first call and grown on it
 * (hipFreeAsync, then hipMallocAsync) when a call needs more; calls on one
 * stream share it in stream order, calls on different streams never share
 * one, and calls on further streams, or on hipStreamPerThread (a different
 * stream in every host thread), allocate per call as before.  This
 * removes the allocation and release packets that otherwise separate
 * consecutive calls on a stream.  Condition while it is on: a stream with
 * calls on this context in flight is not destroyed (a new stream could
 * take its handle and with it a buffer still in use).  enable = 0 waits
 * for the device (hipDeviceSynchronize) and releases the buffers.  Not to
 * be called while other host threads use ctx.  E2_EINVAL for a NULL ctx or
 * enable outside {0, 1}; E2_ENOMEM, E2_EHIP on failure.
 */
int e2_ctx_keep_scratch(e2_ctx *ctx, int32_t enable);

/*
 * Host-only quantisation, same formulas and errors as e2_ctx_create, for
 * inspection: fills HOST arrays t[2][M][N], h[2][M], tau[2][M][M]
 * (diagonal 0).  Makes no HIP call.
 */
int e2_quantise(const e2_problem *prob, uint64_t *t, uint64_t *h, uint64_t *tau);

/*
 * Partition every (individual, cluster) problem of a population
 * (Algorithm 1 per replica, Sec. 3.2).
 *
 *   P            individuals, >= 0 (P = 0 is a no-op)
 *   k_max        cluster ids per genome, in [1, 255]
 *   labels[P][M] device: cluster id of each device; ids >= k_max leave the
 *                device unassigned
 *   roles[P][k_max] device: 0 = prefill replica, nonzero = decode replica
 *   T[P][k_max]  device out: best bottleneck of the cluster (Eq. 1-2 with
 *                the master enumerated), INF when the cluster is empty,
 *                has more devices than blocks, or cannot fit in memory
 *   Lambda[P][k_max] device out: end-to-end forward time of that best
 *                plan, sum of stage times and link times (Sec. 3.2); INF
 *                where T is INF
 *   master[P][k_max] device out: master device id, -1 where T is INF
 *   layers[P][M] device out: blocks placed on each device; 0 for unassigned
 *                devices and devices of infeasible clusters
 *
 * A cluster's device chain is its devices in ascending id order.  Each
 * device holds >= 1 contiguous block; stage k holds blocks j..i with
 * weight bytes (+ head bytes on the master) <= mem_bytes; the bottleneck
 * is the max over stage times (+ head time on the master) and link times
 * of consecutive chain devices; ties go to the smallest master position
 * and, within the recurrence, to the smallest split point j.
 */
int e2_solve_partitions(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                        const uint8_t *labels, const uint8_t *roles,
                        uint64_t *T, uint64_t *Lambda, int16_t *master, uint8_t *layers);

/*
 * Fitness of every individual (Eq. 3-5, Sec. 3.3) from its clusters'
 * partitions.  Same labels/roles layout as e2_solve_partitions.
 *   w[P], phase[P] device out: waiting time (Eq. 5) and bottleneck phase
 *                  (Eq. 3) in ns; both INF for an individual without a
 *                  usable prefill or a usable decode cluster
 *   s_p[P], s_d[P] device out, may be NULL: NP/PS and ND/DS in ns, INF when
 *                  the role has no usable cluster
 * Fixed point with SCALE = 2^50: rho_c = floor(SCALE / max(T_c, 1));
 * S_P = ceil(SCALE / sum_prefill rho); S_D = ND * ceil(SCALE / sum_decode rho);
 * phase = max(S_P, S_D); w = S_P + (phase - T_a) if phase > T_a else 0.
 * A decode cluster is usable only if Lambda <= floor(1e12 / min_tps_milli).
 */
int e2_eval_population(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                       const uint8_t *labels, const uint8_t *roles,
                       const e2_fitness_params *fp,
                       uint64_t *w, uint64_t *phase, uint64_t *s_p, uint64_t *s_d);

/*
 * e2_eval_population without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, allocation-free serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, layouts and results as
 * e2_eval_population.  Instead of a stream-ordered allocation, the call's
 * working memory (counters, the problem list, per-cluster T and Lambda, the
 * DP waves' split-point tables when chains can outgrow their LDS copy) is
 * carved from one fixed 96 MiB device array that the library holds on each
 * GPU it runs on until the process ends.
 *   Limit: P * k_max * 36 bytes plus, when min(M, N) - 1 rows of N split
 *   points exceed 2048 bytes, one DP wave's N * N-byte table must fit in
 *   96 MiB (P * k_max up to about 2.8 million at N = 126); larger inputs
 *   return E2_EINVAL before anything is enqueued.  When the tables of all
 *   of e2_eval_population's DP waves do not fit, fewer waves run (same
 *   results, slower).
 *   Every call on one GPU shares that GPU's array and leaves its contents
 *   behind: calls that overlap on one GPU (several streams or threads) race
 *   and must be serialised by the caller.  The counters are cleared by a
 *   kernel at the start of each call (no memset node).
 * Errors as e2_eval_population; E2_EHIP also when the array's device
 * address could not be resolved.
 */
int e2_eval_population_noalloc(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                               const uint8_t *labels, const uint8_t *roles,
                               const e2_fitness_params *fp,
                               uint64_t *w, uint64_t *phase, uint64_t *s_p, uint64_t *s_d);

/*
 * One GA generation (Algorithm 2: elites, crossover, mutation; Sec. 3.4).
 *   labels_in[P][M], roles_in[P][k_max], w_in[P], phase_in[P]  device in
 *   labels_out[P][M], roles_out[P][k_max]  device out; must not overlap
 *                                          the inputs
 * Individuals are ranked by the key (w, phase, index), smaller is better.
 * Slots 0..n_elite-1 receive the n_elite best in key order, unchanged.
 * Every other slot s breeds one child with the generator
 *   rng(seed, g, s, stream, gene): x = seed; then x = mix(x ^ c) for c in
 *   (g, s, stream, gene), mix = the SplitMix64 output function (Steele,
 *   Lea and Flood, OOPSLA 2014) of x + 0x9E3779B97F4A7C15;
 * parent a = best of tournament_k draws on streams 0.., parent b on
 * streams 64..; draw index = floor(hi32 * P / 2^32);
 * label gene d: from b if lo32(rng(.., 128, d)) < crossover_thresh, else
 * a; then redrawn as floor(lo32 * k_max / 2^32) if hi32(rng(.., 130, d))
 * < mutation_thresh; role gene q: likewise on streams 129 and 131, roles
 * written as 0/1 and flipped on mutation.
 */
int e2_ga_step(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
               const uint8_t *labels_in, const uint8_t *roles_in,
               const uint64_t *w_in, const uint64_t *phase_in, const e2_ga_params *gp,
               uint8_t *labels_out, uint8_t *roles_out);

/*
 * Two-chromosome genomes (App. A, gene definition): per individual an
 * ordering chromosome and a grouping chromosome, plus a role per replica.
 *   order[P][M]   device: a permutation of 0..M-1 (an id >= M makes its
 *                 replica infeasible; a device missing from the ordering
 *                 gets 0 layers; a repeated id gives unspecified layers for
 *                 that device)
 *   sizes[P][k_max] device, u16: replica r holds the devices at ordering
 *                 positions sizes[0] + ... + sizes[r-1] onwards, sizes[r] of
 *                 them, clipped to M; 0 = no replica
 *   roles[P][k_max] device: 0 = prefill replica, nonzero = decode replica
 * A replica's device chain is its run of the ordering, in ordering order
 * (the paper's node ordering, Sec. 3.2).  The paper's example
 * [(0,1,2,3,4,5), (3,1,2)] has replicas {0,1,2}, {3}, {4,5}.
 *
 * e2_solve_partitions_ordered / e2_eval_population_ordered: as
 * e2_solve_partitions / e2_eval_population with replicas in place of
 * clusters (outputs per replica index r < k_max; same layouts, errors and
 * fitness).
 */
int e2_solve_partitions_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                                const uint8_t *order, const uint16_t *sizes,
                                const uint8_t *roles, uint64_t *T, uint64_t *Lambda,
                                int16_t *master, uint8_t *layers);
int e2_eval_population_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                               const uint8_t *order, const uint16_t *sizes, const uint8_t *roles,
                               const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                               uint64_t *s_p, uint64_t *s_d);

/*
 * Parameters of the two-chromosome GA (App. A).
 *   seed, generation, tournament_k, n_elite   as in e2_ga_params
 *   mutation_thresh_u32  a child mutates when a uniform u32 draw is below
 *                        it (about 0.3 * 2^32 in the paper)
 *   max_replica          largest replica size drawn when a grouping
 *                        regrows, in [1, 256]
 */
typedef struct e2_ga2_params {
    uint64_t seed;
    uint32_t generation;
    uint32_t tournament_k;
    uint32_t mutation_thresh_u32;
    uint32_t n_elite;
    uint32_t max_replica;
} e2_ga2_params;

/*
 * One generation of the two-chromosome GA (Algorithm 2, App. A).  Inputs
 * and outputs as above (order, sizes, roles), w_in / phase_in as in
 * e2_ga_step; outputs must not overlap the inputs or each other.
 * Slots 0..n_elite-1 receive the n_elite best individuals (key (w, phase,
 * index)) unchanged.  Every other slot s, with draws rng(seed, generation,
 * s, stream, gene) of the generator of e2_ga_step:
 *   parents a, b      tournaments on streams 0.. and 64.. (as e2_ga_step)
 *   ordering          c = 1 + floor(lo32(rng(.., 140, 0)) * (M-1) / 2^32);
 *                     the child takes a's first c devices, then b's later
 *                     positions; a device of b's part already present
 *                     leaves a hole, and the holes are filled left to right
 *                     with b's first-c devices missing from the child, in
 *                     b's order (M = 1: a copy of a)
 *   grouping, roles   those of b if lo32(rng(.., 141, 0)) < 2^31, else of a
 *                     (roles written as 0/1)
 *   mutation          u = rng(.., 142, 0) fires when hi32(u) <
 *                     mutation_thresh; lo32(u) then picks, below 0.20,
 *                     0.70, 0.85 of 2^32 and above:
 *                     swap ordering positions floor(hi32(v) M / 2^32) and
 *                       floor(lo32(v) M / 2^32), v = rng(.., 143, 0);
 *                     regrow the grouping from replica floor(hi32(rng(..,
 *                       144, 0)) R / 2^32), R = replicas holding devices;
 *                     regrow the whole grouping;
 *                     a new ordering (Fisher-Yates from the identity, step
 *                       t = M-1..1 swapping t with floor(hi32(rng(.., 146,
 *                       t)) (t+1) / 2^32)) and a regrown grouping.
 *   regrowth          replicas before the start keep size and role; each
 *                     later replica r gets size 1 + floor(hi32(u) *
 *                     max_replica / 2^32), capped by the devices left (slot
 *                     k_max-1 takes all that are left), and role
 *                     lo32(u) >= 2^31, u = rng(.., 145, r); unused slots 0.
 * E2_EINVAL for tournament_k outside [1, 64], n_elite > min(256, P),
 * max_replica outside [1, 256] or overlapping buffers.
 */
int e2_ga_step_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                       const uint8_t *order_in, const uint16_t *sizes_in, const uint8_t *roles_in,
                       const uint64_t *w_in, const uint64_t *phase_in, const e2_ga2_params *gp,
                       uint8_t *order_out, uint16_t *sizes_out, uint8_t *roles_out);

/*
 * Role and slot search for label genomes (Algorithm 2's inner loop and its
 * brute-force role assignment, Sec. 3.4).  For every non-empty cluster of
 * every genome (chain in ascending device id): Algorithm 1 with the prefill
 * tables and with the decode tables of each b = 1..b_max of the context
 * (b_max = 1 for a context without a slot model); then
 *   rho_P = floor(2^50 / max(T_prefill, 1)), 0 if infeasible;
 *   b*    = the largest b whose DP is feasible and whose Lambda passes the
 *           QoS floor of fp (floor(1e12 / min_tps_milli) ns, none if 0);
 *   rho_D = floor(b* 2^50 / max(T_b*, 1)), 0 if no b qualifies;
 * and every prefill/decode assignment of the clusters is scored as
 * e2_eval_population scores summed rates (Eq. 3-5); the smallest (w,
 * phase) wins, ties going to the assignment whose decode set, as a bitmask
 * over cluster ids, is smallest.  A cluster with rho_D = 0 is prefill in
 * that winner (w and phase never grow with the prefill sum), so only the F
 * clusters with a decode rate are enumerated (2^F sets); a genome with F >
 * E2_MAX_SEARCH_FREE is not searched (all roles 0, all slots 0xFF, w =
 * phase = INF).
 *   labels[P][M]     device: cluster id per device (ids >= k_max unassigned)
 *   k_max            1..E2_MAX_CLUSTERS
 *   roles_out[P][k_max]  device: 1 decode, 0 prefill or empty cluster
 *   slots_out[P][k_max]  device: b* of a decode cluster (0 if none
 *                    qualified), 0 otherwise; 0xFF throughout for a genome
 *                    that was not searched
 *   w, phase [P]     device: the winning fitness (INF if no assignment has
 *                    both a usable prefill and a usable decode cluster, or
 *                    if the genome was not searched)
 *   T_all, Lambda_all [P][k_max][b_max+1]  device, optional (both or
 *                    neither): every DP result, index 0 prefill, b decode
 *                    with b requests; INF for empty or infeasible
 * Asynchronous on `stream`.  E2_EINVAL for sizes out of range (P below
 * 2^20), nd_tokens > 8192 or a NULL required pointer.
 */
int e2_search_roles(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const uint8_t *labels,
                    const e2_fitness_params *fp, uint8_t *roles_out, uint8_t *slots_out,
                    uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all);

/*
 * The same role and slot search for two-chromosome genomes (App. A gene
 * definition; Algorithm 2's inner loop on the paper's own genome): replica
 * q's chain is its run of the ordering, in ordering order, exactly as in
 * e2_solve_partitions_ordered (an id >= M makes the replica infeasible, an
 * empty replica has no rates); then the same per-replica DPs for prefill and
 * each b = 1..b_max, the same kept slot count b*, rates and brute-force role
 * assignment over the replicas with a decode rate (at most
 * E2_MAX_SEARCH_FREE, else not searched), ties to the smallest decode
 * bitmask over replica slots.
 *   order[P][M], sizes[P][k_max]  device, as e2_solve_partitions_ordered
 *   k_max            1..E2_MAX_CLUSTERS replica slots
 *   outputs          as e2_search_roles, per replica slot
 * E2_EINVAL for sizes out of range (P below 2^20), nd_tokens > 8192 or a
 * NULL required pointer.
 */
int e2_search_roles_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                            const uint8_t *order, const uint16_t *sizes,
                            const e2_fitness_params *fp, uint8_t *roles_out, uint8_t *slots_out,
                            uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all);

/*
 * The adapted-SplitWise role rule (the ablation of Sec. 4.2), on the same
 * per-cluster DP results as e2_search_roles: per genome the R' non-empty
 * clusters split by the token ratio, n_P = R' * np_tokens / (np_tokens +
 * nd_tokens) rounded half up and clamped to [1, R' - 1] (R' when R' <= 1,
 * half of R' rounded up when both token counts are 0); the n_P clusters
 * with the highest prefill rate (ties to the smaller cluster id) prefill,
 * the rest decode at their kept slot count.  Arguments and outputs as
 * e2_search_roles, with k_max up to E2_MAX_CLUSTERS and P below 2^20.
 */
int e2_assign_roles_splitwise(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                              const uint8_t *labels, const e2_fitness_params *fp,
                              uint32_t np_tokens, uint8_t *roles_out, uint8_t *slots_out,
                              uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all);

/*
 * The finishing-time objective (the FT ablation of Sec. 4.2): as
 * e2_solve_partitions / e2_eval_population, but each cluster's master and
 * split points minimise its end-to-end time (stage times plus link times,
 * Eq. 1 with the max replaced by a sum; memory, Eq. 2 and the tie rules
 * unchanged).  T is the bottleneck of that partition (max over stage and
 * link times), Lambda its end-to-end time; fitness by Eq. 3-5 as usual.
 * One DP table per master (O(m^2 N^2) per cluster).
 */
int e2_solve_partitions_ft(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                           const uint8_t *labels, const uint8_t *roles, uint64_t *T,
                           uint64_t *Lambda, int16_t *master, uint8_t *layers);
int e2_eval_population_ft(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                          const uint8_t *labels, const uint8_t *roles,
                          const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                          uint64_t *s_p, uint64_t *s_d);

/*
 * The idle-device relaxation: as e2_solve_partitions / e2_eval_population,
 * but a device of a cluster may hold no block and then sits out of the
 * pipeline; links join consecutive participating devices (tau between any
 * two devices of the cluster); the master always participates, with its
 * head, possibly holding no block (its stage is then the head alone, which
 * must fit its memory).  Clusters with more devices than blocks are solved.
 * Per master mu and x blocks placed, A_k(x) = min over the allowed
 * predecessors k' of max(E_k'(x), tau(k', k)) and E_k(x) = min over stage
 * starts j of max(A_k(j), stage time) (ties: the smallest k', the smallest
 * j, a stage with blocks before the empty one, the smallest last device,
 * the smallest master).  layers[] is 0 for devices that sit out; Lambda
 * sums the participants' stage times (+ head) and links.  Under this
 * relaxation adding a device never raises T.
 */
int e2_solve_partitions_idle(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                             const uint8_t *labels, const uint8_t *roles, uint64_t *T,
                             uint64_t *Lambda, int16_t *master, uint8_t *layers);
int e2_eval_population_idle(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                            const uint8_t *labels, const uint8_t *roles,
                            const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                            uint64_t *s_p, uint64_t *s_d);

/*
 * Profiling of the DP kernel (the dominant cost of e2_solve_partitions and
 * e2_eval_population), for benchmarks and profilers.
 *
 * e2_ctx_dp_timing(ctx, n): for the next n solve/eval calls on ctx, record
 * a HIP event on the call's stream just before and just after its DP
 * kernel (n in [0, 4096]; 0 turns the recording off).  Discards earlier
 * records.  Allocates n event pairs; E2_ENOMEM / E2_EHIP if that fails.
 * e2_ctx_dp_elapsed(ctx, &launches, &ms): waits for the recorded events
 * and returns how many DP launches were recorded and their summed
 * duration in milliseconds.
 * While recording is on, ctx must not be used by several host threads at
 * once (the calls take the next event pair from the context).
 */
int e2_ctx_dp_timing(e2_ctx *ctx, int32_t max_launches);
int e2_ctx_dp_elapsed(e2_ctx *ctx, int32_t *launches, double *total_ms);

/*
 * Failure injection for tests of callers' error handling: the next `calls`
 * library calls that reach a HIP runtime call (context creation, every
 * solve / eval / search / GA call, the timing hook) return E2_EHIP at that
 * point, after their argument checks and before anything is allocated or
 * enqueued; 0 turns it off.  Process-wide.  Returns how many injected
 * failures were still pending before this call (>= 0), or E2_EINVAL for
 * calls < 0.
 */
int e2_debug_inject_hip_error(int32_t calls);

/* Static string for an E2_* code ("unknown error" otherwise). */
const char *e2_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* E2_H */
