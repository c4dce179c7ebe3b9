/*
 * Every entry point of the CPU oracle (oracle/oracle.c) on seeded random
 * inputs of several shapes, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer: any out-of-bounds access, leak or undefined
 * operation aborts the run.  Inputs come from a plain 64-bit LCG (no
 * arithmetic of the method); the results are not checked here (the Python
 * tests pin them), only that every call returns 0 and stays in bounds.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_quantise(int, int, const uint64_t *, const uint64_t *, const uint32_t *, const uint64_t *,
                    const uint64_t *, const uint64_t *, uint64_t *, uint64_t *, uint64_t *);
int oracle_solve(int, int, const uint64_t *, const uint64_t *, const uint64_t *, const uint64_t *,
                 const uint64_t *, uint64_t, int, int, const uint8_t *, const uint8_t *, uint64_t *,
                 uint64_t *, int16_t *, uint8_t *, uint64_t *);
int oracle_solve_obj(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                     const uint64_t *, const uint64_t *, uint64_t, int, int, int, const uint8_t *,
                     const uint8_t *, uint64_t *, uint64_t *, int16_t *, uint8_t *, uint64_t *);
int oracle_fitness(int, int, const uint64_t *, const uint64_t *, const uint8_t *, uint64_t, uint64_t,
                   uint64_t, uint64_t *, uint64_t *, uint64_t *, uint64_t *);
int oracle_ga_step(int, int, int, const uint8_t *, const uint8_t *, const uint64_t *,
                   const uint64_t *, uint64_t, uint32_t, uint32_t, uint32_t, uint32_t, uint32_t,
                   uint8_t *, uint8_t *);
int oracle_solve_ordered(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                         const uint64_t *, const uint64_t *, uint64_t, int, int, const uint8_t *,
                         const uint16_t *, const uint8_t *, uint64_t *, uint64_t *, int16_t *,
                         uint8_t *);
int oracle_ga_step_ordered(int, int, int, const uint8_t *, const uint16_t *, const uint8_t *,
                           const uint64_t *, const uint64_t *, uint64_t, uint32_t, uint32_t,
                           uint32_t, uint32_t, uint32_t, uint8_t *, uint16_t *, uint8_t *);
int oracle_quantise_slots(int, int, const uint64_t *, const uint64_t *, const uint32_t *,
                          const uint64_t *, const uint64_t *, const uint64_t *, int, uint32_t,
                          uint64_t *, uint64_t *, uint64_t *);
int oracle_search_roles(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                        const uint64_t *, const uint64_t *, uint64_t, uint64_t, int, int, int,
                        const uint8_t *, uint64_t, uint64_t, uint64_t, uint64_t *, uint64_t *,
                        uint8_t *, uint8_t *, uint64_t *, uint64_t *);
int oracle_search_roles_ordered(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                                const uint64_t *, const uint64_t *, uint64_t, uint64_t, int, int,
                                int, const uint8_t *, const uint16_t *, uint64_t, uint64_t,
                                uint64_t, uint64_t *, uint64_t *, uint8_t *, uint8_t *,
                                uint64_t *, uint64_t *);
int oracle_assign_roles_splitwise(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                                  const uint64_t *, const uint64_t *, uint64_t, uint64_t, int, int,
                                  int, const uint8_t *, uint64_t, uint64_t, uint64_t, uint64_t,
                                  uint64_t *, uint64_t *, uint8_t *, uint8_t *, uint64_t *,
                                  uint64_t *);
int oracle_solve_idle(int, int, const uint64_t *, const uint64_t *, const uint64_t *,
                      const uint64_t *, const uint64_t *, uint64_t, int, int, const uint8_t *,
                      const uint8_t *, uint64_t *, uint64_t *, int16_t *, uint8_t *);

static uint64_t lcg_state = 0x2606037702606037ull;
static uint64_t next_u64(void)
{
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return lcg_state >> 11;
}
static uint64_t in_range(uint64_t lo, uint64_t hi) { return lo + next_u64() % (hi - lo + 1); }

#define CHECK(call)                                                             \
    do {                                                                        \
        int rc_ = (call);                                                       \
        if (rc_ != 0) {                                                         \
            fprintf(stderr, "%s failed: %d (M=%d N=%d P=%d K=%d)\n", #call, rc_, \
                    M, N, P, K);                                                \
            exit(1);                                                            \
        }                                                                       \
    } while (0)

static void *xmalloc(size_t n)
{
    void *p = calloc(n ? n : 1, 1);
    if (!p) exit(2);
    return p;
}

static void run(int M, int N, int P, int K, int b_max)
{
    uint64_t *speed = xmalloc(8 * M), *mem = xmalloc(8 * M), *bw = xmalloc(8 * (size_t)M * M);
    uint32_t *cong = xmalloc(4 * (size_t)M * M);
    uint64_t *lf = xmalloc(8 * 2 * (size_t)N), *W = xmalloc(8 * (size_t)N);
    uint64_t act[2], head[2];
    for (int d = 0; d < M; d++) {
        speed[d] = in_range(1, 50) * 100000000000ull;
        mem[d] = in_range(1, 40) * 100000000ull;
    }
    for (int i = 0; i < M * M; i++) {
        bw[i] = in_range(0, 4) ? in_range(1000000, 1000000000) : 0;
        cong[i] = (uint32_t)in_range(100000, 1000000);
    }
    for (int n = 0; n < N; n++) {
        lf[n] = in_range(1, 8) * 100000000000ull;
        lf[N + n] = in_range(1, 8) * 100000000ull;
        W[n] = in_range(50000000, 200000000);
    }
    act[0] = in_range(1000000, 100000000);
    act[1] = in_range(1000, 100000);
    head[0] = in_range(0, 2) * 100000000000ull;
    head[1] = head[0] / 7;
    const uint64_t HB = in_range(0, 1) * 100000000ull;
    const int R = b_max + 1;
    uint64_t *t = xmalloc(8 * (size_t)R * M * N), *h = xmalloc(8 * (size_t)R * M);
    uint64_t *tau = xmalloc(8 * (size_t)R * M * M);
    CHECK(oracle_quantise(M, N, speed, bw, cong, lf, act, head, t, h, tau));

    uint8_t *labels = xmalloc((size_t)P * M), *roles = xmalloc((size_t)P * K);
    for (int i = 0; i < P * M; i++) labels[i] = (uint8_t)(in_range(0, 19) ? in_range(0, K - 1) : 250);
    for (int i = 0; i < P * K; i++) roles[i] = (uint8_t)in_range(0, 1);
    uint64_t *T = xmalloc(8 * (size_t)P * K * R), *L = xmalloc(8 * (size_t)P * K * R), ev = 0;
    int16_t *master = xmalloc(2 * (size_t)P * K);
    uint8_t *layers = xmalloc((size_t)P * M);
    CHECK(oracle_solve(M, N, t, h, tau, mem, W, HB, P, K, labels, roles, T, L, master, layers, &ev));
    uint64_t *w = xmalloc(8 * (size_t)P), *ph = xmalloc(8 * (size_t)P);
    uint64_t *sp = xmalloc(8 * (size_t)P), *sd = xmalloc(8 * (size_t)P);
    CHECK(oracle_fitness(P, K, T, L, roles, 100000000, 1024, 7000, w, ph, sp, sd));
    CHECK(oracle_solve_obj(M, N, t, h, tau, mem, W, HB, 1, P, K, labels, roles, T, L, master,
                           layers, &ev));
    CHECK(oracle_solve_idle(M, N, t, h, tau, mem, W, HB, P, K, labels, roles, T, L, master,
                            layers));
    uint8_t *lo = xmalloc((size_t)P * M), *ro = xmalloc((size_t)P * K);
    CHECK(oracle_ga_step(M, P, K, labels, roles, w, ph, 7, 3, 4, 1u << 31, 1u << 28,
                         P < 3 ? (uint32_t)P : 3u, lo, ro));

    /* two-chromosome genomes: a permutation cut into runs (some ids not devices) */
    uint8_t *order = xmalloc((size_t)P * M);
    uint16_t *sizes = xmalloc(2 * (size_t)P * K);
    for (int p = 0; p < P; p++) {
        for (int d = 0; d < M; d++) order[(size_t)p * M + d] = (uint8_t)d;
        for (int d = M - 1; d >= 1; d--) {
            int j = (int)in_range(0, (uint64_t)d);
            uint8_t x = order[(size_t)p * M + d];
            order[(size_t)p * M + d] = order[(size_t)p * M + j];
            order[(size_t)p * M + j] = x;
        }
        if (!in_range(0, 9)) order[(size_t)p * M + in_range(0, M - 1)] = 240;
        int left = M + (int)in_range(0, 4) - 2;
        for (int q = 0; q < K; q++) {
            int s = left > 0 ? (int)in_range(0, 5) : 0;
            if (s > left) s = left;
            sizes[(size_t)p * K + q] = (uint16_t)(s < 0 ? 0 : s);
            left -= s;
        }
    }
    CHECK(oracle_solve_ordered(M, N, t, h, tau, mem, W, HB, P, K, order, sizes, roles, T, L,
                               master, layers));
    uint8_t *oo = xmalloc((size_t)P * M), *qo = xmalloc((size_t)P * K);
    uint16_t *so = xmalloc(2 * (size_t)P * K);
    CHECK(oracle_ga_step_ordered(M, P, K, order, sizes, roles, w, ph, 9, 2, 4, 1288490188u,
                                 P < 2 ? (uint32_t)P : 2u, 5, oo, so, qo));

    /* role and slot search (at most 16 clusters) and the SplitWise rule */
    CHECK(oracle_quantise_slots(M, N, speed, bw, cong, lf, act, head, b_max, 125000, t, h, tau));
    uint8_t *rs = xmalloc((size_t)P * K), *ss = xmalloc((size_t)P * K);
    const uint64_t kv = in_range(0, 1) * 1000000;
    if (K <= 16) {
        CHECK(oracle_search_roles(M, N, t, h, tau, mem, W, HB, kv, b_max, P, K, labels,
                                  100000000, 1024, 7000, T, L, rs, ss, w, ph));
        CHECK(oracle_search_roles_ordered(M, N, t, h, tau, mem, W, HB, kv, b_max, P, K, order,
                                          sizes, 100000000, 1024, 0, T, L, rs, ss, w, ph));
    }
    CHECK(oracle_assign_roles_splitwise(M, N, t, h, tau, mem, W, HB, kv, b_max, P, K, labels,
                                        100000000, 1024, 0, 512, T, L, rs, ss, w, ph));
    void *bufs[] = {speed, mem, bw, cong, lf, W, t, h, tau, labels, roles, T, L, master,
                    layers, w, ph, sp, sd, lo, ro, order, sizes, oo, qo, so, rs, ss};
    for (size_t i = 0; i < sizeof(bufs) / sizeof(bufs[0]); i++) free(bufs[i]);
}

int main(void)
{
    static const int shapes[][5] = {{1, 1, 2, 1, 1},   {3, 2, 3, 2, 2},   {12, 32, 4, 3, 4},
                                    {40, 60, 3, 9, 8},  {64, 80, 2, 16, 3}, {70, 90, 1, 20, 2},
                                    {256, 255, 1, 3, 1}};
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); s++)
        run(shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3], shapes[s][4]);
    printf("oracle driver: %zu shapes ok\n", sizeof(shapes) / sizeof(shapes[0]));
    return 0;
}
