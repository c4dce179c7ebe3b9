/*
 * The host-only paths of libe2 (include/e2.h), for a build whose host code
 * carries AddressSanitizer and UndefinedBehaviorSanitizer: quantisation of
 * seeded random problems (including ones whose times overflow), every
 * argument check of context creation and of the device-facing entry
 * points, and context creation failing at its first HIP call (injected),
 * which must release what it built.  No call here reaches the GPU.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/e2.h"

static uint64_t lcg_state = 0x5eed5eed2606ull;
static uint64_t next_u64()
{
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return lcg_state >> 11;
}
static uint64_t in_range(uint64_t lo, uint64_t hi) { return lo + next_u64() % (hi - lo + 1); }

static int failures = 0;
static void expect(int got, int want, const char *what)
{
    if (got != want) {
        fprintf(stderr, "%s: got %d, want %d\n", what, got, want);
        ++failures;
    }
}

struct Problem {
    int M, N;
    std::vector<uint64_t> speed, mem, bw, lf, W;
    std::vector<uint32_t> cong;
    e2_problem p;
    Problem(int M_, int N_) : M(M_), N(N_), speed(M_), mem(M_), bw((size_t)M_ * M_), lf(2 * N_),
                              W(N_), cong((size_t)M_ * M_)
    {
        for (int d = 0; d < M; ++d) {
            speed[d] = in_range(1, 50) * 100000000000ull;
            mem[d] = in_range(1, 40) * 100000000ull;
        }
        for (size_t i = 0; i < bw.size(); ++i) {
            bw[i] = in_range(0, 4) ? in_range(1000000, 1000000000) : 0;
            cong[i] = (uint32_t)in_range(0, 1000000);
        }
        for (int n = 0; n < N; ++n) {
            lf[n] = in_range(1, 8) * 100000000000ull;
            lf[N + n] = in_range(1, 8) * 100000000ull;
            W[n] = in_range(50000000, 200000000);
        }
        memset(&p, 0, sizeof(p));
        p.n_dev = M;
        p.n_layer = N;
        p.speed_flops = speed.data();
        p.mem_bytes = mem.data();
        p.bw_Bps = bw.data();
        p.congestion_ppm = cong.data();
        p.layer_flops = lf.data();
        p.layer_bytes = W.data();
        p.act_bytes[0] = in_range(1000000, 100000000);
        p.act_bytes[1] = in_range(1000, 100000);
        p.head_flops[0] = in_range(0, 2) * 100000000000ull;
        p.head_flops[1] = p.head_flops[0] / 7;
        p.head_bytes = in_range(0, 1) * 100000000ull;
    }
};

int main()
{
    static const int shapes[][2] = {{1, 1}, {2, 3}, {12, 32}, {64, 80}, {256, 255}};
    for (const auto &s : shapes) {
        Problem pr(s[0], s[1]);
        const int M = s[0], N = s[1];
        std::vector<uint64_t> t(2 * (size_t)M * N), h(2 * (size_t)M), tau(2 * (size_t)M * M);
        expect(e2_quantise(&pr.p, t.data(), h.data(), tau.data()), E2_OK, "quantise");
        // a speed of 1 FLOP/s makes every time overflow 2^48 ns
        pr.speed[0] = 1;
        expect(e2_quantise(&pr.p, t.data(), h.data(), tau.data()), E2_EOVERFLOW, "overflow");
        pr.speed[0] = 0;
        expect(e2_quantise(&pr.p, t.data(), h.data(), tau.data()), E2_EINVAL, "speed 0");
        e2_ctx *ctx = nullptr;
        expect(e2_ctx_create(&pr.p, &ctx), E2_EINVAL, "ctx speed 0");
        pr.speed[0] = 10000000000000ull;
        pr.cong[0] = 1000001;
        expect(e2_ctx_create(&pr.p, &ctx), E2_EINVAL, "ctx congestion");
        pr.cong[0] = 0;
        pr.W[0] = 1ull << 48;
        expect(e2_ctx_create(&pr.p, &ctx), E2_EOVERFLOW, "ctx block bytes");
        pr.W[0] = 100000000;
        // a valid problem fails at its first HIP call: nothing may leak
        expect(e2_debug_inject_hip_error(1), 0, "inject");
        expect(e2_ctx_create(&pr.p, &ctx), E2_EHIP, "ctx injected");
        expect(ctx == nullptr, 1, "no context on failure");
        e2_slot_model sm = {4, 125000, 1000000};
        expect(e2_debug_inject_hip_error(1), 0, "inject slots");
        expect(e2_ctx_create_slots(&pr.p, &sm, &ctx), E2_EHIP, "slots injected");
        sm.b_max = 16;
        expect(e2_ctx_create_slots(&pr.p, &sm, &ctx), E2_EINVAL, "slots b_max");
        expect(e2_debug_inject_hip_error(0), 0, "no pending injection");
    }
    // argument checks of the device-facing entry points (no context)
    e2_fitness_params fp = {100000000, 1024, 7000};
    e2_ga_params gp = {1, 0, 4, 1u << 31, 1u << 24, 1};
    uint8_t b[16];
    uint64_t u[16];
    expect(e2_solve_partitions(nullptr, nullptr, 1, 2, b, b, u, u, nullptr, b), E2_EINVAL, "solve");
    expect(e2_eval_population(nullptr, nullptr, 1, 2, b, b, &fp, u, u, u, u), E2_EINVAL, "eval");
    expect(e2_eval_population_noalloc(nullptr, nullptr, 1, 2, b, b, &fp, u, u, u, u), E2_EINVAL,
           "eval noalloc");
    expect(e2_ga_step(nullptr, nullptr, 1, 2, b, b, u, u, &gp, b, b), E2_EINVAL, "ga");
    expect(e2_search_roles(nullptr, nullptr, 1, 17, b, &fp, b, b, u, u, nullptr, nullptr),
           E2_EINVAL, "search k_max");
    expect(e2_search_roles_ordered(nullptr, nullptr, 1, 2, nullptr, nullptr, &fp, b, b, u, u,
                                   nullptr, nullptr),
           E2_EINVAL, "search ordered");
    expect(e2_ctx_dp_timing(nullptr, 1), E2_EINVAL, "timing");
    expect(e2_ctx_destroy(nullptr), E2_EINVAL, "destroy");
    expect(e2_debug_inject_hip_error(-1), E2_EINVAL, "inject < 0");
    for (int c = -5; c <= 1; ++c)
        if (!e2_strerror(c) || !e2_strerror(c)[0]) ++failures;
    if (failures) return 1;
    printf("library host driver: ok\n");
    return 0;
}
