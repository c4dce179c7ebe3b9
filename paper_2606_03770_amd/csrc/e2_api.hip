// Host side of libe2.so: argument checks, integer quantisation, derived
// tables, device uploads and the stream-ordered launches behind the C ABI
// declared in include/e2.h.

#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <list>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/e2.h"
#include "e2_internal.h"

static_assert(e2_search_max_free == E2_MAX_SEARCH_FREE, "role search bound");

namespace {

typedef unsigned __int128 u128;
constexpr uint64_t kLimit48 = 1ull << 48;

// ceil(a * 1e9 / b) for b > 0 in exact 128-bit arithmetic; saturates to
// UINT64_MAX (which the callers treat as an overflow).
uint64_t ceil_ns(uint64_t a, uint64_t b)
{
    const u128 num = (u128)a * 1000000000u;
    const u128 q = num / b + (num % b != 0);
    return (q >> 64) ? UINT64_MAX : (uint64_t)q;
}

int check_problem(const e2_problem *pr)
{
    if (!pr) return E2_EINVAL;
    const int M = pr->n_dev, N = pr->n_layer;
    if (M < 1 || M > E2_MAX_DEV || N < 1 || N > E2_MAX_LAYER) return E2_EINVAL;
    if (!pr->speed_flops || !pr->mem_bytes || !pr->bw_Bps || !pr->congestion_ppm ||
        !pr->layer_flops || !pr->layer_bytes)
        return E2_EINVAL;
    for (int d = 0; d < M; ++d)
        if (pr->speed_flops[d] == 0) return E2_EINVAL;
    for (int i = 0; i < M * M; ++i)
        if (pr->congestion_ppm[i] > 1000000u) return E2_EINVAL;
    for (int n = 0; n < N; ++n)
        if (pr->layer_bytes[n] >= kLimit48) return E2_EOVERFLOW;
    if (pr->head_bytes >= kLimit48) return E2_EOVERFLOW;
    return E2_OK;
}

// Fill t[2][M][N], h[2][M], tau[2][M][M] (host arrays).
int quantise(const e2_problem *pr, uint64_t *t, uint64_t *h, uint64_t *tau)
{
    const int M = pr->n_dev, N = pr->n_layer;
    for (int r = 0; r < 2; ++r) {
        for (int d = 0; d < M; ++d) {
            const uint64_t S = pr->speed_flops[d];
            for (int n = 0; n < N; ++n) {
                const uint64_t v = ceil_ns(pr->layer_flops[(size_t)r * N + n], S);
                if (v >= kLimit48) return E2_EOVERFLOW;
                t[((size_t)r * M + d) * N + n] = v;
            }
            const uint64_t hv = ceil_ns(pr->head_flops[r], S);
            if (hv >= kLimit48) return E2_EOVERFLOW;
            h[(size_t)r * M + d] = hv;
        }
        for (int d = 0; d < M; ++d) {
            for (int e = 0; e < M; ++e) {
                uint64_t v = 0;
                if (d != e) {
                    const size_t ix = (size_t)d * M + e;
                    const uint64_t beff =
                        (uint64_t)(((u128)pr->bw_Bps[ix] * pr->congestion_ppm[ix]) / 1000000u);
                    if (beff == 0) {
                        v = E2_INF64;
                    } else {
                        v = ceil_ns(pr->act_bytes[r], beff);
                        if (v >= kLimit48) return E2_EOVERFLOW;
                    }
                }
                tau[((size_t)r * M + d) * M + e] = v;
            }
        }
    }
    return E2_OK;
}

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// ---------------------------------------------------------------------------
// Fixed device scratch of e2_eval_population_noalloc: the call's counters,
// problem list, per-cluster T and Lambda and the DP waves' row regions are
// carved from this array instead of a stream-ordered allocation.  Each GPU
// the library runs on holds its own copy until the process ends.  In host
// code `scratch` names a host-side stand-in: only the address returned by
// hipGetSymbolAddress (one per device, kept in g_scratch) is a device
// address.
// ---------------------------------------------------------------------------
constexpr size_t kNoAllocBytes = (size_t)96 << 20;
__device__ __align__(256) uint8_t scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
    std::once_flag once;
    void *ptr = nullptr;
    hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

// Resolve (once per device, with that device current) and return the
// device address of this device's scratch.
int scratch_on(int dev, void **out)
{
    if (dev < 0 || dev >= kMaxDevices) return E2_EINVAL;
    ScratchSlot &sl = g_scratch[dev];
    std::call_once(sl.once, [&sl] {
        sl.err = hipGetSymbolAddress(&sl.ptr, HIP_SYMBOL(scratch));
        if (sl.err != hipSuccess) {
            (void)hipGetLastError();
            sl.ptr = nullptr;
        }
    });
    if (sl.err != hipSuccess || !sl.ptr) return E2_EHIP;
    *out = sl.ptr;
    return E2_OK;
}

// Failure injection (e2_debug_inject_hip_error): calls left that fail with
// E2_EHIP where they would make their first HIP runtime call.
std::atomic<int> g_inject{0};

bool injected_failure()
{
    int n = g_inject.load();
    while (n > 0)
        if (g_inject.compare_exchange_weak(n, n - 1)) return true;
    return false;
}

int check_device(const e2_ctx *ctx)
{
    if (injected_failure()) return E2_EHIP;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return E2_EHIP;
    return cur == ctx->device ? E2_OK : E2_EINVAL;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

// Scratch kept per stream between calls (e2_ctx_keep_scratch).  A call's
// temporary memory is one buffer; calls on one stream run in stream order,
// so they can all use the same buffer, which grows (stream-ordered free,
// then allocation) when a call needs more.  Keeping it removes the per-call
// allocation and release packets from the stream.  Streams are told apart
// by handle: the caller keeps every stream with calls in flight alive, so
// that no new stream takes a handle whose buffer is still in use.  Streams
// past the first kCachedStreams, and the per-thread default stream, allocate
// and free per call.
constexpr int kCachedStreams = 16;
struct StreamScratch {
    hipStream_t stream = nullptr;
    void *base = nullptr;
    size_t bytes = 0;
    std::mutex mu;  // held by a call from its lookup to the end of its launches
};
struct ScratchCache {
    std::mutex mu;
    std::list<StreamScratch> entries;  // stable addresses
};

namespace {

// Scratch for one call: the stream's kept buffer (locked for the call), or
// a stream-ordered allocation of the call's own.
struct Scratch {
    void *base = nullptr;
    hipStream_t stream = nullptr;
    bool owned = false;
    std::unique_lock<std::mutex> held;
    ~Scratch()
    {
        if (owned && base) (void)hipFreeAsync(base, stream);
    }
};

StreamScratch *stream_entry(e2_ctx *ctx, hipStream_t s)
{
    ScratchCache *c = ctx->scratch_cache;
    // hipStreamPerThread names a different stream in every host thread, so
    // one buffer behind that handle could serve two streams at once
    if (!c || s == hipStreamPerThread) return nullptr;
    std::lock_guard<std::mutex> g(c->mu);
    for (StreamScratch &e : c->entries)
        if (e.stream == s) return &e;
    if ((int)c->entries.size() >= kCachedStreams) return nullptr;
    c->entries.emplace_back();
    StreamScratch &e = c->entries.back();
    e.stream = s;
    return &e;
}

int alloc_scratch(e2_ctx *ctx, Scratch &sc, hipStream_t s, size_t bytes)
{
    sc.stream = s;
    if (StreamScratch *e = stream_entry(ctx, s)) {
        sc.held = std::unique_lock<std::mutex>(e->mu);
        if (e->bytes < bytes) {
            if (e->base) (void)hipFreeAsync(e->base, s);
            e->base = nullptr;
            e->bytes = 0;
            if (hipMallocAsync(&e->base, bytes, s) != hipSuccess) {
                e->base = nullptr;
                (void)hipGetLastError();
                return E2_ENOMEM;
            }
            e->bytes = bytes;
        }
        sc.base = e->base;
        return E2_OK;
    }
    sc.owned = true;
    if (hipMallocAsync(&sc.base, bytes, s) != hipSuccess) {
        sc.base = nullptr;
        (void)hipGetLastError();
        return E2_ENOMEM;
    }
    return E2_OK;
}

// Wait for the device, then release every kept buffer.
hipError_t free_scratch_cache(e2_ctx *ctx)
{
    ScratchCache *c = ctx->scratch_cache;
    if (!c) return hipSuccess;
    hipError_t err = hipSuccess;
    bool any = false;
    for (StreamScratch &e : c->entries) any = any || e.base;
    if (any) {
        err = hipDeviceSynchronize();
        for (StreamScratch &e : c->entries)
            if (e.base) {
                const hipError_t f = hipFreeAsync(e.base, nullptr);
                if (err == hipSuccess) err = f;
            }
        const hipError_t f = hipStreamSynchronize(nullptr);
        if (err == hipSuccess) err = f;
    }
    delete c;
    ctx->scratch_cache = nullptr;
    return err;
}

// Lay out counters, the problem list and the split-point fallback.
size_t work_bytes(const e2_ctx *ctx, int P, int k_max, int *slots, size_t *tb_bytes,
                  int n_r = 1, int objective = 0)
{
    const size_t problems = (size_t)P * k_max * n_r;
    const int np = (int)(problems < (size_t)INT32_MAX ? problems : INT32_MAX);
    *slots = objective == 2 ? e2_dp_idle_slots(np, ctx->M, ctx->N) : e2_dp_slots(ctx->N, np);
    const int mcap = ctx->M < ctx->N ? ctx->M : ctx->N;
    // the global split-point table is needed only when some chain's split
    // points (m - 1 rows of at most N cells) can exceed their LDS copy
    const bool need_tb = (size_t)(mcap - 1) * ctx->N > (size_t)e2_dp_lds_tb_cells(ctx->N);
    *tb_bytes = need_tb ? (size_t)(*slots) * ctx->N * ctx->N : 0;
    const size_t idle = objective == 2 ? (size_t)(*slots) * e2_dp_idle_bytes(ctx->M, ctx->N) : 0;
    return kCounterBytes + align256(problems * 4 * kListSegs) + align256(*tb_bytes) +
           align256(idle);
}

void carve_work(void *base, e2_ctx *ctx, int P, int k_max, int slots, size_t tb_bytes,
                E2Work *wk, int n_r = 1, int objective = 0)
{
    char *p = static_cast<char *>(base);
    wk->counters = reinterpret_cast<uint32_t *>(p);
    p += kCounterBytes;
    wk->list = reinterpret_cast<uint32_t *>(p);  // kListSegs segments of P * k_max * n_r
    p += align256((size_t)P * k_max * n_r * 4 * kListSegs);
    wk->tb_global = tb_bytes ? reinterpret_cast<uint8_t *>(p) : nullptr;
    p += align256(tb_bytes);
    wk->idle_stride = objective == 2 ? e2_dp_idle_bytes(ctx->M, ctx->N) : 0;
    wk->idle = objective == 2 ? reinterpret_cast<uint8_t *>(p) : nullptr;
    wk->n_slots = slots;
    wk->ev_begin = wk->ev_end = nullptr;
    if (ctx->dp_events && ctx->dp_events_used < ctx->dp_event_pairs) {
        wk->ev_begin = ctx->dp_events[2 * ctx->dp_events_used];
        wk->ev_end = ctx->dp_events[2 * ctx->dp_events_used + 1];
        ++ctx->dp_events_used;
    }
}

void free_dp_events(e2_ctx *ctx)
{
    if (!ctx->dp_events) return;
    for (int i = 0; i < 2 * ctx->dp_event_pairs; ++i) (void)hipEventDestroy(ctx->dp_events[i]);
    free(ctx->dp_events);
    ctx->dp_events = nullptr;
    ctx->dp_event_pairs = ctx->dp_events_used = 0;
}

int check_pop(int P, int k_max)
{
    if (P < 0 || P >= (1 << 24) || k_max < 1 || k_max > E2_MAX_CLUSTERS) return E2_EINVAL;
    return E2_OK;
}

// ceil(num / den) for den > 0; saturates to UINT64_MAX
uint64_t ceil_div(u128 num, uint64_t den)
{
    const u128 q = num / den + (num % den != 0);
    return (q >> 64) ? UINT64_MAX : (uint64_t)q;
}

// Decode tables for b = 2..b_max (role index b) from the one-request ones
// (role index 1): each further request adds ceil(beta * lone time) to a
// block and to the head, and a link carries b activations.
int extend_slots(const e2_problem *pr, int b_max, uint32_t beta_ppm, uint64_t *t, uint64_t *h,
                 uint64_t *tau)
{
    const int M = pr->n_dev, N = pr->n_layer;
    for (int b = 2; b <= b_max; ++b) {
        for (int d = 0; d < M; ++d) {
            for (int n = 0; n < N; ++n) {
                const uint64_t one = t[((size_t)M + d) * N + n];
                const uint64_t v = one + (uint64_t)(b - 1) * ceil_div((u128)one * beta_ppm, 1000000u);
                if (v >= kLimit48) return E2_EOVERFLOW;
                t[((size_t)b * M + d) * N + n] = v;
            }
            const uint64_t one = h[(size_t)M + d];
            const uint64_t hv = one + (uint64_t)(b - 1) * ceil_div((u128)one * beta_ppm, 1000000u);
            if (hv >= kLimit48) return E2_EOVERFLOW;
            h[(size_t)b * M + d] = hv;
        }
        for (int d = 0; d < M; ++d)
            for (int e = 0; e < M; ++e) {
                uint64_t v = 0;
                if (d != e) {
                    const size_t ix = (size_t)d * M + e;
                    const uint64_t beff =
                        (uint64_t)(((u128)pr->bw_Bps[ix] * pr->congestion_ppm[ix]) / 1000000u);
                    if (beff == 0) {
                        v = E2_INF64;
                    } else {
                        v = ceil_div((u128)pr->act_bytes[1] * (uint64_t)b * 1000000000u, beff);
                        if (v >= kLimit48) return E2_EOVERFLOW;
                    }
                }
                tau[((size_t)b * M + d) * M + e] = v;
            }
    }
    return E2_OK;
}

// Build a context: R = b_max + 1 role indices of time tables and, with KV
// bytes, one memory class per role index (block bytes W[n] + kv * slots,
// slots = 1 for prefill and b for decode with b requests).
int build_ctx(const e2_problem *prob, int b_max, uint32_t beta_ppm, uint64_t kv, e2_ctx **out)
{
    if (!out) return E2_EINVAL;
    *out = nullptr;
    int rc = check_problem(prob);
    if (rc) return rc;
    const int M = prob->n_dev, N = prob->n_layer;
    const int R = b_max + 1;
    const int C = kv ? R : 1;
    // kv * slots below must not wrap: with kv < 2^48 and slots <= 15 it
    // stays below 2^52, and the per-block test then catches 2^48 and above
    if (kv >= kLimit48) return E2_EOVERFLOW;
    std::vector<uint64_t> t((size_t)R * M * N), h((size_t)R * M), tau((size_t)R * M * M);
    rc = quantise(prob, t.data(), h.data(), tau.data());
    if (rc) return rc;
    if ((rc = extend_slots(prob, b_max, beta_ppm, t.data(), h.data(), tau.data()))) return rc;

    // prefix sums of block times per role and device
    std::vector<uint64_t> pref((size_t)R * M * (N + 1));
    for (int r = 0; r < R; ++r)
        for (int d = 0; d < M; ++d) {
            uint64_t *row = &pref[((size_t)r * M + d) * (N + 1)];
            row[0] = 0;
            for (int n = 0; n < N; ++n) row[n + 1] = row[n] + t[((size_t)r * M + d) * N + n];
        }
    // per memory class: block-byte prefix sums, then windows (smallest start
    // j such that bytes(j..i) (+ head) <= mem) forward and over reversed blocks
    std::vector<uint8_t> win((size_t)C * 2 * M * N), cap0((size_t)C * M), capH((size_t)C * M);
    std::vector<uint8_t> winR((size_t)C * M * N);
    std::vector<uint64_t> wpref(N + 1, 0);
    for (int c = 0; c < C; ++c) {
        const uint64_t extra_kv = kv * (uint64_t)(c == 0 ? 1 : c);
        for (int n = 0; n < N; ++n) {
            const uint64_t wb = prob->layer_bytes[n] + extra_kv;
            if (extra_kv >= kLimit48 || wb >= kLimit48) return E2_EOVERFLOW;
            wpref[n + 1] = wpref[n] + wb;
        }
        for (int f = 0; f < 2; ++f)
            for (int d = 0; d < M; ++d) {
                const uint64_t extra = f ? prob->head_bytes : 0;
                const uint64_t mem = prob->mem_bytes[d];
                int j = 0, best = 0;
                for (int i = 0; i < N; ++i) {
                    // advance j until blocks j..i (+ extra) fit or j passes i
                    while (j <= i && wpref[i + 1] - wpref[j] + extra > mem) ++j;
                    uint8_t v = E2_NO_START;
                    if (j <= i) {
                        v = (uint8_t)j;
                        if (i - j + 1 > best) best = i - j + 1;
                    }
                    win[(((size_t)c * 2 + f) * M + d) * N + i] = v;
                }
                (f ? capH : cap0)[(size_t)c * M + d] = (uint8_t)best;
            }
        for (int d = 0; d < M; ++d) {
            const uint64_t mem = prob->mem_bytes[d];
            // reversed blocks y..x are original blocks N-1-x..N-1-y
            int y = 0;
            for (int x = 0; x < N; ++x) {
                while (y <= x && wpref[N - y] - wpref[N - 1 - x] > mem) ++y;
                winR[((size_t)c * M + d) * N + x] = (y <= x) ? (uint8_t)y : E2_NO_START;
            }
        }
    }
    // reversed blocks (block N-1 first): prefix sums, used by the backward
    // rows of the DP, which run as forward rows on them
    std::vector<uint64_t> prefR((size_t)R * M * (N + 1));
    for (int r = 0; r < R; ++r)
        for (int d = 0; d < M; ++d) {
            const uint64_t *row = &pref[((size_t)r * M + d) * (N + 1)];
            uint64_t *rev = &prefR[((size_t)r * M + d) * (N + 1)];
            for (int x = 0; x <= N; ++x) rev[x] = row[N] - row[N - x];
        }

    // lower bounds of window lengths over cells i >= x (0 = no fitting cell)
    std::vector<uint8_t> minwin((size_t)C * 2 * M * N), minwinR((size_t)C * M * N);
    auto suffix_min = [N](const uint8_t *w, uint8_t *o) {
        int best = 0;  // 0 encodes "none yet"
        for (int x = N - 1; x >= 0; --x) {
            if (w[x] != E2_NO_START) {
                const int len = x - w[x] + 1;
                best = (best == 0 || len < best) ? len : best;
            }
            o[x] = (uint8_t)best;
        }
    };
    for (size_t row = 0; row < (size_t)C * 2 * M; ++row)
        suffix_min(&win[row * N], &minwin[row * N]);
    for (size_t row = 0; row < (size_t)C * M; ++row) suffix_min(&winR[row * N], &minwinR[row * N]);

    // largest cost of a memory-fitting stage per role and device (with the
    // head time for stages that carry the head bytes): every finite value a
    // DP over a chain produces is at most the largest of these over its
    // devices and its largest finite link time
    std::vector<uint64_t> vmax((size_t)R * M, 0);
    for (int r = 0; r < R; ++r) {
        const int c = C > 1 ? r : 0;
        for (int d = 0; d < M; ++d) {
            const uint64_t *row = &pref[((size_t)r * M + d) * (N + 1)];
            uint64_t best = 0;
            for (int f = 0; f < 2; ++f)
                for (int i = 0; i < N; ++i) {
                    const uint8_t j = win[(((size_t)c * 2 + f) * M + d) * N + i];
                    if (j == E2_NO_START) continue;
                    const uint64_t v = row[i + 1] - row[j] + (f ? h[(size_t)r * M + d] : 0);
                    if (v > best) best = v;
                }
            vmax[(size_t)r * M + d] = best;
        }
    }
    // largest prefix sum (+ head time) per role and device: every shifted
    // prefix sum of a chain stays below 2^53 when these and its link times
    // are below 2^45
    std::vector<uint8_t> hfit((size_t)M);
    for (int d = 0; d < M; ++d) hfit[d] = prob->head_bytes <= prob->mem_bytes[d];
    std::vector<uint64_t> vtot((size_t)R * M, 0);
    for (int r = 0; r < R; ++r)
        for (int d = 0; d < M; ++d)
            vtot[(size_t)r * M + d] =
                pref[((size_t)r * M + d) * (N + 1) + N] + h[(size_t)r * M + d];

    // one prefix row block per role index and device: P, PR, P x 256 and
    // PR x 256 as doubles, P << 8 and PR << 8 modulo 2^32 (the DP's packed
    // keys, value << 8 | index)
    const size_t X = (size_t)N + 1;
    std::vector<uint8_t> prow((size_t)R * M * kRowBlock * X);
    for (size_t b = 0; b < (size_t)R * M; ++b) {
        uint8_t *blk = &prow[b * kRowBlock * X];
        const uint64_t *P = &pref[b * X], *PR = &prefR[b * X];
        for (size_t x = 0; x < X; ++x) {
            const uint32_t p8 = (uint32_t)(P[x] << 8), pr8 = (uint32_t)(PR[x] << 8);
            const double p8d = (double)P[x] * 256.0, pr8d = (double)PR[x] * 256.0;
            memcpy(blk + kRowPref * X + 8 * x, &P[x], 8);
            memcpy(blk + kRowPrefR * X + 8 * x, &PR[x], 8);
            memcpy(blk + kRowPref8d * X + 8 * x, &p8d, 8);
            memcpy(blk + kRowPrefR8d * X + 8 * x, &pr8d, 8);
            memcpy(blk + kRowPref8u * X + 4 * x, &p8, 4);
            memcpy(blk + kRowPrefR8u * X + 4 * x, &pr8, 4);
        }
    }
    // one memory-window block per class: win, minwin, winR, minwinR
    const size_t MN = (size_t)M * N;
    std::vector<uint8_t> wtab((size_t)C * 6 * MN);
    for (int c = 0; c < C; ++c) {
        uint8_t *blk = &wtab[(size_t)c * 6 * MN];
        memcpy(blk, &win[(size_t)c * 2 * MN], 2 * MN);
        memcpy(blk + 2 * MN, &minwin[(size_t)c * 2 * MN], 2 * MN);
        memcpy(blk + 4 * MN, &winR[(size_t)c * MN], MN);
        memcpy(blk + 5 * MN, &minwinR[(size_t)c * MN], MN);
    }

    struct Part {
        const void *src;
        size_t bytes;
        char *dst;
    };
    Part parts[] = {{prow.data(), prow.size(), nullptr},       {h.data(), h.size() * 8, nullptr},
                    {tau.data(), tau.size() * 8, nullptr},     {wtab.data(), wtab.size(), nullptr},
                    {cap0.data(), cap0.size(), nullptr},       {capH.data(), capH.size(), nullptr},
                    {vmax.data(), vmax.size() * 8, nullptr},   {vtot.data(), vtot.size() * 8, nullptr},
                    {hfit.data(), hfit.size(), nullptr}};
    size_t total = 0;
    for (const Part &pt : parts) total += align256(pt.bytes);
    e2_ctx *ctx = static_cast<e2_ctx *>(calloc(1, sizeof(e2_ctx)));
    if (!ctx) return E2_ENOMEM;
    if (injected_failure()) {
        free(ctx);
        return E2_EHIP;
    }
    if (hipGetDevice(&ctx->device) != hipSuccess) {
        free(ctx);
        return E2_EHIP;
    }
    // the allocation-free entry point's scratch address on this device; a
    // failure is reported by that entry point, not here
    {
        void *unused = nullptr;
        (void)scratch_on(ctx->device, &unused);
    }
    if (hipMalloc(&ctx->blob, total) != hipSuccess) {
        (void)hipGetLastError();
        free(ctx);
        return E2_ENOMEM;
    }
    char *p = static_cast<char *>(ctx->blob);
    hipError_t e = hipSuccess;
    for (Part &pt : parts) {
        pt.dst = p;
        p += align256(pt.bytes);
        if (e == hipSuccess) e = hipMemcpy(pt.dst, pt.src, pt.bytes, hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        (void)hipFree(ctx->blob);
        free(ctx);
        return E2_EHIP;
    }
    ctx->M = M;
    ctx->N = N;
    ctx->b_max = b_max;
    ctx->head_bytes = prob->head_bytes;
    E2Tables &tb = ctx->tables;
    tb.prow = reinterpret_cast<const uint8_t *>(parts[0].dst);
    tb.head = reinterpret_cast<const uint64_t *>(parts[1].dst);
    tb.tau = reinterpret_cast<const uint64_t *>(parts[2].dst);
    tb.wtab = reinterpret_cast<const uint8_t *>(parts[3].dst);
    tb.cap0 = reinterpret_cast<const uint8_t *>(parts[4].dst);
    tb.capH = reinterpret_cast<const uint8_t *>(parts[5].dst);
    tb.vmax = reinterpret_cast<const uint64_t *>(parts[6].dst);
    tb.vtot = reinterpret_cast<const uint64_t *>(parts[7].dst);
    tb.hfit = reinterpret_cast<const uint8_t *>(parts[8].dst);
    tb.M = M;
    tb.N = N;
    tb.R = R;
    tb.n_mem = C;
    *out = ctx;
    return E2_OK;
}

}  // namespace

extern "C" {

const char *e2_strerror(int code)
{
    switch (code) {
    case E2_OK: return "ok";
    case E2_EINVAL: return "invalid argument";
    case E2_EOVERFLOW: return "quantised value reaches 2^48";
    case E2_ENOMEM: return "out of memory";
    case E2_EHIP: return "HIP runtime error";
    default: return "unknown error";
    }
}

int e2_debug_inject_hip_error(int32_t calls)
{
    if (calls < 0) return E2_EINVAL;
    return g_inject.exchange(calls);
}

int e2_quantise(const e2_problem *prob, uint64_t *t, uint64_t *h, uint64_t *tau)
{
    const int rc = check_problem(prob);
    if (rc) return rc;
    if (!t || !h || !tau) return E2_EINVAL;
    return quantise(prob, t, h, tau);
}

int e2_ctx_create(const e2_problem *prob, e2_ctx **out)
{
    return build_ctx(prob, 1, 0, 0, out);
}

int e2_ctx_create_slots(const e2_problem *prob, const e2_slot_model *sm, e2_ctx **out)
{
    if (!out) return E2_EINVAL;
    *out = nullptr;
    if (!sm || sm->b_max < 1 || sm->b_max > E2_MAX_SLOTS || sm->beta_ppm > 1000000u)
        return E2_EINVAL;
    return build_ctx(prob, sm->b_max, sm->beta_ppm, sm->kv_bytes_per_block_slot, out);
}

int e2_ctx_destroy(e2_ctx *ctx)
{
    if (!ctx) return E2_EINVAL;
    free_dp_events(ctx);
    const hipError_t es = free_scratch_cache(ctx);
    const hipError_t e = hipFree(ctx->blob);
    free(ctx);
    return e == hipSuccess && es == hipSuccess ? E2_OK : E2_EHIP;
}

int e2_ctx_keep_scratch(e2_ctx *ctx, int32_t enable)
{
    if (!ctx || (enable != 0 && enable != 1)) return E2_EINVAL;
    int rc = check_device(ctx);
    if (rc) return rc;
    if (!enable) return free_scratch_cache(ctx) == hipSuccess ? E2_OK : E2_EHIP;
    if (!ctx->scratch_cache) ctx->scratch_cache = new (std::nothrow) ScratchCache;
    return ctx->scratch_cache ? E2_OK : E2_ENOMEM;
}

int e2_ctx_dp_timing(e2_ctx *ctx, int32_t max_launches)
{
    if (!ctx || max_launches < 0 || max_launches > 4096) return E2_EINVAL;
    int rc = check_device(ctx);
    if (rc) return rc;
    free_dp_events(ctx);
    if (max_launches == 0) return E2_OK;
    ctx->dp_events = static_cast<hipEvent_t *>(calloc(2 * (size_t)max_launches, sizeof(hipEvent_t)));
    if (!ctx->dp_events) return E2_ENOMEM;
    for (int i = 0; i < 2 * max_launches; ++i)
        if (hipEventCreate(&ctx->dp_events[i]) != hipSuccess) {
            (void)hipGetLastError();
            for (int k = 0; k < i; ++k) (void)hipEventDestroy(ctx->dp_events[k]);
            free(ctx->dp_events);
            ctx->dp_events = nullptr;
            return E2_EHIP;
        }
    ctx->dp_event_pairs = max_launches;
    ctx->dp_events_used = 0;
    return E2_OK;
}

int e2_ctx_dp_elapsed(e2_ctx *ctx, int32_t *launches, double *total_ms)
{
    if (!ctx || !launches || !total_ms) return E2_EINVAL;
    int rc = check_device(ctx);
    if (rc) return rc;
    double sum = 0;
    for (int i = 0; i < ctx->dp_events_used; ++i) {
        float ms = 0;
        if (hipEventSynchronize(ctx->dp_events[2 * i + 1]) != hipSuccess ||
            hipEventElapsedTime(&ms, ctx->dp_events[2 * i], ctx->dp_events[2 * i + 1]) !=
                hipSuccess) {
            (void)hipGetLastError();
            return E2_EHIP;
        }
        sum += ms;
    }
    *launches = ctx->dp_events_used;
    *total_ms = sum;
    return E2_OK;
}

}  // extern "C"

namespace {

int solve_impl(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const E2Genomes &gen,
               const uint8_t *roles, uint64_t *T, uint64_t *Lambda, int16_t *master,
               uint8_t *layers, int objective = 0)
{
    if (!ctx) return E2_EINVAL;
    int rc = check_pop(P, k_max);
    if (rc) return rc;
    if (P == 0) return E2_OK;
    if (!roles || !T || !Lambda || !master || !layers) return E2_EINVAL;
    if ((rc = check_device(ctx))) return rc;
    hipStream_t s = as_stream(stream);
    int slots;
    size_t tbb;
    const size_t bytes = work_bytes(ctx, P, k_max, &slots, &tbb, 1, objective);
    Scratch sc;
    if ((rc = alloc_scratch(ctx, sc, s, bytes))) return rc;
    E2Work wk;
    carve_work(sc.base, ctx, P, k_max, slots, tbb, &wk, 1, objective);
    const hipError_t e = e2_launch_partitions(ctx->tables, s, P, k_max, gen, roles, wk, T,
                                              Lambda, master, layers, objective);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

int eval_impl(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const E2Genomes &gen,
              const uint8_t *roles, const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
              uint64_t *s_p, uint64_t *s_d, int objective = 0)
{
    if (!ctx || !fp) return E2_EINVAL;
    int rc = check_pop(P, k_max);
    if (rc) return rc;
    if (fp->nd_tokens > 8192) return E2_EINVAL;
    if (P == 0) return E2_OK;
    if (!roles || !w || !phase) return E2_EINVAL;
    if ((rc = check_device(ctx))) return rc;
    hipStream_t s = as_stream(stream);
    int slots;
    size_t tbb;
    const size_t wb = work_bytes(ctx, P, k_max, &slots, &tbb, 1, objective);
    const size_t tl = align256((size_t)P * k_max * 8);
    Scratch sc;
    if ((rc = alloc_scratch(ctx, sc, s, wb + 2 * tl))) return rc;
    E2Work wk;
    carve_work(sc.base, ctx, P, k_max, slots, tbb, &wk, 1, objective);
    uint64_t *Ts = reinterpret_cast<uint64_t *>(static_cast<char *>(sc.base) + wb);
    uint64_t *Ls = reinterpret_cast<uint64_t *>(static_cast<char *>(sc.base) + wb + tl);
    hipError_t e = e2_launch_partitions(ctx->tables, s, P, k_max, gen, roles, wk, Ts, Ls,
                                        nullptr, nullptr, objective);
    if (e != hipSuccess) return E2_EHIP;
    const uint64_t lam_max =
        fp->min_tps_milli ? 1000000000000ull / fp->min_tps_milli : E2_INF64;
    e = e2_launch_fitness(s, P, k_max, Ts, Ls, roles, fp->t_arrival_ns, fp->nd_tokens, lam_max,
                          w, phase, s_p, s_d);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

// Every cluster for every role index, then the role assignment of policy
// 0 (brute force) or 1 (adapted SplitWise).
int roles_impl(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const E2Genomes &gen,
               const e2_fitness_params *fp, int policy, uint32_t np_tokens, uint8_t *roles_out,
               uint8_t *slots_out, uint64_t *w, uint64_t *phase, uint64_t *T_all,
               uint64_t *Lambda_all)
{
    if (!ctx || !fp) return E2_EINVAL;
    if (P < 0 || P >= (1 << 20) || k_max < 1 || k_max > E2_MAX_CLUSTERS) return E2_EINVAL;
    if (fp->nd_tokens > 8192) return E2_EINVAL;
    if ((T_all == nullptr) != (Lambda_all == nullptr)) return E2_EINVAL;
    if (P == 0) return E2_OK;
    if (!(gen.labels || (gen.order && gen.sizes)) || !roles_out || !slots_out || !w || !phase)
        return E2_EINVAL;
    int rc = check_device(ctx);
    if (rc) return rc;
    const int R = ctx->b_max + 1;
    hipStream_t s = as_stream(stream);
    int slots;
    size_t tbb;
    const size_t wb = work_bytes(ctx, P, k_max, &slots, &tbb, R);
    const size_t tl = T_all ? 0 : align256((size_t)P * k_max * R * 8);
    Scratch sc;
    if ((rc = alloc_scratch(ctx, sc, s, wb + 2 * tl))) return rc;
    E2Work wk;
    carve_work(sc.base, ctx, P, k_max, slots, tbb, &wk, R);
    uint64_t *Ts = T_all ? T_all : reinterpret_cast<uint64_t *>(static_cast<char *>(sc.base) + wb);
    uint64_t *Ls = Lambda_all ? Lambda_all
                              : reinterpret_cast<uint64_t *>(static_cast<char *>(sc.base) + wb + tl);
    hipError_t e = e2_launch_partitions(ctx->tables, s, P, k_max, gen, nullptr, wk, Ts, Ls,
                                        nullptr, nullptr);
    if (e != hipSuccess) return E2_EHIP;
    const uint64_t lam_max =
        fp->min_tps_milli ? 1000000000000ull / fp->min_tps_milli : E2_INF64;
    e = e2_launch_roles(s, P, ctx->M, k_max, R, policy, np_tokens, gen.labels, Ts, Ls,
                        fp->t_arrival_ns, fp->nd_tokens, lam_max, roles_out, slots_out, w, phase);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

bool overlap(const void *a, size_t na, const void *b, size_t nb)
{
    const char *x = static_cast<const char *>(a), *y = static_cast<const char *>(b);
    return x < y + nb && y < x + na;
}

}  // namespace

extern "C" {

int e2_solve_partitions(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                        const uint8_t *labels, const uint8_t *roles, uint64_t *T,
                        uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return solve_impl(ctx, stream, P, k_max, gen, roles, T, Lambda, master, layers);
}

int e2_eval_population(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                       const uint8_t *labels, const uint8_t *roles, const e2_fitness_params *fp,
                       uint64_t *w, uint64_t *phase, uint64_t *s_p, uint64_t *s_d)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return eval_impl(ctx, stream, P, k_max, gen, roles, fp, w, phase, s_p, s_d);
}

int e2_solve_partitions_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                                const uint8_t *order, const uint16_t *sizes,
                                const uint8_t *roles, uint64_t *T, uint64_t *Lambda,
                                int16_t *master, uint8_t *layers)
{
    if (P > 0 && (!order || !sizes)) return E2_EINVAL;
    const E2Genomes gen = {nullptr, order, sizes};
    return solve_impl(ctx, stream, P, k_max, gen, roles, T, Lambda, master, layers);
}

int e2_eval_population_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                               const uint8_t *order, const uint16_t *sizes, const uint8_t *roles,
                               const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                               uint64_t *s_p, uint64_t *s_d)
{
    if (P > 0 && (!order || !sizes)) return E2_EINVAL;
    const E2Genomes gen = {nullptr, order, sizes};
    return eval_impl(ctx, stream, P, k_max, gen, roles, fp, w, phase, s_p, s_d);
}

int e2_ga_step_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                       const uint8_t *order_in, const uint16_t *sizes_in, const uint8_t *roles_in,
                       const uint64_t *w_in, const uint64_t *phase_in, const e2_ga2_params *gp,
                       uint8_t *order_out, uint16_t *sizes_out, uint8_t *roles_out)
{
    if (!ctx || !gp) return E2_EINVAL;
    int rc = check_pop(P, k_max);
    if (rc) return rc;
    if (P == 0) return E2_OK;
    if (!order_in || !sizes_in || !roles_in || !w_in || !phase_in || !order_out || !sizes_out ||
        !roles_out)
        return E2_EINVAL;
    if (gp->tournament_k < 1 || gp->tournament_k > 64 || gp->n_elite > 256 ||
        gp->n_elite > (uint32_t)P || gp->max_replica < 1 || gp->max_replica > 256)
        return E2_EINVAL;
    const size_t no = (size_t)P * ctx->M, ns = (size_t)P * k_max * 2, nr = (size_t)P * k_max;
    const size_t nk = (size_t)P * 8;
    const void *ins[5] = {order_in, sizes_in, roles_in, w_in, phase_in};
    const size_t nin[5] = {no, ns, nr, nk, nk};
    void *outs[3] = {order_out, sizes_out, roles_out};
    for (int i = 0; i < 3; ++i) {
        for (int j = 0; j < 5; ++j)
            if (overlap(outs[i], nin[i], ins[j], nin[j])) return E2_EINVAL;
        for (int j = i + 1; j < 3; ++j)
            if (overlap(outs[i], nin[i], outs[j], nin[j])) return E2_EINVAL;
    }
    if ((rc = check_device(ctx))) return rc;
    hipStream_t s = as_stream(stream);
    Scratch sc;
    if ((rc = alloc_scratch(ctx, sc, s, align256(256 * 4)))) return rc;
    const hipError_t e = e2_launch_ga_ordered(
        s, ctx->M, P, k_max, order_in, sizes_in, roles_in, w_in, phase_in, gp->seed,
        gp->generation, gp->tournament_k, gp->mutation_thresh_u32, gp->n_elite, gp->max_replica,
        static_cast<uint32_t *>(sc.base), order_out, sizes_out, roles_out);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

int e2_search_roles(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const uint8_t *labels,
                    const e2_fitness_params *fp, uint8_t *roles_out, uint8_t *slots_out,
                    uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return roles_impl(ctx, stream, P, k_max, gen, fp, 0, 0, roles_out, slots_out, w, phase,
                      T_all, Lambda_all);
}

int e2_search_roles_ordered(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                            const uint8_t *order, const uint16_t *sizes,
                            const e2_fitness_params *fp, uint8_t *roles_out, uint8_t *slots_out,
                            uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all)
{
    if (P > 0 && (!order || !sizes)) return E2_EINVAL;
    const E2Genomes gen = {nullptr, order, sizes};
    return roles_impl(ctx, stream, P, k_max, gen, fp, 0, 0, roles_out, slots_out, w, phase,
                      T_all, Lambda_all);
}

int e2_assign_roles_splitwise(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                              const uint8_t *labels, const e2_fitness_params *fp,
                              uint32_t np_tokens, uint8_t *roles_out, uint8_t *slots_out,
                              uint64_t *w, uint64_t *phase, uint64_t *T_all, uint64_t *Lambda_all)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return roles_impl(ctx, stream, P, k_max, gen, fp, 1, np_tokens, roles_out, slots_out, w,
                      phase, T_all, Lambda_all);
}

int e2_solve_partitions_ft(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                           const uint8_t *labels, const uint8_t *roles, uint64_t *T,
                           uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return solve_impl(ctx, stream, P, k_max, gen, roles, T, Lambda, master, layers, 1);
}

int e2_solve_partitions_idle(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                             const uint8_t *labels, const uint8_t *roles, uint64_t *T,
                             uint64_t *Lambda, int16_t *master, uint8_t *layers)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return solve_impl(ctx, stream, P, k_max, gen, roles, T, Lambda, master, layers, 2);
}

int e2_eval_population_idle(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                            const uint8_t *labels, const uint8_t *roles,
                            const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                            uint64_t *s_p, uint64_t *s_d)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return eval_impl(ctx, stream, P, k_max, gen, roles, fp, w, phase, s_p, s_d, 2);
}

int e2_eval_population_ft(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                          const uint8_t *labels, const uint8_t *roles,
                          const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                          uint64_t *s_p, uint64_t *s_d)
{
    if (P > 0 && !labels) return E2_EINVAL;
    const E2Genomes gen = {labels, nullptr, nullptr};
    return eval_impl(ctx, stream, P, k_max, gen, roles, fp, w, phase, s_p, s_d, 1);
}

int e2_eval_population_noalloc(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max,
                               const uint8_t *labels, const uint8_t *roles,
                               const e2_fitness_params *fp, uint64_t *w, uint64_t *phase,
                               uint64_t *s_p, uint64_t *s_d)
{
    if (!ctx || !fp) return E2_EINVAL;
    int rc = check_pop(P, k_max);
    if (rc) return rc;
    if (fp->nd_tokens > 8192) return E2_EINVAL;
    if (P == 0) return E2_OK;
    if (!labels || !roles || !w || !phase) return E2_EINVAL;
    if ((rc = check_device(ctx))) return rc;
    // layout of the fixed scratch: counters, list, T and Lambda, then as
    // many DP waves' row regions (and split-point tables) as still fit
    const size_t problems = (size_t)P * k_max;
    const size_t tl = align256(problems * 8);
    const size_t fixed = kCounterBytes + align256(problems * 4 * kListSegs) + 2 * tl;
    const int mcap = ctx->M < ctx->N ? ctx->M : ctx->N;
    const bool need_tb = (size_t)(mcap - 1) * ctx->N > (size_t)e2_dp_lds_tb_cells(ctx->N);
    const size_t per_wave = need_tb ? (size_t)ctx->N * ctx->N : 0;
    if (fixed + per_wave + 256 > kNoAllocBytes) return E2_EINVAL;  // beyond the maximum
    const int np = (int)(problems < (size_t)INT32_MAX ? problems : INT32_MAX);
    int slots = e2_dp_slots(ctx->N, np);
    if (per_wave) {
        const size_t fit = (kNoAllocBytes - fixed - 256) / per_wave;
        if ((size_t)slots > fit) slots = (int)fit;
    }
    const size_t tbb = need_tb ? (size_t)slots * ctx->N * ctx->N : 0;
    void *base = nullptr;
    if ((rc = scratch_on(ctx->device, &base))) return rc;
    E2Work wk;
    carve_work(base, ctx, P, k_max, slots, tbb, &wk);
    char *after = static_cast<char *>(base) + kCounterBytes + align256(problems * 4 * kListSegs) +
                  align256(tbb);
    uint64_t *Ts = reinterpret_cast<uint64_t *>(after);
    uint64_t *Ls = reinterpret_cast<uint64_t *>(after + tl);
    hipStream_t s = as_stream(stream);
    hipError_t e = e2_launch_partitions(ctx->tables, s, P, k_max, {labels, nullptr, nullptr},
                                        roles, wk, Ts, Ls, nullptr, nullptr);
    if (e != hipSuccess) return E2_EHIP;
    const uint64_t lam_max =
        fp->min_tps_milli ? 1000000000000ull / fp->min_tps_milli : E2_INF64;
    e = e2_launch_fitness(s, P, k_max, Ts, Ls, roles, fp->t_arrival_ns, fp->nd_tokens, lam_max,
                          w, phase, s_p, s_d);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

int e2_ga_step(e2_ctx *ctx, void *stream, int32_t P, int32_t k_max, const uint8_t *labels_in,
               const uint8_t *roles_in, const uint64_t *w_in, const uint64_t *phase_in,
               const e2_ga_params *gp, uint8_t *labels_out, uint8_t *roles_out)
{
    if (!ctx || !gp) return E2_EINVAL;
    int rc = check_pop(P, k_max);
    if (rc) return rc;
    if (P == 0) return E2_OK;
    if (!labels_in || !roles_in || !w_in || !phase_in || !labels_out || !roles_out)
        return E2_EINVAL;
    if (gp->tournament_k < 1 || gp->tournament_k > 64 || gp->n_elite > 256 ||
        gp->n_elite > (uint32_t)P)
        return E2_EINVAL;
    const size_t M = (size_t)ctx->M;
    // outputs must not overlap the inputs
    const size_t nl = (size_t)P * M, nr = (size_t)P * k_max, nk = (size_t)P * 8;
    const void *ins[4] = {labels_in, roles_in, w_in, phase_in};
    const size_t nin[4] = {nl, nr, nk, nk};
    for (int j = 0; j < 4; ++j)
        if (overlap(labels_out, nl, ins[j], nin[j]) || overlap(roles_out, nr, ins[j], nin[j]))
            return E2_EINVAL;
    if (overlap(labels_out, nl, roles_out, nr)) return E2_EINVAL;
    if ((rc = check_device(ctx))) return rc;
    hipStream_t s = as_stream(stream);
    Scratch sc;
    if ((rc = alloc_scratch(ctx, sc, s, align256(256 * 4)))) return rc;
    const hipError_t e = e2_launch_ga(s, ctx->M, P, k_max, labels_in, roles_in, w_in, phase_in,
                                      gp->seed, gp->generation, gp->tournament_k,
                                      gp->crossover_thresh_u32, gp->mutation_thresh_u32,
                                      gp->n_elite, static_cast<uint32_t *>(sc.base), labels_out,
                                      roles_out);
    return e == hipSuccess ? E2_OK : E2_EHIP;
}

}  // extern "C"
