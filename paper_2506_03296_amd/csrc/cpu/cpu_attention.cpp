// cpu_attention.cpp -- host side of include/apex_cpu_attention.h.
//
// Validates arguments, cuts the batch into work items, runs them on a
// persistent thread pool with a shared atomic item counter (longest items
// first), merges split pairs with the log-sum-exp identity and writes fp16
// rows.  The SIMD inner loops live in attend_simd.cpp (one build per ISA);
// this file is compiled for baseline x86-64 and picks the ISA with cpuid.
#include <cpuid.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include <sched.h>

#include "apex_cpu_attention.h"
#include "attend.h"

namespace {

thread_local char g_last_error[512] = "";

__attribute__((format(printf, 2, 3))) int fail(int code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

}  // namespace

namespace apex_cpu {
// error reporting shared with the scheduler (scheduler.cpp)
__attribute__((visibility("hidden"), format(printf, 2, 3))) int sched_fail(int code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}
}  // namespace apex_cpu

namespace {

constexpr int kMaxD = 512;
constexpr int kMaxG = 64;
constexpr int kDefaultMinChunk = 512;
constexpr int kItemsPerThread = 4;

// ---------------------------------------------------------------------------
// ISA selection
// ---------------------------------------------------------------------------

int detect_isa()
{
    unsigned a, b, c, d;
    if (!__get_cpuid(1, &a, &b, &c, &d)) return 0;
    const bool f16c = (c >> 29) & 1u;
    const bool fma = (c >> 12) & 1u;
    __builtin_cpu_init();
    if (!f16c || !fma || !__builtin_cpu_supports("avx2")) return 0;
    if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
        __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512dq"))
        return 2;
    return 1;
}

int isa()
{
    static const int v = detect_isa();
    return v;
}

struct Kernels {
    void (*attend)(const apex_cpu::Problem&, int, int, int, int, apex_cpu::State, float*);
    void (*finish)(const float*, const float*, const float*, int, int, uint16_t*, float*);
    void (*merge)(const float* const*, const float* const*, const float* const*, int, int, int,
                  float*, float*, float*);
};

Kernels kernels_for(int level)
{
    if (level == 2)
        return {apex_cpu::simd_avx512::attend, apex_cpu::simd_avx512::finish, apex_cpu::simd_avx512::merge};
    return {apex_cpu::simd_avx2::attend, apex_cpu::simd_avx2::finish, apex_cpu::simd_avx2::merge};
}

// ---------------------------------------------------------------------------
// persistent thread pool: run(n_threads, fn) calls fn(thread_index) on the
// caller (index 0) and n_threads - 1 workers, and returns when all are done
// ---------------------------------------------------------------------------

class Pool {
public:
    ~Pool() { stop(); }

    int size()
    {
        std::lock_guard<std::mutex> lk(m_);
        return (int)workers_.size() + 1;
    }

    void resize(int n)
    {
        stop();
        std::lock_guard<std::mutex> lk(m_);
        stopping_ = false;
        // a new worker waits for the next job, not one that already ran
        const uint64_t current = generation_;
        for (int i = 1; i < n; ++i) workers_.emplace_back([this, i, current] { loop(i, current); });
    }

    void run(int n_threads, const std::function<void(int)>& fn)
    {
        {
            std::lock_guard<std::mutex> lk(m_);
            job_ = &fn;
            active_ = n_threads;
            remaining_ = n_threads - 1;
            ++generation_;
        }
        cv_.notify_all();
        fn(0);
        std::unique_lock<std::mutex> lk(m_);
        done_.wait(lk, [this] { return remaining_ == 0; });
        job_ = nullptr;
    }

private:
    void loop(int index, uint64_t seen)
    {
        for (;;) {
            const std::function<void(int)>* job;
            {
                std::unique_lock<std::mutex> lk(m_);
                cv_.wait(lk, [&] { return stopping_ || generation_ != seen; });
                if (stopping_) return;
                seen = generation_;
                if (index >= active_) continue;
                job = job_;
            }
            (*job)(index);
            {
                std::lock_guard<std::mutex> lk(m_);
                if (--remaining_ == 0) done_.notify_one();
            }
        }
    }

    void stop()
    {
        {
            std::lock_guard<std::mutex> lk(m_);
            stopping_ = true;
        }
        cv_.notify_all();
        for (auto& t : workers_) t.join();
        workers_.clear();
    }

    std::mutex m_;
    std::condition_variable cv_, done_;
    std::vector<std::thread> workers_;
    const std::function<void(int)>* job_ = nullptr;
    uint64_t generation_ = 0;
    int active_ = 0;
    int remaining_ = 0;
    bool stopping_ = false;
};

std::mutex g_call_mutex;   // one call at a time uses the pool and the scratch
Pool g_pool;
bool g_pool_ready = false;

int available_cores()
{
    cpu_set_t set;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) {
        const int n = CPU_COUNT(&set);
        if (n > 0) return n;
    }
    const unsigned n = std::thread::hardware_concurrency();
    return n > 0 ? (int)n : 1;
}

void ensure_pool()
{
    if (!g_pool_ready) {
        g_pool.resize(available_cores());
        g_pool_ready = true;
    }
}

// per-call scratch, reused across calls (guarded by g_call_mutex)
std::vector<float> g_partials;
std::vector<float> g_thread_scratch;

struct Split {
    int b, g;
    int64_t first_slot;
    int chunks;
};

int run(const apex_cpu_args& a)
{
    const int G = a.Hq / a.Hkv;
    const int level = (a.flags & APEX_CPU_FLAG_FORCE_AVX2) ? std::min(isa(), 1) : isa();
    if (level == 0) return fail(APEX_ERR_UNSUPPORTED, "this CPU lacks AVX2 + FMA + F16C");
    const Kernels K = kernels_for(level);

    int64_t max_len = 0;
    for (int b = 0; b < a.B; ++b) max_len = std::max<int64_t>(max_len, a.context_lens[b]);
    const int64_t stride =
        a.block_table_stride ? a.block_table_stride : std::max<int64_t>(1, (max_len + a.block_size - 1) / a.block_size);

    apex_cpu::Problem p;
    p.q = (const uint16_t*)a.q;
    p.k = (const uint16_t*)a.k_cache;
    p.v = (const uint16_t*)a.v_cache;
    p.block_table = a.block_table;
    p.stride = stride;
    p.Hq = a.Hq;
    p.Hkv = a.Hkv;
    p.G = G;
    p.d = a.d;
    p.bs = a.block_size;
    p.scale_log2 = a.scale * 1.4426950408889634f;

    ensure_pool();
    int threads = g_pool.size();
    if (a.num_threads > 0) threads = std::min(threads, a.num_threads);

    // zero rows for empty requests; count the work
    uint16_t* out = (uint16_t*)a.out;
    int64_t pairs = 0, tokens = 0;
    for (int b = 0; b < a.B; ++b) {
        const int L = a.context_lens[b];
        if (L <= 0) {
            memset(out + (int64_t)b * a.Hq * a.d, 0, sizeof(uint16_t) * (size_t)a.Hq * a.d);
            if (a.lse_out)
                for (int h = 0; h < a.Hq; ++h) a.lse_out[(int64_t)b * a.Hq + h] = -INFINITY;
            continue;
        }
        pairs += a.Hkv;
        tokens += (int64_t)L * a.Hkv;
    }
    if (pairs == 0) return APEX_OK;

    // chunk size: whole pairs when there are enough of them to balance the
    // threads, otherwise block-aligned chunks so that there are about
    // kItemsPerThread items per thread
    int64_t chunk = INT64_MAX;
    const int64_t want = (int64_t)kItemsPerThread * threads;
    if (pairs < want) {
        const int64_t min_chunk = a.min_chunk_tokens > 0 ? a.min_chunk_tokens : kDefaultMinChunk;
        chunk = std::max<int64_t>(min_chunk, (tokens + want - 1) / want);
        chunk = (chunk + a.block_size - 1) / a.block_size * a.block_size;
    }
    std::vector<apex_cpu::Item> items;
    std::vector<Split> splits;
    int64_t slots = 0;
    for (int b = 0; b < a.B; ++b) {
        const int L = a.context_lens[b];
        if (L <= 0) continue;
        const int64_t n = L <= chunk ? 1 : (L + chunk - 1) / chunk;
        for (int g = 0; g < a.Hkv; ++g) {
            if (n == 1) {
                items.push_back({b, g, 0, L, -1});
                continue;
            }
            splits.push_back({b, g, slots, (int)n});
            for (int64_t c = 0; c < n; ++c) {
                const int t0 = (int)(c * chunk);
                const int t1 = (int)std::min<int64_t>(L, (c + 1) * chunk);
                items.push_back({b, g, t0, t1, slots++});
            }
        }
    }
    std::stable_sort(items.begin(), items.end(), [](const apex_cpu::Item& x, const apex_cpu::Item& y) {
        return x.t1 - x.t0 > y.t1 - y.t0;
    });

    const int64_t per_state = (int64_t)G * (a.d + 2);
    g_partials.resize((size_t)std::max<int64_t>(1, slots * per_state));
    const int64_t scratch_each = apex_cpu::scratch_floats(G, a.d) + (int64_t)G * (a.d + 2);
    g_thread_scratch.resize((size_t)(scratch_each * threads));

    std::atomic<int64_t> next(0);
    const int64_t n_items = (int64_t)items.size();
    float* partials = g_partials.data();
    const int d = a.d, Hq = a.Hq;
    float* lse = a.lse_out;
    g_pool.run(threads, [&](int tid) {
        float* scratch = g_thread_scratch.data() + scratch_each * tid;
        float* own = scratch + apex_cpu::scratch_floats(G, d);   // m, l, acc of a direct item
        for (;;) {
            const int64_t i = next.fetch_add(1, std::memory_order_relaxed);
            if (i >= n_items) break;
            const apex_cpu::Item& it = items[(size_t)i];
            float* base = it.slot >= 0 ? partials + it.slot * per_state : own;
            apex_cpu::State st{base, base + G, base + 2 * G};
            K.attend(p, it.b, it.g, it.t0, it.t1, st, scratch);
            if (it.slot < 0) {
                const int64_t row = (int64_t)it.b * Hq + (int64_t)it.g * G;
                K.finish(st.m, st.l, st.acc, G, d, out + row * d, lse ? lse + row : nullptr);
            }
        }
    });

    if (!splits.empty()) {
        // the chunks of a split occupy consecutive partial slots; the pointer
        // arrays are built here so that the workers allocate nothing
        std::vector<const float*> ms((size_t)slots), ls((size_t)slots), accs((size_t)slots);
        for (int64_t i = 0; i < slots; ++i) {
            const float* base = partials + i * per_state;
            ms[(size_t)i] = base;
            ls[(size_t)i] = base + G;
            accs[(size_t)i] = base + 2 * G;
        }
        std::atomic<int64_t> next_split(0);
        const int64_t n_splits = (int64_t)splits.size();
        g_pool.run(threads, [&](int tid) {
            float* merged = g_thread_scratch.data() + scratch_each * tid;
            for (;;) {
                const int64_t i = next_split.fetch_add(1, std::memory_order_relaxed);
                if (i >= n_splits) break;
                const Split& s = splits[(size_t)i];
                const size_t f = (size_t)s.first_slot;
                float* mm = merged;
                float* ll = merged + G;
                float* aa = merged + 2 * G;
                K.merge(&ms[f], &ls[f], &accs[f], s.chunks, G, d, mm, ll, aa);
                const int64_t row = (int64_t)s.b * Hq + (int64_t)s.g * G;
                K.finish(mm, ll, aa, G, d, out + row * d, lse ? lse + row : nullptr);
            }
        });
    }
    return APEX_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

int validate(const apex_cpu_args& a)
{
    if (a.B < 0) return fail(APEX_ERR_INVALID_ARG, "B = %d is negative", a.B);
    if (a.Hq <= 0 || a.Hkv <= 0) return fail(APEX_ERR_INVALID_ARG, "Hq and Hkv must be positive");
    if (a.Hq % a.Hkv != 0) return fail(APEX_ERR_INVALID_ARG, "Hq = %d is not a multiple of Hkv = %d", a.Hq, a.Hkv);
    if (a.block_size <= 0) return fail(APEX_ERR_INVALID_ARG, "block_size must be positive");
    if (a.d <= 0 || a.d % 16 != 0 || a.d > kMaxD)
        return fail(APEX_ERR_UNSUPPORTED, "head dim %d unsupported (a multiple of 16 up to %d)", a.d, kMaxD);
    if (a.Hq / a.Hkv > kMaxG) return fail(APEX_ERR_UNSUPPORTED, "group size %d above %d", a.Hq / a.Hkv, kMaxG);
    if (a.block_table_stride < 0) return fail(APEX_ERR_INVALID_ARG, "block_table_stride is negative");
    if (a.num_threads < 0 || a.min_chunk_tokens < 0)
        return fail(APEX_ERR_INVALID_ARG, "num_threads and min_chunk_tokens must be >= 0");
    if (a.flags & ~APEX_CPU_FLAG_FORCE_AVX2) return fail(APEX_ERR_INVALID_ARG, "unknown flags");
    if (a.B == 0) return APEX_OK;
    if (!a.q || !a.k_cache || !a.v_cache || !a.block_table || !a.context_lens || !a.out)
        return fail(APEX_ERR_INVALID_ARG, "a pointer is NULL");
    const size_t qo = (size_t)a.B * a.Hq * a.d * 2;
    if (overlaps(a.out, qo, a.q, qo)) return fail(APEX_ERR_INVALID_ARG, "out overlaps q");
    if (overlaps(a.out, qo, a.context_lens, (size_t)a.B * 4))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps context_lens");
    if (a.lse_out && overlaps(a.lse_out, (size_t)a.B * a.Hq * 4, a.out, qo))
        return fail(APEX_ERR_INVALID_ARG, "lse_out overlaps out");
    if (a.block_table_stride > 0) {
        for (int b = 0; b < a.B; ++b) {
            const int64_t nb = a.context_lens[b] > 0 ? (a.context_lens[b] + (int64_t)a.block_size - 1) / a.block_size : 0;
            if (nb > a.block_table_stride)
                return fail(APEX_ERR_INVALID_ARG, "request %d needs %lld blocks, table rows hold %lld", b,
                            (long long)nb, (long long)a.block_table_stride);
        }
    }
    return APEX_OK;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

int apex_cpu_decode_attention_ex(const apex_cpu_args* args)
{
    g_last_error[0] = 0;
    if (!args) return fail(APEX_ERR_INVALID_ARG, "args is NULL");
    int rc = validate(*args);
    if (rc != APEX_OK || args->B == 0) return rc;
    std::lock_guard<std::mutex> lk(g_call_mutex);
    try {
        return run(*args);
    } catch (const std::exception& e) {
        return fail(APEX_ERR_OUT_OF_MEMORY, "host allocation failed: %s", e.what());
    }
}

int apex_cpu_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* block_table, const int32_t* context_lens, void* out,
                              int B, int Hq, int Hkv, int d, int block_size, float scale)
{
    apex_cpu_args a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k_cache = k_cache;
    a.v_cache = v_cache;
    a.block_table = block_table;
    a.context_lens = context_lens;
    a.out = out;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.d = d;
    a.block_size = block_size;
    a.scale = scale;
    return apex_cpu_decode_attention_ex(&a);
}

int apex_cpu_set_threads(int n)
{
    g_last_error[0] = 0;
    if (n < 0) return fail(APEX_ERR_INVALID_ARG, "thread count %d is negative", n);
    std::lock_guard<std::mutex> lk(g_call_mutex);
    try {
        g_pool.resize(n == 0 ? available_cores() : n);
        g_pool_ready = true;
    } catch (const std::exception& e) {
        return fail(APEX_ERR_OUT_OF_MEMORY, "could not start threads: %s", e.what());
    }
    return APEX_OK;
}

int apex_cpu_threads(void)
{
    std::lock_guard<std::mutex> lk(g_call_mutex);
    ensure_pool();
    return g_pool.size();
}

int apex_cpu_isa(void) { return isa(); }

double apex_cpu_read_bandwidth(size_t bytes, int threads, int reps)
{
    g_last_error[0] = 0;
    if (bytes < 4096 || threads <= 0 || reps <= 0) {
        fail(APEX_ERR_INVALID_ARG, "bad probe arguments");
        return -1.0;
    }
    std::lock_guard<std::mutex> lk(g_call_mutex);
    const size_t n = bytes / 8 / threads * threads;
    std::vector<uint64_t> buf;
    try {
        buf.assign(n, 1);
    } catch (const std::exception&) {
        fail(APEX_ERR_OUT_OF_MEMORY, "could not allocate %zu bytes", bytes);
        return -1.0;
    }
    ensure_pool();
    threads = std::min(threads, g_pool.size());
    const size_t per = n / threads;
    std::vector<uint64_t> sums((size_t)threads * 8, 0);
    auto body = [&](int tid) {
        const uint64_t* p = buf.data() + per * tid;
        uint64_t s0 = 0, s1 = 0, s2 = 0, s3 = 0;
        for (size_t i = 0; i + 4 <= per; i += 4) {
            s0 += p[i];
            s1 += p[i + 1];
            s2 += p[i + 2];
            s3 += p[i + 3];
        }
        sums[(size_t)tid * 8] += s0 + s1 + s2 + s3;
    };
    g_pool.run(threads, body);   // touch once
    const auto t0 = std::chrono::steady_clock::now();
    for (int r = 0; r < reps; ++r) g_pool.run(threads, body);
    const double s = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    uint64_t total = 0;
    for (int t = 0; t < threads; ++t) total += sums[(size_t)t * 8];
    if (total == 0) return -1.0;   // keeps the reads alive
    return (double)(per * threads * 8) * reps / s / 1e9;
}

const char* apex_cpu_last_error(void) { return g_last_error; }

}  // extern "C"
#pragma GCC visibility pop
