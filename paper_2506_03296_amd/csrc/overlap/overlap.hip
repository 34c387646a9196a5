// overlap.hip -- host side of the Asynchronous Overlap runtime
// (include/apex_overlap.h).  No device code: HIP runtime calls for the
// pinned staging copies and their events, a compute thread that appends the
// new K/V rows to the host cache and runs the host attention of
// libapex_cpu.so, and the non-blocking readiness check of the main thread.
//
// Per result slot the states run FREE -> QUEUED (copies to the host enqueued
// on the caller's stream, job queued) -> DONE (compute thread finished) ->
// COLLECTED (copy back enqueued).  A collected slot takes the next submit at
// once: that submit's stream first waits for the copy-back's event, so its
// copies to the host -- and the compute thread, which waits for those --
// come after the previous result has left the staging buffer.
#include <hip/hip_runtime.h>

#include <sched.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "apex_cpu_attention.h"
#include "apex_overlap.h"

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

enum SlotState : int { kFree = 0, kQueued = 1, kDone = 2, kCollected = 3 };

constexpr int kSpinPolls = 2000;   // event queries (with a yield) before sleeping on it

struct Slot {
    uint16_t* q = nullptr;     // pinned: [B][Hq][d] q, then [B][Hkv][d] kn and vn
    uint16_t* kn = nullptr;    // inside the q allocation, placed per submit
    uint16_t* vn = nullptr;
    uint16_t* out = nullptr;   // pinned [max_requests][Hq][d]
    hipEvent_t in_done = nullptr;
    hipEvent_t out_done = nullptr;
    std::vector<int32_t> table;
    std::vector<int32_t> lens;
    std::vector<int64_t> slots;
    int64_t stride = 0;
    int B = 0;
    int layer = 0;
    int64_t ticket = -1;
    std::atomic<int> state{kFree};
    int rc = APEX_OK;
    char msg[256] = "";
};

}  // namespace

struct apex_overlap {
    apex_overlap_config cfg;
    int device = 0;
    int per_layer = 2;
    std::vector<void*> host_k, host_v;   // pinned caches, one pair per layer
    std::vector<Slot> slots;
    std::vector<int64_t> next_seq;       // per layer
    std::mutex m;
    std::condition_variable work_cv, done_cv;
    std::deque<int> queue;
    int pending = 0;
    bool hold = false;
    bool stop = false;
    std::thread worker;

    size_t q_bytes(int B) const { return (size_t)B * cfg.Hq * cfg.d * 2; }
    size_t kv_bytes(int B) const { return (size_t)B * cfg.Hkv * cfg.d * 2; }
    size_t cache_bytes() const { return (size_t)cfg.num_blocks * cfg.Hkv * cfg.block_size * cfg.d * 2; }

    // Waits for the copies of a job: polls briefly (the GPU is usually about
    // to deliver), then sleeps on the event.
    static hipError_t wait_copies(hipEvent_t ev)
    {
        for (int i = 0; i < kSpinPolls; ++i) {
            const hipError_t e = hipEventQuery(ev);
            if (e != hipErrorNotReady) return e;
            sched_yield();
        }
        return hipEventSynchronize(ev);
    }

    void run_job(Slot& s)
    {
        hipError_t e = wait_copies(s.in_done);
        if (e != hipSuccess) {
            s.rc = APEX_ERR_HIP;
            snprintf(s.msg, sizeof(s.msg), "copy of the new rows to the host failed: %s", hipGetErrorString(e));
            return;
        }
        // append this token's K/V rows to the layer's host cache
        const int Hkv = cfg.Hkv, d = cfg.d, bs = cfg.block_size;
        uint16_t* kc = (uint16_t*)host_k[s.layer];
        uint16_t* vc = (uint16_t*)host_v[s.layer];
        const int64_t capacity = cfg.num_blocks * bs;
        for (int t = 0; t < s.B; ++t) {
            const int64_t slot = s.slots[t];
            if (slot < 0 || slot >= capacity) continue;
            const int64_t block = slot / bs, pos = slot % bs;
            for (int g = 0; g < Hkv; ++g) {
                const int64_t dst = ((block * Hkv + g) * bs + pos) * d;
                const int64_t src = ((int64_t)t * Hkv + g) * d;
                memcpy(kc + dst, s.kn + src, (size_t)d * 2);
                memcpy(vc + dst, s.vn + src, (size_t)d * 2);
            }
        }
        apex_cpu_args a;
        memset(&a, 0, sizeof(a));
        a.q = s.q;
        a.k_cache = kc;
        a.v_cache = vc;
        a.block_table = s.table.data();
        a.context_lens = s.lens.data();
        a.out = s.out;
        a.B = s.B;
        a.Hq = cfg.Hq;
        a.Hkv = Hkv;
        a.d = d;
        a.block_size = bs;
        a.scale = cfg.scale;
        a.block_table_stride = s.stride;
        a.num_threads = cfg.threads;
        const int rc = apex_cpu_decode_attention_ex(&a);
        if (rc != APEX_OK) {
            s.rc = rc;
            snprintf(s.msg, sizeof(s.msg), "host attention failed: %s", apex_cpu_last_error());
        }
    }

    void loop()
    {
        (void)hipSetDevice(device);
        for (;;) {
            int idx;
            {
                std::unique_lock<std::mutex> lk(m);
                work_cv.wait(lk, [&] { return (!queue.empty() && (!hold || stop)) || (stop && queue.empty()); });
                if (queue.empty()) return;   // stopping, nothing left
                idx = queue.front();
                queue.pop_front();
            }
            Slot& s = slots[(size_t)idx];
            s.rc = APEX_OK;
            s.msg[0] = 0;
            run_job(s);
            {
                std::lock_guard<std::mutex> lk(m);
                s.state.store(kDone, std::memory_order_release);
                --pending;
            }
            done_cv.notify_all();
        }
    }
};

namespace {

void free_all(apex_overlap* rt)
{
    for (Slot& s : rt->slots) {
        if (s.q) (void)hipHostFree(s.q);
        if (s.out) (void)hipHostFree(s.out);
        if (s.in_done) (void)hipEventDestroy(s.in_done);
        if (s.out_done) (void)hipEventDestroy(s.out_done);
    }
    for (void* p : rt->host_k)
        if (p) (void)hipHostFree(p);
    for (void* p : rt->host_v)
        if (p) (void)hipHostFree(p);
}

int host_alloc(void** p, size_t bytes)
{
    *p = nullptr;
    hipError_t e = hipHostMalloc(p, bytes < 64 ? 64 : bytes, hipHostMallocDefault);
    if (e != hipSuccess || !*p) {
        (void)hipGetLastError();
        *p = nullptr;
        return fail(APEX_ERR_OUT_OF_MEMORY, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    return APEX_OK;
}

Slot* find(apex_overlap* rt, int64_t ticket)
{
    if (ticket < 0) return nullptr;
    const int layer = (int)(ticket & 0xffff);
    const int64_t seq = ticket >> 16;
    if (layer >= rt->cfg.layers) return nullptr;
    Slot& s = rt->slots[(size_t)layer * rt->per_layer + (size_t)(seq % rt->per_layer)];
    return s.ticket == ticket ? &s : nullptr;
}

int collect(apex_overlap* rt, Slot& s, void* out, hipStream_t stream)
{
    s.state.store(kCollected, std::memory_order_relaxed);
    if (s.rc != APEX_OK) return fail(s.rc, "%s", s.msg);
    hipError_t e = hipMemcpyAsync(out, s.out, rt->q_bytes(s.B), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipEventRecord(s.out_done, stream);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "copy of the result to the GPU failed: %s", hipGetErrorString(e));
    return APEX_OK;
}

}  // namespace

extern "C" {

const char* apex_overlap_last_error(void) { return g_last_error; }

int apex_overlap_create(const apex_overlap_config* cfg, apex_overlap** out)
{
    g_last_error[0] = 0;
    if (!cfg || !out) return fail(APEX_ERR_INVALID_ARG, "NULL argument");
    *out = nullptr;
    const apex_overlap_config& c = *cfg;
    if (c.layers <= 0 || c.layers > 0xffff) return fail(APEX_ERR_INVALID_ARG, "layers must be in [1, 65535]");
    if (c.max_requests <= 0) return fail(APEX_ERR_INVALID_ARG, "max_requests must be positive");
    if (c.Hq <= 0 || c.Hkv <= 0 || c.Hq % c.Hkv != 0) return fail(APEX_ERR_INVALID_ARG, "bad head counts");
    // the host attention's supported set (apex_cpu_attention.h), checked here
    // so that a runtime which cannot serve any job is never created
    if (c.d <= 0 || c.d % 16 != 0 || c.d > 512) return fail(APEX_ERR_UNSUPPORTED, "head dim %d unsupported", c.d);
    if (c.Hq / c.Hkv > 64) return fail(APEX_ERR_UNSUPPORTED, "group size %d above 64", c.Hq / c.Hkv);
    if (c.block_size <= 0 || c.num_blocks <= 0 || c.max_blocks_per_request <= 0)
        return fail(APEX_ERR_INVALID_ARG, "block_size, num_blocks and max_blocks_per_request must be positive");
    if (c.threads < 0 || c.slots_per_layer < 0) return fail(APEX_ERR_INVALID_ARG, "threads and slots must be >= 0");

    apex_overlap* rt = new (std::nothrow) apex_overlap();
    if (!rt) return fail(APEX_ERR_OUT_OF_MEMORY, "out of host memory");
    rt->cfg = c;
    rt->per_layer = c.slots_per_layer ? c.slots_per_layer : 2;
    hipError_t e = hipGetDevice(&rt->device);
    if (e != hipSuccess) {
        delete rt;
        return fail(APEX_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    }
    int rc = APEX_OK;
    try {
        rt->host_k.assign((size_t)c.layers, nullptr);
        rt->host_v.assign((size_t)c.layers, nullptr);
        rt->slots = std::vector<Slot>((size_t)c.layers * rt->per_layer);
        rt->next_seq.assign((size_t)c.layers, 0);
    } catch (const std::exception&) {
        delete rt;
        return fail(APEX_ERR_OUT_OF_MEMORY, "out of host memory");
    }
    for (int l = 0; l < c.layers && rc == APEX_OK; ++l) {
        rc = host_alloc(&rt->host_k[l], rt->cache_bytes());
        if (rc == APEX_OK) rc = host_alloc(&rt->host_v[l], rt->cache_bytes());
        if (rc == APEX_OK) {
            memset(rt->host_k[l], 0, rt->cache_bytes());
            memset(rt->host_v[l], 0, rt->cache_bytes());
        }
    }
    for (size_t i = 0; i < rt->slots.size() && rc == APEX_OK; ++i) {
        Slot& s = rt->slots[i];
        s.layer = (int)(i / rt->per_layer);
        // q, kn, vn share one allocation; submit() places kn and vn right
        // after the B rows of q so that packed device rows copy in one go
        if ((rc = host_alloc((void**)&s.q, rt->q_bytes(c.max_requests) + 2 * rt->kv_bytes(c.max_requests))) != APEX_OK)
            break;
        if ((rc = host_alloc((void**)&s.out, rt->q_bytes(c.max_requests))) != APEX_OK) break;
        // the compute thread sleeps on in_done instead of spinning a core
        e = hipEventCreateWithFlags(&s.in_done, hipEventDisableTiming | hipEventBlockingSync);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&s.out_done, hipEventDisableTiming);
        if (e != hipSuccess) rc = fail(APEX_ERR_HIP, "hipEventCreate: %s", hipGetErrorString(e));
    }
    if (rc != APEX_OK) {
        free_all(rt);
        delete rt;
        return rc;
    }
    try {
        rt->worker = std::thread([rt] { rt->loop(); });
    } catch (const std::exception& ex) {
        free_all(rt);
        delete rt;
        return fail(APEX_ERR_OUT_OF_MEMORY, "could not start the compute thread: %s", ex.what());
    }
    *out = rt;
    return APEX_OK;
}

int apex_overlap_host_cache(apex_overlap* rt, int layer, void** k_cache, void** v_cache)
{
    g_last_error[0] = 0;
    if (!rt || !k_cache || !v_cache) return fail(APEX_ERR_INVALID_ARG, "NULL argument");
    if (layer < 0 || layer >= rt->cfg.layers) return fail(APEX_ERR_INVALID_ARG, "layer %d out of range", layer);
    *k_cache = rt->host_k[layer];
    *v_cache = rt->host_v[layer];
    return APEX_OK;
}

int apex_overlap_submit(apex_overlap* rt, int layer, const void* q, const void* k_new,
                        const void* v_new, const int64_t* slot_mapping,
                        const int32_t* block_table, int64_t block_table_stride,
                        const int32_t* context_lens, int B, void* stream, int64_t* ticket)
{
    g_last_error[0] = 0;
    if (!rt || !ticket) return fail(APEX_ERR_INVALID_ARG, "NULL argument");
    const apex_overlap_config& c = rt->cfg;
    if (layer < 0 || layer >= c.layers) return fail(APEX_ERR_INVALID_ARG, "layer %d out of range", layer);
    if (B <= 0 || B > c.max_requests) return fail(APEX_ERR_INVALID_ARG, "B = %d outside [1, %d]", B, c.max_requests);
    if (!q || !k_new || !v_new || !slot_mapping || !block_table || !context_lens)
        return fail(APEX_ERR_INVALID_ARG, "a pointer is NULL");
    int64_t maxb = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t nb = context_lens[b] > 0 ? (context_lens[b] + (int64_t)c.block_size - 1) / c.block_size : 0;
        maxb = nb > maxb ? nb : maxb;
    }
    const int64_t stride = block_table_stride ? block_table_stride : (maxb ? maxb : 1);
    if (stride < maxb || stride > c.max_blocks_per_request)
        return fail(APEX_ERR_INVALID_ARG, "block table stride %lld outside [%lld, %d]", (long long)stride,
                    (long long)maxb, c.max_blocks_per_request);
    for (int b = 0; b < B; ++b) {
        const int64_t nb = context_lens[b] > 0 ? (context_lens[b] + (int64_t)c.block_size - 1) / c.block_size : 0;
        for (int64_t i = 0; i < nb; ++i) {
            const int32_t id = block_table[b * stride + i];
            if (id < 0 || id >= c.num_blocks)
                return fail(APEX_ERR_INVALID_ARG, "request %d: block id %d outside the host cache", b, id);
        }
    }
    const int64_t seq = rt->next_seq[(size_t)layer];
    Slot& s = rt->slots[(size_t)layer * rt->per_layer + (size_t)(seq % rt->per_layer)];
    const int st = s.state.load(std::memory_order_acquire);
    if (st == kQueued || st == kDone)
        return fail(APEX_ERR_BUSY, "layer %d: the result of ticket %lld is not collected yet", layer, (long long)s.ticket);
    hipStream_t st_ = (hipStream_t)stream;
    if (st == kCollected) {
        // the copy-back of the slot's previous result may still be queued:
        // order this submit's copies (and so the compute thread, which waits
        // for them) after it, on the device, without blocking the host
        hipError_t e = hipStreamWaitEvent(st_, s.out_done, 0);
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipStreamWaitEvent: %s", hipGetErrorString(e));
    }
    try {
        s.table.assign(block_table, block_table + (size_t)B * stride);
        s.lens.assign(context_lens, context_lens + B);
        s.slots.assign(slot_mapping, slot_mapping + B);
    } catch (const std::exception&) {
        return fail(APEX_ERR_OUT_OF_MEMORY, "out of host memory");
    }
    s.stride = stride;
    s.B = B;
    s.kn = s.q + rt->q_bytes(B) / 2;
    s.vn = s.kn + rt->kv_bytes(B) / 2;
    hipError_t e;
    if ((const char*)k_new == (const char*)q + rt->q_bytes(B) &&
        (const char*)v_new == (const char*)k_new + rt->kv_bytes(B)) {
        // q, k_new and v_new back to back on the device: one copy into the
        // (equally back-to-back) staging buffers
        e = hipMemcpyAsync(s.q, q, rt->q_bytes(B) + 2 * rt->kv_bytes(B), hipMemcpyDeviceToHost, st_);
    } else {
        e = hipMemcpyAsync(s.q, q, rt->q_bytes(B), hipMemcpyDeviceToHost, st_);
        if (e == hipSuccess) e = hipMemcpyAsync(s.kn, k_new, rt->kv_bytes(B), hipMemcpyDeviceToHost, st_);
        if (e == hipSuccess) e = hipMemcpyAsync(s.vn, v_new, rt->kv_bytes(B), hipMemcpyDeviceToHost, st_);
    }
    if (e == hipSuccess) e = hipEventRecord(s.in_done, st_);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "copy of the new rows to the host failed: %s", hipGetErrorString(e));
    s.ticket = (seq << 16) | layer;
    rt->next_seq[(size_t)layer] = seq + 1;
    {
        std::lock_guard<std::mutex> lk(rt->m);
        s.state.store(kQueued, std::memory_order_relaxed);
        rt->queue.push_back((int)(&s - rt->slots.data()));
        ++rt->pending;
    }
    rt->work_cv.notify_one();
    *ticket = s.ticket;
    return APEX_OK;
}

int apex_overlap_poll(apex_overlap* rt, int64_t ticket, void* out, void* stream, int* ready)
{
    g_last_error[0] = 0;
    if (!rt || !out || !ready) return fail(APEX_ERR_INVALID_ARG, "NULL argument");
    *ready = 0;
    Slot* s = find(rt, ticket);
    if (!s) return fail(APEX_ERR_INVALID_ARG, "unknown or superseded ticket %lld", (long long)ticket);
    const int st = s->state.load(std::memory_order_acquire);
    if (st == kCollected) return fail(APEX_ERR_INVALID_ARG, "ticket %lld was already collected", (long long)ticket);
    if (st != kDone) return APEX_OK;
    *ready = 1;
    return collect(rt, *s, out, (hipStream_t)stream);
}

int apex_overlap_wait(apex_overlap* rt, int64_t ticket, void* out, void* stream)
{
    g_last_error[0] = 0;
    if (!rt || !out) return fail(APEX_ERR_INVALID_ARG, "NULL argument");
    Slot* s = find(rt, ticket);
    if (!s) return fail(APEX_ERR_INVALID_ARG, "unknown or superseded ticket %lld", (long long)ticket);
    {
        std::unique_lock<std::mutex> lk(rt->m);
        const int st = s->state.load(std::memory_order_acquire);
        if (st == kCollected) return fail(APEX_ERR_INVALID_ARG, "ticket %lld was already collected", (long long)ticket);
        if (st != kDone && rt->hold)
            return fail(APEX_ERR_BUSY, "the compute thread is held; ticket %lld cannot finish", (long long)ticket);
        rt->done_cv.wait(lk, [&] { return s->state.load(std::memory_order_acquire) == kDone; });
    }
    return collect(rt, *s, out, (hipStream_t)stream);
}

int apex_overlap_hold(apex_overlap* rt, int hold)
{
    g_last_error[0] = 0;
    if (!rt) return fail(APEX_ERR_INVALID_ARG, "NULL runtime");
    {
        std::lock_guard<std::mutex> lk(rt->m);
        rt->hold = hold != 0;
    }
    rt->work_cv.notify_all();
    return APEX_OK;
}

int apex_overlap_pending(apex_overlap* rt)
{
    if (!rt) return 0;
    std::lock_guard<std::mutex> lk(rt->m);
    return rt->pending;
}

int apex_overlap_destroy(apex_overlap* rt)
{
    g_last_error[0] = 0;
    if (!rt) return APEX_OK;
    {
        std::lock_guard<std::mutex> lk(rt->m);
        rt->stop = true;
        rt->hold = false;
    }
    rt->work_cv.notify_all();
    if (rt->worker.joinable()) rt->worker.join();
    int rc = APEX_OK;
    for (Slot& s : rt->slots) {
        if (s.state.load() == kCollected && s.out_done) {
            hipError_t e = hipEventSynchronize(s.out_done);
            if (e != hipSuccess) rc = fail(APEX_ERR_HIP, "waiting for a result copy: %s", hipGetErrorString(e));
        }
    }
    free_all(rt);
    delete rt;
    return rc;
}

}  // extern "C"
