// apex_decode.hip -- host side of the C ABI declared in include/apex_decode.h.
//
// Validates arguments, finds or grows the per-device workspace, and enqueues
// the planner, attention and combine kernels on the caller's stream.  No host
// synchronisation happens on the call path (the workspace only grows when a
// call needs more than any earlier call on that device, and growing waits for
// the device before the old buffer is freed).
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "apex_decode.h"
#include "kernels.h"
#include "plan_policy.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

constexpr int kMaxDevices = 64;

struct DeviceState {
    int num_cu = 0;
    void* ws = nullptr;
    size_t ws_bytes = 0;
};

std::mutex g_mutex;
DeviceState g_dev[kMaxDevices];

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct WsLayout {
    size_t hdr, req, items, pacc, pml, total;
};

WsLayout ws_layout(int B, int G, int64_t max_items)
{
    WsLayout w;
    size_t off = 0;
    w.hdr = off;
    off = align_up(off + sizeof(apex::WsHeader), 256);
    w.req = off;
    off = align_up(off + sizeof(apex::ReqInfo) * (size_t)(B > 0 ? B : 1), 256);
    w.items = off;
    off = align_up(off + sizeof(apex::Item) * (size_t)max_items, 256);
    w.pacc = off;
    off = align_up(off + sizeof(float) * (size_t)max_items * G * apex::kHeadDim, 256);
    w.pml = off;
    off = align_up(off + sizeof(float) * 2 * (size_t)max_items * G, 256);
    w.total = off;
    return w;
}

int device_cu_count(int dev, int* num_cu)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(APEX_ERR_HIP, "device ordinal %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_mutex);
    if (g_dev[dev].num_cu == 0) {
        int n = 0;
        hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess || n <= 0)
            return fail(APEX_ERR_HIP, "hipDeviceGetAttribute(CU count): %s", hipGetErrorString(e));
        g_dev[dev].num_cu = n;
    }
    *num_cu = g_dev[dev].num_cu;
    return APEX_OK;
}

int library_workspace(int dev, size_t need, void** out)
{
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState& s = g_dev[dev];
    if (s.ws_bytes < need) {
        if (s.ws) {
            hipError_t e = hipDeviceSynchronize();
            if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipDeviceSynchronize: %s", hipGetErrorString(e));
            (void)hipFree(s.ws);
            s.ws = nullptr;
            s.ws_bytes = 0;
        }
        const size_t bytes = align_up(need + need / 4, 1 << 20);
        void* p = nullptr;
        hipError_t e = hipMalloc(&p, bytes);
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(APEX_ERR_OUT_OF_MEMORY, "hipMalloc(%zu) for the workspace failed: %s", bytes,
                        hipGetErrorString(e));
        }
        s.ws = p;
        s.ws_bytes = bytes;
    }
    *out = s.ws;
    return APEX_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

int check_shapes(int B, int Hq, int Hkv, int d, int block_size)
{
    if (B < 0) return fail(APEX_ERR_INVALID_ARG, "B = %d is negative", B);
    if (Hq <= 0 || Hkv <= 0) return fail(APEX_ERR_INVALID_ARG, "Hq = %d and Hkv = %d must be positive", Hq, Hkv);
    if (Hq % Hkv != 0) return fail(APEX_ERR_INVALID_ARG, "Hq = %d is not a multiple of Hkv = %d", Hq, Hkv);
    const int G = Hq / Hkv;
    if (d != apex::kHeadDim) return fail(APEX_ERR_UNSUPPORTED, "head dim %d unsupported (only 128)", d);
    if (block_size != apex::kBlockSize)
        return fail(APEX_ERR_UNSUPPORTED, "block_size %d unsupported (only 16)", block_size);
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(APEX_ERR_UNSUPPORTED, "group size Hq/Hkv = %d unsupported (1, 2, 4, 8)", G);
    return APEX_OK;
}

template <int G>
int launch(const apex_decode_args& a, const apex::WsPtrs& ws, int64_t target, int64_t max_items,
           hipStream_t stream)
{
    apex::plan_kernel<<<1, apex::kPlanThreads, 0, stream>>>(a.context_lens, a.B, a.Hkv, target,
                                                            a.num_splits, ws);
    apex::AttnParams p;
    p.q = (const apex::f16*)a.q;
    p.k = (const apex::f16*)a.k_cache;
    p.v = (const apex::f16*)a.v_cache;
    p.bt = a.block_table;
    p.out = (apex::f16*)a.out;
    p.lse = a.lse_out;
    p.bt_stride = a.block_table_stride;
    p.ws = ws;
    p.scale_log2 = a.scale * 1.4426950408889634f;
    p.Hq = a.Hq;
    p.Hkv = a.Hkv;
    if (a.attn_kernel_events[0]) {
        hipError_t e = hipEventRecord((hipEvent_t)a.attn_kernel_events[0], stream);
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    apex::attn_kernel<G><<<(unsigned)max_items, apex::kAttnThreads, 0, stream>>>(p);
    if (a.attn_kernel_events[1]) {
        hipError_t e = hipEventRecord((hipEvent_t)a.attn_kernel_events[1], stream);
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    apex::CombineParams cp;
    cp.out = (apex::f16*)a.out;
    cp.lse = a.lse_out;
    cp.ws = ws;
    cp.Hq = a.Hq;
    cp.Hkv = a.Hkv;
    apex::combine_kernel<G><<<(unsigned)((int64_t)a.B * a.Hkv), apex::kAttnThreads, 0, stream>>>(cp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return APEX_OK;
}

}  // namespace

extern "C" {

int apex_decode_version(void) { return 100; }

const char* apex_decode_last_error(void) { return g_last_error; }

size_t apex_decode_workspace_bytes(int B, int Hq, int Hkv, int d, int block_size, int num_splits,
                                   int items_per_cu)
{
    if (check_shapes(B, Hq, Hkv, d, block_size) != APEX_OK || num_splits < 0 || items_per_cu < 0)
        return 0;
    int dev = 0, num_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess || device_cu_count(dev, &num_cu) != APEX_OK) return 0;
    const int64_t mi = apex::max_items(B, Hkv, num_cu, items_per_cu, num_splits);
    return ws_layout(B, Hq / Hkv, mi).total;
}

int apex_decode_plan_host(const int32_t* context_lens, int B, int Hkv, int block_size, int num_cu,
                          int num_splits, int items_per_cu, int32_t* splits_out,
                          int32_t* blocks_per_split_out, int64_t* chunk_out, int64_t* items_out,
                          int64_t* partial_slots_out)
{
    g_last_error[0] = 0;
    if (B < 0 || Hkv <= 0 || num_cu <= 0 || num_splits < 0 || items_per_cu < 0)
        return fail(APEX_ERR_INVALID_ARG, "bad planner arguments");
    if (B > 0 && !context_lens) return fail(APEX_ERR_INVALID_ARG, "context_lens is NULL");
    if (block_size != apex::kBlockSize)
        return fail(APEX_ERR_UNSUPPORTED, "block_size %d unsupported (only 16)", block_size);
    int64_t units = 0;
    for (int b = 0; b < B; ++b) units += apex::blocks_of(context_lens[b], block_size);
    units *= Hkv;
    const int64_t chunk = apex::chunk_blocks(units, apex::target_items(num_cu, items_per_cu));
    int64_t items = 0, slots = 0;
    for (int b = 0; b < B; ++b) {
        const apex::SplitPlan sp =
            apex::split_request(apex::blocks_of(context_lens[b], block_size), chunk, num_splits);
        if (splits_out) splits_out[b] = sp.n;
        if (blocks_per_split_out) blocks_per_split_out[b] = sp.per;
        items += (int64_t)sp.n * Hkv;
        if (sp.n > 1) slots += (int64_t)sp.n * Hkv;
    }
    if (chunk_out) *chunk_out = chunk;
    if (items_out) *items_out = items;
    if (partial_slots_out) *partial_slots_out = slots;
    return APEX_OK;
}

int apex_decode_attention_ex(const apex_decode_args* args)
{
    g_last_error[0] = 0;
    if (!args) return fail(APEX_ERR_INVALID_ARG, "args is NULL");
    const apex_decode_args& a = *args;
    int rc = check_shapes(a.B, a.Hq, a.Hkv, a.d, a.block_size);
    if (rc != APEX_OK) return rc;
    if (a.flags != 0) return fail(APEX_ERR_INVALID_ARG, "flags must be 0");
    if (a.num_splits < 0) return fail(APEX_ERR_INVALID_ARG, "num_splits = %d is negative", a.num_splits);
    if (a.items_per_cu < 0) return fail(APEX_ERR_INVALID_ARG, "items_per_cu is negative");
    if (a.block_table_stride < 0) return fail(APEX_ERR_INVALID_ARG, "block_table_stride is negative");
    if (a.B == 0) return APEX_OK;
    if (!a.q || !a.k_cache || !a.v_cache || !a.block_table || !a.context_lens || !a.out)
        return fail(APEX_ERR_INVALID_ARG, "a tensor pointer is NULL");
    if (!aligned(a.q, 16) || !aligned(a.k_cache, 16) || !aligned(a.v_cache, 16) || !aligned(a.out, 16))
        return fail(APEX_ERR_INVALID_ARG, "q, k_cache, v_cache and out must be 16-byte aligned");
    if (!aligned(a.block_table, 4) || !aligned(a.context_lens, 4) || (a.lse_out && !aligned(a.lse_out, 4)))
        return fail(APEX_ERR_INVALID_ARG, "block_table, context_lens and lse_out must be 4-byte aligned");
    const size_t qo_bytes = (size_t)a.B * a.Hq * a.d * 2;
    if (overlaps(a.out, qo_bytes, a.q, qo_bytes))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps q");
    if (overlaps(a.out, qo_bytes, a.context_lens, (size_t)a.B * 4))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps context_lens");
    if (a.lse_out && overlaps(a.lse_out, (size_t)a.B * a.Hq * 4, a.out, qo_bytes))
        return fail(APEX_ERR_INVALID_ARG, "lse_out overlaps out");

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    int num_cu = 0;
    rc = device_cu_count(dev, &num_cu);
    if (rc != APEX_OK) return rc;

    const int G = a.Hq / a.Hkv;
    const int64_t target = apex::target_items(num_cu, a.items_per_cu);
    const int64_t mi = apex::max_items(a.B, a.Hkv, num_cu, a.items_per_cu, a.num_splits);
    if (mi > 0x7fffffff) return fail(APEX_ERR_UNSUPPORTED, "too many work items (%lld)", (long long)mi);
    const WsLayout lay = ws_layout(a.B, G, mi);
    void* ws = a.workspace;
    if (ws) {
        if (a.workspace_bytes < lay.total)
            return fail(APEX_ERR_OUT_OF_MEMORY, "caller workspace holds %zu bytes, %zu needed",
                        a.workspace_bytes, lay.total);
        if (!aligned(ws, 256)) return fail(APEX_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    } else {
        rc = library_workspace(dev, lay.total, &ws);
        if (rc != APEX_OK) return rc;
    }
    apex::WsPtrs wp;
    char* base = (char*)ws;
    wp.hdr = (apex::WsHeader*)(base + lay.hdr);
    wp.req = (apex::ReqInfo*)(base + lay.req);
    wp.items = (apex::Item*)(base + lay.items);
    wp.pacc = (float*)(base + lay.pacc);
    wp.pml = (float*)(base + lay.pml);

    hipStream_t stream = (hipStream_t)a.stream;
    switch (G) {
        case 1: return launch<1>(a, wp, target, mi, stream);
        case 2: return launch<2>(a, wp, target, mi, stream);
        case 4: return launch<4>(a, wp, target, mi, stream);
        default: return launch<8>(a, wp, target, mi, stream);
    }
}

int apex_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* block_table, const int32_t* context_lens, void* out, int B,
                          int Hq, int Hkv, int d, int block_size, float scale, void* stream)
{
    apex_decode_args a;
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
    a.stream = stream;
    return apex_decode_attention_ex(&a);
}

int apex_decode_release_workspace(void)
{
    g_last_error[0] = 0;
    std::lock_guard<std::mutex> lock(g_mutex);
    int rc = APEX_OK;
    for (int d = 0; d < kMaxDevices; ++d) {
        if (!g_dev[d].ws) continue;
        int prev = 0;
        (void)hipGetDevice(&prev);
        if (hipSetDevice(d) == hipSuccess && hipDeviceSynchronize() == hipSuccess) {
            (void)hipFree(g_dev[d].ws);
            g_dev[d].ws = nullptr;
            g_dev[d].ws_bytes = 0;
        } else {
            rc = fail(APEX_ERR_HIP, "could not release the workspace of device %d", d);
        }
        (void)hipSetDevice(prev);
    }
    return rc;
}

}  // extern "C"
