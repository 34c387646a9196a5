// apex_decode.hip -- host side of the C ABI declared in include/apex_decode.h.
//
// Validates arguments, finds or grows the per-device workspaces, and enqueues
// the single persistent attention kernel on the caller's stream.  No host
// synchronisation happens on the call path (a library workspace only grows
// when a call needs more than any earlier call on that device, and growing
// waits for the device before the old buffer is freed).
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "apex_decode.h"
#ifdef APEX_TRACE_WORK_GROUPS
#include "apex_decode_trace.h"
#endif
#include "kernels.h"
#include "plan_policy.h"
#include "status.h"

namespace {

// Static scratch of apex_decode_attention_noalloc: arrival counters for up to
// kScratchPairs (request, kv-head) pairs, then the partial accumulators and
// (max, sum) pairs of up to kScratchWorkerHeads (work group, q-head) pairs,
// two slots each -- the layout of a workspace of that size, at fixed offsets.
constexpr int64_t kScratchPairs = 1 << 16;
constexpr int64_t kScratchWorkerHeads = 4096;
constexpr size_t kScratchCounterBytes = kScratchPairs * sizeof(int32_t);
constexpr size_t kScratchAccBytes = 2 * kScratchWorkerHeads * apex::kHeadDim * sizeof(float);
constexpr size_t kScratchMlBytes = 2 * kScratchWorkerHeads * 2 * sizeof(float);
constexpr size_t kScratchBytes = kScratchCounterBytes + kScratchAccBytes + kScratchMlBytes;
static_assert(kScratchCounterBytes % 256 == 0 && kScratchAccBytes % 256 == 0, "256-byte aligned parts");
}  // namespace

// The array, 4.3 MiB: one copy per device that loads the library, held until
// the process ends.  Host code never uses this name as an address: its device
// address comes from hipGetSymbolAddress (scratch_for), once per device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

using apex::fail;

constexpr int kMaxDevices = 64;
constexpr int kGroupKinds = 4;   // G = 1, 2, 4, 8
constexpr int kMaxWorkers = 1 << 20;

struct Buffer {
    void* ptr = nullptr;
    size_t bytes = 0;
};

struct DeviceState {
    int num_cu = 0;
    int resident[kGroupKinds] = {0, 0, 0, 0};   // work groups per CU, per G
    Buffer counters;   // zeroed at allocation; calls leave it zero
    Buffer partials;
    Buffer error_word;   // input-check error bits, zeroed at allocation and when read
    char* scratch_addr = nullptr;   // device address of this device's static scratch array
};

std::mutex g_mutex;
DeviceState g_dev[kMaxDevices];

#ifdef APEX_TRACE_WORK_GROUPS
// work-group timeline buffer of the diagnostic build (apex_decode_trace.h)
uint64_t* g_trace = nullptr;
int64_t g_trace_groups = 0;
#endif


__global__ void clear_words(int32_t* words, int n)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) words[i] = 0;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int group_index(int G) { return G == 1 ? 0 : G == 2 ? 1 : G == 4 ? 2 : 3; }

size_t counter_bytes(int B, int Hkv) { return align_up((size_t)B * Hkv * sizeof(int32_t), 256); }

size_t partial_bytes(int64_t workers, int G)
{
    return align_up(sizeof(float) * 2 * (size_t)workers * G * apex::kHeadDim, 256) +
           align_up(sizeof(float) * 2 * 2 * (size_t)workers * G, 256);
}

int resident_groups(int G, int* out)
{
    int n = 0;
    hipError_t e;
    switch (G) {
        case 1: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, apex::attn_kernel<1, false, false>, apex::kAttnThreads, 0); break;
        case 2: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, apex::attn_kernel<2, false, false>, apex::kAttnThreads, 0); break;
        case 4: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, apex::attn_kernel<4, false, false>, apex::kAttnThreads, 0); break;
        default: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, apex::attn_kernel<8, false, false>, apex::kAttnThreads, 0); break;
    }
    if (e != hipSuccess || n <= 0)
        return fail(APEX_ERR_HIP, "occupancy query failed: %s", hipGetErrorString(e));
    *out = n;
    return APEX_OK;
}

// Default persistent grid for group size G on device dev: CUs x resident
// groups (and the CU count, if cus is not NULL).
int default_workers(int dev, int G, int64_t* out, int* cus = nullptr)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(APEX_ERR_HIP, "device ordinal %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState& s = g_dev[dev];
    if (s.num_cu == 0) {
        int n = 0;
        hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess || n <= 0)
            return fail(APEX_ERR_HIP, "hipDeviceGetAttribute(CU count): %s", hipGetErrorString(e));
        s.num_cu = n;
    }
    const int gi = group_index(G);
    if (s.resident[gi] == 0) {
        int rc = resident_groups(G, &s.resident[gi]);
        if (rc != APEX_OK) return rc;
    }
    *out = (int64_t)s.num_cu * s.resident[gi];
    if (cus) *cus = s.num_cu;
    return APEX_OK;
}

// Device address of the static scratch on device dev (current), looked up on
// the device's first no-allocation call; that call also clears the counters
// with a kernel on `stream` (a kernel, not a memset, so that a call under
// stream capture records nothing the graph cannot replay).  The array starts
// zeroed and every launch leaves the counters zero.
int scratch_for(int dev, hipStream_t stream, char** out)
{
    if (dev < 0 || dev >= kMaxDevices) return fail(APEX_ERR_HIP, "device ordinal %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState& s = g_dev[dev];
    if (!s.scratch_addr) {
        void* ptr = nullptr;
        hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(::scratch));
        if (e != hipSuccess || !ptr)
            return fail(APEX_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        clear_words<<<64, 256, 0, stream>>>((int32_t*)ptr, (int)kScratchPairs);
        e = hipGetLastError();
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "clearing the scratch counters: %s", hipGetErrorString(e));
        s.scratch_addr = (char*)ptr;
    }
    *out = s.scratch_addr;
    return APEX_OK;
}

int grow(Buffer& buf, size_t need, bool zero)
{
    if (buf.bytes >= need) return APEX_OK;
    if (buf.ptr) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipDeviceSynchronize: %s", hipGetErrorString(e));
        (void)hipFree(buf.ptr);
        buf.ptr = nullptr;
        buf.bytes = 0;
    }
    const size_t bytes = align_up(need + need / 4, 1 << 20);
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess || !p) {
        (void)hipGetLastError();
        return fail(APEX_ERR_OUT_OF_MEMORY, "hipMalloc(%zu) for a workspace failed: %s", bytes,
                    hipGetErrorString(e));
    }
    if (zero) {
        e = hipMemset(p, 0, bytes);
        if (e != hipSuccess) {
            (void)hipFree(p);
            return fail(APEX_ERR_HIP, "hipMemset of the counters failed: %s", hipGetErrorString(e));
        }
    }
    buf.ptr = p;
    buf.bytes = bytes;
    return APEX_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// a * b, saturated at the largest size (an extent past the address space
// still overlaps everything above its start)
size_t sat_mul(size_t a, size_t b)
{
    return b != 0 && a > SIZE_MAX / b ? SIZE_MAX : a * b;
}

size_t sat_extent(const void* base, size_t bytes)
{
    const size_t room = SIZE_MAX - (uintptr_t)base;
    return bytes < room ? bytes : room;
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

template <int G, bool kCheck, bool kAppend>
int launch(const apex::AttnParams& p, const int32_t* bt, const int32_t* lens, int64_t workers,
           void* const* events, hipStream_t stream)
{
    if (events[0]) {
        hipError_t e = hipEventRecord((hipEvent_t)events[0], stream);
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    apex::attn_kernel<G, kCheck, kAppend><<<(unsigned)workers, apex::kAttnThreads, 0, stream>>>(p, bt, lens);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    if (events[1]) {
        e = hipEventRecord((hipEvent_t)events[1], stream);
        if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    }
    return APEX_OK;
}

template <bool kCheck, bool kAppend>
int dispatch_g(int G, const apex::AttnParams& p, const int32_t* bt, const int32_t* lens, int64_t workers,
               void* const* ev, hipStream_t stream)
{
    switch (G) {
        case 1: return launch<1, kCheck, kAppend>(p, bt, lens, workers, ev, stream);
        case 2: return launch<2, kCheck, kAppend>(p, bt, lens, workers, ev, stream);
        case 4: return launch<4, kCheck, kAppend>(p, bt, lens, workers, ev, stream);
        default: return launch<8, kCheck, kAppend>(p, bt, lens, workers, ev, stream);
    }
}

// One kernel build per (group size, input check, fused append): the default
// path compiles without the other two.
int dispatch(int G, bool check, bool append, const apex::AttnParams& p, const int32_t* bt,
             const int32_t* lens, int64_t workers, void* const* ev, hipStream_t stream)
{
    if (check) return append ? dispatch_g<true, true>(G, p, bt, lens, workers, ev, stream)
                             : dispatch_g<true, false>(G, p, bt, lens, workers, ev, stream);
    return append ? dispatch_g<false, true>(G, p, bt, lens, workers, ev, stream)
                  : dispatch_g<false, false>(G, p, bt, lens, workers, ev, stream);
}

// Validates a call and enqueues its kernel.  The arrival counters and the
// partials come from the caller's workspace, the library-owned workspace of
// the device, or (noalloc) the device's static scratch array.
int enqueue(const apex_decode_args& a, bool noalloc)
{
    int rc = check_shapes(a.B, a.Hq, a.Hkv, a.d, a.block_size);
    if (rc != APEX_OK) return rc;
    if (a.flags & ~APEX_DECODE_FLAG_CHECK_INPUTS) return fail(APEX_ERR_INVALID_ARG, "unknown flags");
    const bool check = (a.flags & APEX_DECODE_FLAG_CHECK_INPUTS) != 0;
    if (a.num_blocks < 0) return fail(APEX_ERR_INVALID_ARG, "num_blocks is negative");
    if (check && a.num_blocks <= 0)
        return fail(APEX_ERR_INVALID_ARG, "the input check needs num_blocks > 0");
    if (a.num_workers < 0 || a.num_workers > kMaxWorkers)
        return fail(APEX_ERR_INVALID_ARG, "num_workers = %d out of range", a.num_workers);
    if (a.block_table_stride < 0) return fail(APEX_ERR_INVALID_ARG, "block_table_stride is negative");
    const bool append = a.k_new || a.v_new;
    const int64_t new_row = (int64_t)a.Hkv * a.d;
    const int64_t new_stride = a.new_token_stride ? a.new_token_stride : new_row;
    if (append) {
        if (!a.k_new || !a.v_new) return fail(APEX_ERR_INVALID_ARG, "the fused append needs both k_new and v_new");
        if (new_stride < new_row || new_stride % 8 != 0)
            return fail(APEX_ERR_INVALID_ARG, "new_token_stride %lld must be 0 or a multiple of 8 >= Hkv * d",
                        (long long)a.new_token_stride);
    } else if (a.new_token_stride != 0) {
        return fail(APEX_ERR_INVALID_ARG, "new_token_stride without k_new/v_new");
    }
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
    // the caches and the table over the extents the host knows: num_blocks
    // blocks when given (else the first block), the rows of an explicit
    // stride (else one entry per request)
    const size_t block_bytes = (size_t)a.Hkv * a.block_size * a.d * 2;
    const size_t cache_bytes = sat_mul(block_bytes, a.num_blocks > 0 ? (size_t)a.num_blocks : 1);
    const size_t bt_bytes =
        sat_mul((size_t)a.B * 4, a.block_table_stride > 0 ? (size_t)a.block_table_stride : 1);
    if (overlaps(a.out, qo_bytes, a.k_cache, sat_extent(a.k_cache, cache_bytes)))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps k_cache");
    if (overlaps(a.out, qo_bytes, a.v_cache, sat_extent(a.v_cache, cache_bytes)))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps v_cache");
    if (overlaps(a.out, qo_bytes, a.block_table, sat_extent(a.block_table, bt_bytes)))
        return fail(APEX_ERR_INVALID_ARG, "out overlaps block_table");
    if (append) {
        if (!aligned(a.k_new, 16) || !aligned(a.v_new, 16))
            return fail(APEX_ERR_INVALID_ARG, "k_new and v_new must be 16-byte aligned");
        const size_t new_bytes = ((size_t)(a.B - 1) * new_stride + new_row) * 2;
        if (overlaps(a.out, qo_bytes, a.k_new, new_bytes) || overlaps(a.out, qo_bytes, a.v_new, new_bytes))
            return fail(APEX_ERR_INVALID_ARG, "out overlaps k_new or v_new");
    }

    if (noalloc && (int64_t)a.B * a.Hkv > kScratchPairs)
        return fail(APEX_ERR_UNSUPPORTED,
                    "B * Hkv = %lld (request, kv-head) pairs exceed the static scratch's %lld",
                    (long long)a.B * a.Hkv, (long long)kScratchPairs);

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    const int G = a.Hq / a.Hkv;
    int64_t workers = a.num_workers;
    int cus = 0;   // the one-group-per-CU rule applies to the default grid only
    if (workers == 0) {
        rc = default_workers(dev, G, &workers, &cus);
        if (rc != APEX_OK) return rc;
    }
    // the static scratch holds the partials of kScratchWorkerHeads / G work groups
    if (noalloc && workers > kScratchWorkerHeads / G) workers = kScratchWorkerHeads / G;

    const size_t cbytes = counter_bytes(a.B, a.Hkv);
    const size_t pbytes = partial_bytes(workers, G);
    void* counters = nullptr;
    void* partials = nullptr;
    void* part_ml = nullptr;
    if (noalloc) {
        char* base = nullptr;
        rc = scratch_for(dev, (hipStream_t)a.stream, &base);
        if (rc != APEX_OK) return rc;
        counters = base;
        partials = base + kScratchCounterBytes;
        part_ml = base + kScratchCounterBytes + kScratchAccBytes;
    } else if (a.workspace) {
        if (a.workspace_bytes < cbytes + pbytes)
            return fail(APEX_ERR_OUT_OF_MEMORY, "caller workspace holds %zu bytes, %zu needed",
                        a.workspace_bytes, cbytes + pbytes);
        if (!aligned(a.workspace, 256)) return fail(APEX_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
        counters = a.workspace;
        partials = (char*)a.workspace + cbytes;
    } else {
        std::lock_guard<std::mutex> lock(g_mutex);
        DeviceState& s = g_dev[dev];
        rc = grow(s.counters, cbytes, true);
        if (rc != APEX_OK) return rc;
        rc = grow(s.partials, pbytes, false);
        if (rc != APEX_OK) return rc;
        counters = s.counters.ptr;
        partials = s.partials.ptr;
    }
    void* error_word = nullptr;
    if (check) {
        std::lock_guard<std::mutex> lock(g_mutex);
        rc = grow(g_dev[dev].error_word, 4, true);
        if (rc != APEX_OK) return rc;
        error_word = g_dev[dev].error_word.ptr;
    }

    apex::AttnParams p;
    p.q = (const apex::f16*)a.q;
    p.k = (const apex::f16*)a.k_cache;
    p.v = (const apex::f16*)a.v_cache;
    p.out = (apex::f16*)a.out;
    p.lse = a.lse_out;
    p.counters = (int32_t*)counters;
    p.pacc = (float*)partials;
    p.pml = part_ml ? (float*)part_ml
                    : (float*)((char*)partials +
                               align_up(sizeof(float) * 2 * (size_t)workers * G * apex::kHeadDim, 256));
    p.bt_stride = a.block_table_stride;
    p.scale_log2 = a.scale * 1.4426950408889634f;
    p.B = a.B;
    p.Hq = a.Hq;
    p.Hkv = a.Hkv;
    p.min_units = a.num_workers > 0 ? 1 : apex::kMinUnitsPerWorker;
    p.seg_cost = a.num_workers > 0 ? 0 : apex::kSegmentCostUnits;
    p.cus = cus;
    p.launched = (int)workers;
    p.num_blocks = check ? a.num_blocks : 0;
    p.error_word = (unsigned*)error_word;
    p.k_new = (const apex::f16*)a.k_new;
    p.v_new = (const apex::f16*)a.v_new;
    p.new_stride = new_stride;
    p.k_store = (apex::f16*)a.k_cache;
    p.v_store = (apex::f16*)a.v_cache;
#ifdef APEX_TRACE_WORK_GROUPS
    {
        std::lock_guard<std::mutex> lock(g_mutex);
        p.trace = g_trace;
        p.trace_groups = g_trace_groups;
    }
#endif

    hipStream_t stream = (hipStream_t)a.stream;
    const int32_t* bt = a.block_table;
    const int32_t* lens = a.context_lens;
    void* const* ev = a.attn_kernel_events;
    return dispatch(G, check, append, p, bt, lens, workers, ev, stream);
}

}  // namespace

extern "C" {

int apex_decode_version(void) { return 310; }

const char* apex_decode_last_error(void) { return apex::last_error_message(); }

size_t apex_decode_counter_bytes(int B, int Hkv)
{
    if (B < 0 || Hkv <= 0) return 0;
    return counter_bytes(B, Hkv);
}

size_t apex_decode_workspace_bytes(int B, int Hq, int Hkv, int d, int block_size, int num_workers)
{
    if (check_shapes(B, Hq, Hkv, d, block_size) != APEX_OK || num_workers < 0) return 0;
    int64_t workers = num_workers;
    if (workers == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || default_workers(dev, Hq / Hkv, &workers) != APEX_OK)
            return 0;
    }
    return counter_bytes(B, Hkv) + partial_bytes(workers, Hq / Hkv);
}

int apex_decode_attention_ex(const apex_decode_args* args)
{
    apex::clear_error();
    if (!args) return fail(APEX_ERR_INVALID_ARG, "args is NULL");
    return enqueue(*args, false);
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

int apex_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* block_table, const int32_t* context_lens, void* out,
                                  int B, int Hq, int Hkv, int d, int block_size, float scale,
                                  void* stream)
{
    apex::clear_error();
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
    return enqueue(a, true);
}

#ifdef APEX_TRACE_WORK_GROUPS
int apex_decode_trace_buffer(void* device_words, int64_t max_work_groups)
{
    apex::clear_error();
    if (max_work_groups < 0) return fail(APEX_ERR_INVALID_ARG, "max_work_groups is negative");
    if (device_words && !aligned(device_words, 8))
        return fail(APEX_ERR_INVALID_ARG, "the trace buffer must be 8-byte aligned");
    std::lock_guard<std::mutex> lock(g_mutex);
    g_trace = device_words ? (uint64_t*)device_words : nullptr;
    g_trace_groups = device_words ? max_work_groups : 0;
    return APEX_OK;
}
#endif

int apex_decode_check_device_error(uint32_t* error_bits)
{
    apex::clear_error();
    if (!error_bits) return fail(APEX_ERR_INVALID_ARG, "error_bits is NULL");
    *error_bits = 0;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return fail(APEX_ERR_HIP, "device ordinal %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_mutex);
    Buffer& w = g_dev[dev].error_word;
    if (!w.ptr) return APEX_OK;   // no checked call ran on this device
    e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(error_bits, w.ptr, 4, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemset(w.ptr, 0, 4);
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "reading the error word: %s", hipGetErrorString(e));
    return APEX_OK;
}

int apex_decode_release_workspace(void)
{
    apex::clear_error();
    std::lock_guard<std::mutex> lock(g_mutex);
    int rc = APEX_OK;
    for (int d = 0; d < kMaxDevices; ++d) {
        DeviceState& s = g_dev[d];
        if (!s.counters.ptr && !s.partials.ptr && !s.error_word.ptr) continue;
        int prev = 0;
        (void)hipGetDevice(&prev);
        if (hipSetDevice(d) == hipSuccess && hipDeviceSynchronize() == hipSuccess) {
            if (s.counters.ptr) (void)hipFree(s.counters.ptr);
            if (s.partials.ptr) (void)hipFree(s.partials.ptr);
            if (s.error_word.ptr) (void)hipFree(s.error_word.ptr);
            s.counters = Buffer();
            s.partials = Buffer();
            s.error_word = Buffer();
        } else {
            rc = fail(APEX_ERR_HIP, "could not release the workspaces of device %d", d);
        }
        (void)hipSetDevice(prev);
    }
    return rc;
}

}  // extern "C"
