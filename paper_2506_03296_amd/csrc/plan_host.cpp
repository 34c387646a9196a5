// plan_host.cpp -- host mirror of the work partition (apex_decode_plan_host in
// include/apex_decode.h): the same plan_policy.h arithmetic the kernel's
// prologue runs, over host context_lens, for inspection and tests.  Plain
// host C++ (no HIP kernels), so it also builds with g++ under sanitizers.
#include <stdint.h>

#include "apex_decode.h"
#include "plan_policy.h"
#include "status.h"

using apex::fail;

extern "C" {

int apex_decode_plan_host(const int32_t* context_lens, int B, int Hkv, int block_size,
                          int launched_workers, int forced, int cus, int32_t* contributors_out,
                          int64_t* units_out, int64_t* active_out, int64_t* partials_out)
{
    apex::clear_error();
    if (B < 0 || Hkv <= 0 || launched_workers <= 0 || cus < 0)
        return fail(APEX_ERR_INVALID_ARG, "bad partition arguments");
    if (B > 0 && !context_lens) return fail(APEX_ERR_INVALID_ARG, "context_lens is NULL");
    if (block_size != apex::kBlockSize)
        return fail(APEX_ERR_UNSUPPORTED, "block_size %d unsupported (only 16)", block_size);
    int64_t blocks = 0, nonempty = 0;
    for (int b = 0; b < B; ++b) {
        blocks += apex::blocks_of(context_lens[b], block_size);
        nonempty += context_lens[b] > 0;
    }
    const int64_t units = blocks * Hkv;
    const int64_t pairs = nonempty * Hkv;
    const int64_t W = apex::active_workers(units, launched_workers,
                                           forced ? 1 : apex::kMinUnitsPerWorker, pairs,
                                           forced ? 0 : cus);
    const int64_t K = forced ? 0 : apex::kSegmentCostUnits;
    const int64_t V = units + K * pairs;
    int64_t partials = 0, pre = 0, pp = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t nb = apex::blocks_of(context_lens[b], block_size);
        for (int g = 0; g < Hkv; ++g) {
            int64_t n = 0;
            if (nb > 0) {
                const int64_t vf = apex::first_block_position(pre * Hkv + (int64_t)g * nb, pp * Hkv + g, K);
                n = apex::worker_of(vf + nb - 1, V, W) - apex::worker_of(vf, V, W) + 1;
                if (n > 1) partials += n;
            }
            if (contributors_out) contributors_out[(size_t)b * Hkv + g] = (int32_t)n;
        }
        pre += nb;
        pp += nb > 0;
    }
    if (units_out) *units_out = units;
    if (active_out) *active_out = units > 0 ? W : 0;
    if (partials_out) *partials_out = partials;
    return APEX_OK;
}

}  // extern "C"
