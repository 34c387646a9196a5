// driver.cpp -- the library's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer, or ThreadSanitizer (built and run by
// tests/test_sanitizers.py, never part of the product).
//
// Seeded random inputs for:
//   - the fp64 oracle (test infrastructure) and the host paged-attention
//     backend, compared with each other (max-abs <= 2e-3): both SIMD paths,
//     whole and chunked pairs, several thread counts and pool resizes;
//   - the partition's host mirror, against an explicit line of positions
//     (every non-empty pair's cost positions, then its blocks);
//   - the strategy selection (Eq. 1-8, Alg. 1-2) on random valid inputs;
//   - the partition's 32-bit arithmetic (the kernel's path when
//     V (launched + 1) < 2^32) against its 64-bit form.
// Usage: driver <cases> <mode: all | threads>; exit status 0 when every
// check holds.
#include <immintrin.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <random>
#include <vector>

#include "apex_cpu_attention.h"
#include "apex_decode.h"
#include "apex_sched.h"
#include "plan_policy.h"

extern "C" int apex_oracle_decode_attention_f64(const uint16_t* q, const uint16_t* k_cache,
                                                const uint16_t* v_cache, const int32_t* block_table,
                                                long stride, const int32_t* context_lens, int B, int Hq,
                                                int Hkv, int d, int bs, float scale, double* out,
                                                double* lse, int num_threads);
extern "C" double apex_oracle_f16_to_f64(uint16_t bits);

namespace {

int g_failures = 0;

void check(bool ok, const char* what, long a = 0, long b = 0)
{
    if (!ok) {
        ++g_failures;
        fprintf(stderr, "FAIL %s (%ld, %ld)\n", what, a, b);
    }
}

uint16_t to_half(float x) { return (uint16_t)_cvtss_sh(x, 0); }   // round to nearest even

// oracle threads: 1 under ThreadSanitizer (it does not see OpenMP's own
// synchronisation), 2 otherwise
int g_oracle_threads = 2;

// One attention case: the oracle against the host backend.
void attention_case(std::mt19937_64& rng, int threads, bool force_avx2, int min_chunk)
{
    std::uniform_int_distribution<int> pick(0, 1 << 30);
    const int Gs[] = {1, 2, 4, 8}, Hkvs[] = {1, 2, 4, 8}, ds[] = {64, 128}, bss[] = {8, 16};
    const int G = Gs[pick(rng) % 4], Hkv = Hkvs[pick(rng) % 4], d = ds[pick(rng) % 2];
    const int bs = bss[pick(rng) % 2], Hq = G * Hkv, B = 1 + pick(rng) % 12;
    std::vector<int32_t> lens(B);
    int maxb = 1;
    for (int b = 0; b < B; ++b) {
        const int kind = pick(rng) % 5;
        lens[b] = kind == 0 ? 0 : kind == 1 ? 1 + pick(rng) % 20 : kind == 2 ? bs * (1 + pick(rng) % 30)
                : kind == 3 ? 200 + pick(rng) % 1500 : -(pick(rng) % 3);
        if (lens[b] > 0) maxb = std::max(maxb, (lens[b] + bs - 1) / bs);
    }
    const int stride = maxb + pick(rng) % 3;
    int nblocks = 1;   // block 0 is the pad target of unused table entries
    std::vector<int32_t> table((size_t)B * stride, 0);
    for (int b = 0; b < B; ++b)
        for (int j = 0; j < (lens[b] + bs - 1) / bs; ++j) table[(size_t)b * stride + j] = nblocks++;
    std::normal_distribution<float> nrm(0.f, 1.f);
    const size_t nkv = (size_t)nblocks * Hkv * bs * d;
    std::vector<uint16_t> q((size_t)B * Hq * d), k(nkv), v(nkv);
    for (auto& x : q) x = to_half(nrm(rng));
    for (auto& x : k) x = to_half(nrm(rng));
    for (auto& x : v) x = to_half(nrm(rng));
    const float scale = 1.f / sqrtf((float)d);

    std::vector<double> ref((size_t)B * Hq * d), lse_ref((size_t)B * Hq);
    check(apex_oracle_decode_attention_f64(q.data(), k.data(), v.data(), table.data(), stride, lens.data(), B,
                                           Hq, Hkv, d, bs, scale, ref.data(), lse_ref.data(), g_oracle_threads) == 0,
          "oracle rejected a valid case");
    std::vector<uint16_t> out((size_t)B * Hq * d, 0xffff);
    std::vector<float> lse((size_t)B * Hq);
    apex_cpu_args a;
    memset(&a, 0, sizeof(a));
    a.q = q.data();
    a.k_cache = k.data();
    a.v_cache = v.data();
    a.block_table = table.data();
    a.context_lens = lens.data();
    a.out = out.data();
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.d = d;
    a.block_size = bs;
    a.scale = scale;
    a.block_table_stride = stride;
    a.lse_out = lse.data();
    a.num_threads = threads;
    a.min_chunk_tokens = min_chunk;
    a.flags = force_avx2 ? APEX_CPU_FLAG_FORCE_AVX2 : 0;
    const int rc = apex_cpu_decode_attention_ex(&a);
    check(rc == APEX_OK, "host attention failed", rc);
    if (rc != APEX_OK) return;
    double worst = 0.;
    for (size_t i = 0; i < out.size(); ++i) {
        const double g = apex_oracle_f16_to_f64(out[i]);
        worst = std::max(worst, std::isfinite(g) ? fabs(g - ref[i]) : 1e30);
    }
    check(worst <= 2e-3, "host attention off the oracle", (long)(worst * 1e6), B);
}

// One partition case: the host mirror against an explicit line of positions.
void partition_case(std::mt19937_64& rng)
{
    std::uniform_int_distribution<int> pick(0, 1 << 30);
    const int B = pick(rng) % 300, Hkvs[] = {1, 2, 8, 32}, Hkv = Hkvs[pick(rng) % 4];
    const bool forced = pick(rng) % 3 == 0;
    const int launched_opts[] = {1, 3, 7, 64, 256, 512, 1024, 100000};
    const int launched = launched_opts[pick(rng) % 8];
    const int cus = pick(rng) % 2 ? 256 : 0;
    std::vector<int32_t> lens(B);
    for (auto& L : lens) {
        const int kind = pick(rng) % 4;
        L = kind == 0 ? -(pick(rng) % 3) : kind == 1 ? pick(rng) % 40 : kind == 2 ? pick(rng) % 5000
          : 16 * (pick(rng) % 100);
    }
    std::vector<int32_t> contrib((size_t)std::max(1, B * Hkv));
    int64_t units = -1, active = -1, partials = -1;
    const int rc = apex_decode_plan_host(B ? lens.data() : nullptr, B, Hkv, 16, launched, forced, cus,
                                         contrib.data(), &units, &active, &partials);
    check(rc == APEX_OK, "plan_host failed", rc);
    if (rc != APEX_OK) return;

    // the line: every non-empty pair's K cost positions, then its blocks
    int64_t U = 0, P = 0;
    for (int L : lens) {
        const int64_t nb = L > 0 ? (L + 15) / 16 : 0;
        U += nb * Hkv;
        P += nb > 0 ? Hkv : 0;
    }
    int64_t lw = launched;
    if (!forced && cus > 0 && P <= cus && U <= 1024LL * cus) lw = std::min<int64_t>(lw, cus);
    const int64_t W = std::min<int64_t>(lw, std::max<int64_t>({1, U / (forced ? 1 : 16), P}));
    const int64_t K = forced ? 0 : 8, V = U + K * P;
    check(units == U, "units", (long)units, (long)U);
    check(active == (U ? W : 0), "active workers", (long)active, (long)W);
    int64_t pos = 0, split = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t nb = lens[b] > 0 ? (lens[b] + 15) / 16 : 0;
        for (int g = 0; g < Hkv; ++g) {
            int64_t n = 0;
            if (nb > 0) {
                pos += K;
                // owner of position p: the w with floor(w V / W) <= p < floor((w + 1) V / W)
                auto owner = [&](int64_t p) {
                    int64_t w = (int64_t)((__int128)p * W / V);
                    while (w > 0 && (__int128)w * V / W > p) --w;
                    while ((__int128)(w + 1) * V / W <= p) ++w;
                    return w;
                };
                n = owner(pos + nb - 1) - owner(pos) + 1;
                pos += nb;
                if (n > 1) split += n;
            }
            check(contrib[(size_t)b * Hkv + g] == n, "contributors", (long)contrib[(size_t)b * Hkv + g], (long)n);
        }
    }
    check(pos == V, "line length", (long)pos, (long)V);
    check(partials == split, "partials", (long)partials, (long)split);
}

// One case of the partition in 32-bit arithmetic, drawn inside the bound the
// kernel uses it under (V (launched + 1) <= 2^32 - 1, half the draws close to
// it): the worker count and every sampled range end must equal the 64-bit
// form's.
void width_case(std::mt19937_64& rng)
{
    std::uniform_int_distribution<int64_t> pick(0, (int64_t)1 << 40);
    const int64_t launched = 1 + pick(rng) % ((int64_t)1 << 20);
    const int64_t max_v = (int64_t)(0xffffffffull / (uint64_t)(launched + 1));
    const int64_t K = pick(rng) % 2 ? 8 : 0;
    int64_t units = 0, pairs = 0;
    for (int tries = 0; tries < 100; ++tries) {
        units = pick(rng) % 2 ? max_v - pick(rng) % 64 : 1 + pick(rng) % std::max<int64_t>(1, max_v);
        if (units < 1) continue;
        pairs = 1 + pick(rng) % units;
        if (units + K * pairs <= max_v) break;
        units = 0;
    }
    if (units == 0) return;
    const int64_t V = units + K * pairs;
    check((uint64_t)V * (uint64_t)(launched + 1) <= 0xffffffffull, "width case outside the bound", (long)V);
    const int64_t cus = pick(rng) % 2 ? 256 : 0;
    const int min_units = pick(rng) % 2 ? 16 : 1;
    const int64_t W = apex::active_workers(units, launched, min_units, pairs, cus);
    const uint32_t W32 = apex::active_workers_t<uint32_t>((uint32_t)units, (uint32_t)launched, (uint32_t)min_units,
                                                          (uint32_t)pairs, (uint32_t)cus);
    check((int64_t)W32 == W, "32-bit worker count", (long)W32, (long)W);
    for (int i = 0; i < 16; ++i) {
        const int64_t w = i < 2 ? (i == 0 ? 0 : W - 1) : pick(rng) % W;
        for (int64_t e = w; e <= w + 1; ++e) {
            const uint32_t end32 = (uint32_t)e * (uint32_t)V / W32;   // the kernel's 32-bit range end
            check((int64_t)end32 == apex::worker_start(e, V, W), "32-bit range end", (long)e, (long)end32);
        }
    }
}

// One strategy-selection case on random valid inputs (exercised for
// undefined behaviour; the decisions are checked against the oracle in
// tests/test_sched.py).
void sched_case(std::mt19937_64& rng)
{
    std::uniform_real_distribution<double> u(1e-6, 1e-2);
    apex_sched_inputs in;
    memset(&in, 0, sizeof(in));
    in.n_g = 1e5 + 1e9 * u(rng);
    in.n_c = 1e7 * u(rng);
    in.t_glinear = u(rng);
    in.t_gatt = u(rng);
    in.t_glinear_pref = u(rng);
    in.t_gatt_pref = u(rng);
    in.prefill = (int)(rng() % 2);
    in.mixed_form = (int)(rng() % 2);
    apex_sched_result r;
    check(apex_sched_select(&in, &r) == APEX_OK, "apex_sched_select");
    const int waiting = (int)(rng() % 64);
    const int scheduled = std::min(waiting, (int)(rng() % 4));
    check(apex_sched_main((int)(rng() % 3), 1 + (int)(rng() % 64), waiting, scheduled, &in, &r) == APEX_OK,
          "apex_sched_main");
    // more CPU requests scheduled than waiting is refused
    check(apex_sched_main(0, 1, waiting, waiting + 1, &in, &r) == APEX_ERR_INVALID_ARG,
          "apex_sched_main accepted more scheduled than waiting");
    check(std::isfinite(apex_sched_ratio_bound(in.t_glinear, in.t_gatt)), "ratio bound");
}

}  // namespace

int main(int argc, char** argv)
{
    const int cases = argc > 1 ? atoi(argv[1]) : 50;
    const bool threads_only = argc > 2 && strcmp(argv[2], "threads") == 0;
    if (threads_only) g_oracle_threads = 1;
    std::mt19937_64 rng(2026);
    const int thread_opts[] = {1, 2, 3, 4};
    for (int i = 0; i < cases; ++i) {
        if (i % 10 == 0) check(apex_cpu_set_threads(1 + i / 10 % 4) == APEX_OK, "pool resize");
        attention_case(rng, thread_opts[i % 4], i % 2 == 1, i % 3 == 0 ? 16 : 0);
        if (!threads_only) {
            partition_case(rng);
            sched_case(rng);
            for (int j = 0; j < 20; ++j) width_case(rng);
        }
    }
    printf("%d cases, %d failures\n", cases, g_failures);
    return g_failures ? 1 : 0;
}
