// attend.h -- the per-ISA inner loops of the host paged decode attention.
//
// attend_simd.cpp is compiled once per instruction set (AVX-512 and AVX2),
// each time into its own namespace; cpu_attention.cpp picks one at run time.
#pragma once

#include <stdint.h>

namespace apex_cpu {

// One call's shapes and pointers (host memory).
struct Problem {
    const uint16_t* q;          // fp16 [B][Hq][d]
    const uint16_t* k;          // fp16 [NB][Hkv][bs][d]
    const uint16_t* v;
    const int32_t* block_table; // [B][stride]
    int64_t stride;
    int Hq, Hkv, G, d, bs;
    float scale_log2;           // scale * log2(e): scores are kept in base 2
};

// Running state of one (request, kv-head) range, base-2 units:
// m[G] running max, l[G] normaliser, acc[G][d] unnormalised output.
struct State {
    float* m;
    float* l;
    float* acc;
};

// Work item: tokens [t0, t1) of request b against kv-head g.
struct Item {
    int b, g;
    int t0, t1;
    int64_t slot;   // partial slot, or -1 when the item covers the whole pair
};

#define APEX_CPU_DECLARE(NS)                                                                   \
    namespace NS {                                                                              \
    /* Attends tokens [t0, t1) of (b, g); state starts empty.  scratch holds at least          \
       scratch_floats(G, d) floats. */                                                          \
    void attend(const Problem& p, int b, int g, int t0, int t1, State st, float* scratch);     \
    /* out[h][:] = acc[h][:] / l[h] as fp16 (nearest even); lse[h] (natural log) if lse. */     \
    void finish(const float* m, const float* l, const float* acc, int G, int d, uint16_t* out,  \
                float* lse);                                                                    \
    /* Merges n partial states (each G heads) into one, log-sum-exp identity. */                \
    void merge(const float* const* m, const float* const* l, const float* const* acc, int n,   \
               int G, int d, float* m_out, float* l_out, float* acc_out);                      \
    }

APEX_CPU_DECLARE(simd_avx512)
APEX_CPU_DECLARE(simd_avx2)

// Scratch floats an attend() call needs for G heads of dimension d (query
// rows, tile weights, a 16-row K tile and G x 16 partial score vectors of
// 16 floats), with room to align the vectors to 64 bytes.
inline int64_t scratch_floats(int G, int d) { return (int64_t)G * d + (int64_t)G * 16 + 16 * (int64_t)d + (int64_t)G * 256 + 64; }

}  // namespace apex_cpu
