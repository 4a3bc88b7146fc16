// Shared device-side definitions of the RNNLM frame scorer (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rnnlm.h"

namespace rn {

typedef unsigned long long u64;   // the integer type HIP 64-bit atomics take

constexpr u64 kPhi = 0x9E3779B97F4A7C15ull;   // SplitMix64 increment (2^64 / golden ratio)
constexpr int kMaxLH = 2048;                       // largest L*H (codes staged in LDS)
constexpr int kMaxCW = kMaxLH / 2;                 // largest code-word count (EXACT: 2 per word)

// Counter slots in the device counter array (int64 each).
enum Ctr {
    C_HC_SIZE = 0, C_SC_SIZE, C_FRAMES, C_QUERIES, C_SCORE_HITS, C_QUERY_DUPS, C_COMPUTED,
    C_HISTS, C_HIST_HITS, C_HIST_DUPS, C_GRU_ROWS, C_HIST_INS, C_HIST_REJ, C_SCORE_INS,
    C_SCORE_REJ, C_FRAME_M, C_N
};

// Frame arguments as the kernels see them.
struct FrameArgs {
    int n_hist, n_query;
    const float *hist_vec;
    const int32_t *hist_words, *q_hist, *q_tgt;
    float *scores, *hnew;
    uint8_t *q_status, *h_status;
    int32_t *q_rep, *h_rep;
    u64 *h_hash;
};

// smallest fp32 bit pattern >= 10^-j, j = 0..20 (decimal decade boundaries)
struct DecadeTab {
    uint32_t lo[21];
};

// Everything a kernel needs to know about one context (passed by value).
struct Dev {
    // configuration
    int V, E, H, L, LH, wdtype, me_log2, me_order, qmode, qdigits, max_hist, max_query, CW;
    long long cap_hist, cap_query;
    unsigned long long seed;
    uint32_t hi_mask, si_mask, ft_mask, qt_mask;
    // weights (borrowed) and packed GRU weights [3H][Kx + H] per layer
    const void *emb;
    const void *Wp[2];
    const float *b_ih[2];
    const void *U_out;
    const float *b_out;
    const float *maxent;
    // history cache: open-addressing index (slot id, key hash) + dense entries
    int *hc_islot;
    u64 *hc_ihash;
    u64 *hc_codes;   // [cap_hist][CW]
    int *hc_word;                   // [cap_hist]
    float *hc_val;                  // [cap_hist][LH]
    // LM-query (score) cache: index + dense entries (hist slot, w-2, w-3, target) -> score
    int *sc_islot;
    u64 *sc_ihash;
    int4 *sc_key;
    float *sc_val;
    // statistics and sticky error bits
    long long *ctr;
    unsigned *derr;
    // per-frame history scratch
    u64 *f_codes;    // [max_hist][CW]
    u64 *f_hhash;
    int *f_words;                   // [max_hist][3], ids clamped into [0, V)
    int *f_hcslot;                  // cache slot found before the frame, or -1
    int *f_hrep, *f_hstat, *f_hslot, *f_ftpos;
    u64 *f_hptr;     // device address of each history's h' (all layers)
    int *f_rows;                    // GRU work list: history index of row r
    u64 *f_rowdst;   // where row r writes its h'
    float *f_hval;                  // [max_hist][LH] h' of rows the cache did not admit
    u64 *ft_hash;    // per-frame history table (cleared after the frame)
    int *ft_min;
    // per-frame query scratch
    int4 *f_qkey;                   // (history representative, w-2, w-3, target)
    int *f_qhist, *f_qsc, *f_qrep, *f_qstat, *f_qcand, *f_qadmit, *f_qtpos;
    u64 *qt_hash;
    int *qt_min;
    // normaliser partials [max_hist][n_tiles] of (max, sum exp)
    float2 *ln_part;
};

__device__ __forceinline__ u64 mix64(u64 z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// round-to-nearest-even fp32 -> bf16 (inputs are finite)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// butterfly sum over the 64 lanes; every lane ends with the same value
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ u64 wave_sum_u64(u64 v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// 64-bit hash of a query key (for table placement only)
__device__ __forceinline__ u64 query_hash(int a, int b, int c, int d) {
    u64 g = mix64((u64)(uint32_t)a + kPhi);
    g = mix64(g ^ (u64)(uint32_t)(b + 2));
    g = mix64(g ^ (u64)(uint32_t)(c + 2));
    return mix64(g ^ (u64)(uint32_t)(d + 1));
}

// slot of the order-n MaxEnt n-gram (w-1 .. w-(n-1), target) in a 2^log2 table
__device__ __forceinline__ uint32_t maxent_slot(int order, int w1, int w2, int w3, int tgt, int log2) {
    u64 g = mix64((u64)order * kPhi);
    g = mix64(g ^ (u64)(w1 + 1));
    if (order >= 3) g = mix64(g ^ (u64)(w2 + 1));
    if (order >= 4) g = mix64(g ^ (u64)(w3 + 1));
    g = mix64(g ^ (u64)(tgt + 1));
    return (uint32_t)(g & ((1ull << log2) - 1));
}

}  // namespace rn
