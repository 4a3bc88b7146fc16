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
constexpr int kPlanMaxHist = 2048;                 // frame planner limits (LDS tables)
constexpr int kPlanMaxQuery = 8192;

// Counter slots in the device counter array (int64 each).
enum Ctr {
    C_HC_SIZE = 0, C_SC_SIZE, C_FRAMES, C_QUERIES, C_SCORE_HITS, C_QUERY_DUPS, C_COMPUTED,
    C_HISTS, C_HIST_HITS, C_HIST_DUPS, C_GRU_ROWS, C_HIST_INS, C_HIST_REJ, C_SCORE_INS,
    C_SCORE_REJ, C_FRAME_M, C_STAGED, C_NEAR_CAP, C_DONE, C_N
};

// QRec flag bits above the 2-bit base status (COMPUTED or Q_DUP)
constexpr int QF_CAND = 16;    // first of its key with a cached history key: may be admitted
constexpr int QF_PROBE = 32;   // the history key was cached before the frame: probe the LM cache

// Frame arguments as the kernels see them.
struct FrameArgs {
    int n_hist, n_query;
    const float *hist_vec;
    const u64 *hist_ptr;   // optional per-history row addresses (replace hist_vec)
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

// History-cache index record (open addressing, 16 B): slot -1 = empty.
struct HcIdx {
    u64 hash;
    int slot;   // dense entry (codes + h') of this key
    int word;   // GRU input word of the key
};

// LM-query cache entry (open addressing, 32 B, key stored in place): hs -1 = empty.
struct ScEnt {
    int hs;     // history-cache slot of the query's history key
    int w2, w3; // MaxEnt context words of the key (-1 where the orders do not use them)
    int t;      // target word
    float val;  // stored fp32 score
    int pad[3];
};

// What the scorer needs per query beyond its words, written by the frame
// planner (16 B); the words (f_qwords) come from the keys kernel.
struct QRec {
    u64 hptr;   // address of the history's top-layer h'
    int flags;  // bits 0-1 base status (COMPUTED / Q_DUP), QF_CAND, QF_PROBE; bits 6.. staging slot
    int hs;     // history-cache slot after the frame (-1: not cached)
};

// What the frame planner reads per history, written by the keys kernel as
// one 16-byte record.
struct HistRec {
    u64 hash;   // 64-bit key hash
    int slot;   // history-cache slot found before the frame, or -1
    int w1;     // GRU input word (clamped into [0, V))
};

// Cache probes read the linear-probe sequence kProbeWin records at a time,
// one record per lane (tables have at least 64 slots).
constexpr int kProbeShift = 4;
constexpr int kProbeWin = 1 << kProbeShift;

// Independent decode sessions per context (one frame each per launch).
constexpr int kMaxSessions = 8;

// Everything a kernel needs to know about one context (passed by value). The
// per-session state (caches, counters, per-frame scratch) of session s lives
// s * sess_stride bytes after session 0's; session_view() shifts the pointers.
struct Dev {
    // configuration
    int V, E, H, L, LH, wdtype, me_log2, me_order, qmode, qdigits, max_hist, max_query, CW;
    int sessions;
    long long sess_stride;
    long long cap_hist, cap_query;
    unsigned long long seed;
    uint32_t hi_mask, si_mask;
    // weights (borrowed) and packed GRU weights [3H][Kx + H] per layer
    const void *emb;
    const void *Wp[2];
    const float *b_ih[2];
    const void *Wl;    // the layer a GRU launch computes: Wp[layer], b_ih[layer] (set per launch, so
    const float *bl;   // that no argument load waits for the layer index)
    const void *U_out;
    const float *b_out;
    const float *maxent;
    // history cache: index + dense entries
    HcIdx *hc_idx;
    u64 *hc_codes;    // [cap_hist][CW]
    float *hc_val;    // [cap_hist][LH]
    // LM-query cache, and the scores admitted this frame (entered into the
    // table by the next frame's keys kernel, so probes always see the cache as
    // it was before the frame)
    ScEnt *sc_tab;
    ScEnt *sc_stage;  // [max_query]
    // statistics and sticky error bits
    long long *ctr;
    unsigned *derr;
    // per-frame history scratch
    u64 *f_codes;     // [max_hist][CW]
    HistRec *f_hrec;  // key hash, cache slot before the frame, input word
    int *f_hstat, *f_hslot;
    u64 *f_hptr;      // device address of each history's h' (all layers)
    int *f_roww;      // GRU input word (w-1) of row r
    u64 *f_rowh;      // address of row r's history vector (all layers)
    u64 *f_rowdst;    // where row r writes its h'
    float *f_hval;    // [max_hist][LH] h' of rows the cache did not admit
    // bf16 weights: the GEMM's A operand, rounded to bf16 once per frame
    uint16_t *f_hbf;  // [max_hist][LH] each history row (written by the keys kernel)
    u64 *f_rowhb;     // address of row r's bf16 history row
    uint16_t *f_xbf;  // two layers: [max_hist][H] the first layer's h' of row r (its tiles' epilogue)
    // per-frame query scratch
    int4 *f_qkey;     // (history index, w-2, w-3, target) for exact key checks
    int4 *f_qwords;   // (w-1, w-2, w-3, target) of each query, as the scorer reads them
    QRec *f_qrec;
    int *f_qcand;     // admission candidates (used when the cache is nearly full)
    int4 *f_part;     // per scoring block: (computed, duplicates, hits, admitted), folded later
    // normaliser partials [256][n_tiles] of (max, sum exp)
    float2 *ln_part;
};

template <class T>
__host__ __device__ __forceinline__ T *shift_ptr(T *p, long long o) {
    return reinterpret_cast<T *>(reinterpret_cast<uintptr_t>(p) + o);
}

// The context as seen by session s: its own caches, counters and scratch.
// The host applies it to the first frame of a launch, and kernels to later
// frames relative to that one, so a one-frame launch reads every pointer
// straight from its arguments.
__host__ __device__ __forceinline__ Dev session_view(const Dev &d0, int s) {
    Dev d = d0;
    const long long o = (long long)s * d0.sess_stride;
    d.hc_idx = shift_ptr(d.hc_idx, o);
    d.hc_codes = shift_ptr(d.hc_codes, o);
    d.hc_val = shift_ptr(d.hc_val, o);
    d.sc_tab = shift_ptr(d.sc_tab, o);
    d.sc_stage = shift_ptr(d.sc_stage, o);
    d.ctr = shift_ptr(d.ctr, o);
    d.derr = shift_ptr(d.derr, o);
    d.f_codes = shift_ptr(d.f_codes, o);
    d.f_hrec = shift_ptr(d.f_hrec, o);
    d.f_hstat = shift_ptr(d.f_hstat, o);
    d.f_hslot = shift_ptr(d.f_hslot, o);
    d.f_hptr = shift_ptr(d.f_hptr, o);
    d.f_roww = shift_ptr(d.f_roww, o);
    d.f_rowh = shift_ptr(d.f_rowh, o);
    d.f_rowdst = shift_ptr(d.f_rowdst, o);
    d.f_hval = shift_ptr(d.f_hval, o);
    d.f_hbf = shift_ptr(d.f_hbf, o);
    d.f_rowhb = shift_ptr(d.f_rowhb, o);
    d.f_xbf = shift_ptr(d.f_xbf, o);
    d.f_qkey = shift_ptr(d.f_qkey, o);
    d.f_qwords = shift_ptr(d.f_qwords, o);
    d.f_qrec = shift_ptr(d.f_qrec, o);
    d.f_qcand = shift_ptr(d.f_qcand, o);
    d.f_part = shift_ptr(d.f_part, o);
    return d;
}

// The frames of one launch (at most one per session), with each kernel's
// block ranges: entry e's blocks of a role start at off[e] (off[n] = total).
struct FrameBlock {
    FrameArgs f[kMaxSessions];
    int sess[kMaxSessions];          // session of entry e, relative to entry 0's (the launch's Dev)
    int n;                           // entries
    int hoff[kMaxSessions + 1];      // keys kernel: history blocks
    int qoff[kMaxSessions + 1];      // keys kernel: query-key blocks
    int soff[kMaxSessions + 1];      // keys kernel: staged-insert blocks
    int npart[kMaxSessions];         // scoring blocks of the session's last frame still to fold
    int boff[kMaxSessions + 1];      // scoring kernel: entry e's blocks (its query blocks, then its
    int qblk[kMaxSessions];          //   qblk[e] = ... history blocks) start at boff[e]
};

// scoring blocks of each session's last frame whose counts are still to fold
struct FoldParts {
    int npart[kMaxSessions];
};

// entry whose range [off[e], off[e+1]) holds b (off[0] = 0 <= b < off[n])
__device__ __forceinline__ int entry_of(const int *off, int n, int b) {
    int e = 0;
    while (e + 1 < n && b >= off[e + 1]) ++e;
    return e;
}

__device__ __forceinline__ u64 mix64(u64 z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// round-to-nearest-even fp32 -> bf16 (inputs are finite)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// four fp32 as four bf16 (RNE), lowest element in the lowest half-word
__device__ __forceinline__ uint2 pack_bf16x4(float4 a) {
    uint2 r;
    r.x = (uint32_t)f32_to_bf16(a.x) | ((uint32_t)f32_to_bf16(a.y) << 16);
    r.y = (uint32_t)f32_to_bf16(a.z) | ((uint32_t)f32_to_bf16(a.w) << 16);
    return r;
}

// A history handle is bad when null or not 16-byte aligned.
__device__ __forceinline__ bool bad_handle(u64 p) { return p == 0 || (p & 15); }

// The row a history handle names; a bad handle is replaced by a row of the
// workspace, so that no access leaves valid memory.
__device__ __forceinline__ const float *handle_row(const Dev &d, u64 p) {
    return bad_handle(p) ? d.f_hval : reinterpret_cast<const float *>(p);
}

// Address of history i's L*H vector: a row of hist_vec, or its handle (a bad
// one is replaced as above and reported through *bad).
__device__ __forceinline__ const float *hist_row(const Dev &d, const FrameArgs &f, int i, bool &bad) {
    if (!f.hist_ptr) return f.hist_vec + (size_t)i * d.LH;
    const u64 p = f.hist_ptr[i];
    bad = bad_handle(p);
    return handle_row(d, p);
}

// Index of the calling wave in its block, as a scalar. The compiler cannot
// prove threadIdx.x >> 6 uniform across a wave; branches on a value it takes
// for divergent become exec-masked regions, and a matrix instruction inside
// such a region still writes its accumulator when no lane is active. Every
// branch around an MFMA must therefore depend on scalars only.
// Load through a pointer known to address global memory. Pointers read from
// memory or chosen by a select are generic to the compiler, which then emits
// flat loads (they also count against the LDS wait counter); this spells out
// the global address space.
template <typename T>
__device__ __forceinline__ T ldg(const void *p) {
    static_assert(sizeof(T) == 16 || sizeof(T) == 8 || sizeof(T) == 4, "16-, 8- or 4-byte loads");
    if constexpr (sizeof(T) == 4) {
        const unsigned v = *reinterpret_cast<const __attribute__((address_space(1))) unsigned *>(reinterpret_cast<uintptr_t>(p));
        return __builtin_bit_cast(T, v);
    } else {
        typedef unsigned int raw __attribute__((ext_vector_type(sizeof(T) / 4)));
        const raw v = *reinterpret_cast<const __attribute__((address_space(1))) raw *>(reinterpret_cast<uintptr_t>(p));
        return __builtin_bit_cast(T, v);
    }
}

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

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

// 64-bit hash of a query key (for table placement only); `a` identifies the
// history key (its cache slot, or its 64-bit key hash within a frame)
__device__ __forceinline__ u64 query_hash(u64 a, int b, int c, int d) {
    u64 g = mix64(a + kPhi);
    g = mix64(g ^ (u64)(uint32_t)(b + 2));
    g = mix64(g ^ (u64)(uint32_t)(c + 2));
    return mix64(g ^ (u64)(uint32_t)(d + 1));
}

// Counts of the last frame's scoring blocks (per-block records, written
// without atomics), added into a copy of the counters `c` held in LDS. Run by
// one block; every thread must call it.
__device__ __forceinline__ void fold_partials(const Dev &d, int n, long long *c, int *s_red) {
    int a0 = 0, a1 = 0, a2 = 0, a3 = 0;
    for (int b = threadIdx.x; b < n; b += blockDim.x) {
        const int4 p = d.f_part[b];
        a0 += p.x; a1 += p.y; a2 += p.z; a3 += p.w;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        a0 += __shfl_xor(a0, o, 64);
        a1 += __shfl_xor(a1, o, 64);
        a2 += __shfl_xor(a2, o, 64);
        a3 += __shfl_xor(a3, o, 64);
    }
    if (threadIdx.x < 4) s_red[threadIdx.x] = 0;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
        atomicAdd(&s_red[0], a0);
        atomicAdd(&s_red[1], a1);
        atomicAdd(&s_red[2], a2);
        atomicAdd(&s_red[3], a3);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        c[C_COMPUTED] += s_red[0];
        c[C_QUERY_DUPS] += s_red[1];
        c[C_SCORE_HITS] += s_red[2];
        c[C_SCORE_INS] += s_red[3];
        c[C_SC_SIZE] += s_red[3];
    }
    __syncthreads();
}

// slot of the order-n MaxEnt n-gram (w-1 .. w-(n-1), target) in a 2^log2 table
// order-n MaxEnt feature: the order seeds a fold of the n-1 context words
// (most recent first), then the target; the prefix (everything before the
// target) is shared by all targets after the same context
__device__ __forceinline__ u64 maxent_prefix(int order, int w1, int w2, int w3) {
    u64 g = mix64((u64)order * kPhi);
    g = mix64(g ^ (u64)(w1 + 1));
    if (order >= 3) g = mix64(g ^ (u64)(w2 + 1));
    if (order >= 4) g = mix64(g ^ (u64)(w3 + 1));
    return g;
}

__device__ __forceinline__ uint32_t maxent_slot(int order, int w1, int w2, int w3, int tgt, int log2) {
    const u64 g = mix64(maxent_prefix(order, w1, w2, w3) ^ (u64)(tgt + 1));
    return (uint32_t)(g & ((1ull << log2) - 1));
}

}  // namespace rn
