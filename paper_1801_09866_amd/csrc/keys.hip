// History and query keys: quantise, hash, de-duplicate, probe and fill the
// two caches (Sec. 2.4 LM-query cache; Sec. 3 history cache of quantised
// history vectors). All decisions are integer-exact.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

// k-significant-digit code of one fp32 element (Sec. 3 "rounding"), ties away
// from zero. Code = sign<<15 | (e+20)<<10 | m for +-m*10^(e-k+1), zero -> 0.
// |x| = M * 2^-s. Its decade j (10^-j <= |x| < 10^(1-j), i.e. j =
// ceil(-log10 |x|)) is j1 = floor(n log10 2) + 1 or j1 + 1, where 2^-(n+1)
// <= |x| < 2^-n; one exact comparison, M 5^j1 >= 2^(s-j1) in 128-bit
// integers, decides. Then m = floor(M*10^p/2^s + 1/2) with 10^p = 5^p * 2^p,
// p = k - 1 + j, from the same product. floor(n log10 2) is n * 1233 >> 12
// for every n here (-1 .. 66). Everything is computed in registers: 5^j1 is
// a product of 5^(2^b) over the bits b of j1, and the only table entry read
// (10^-20, the smallest code) is uniform.
__device__ __forceinline__ uint32_t sigdig_code(float x, int k, const DecadeTab &T, bool &bad) {
    uint32_t b = __float_as_uint(x);
    uint32_t neg = b >> 31, mag = b & 0x7FFFFFFFu;
    if (mag > 0x3F800000u) { bad = true; return 0u; }   // |x| > 1, inf, nan
    if (mag < T.lo[20]) return 0u;                       // |x| < 1e-20
    const int ex = (int)(mag >> 23);                     // normal: |x| >= 1e-20
    const u64 M = (u64)((mag & 0x7FFFFFu) | 0x800000u);
    const int s = 150 - ex;
    const int n = 126 - ex;                              // -1 .. 66
    const int j1 = ((n * 1233) >> 12) + 1;               // 0 .. 20
    u64 p5 = (j1 & 1) ? 5ull : 1ull;
    p5 *= (j1 & 2) ? 25ull : 1ull;
    p5 *= (j1 & 4) ? 625ull : 1ull;
    p5 *= (j1 & 8) ? 390625ull : 1ull;
    p5 *= (j1 & 16) ? 152587890625ull : 1ull;
    const unsigned __int128 t = (unsigned __int128)M * p5;   // |x| 10^j1 = t 2^-(s - j1)
    const bool ge = (t >> (s - j1)) != 0;                // |x| >= 10^-j1
    const int j = ge ? j1 : j1 + 1;
    const u64 f = (k == 1 ? 1ull : k == 2 ? 5ull : 25ull) * (ge ? 1ull : 5ull);   // 5^(p - j1)
    const int sh = s - (k - 1 + j);                      // >= 18 for |x| <= 1
    const unsigned __int128 v = t * f + ((unsigned __int128)1 << (sh - 1));
    uint32_t m = (uint32_t)(v >> sh);
    int e = -j;
    const uint32_t top = k == 1 ? 10u : k == 2 ? 100u : 1000u;   // 10^k
    if (m == top) { m = top / 10u; e += 1; }
    return (neg << 15) | ((uint32_t)(e + 20) << 10) | m;
}

__device__ __forceinline__ uint32_t exact_code(float x, bool &bad) {
    uint32_t b = __float_as_uint(x);
    if ((b & 0x7FFFFFFFu) >= 0x7F800000u) bad = true;
    return b == 0x80000000u ? 0u : b;
}

__device__ __forceinline__ bool nonfinite(float x) {
    return (__float_as_uint(x) & 0x7FFFFFFFu) >= 0x7F800000u;
}

// ---------------------------------------------------------------------------
// K1: one wave per history (sign and exact keys; k significant digits take a
// block per history, below): validate, quantise into code words, hash the
// key (codes, GRU input word), and probe the history cache with an exact
// code comparison. Each lane keeps its code words in registers:
//   SIGN   word w (64 elements, one ballot) is held by lane w      (CW <= 32)
//   EXACT  word w = elements 2w, 2w+1, held by lane w % 64, slot w / 64
// ---------------------------------------------------------------------------
constexpr int kWordsPerLane = kMaxCW / 64;   // 16
constexpr int kSignWords = kMaxLH / 64;      // sign code words of the longest vector

// Block roles (independent work, so one launch runs them side by side):
//   [0, hb)            one wave per history, or one block for k significant digits
//   [hb, hb+qb)        one thread per query: its key, validated
//   [hb+qb, hb+qb+sb)  enter the scores the previous frame admitted into the
//                      LM-query cache
//   last block         fold the previous frame's per-block scoring counts
//                      into the counters
__device__ void insert_staged(const Dev &d, int b, int sb) {
    const long long ns = d.ctr[C_STAGED];
    for (long long e = (long long)b * blockDim.x + threadIdx.x; e < ns; e += (long long)sb * blockDim.x) {
        const ScEnt en = d.sc_stage[e];
        if (en.hs < 0) continue;   // a candidate that turned out to be a cache hit
        unsigned pos = (unsigned)(query_hash((u64)en.hs, en.w2, en.w3, en.t) & d.si_mask);
        for (unsigned n = 0; n <= d.si_mask; ++n) {
            ScEnt *slot = d.sc_tab + pos;
            if (atomicCAS(&slot->hs, -1, en.hs) == -1) {
                slot->w2 = en.w2;
                slot->w3 = en.w3;
                slot->t = en.t;
                slot->val = en.val;
                break;
            }
            pos = (pos + 1) & d.si_mask;
        }
    }
}

__device__ void query_key(const Dev &d, const FrameArgs &f, int q) {
    if (q >= f.n_query) return;
    unsigned qerr = 0;
    int i = f.q_hist[q];
    if (i < 0 || i >= f.n_hist) { qerr |= RNNLM_DERR_QHIST; i = 0; }
    int t = f.q_tgt[q];
    if (t < 0 || t >= d.V) { qerr |= RNNLM_DERR_WORD; t = 0; }
    int w[3];
#pragma unroll
    for (int c = 0; c < 3; ++c) {   // same clamping as the history waves
        w[c] = f.hist_words[(size_t)i * 3 + c];
        if (w[c] < 0 || w[c] >= d.V) w[c] = 0;
    }
    d.f_qkey[q] = make_int4(i, d.me_order >= 3 ? w[1] : -1, d.me_order >= 4 ? w[2] : -1, t);
    d.f_qwords[q] = make_int4(w[0], d.me_order >= 3 ? w[1] : -1, d.me_order >= 4 ? w[2] : -1, t);
    if (qerr) atomicOr(d.derr, qerr);
}

__device__ void fold_counts(const Dev &d, int npart) {
    __shared__ int s_red[4];
    __shared__ long long c[C_N];
    if (threadIdx.x < C_N) c[threadIdx.x] = d.ctr[threadIdx.x];
    __syncthreads();
    fold_partials(d, npart, c, s_red);
    if (threadIdx.x == 0) {   // only the fields the fold changes
        d.ctr[C_COMPUTED] = c[C_COMPUTED];
        d.ctr[C_QUERY_DUPS] = c[C_QUERY_DUPS];
        d.ctr[C_SCORE_HITS] = c[C_SCORE_HITS];
        d.ctr[C_SCORE_INS] = c[C_SCORE_INS];
        d.ctr[C_SC_SIZE] = c[C_SC_SIZE];
    }
}

// one wave: history i of a frame. BF16: the model's GEMM takes bf16 rows, so
// the wave also writes the row's bf16 copy (fp32 models keep no row elements
// live across the cache probe, and more waves fit).
template <bool BF16>
__device__ void hist_wave(const Dev &d, const FrameArgs &f, int i) {
    const int lane = threadIdx.x & 63;
    if (i >= f.n_hist) return;
    // the record's words are loaded with the row, not after it
    int w3[3];
#pragma unroll
    for (int c = 0; c < 3; ++c) w3[c] = f.hist_words[(size_t)i * 3 + c];
    bool hbad = false;   // wave-uniform: one history per wave
    const float *x = hist_row(d, f, i, hbad);
    const int CW = d.CW;
    u64 words[kWordsPerLane];
    bool bad = false;
    u64 hs = 0;
    // the lane's row elements, kept for the GEMM's bf16 copy of the row:
    // sign v[u] = element 64 u + lane; exact float2 s = elements
    // 2 (lane + 64 s) ..
    static_assert(kSignWords <= 32 && 2 * kWordsPerLane <= 32, "row elements per lane");
    __attribute__((aligned(16))) float rv[32];   // registers: indexed only by constants
    if (d.qmode == RNNLM_Q_SIGN) {
        // the whole row in flight at once (one coalesced load per 64
        // elements), then one ballot per code word
        float *v = rv;
#pragma unroll
        for (int u = 0; u < kSignWords; ++u) v[u] = u < CW ? ldg<float>(x + u * 64 + lane) : 0.0f;
        words[0] = 0;
#pragma unroll
        for (int u = 0; u < kSignWords; ++u) {
            if (u < CW) {   // wave-uniform
                bad |= nonfinite(v[u]);
                const u64 b = __ballot(v[u] < 0.0f);
                if (lane == u) words[0] = b;
            }
        }
        if (lane < CW) hs = mix64(words[0] ^ ((u64)(lane + 1) * kPhi));
    } else {
        // all of the row's loads first (2 elements per code word), then the codes
        float2 *v = reinterpret_cast<float2 *>(rv);
#pragma unroll
        for (int s = 0; s < kWordsPerLane; ++s)
            v[s] = lane + 64 * s < CW ? ldg<float2>(x + 2 * (lane + 64 * s)) : make_float2(0.f, 0.f);
#pragma unroll
        for (int s = 0; s < kWordsPerLane; ++s) {
            const int w = lane + 64 * s;
            if (w < CW) {
                words[s] = (u64)exact_code(v[s].x, bad) | ((u64)exact_code(v[s].y, bad) << 32);
                hs += mix64(words[s] ^ ((u64)(w + 1) * kPhi));
            }
        }
    }
    const u64 S = wave_sum_u64(hs);
    const bool anybad = __ballot(bad) != 0ull;

    // words of the history record (validated, clamped)
    // a bad handle read a placeholder row: report the handle, not its values
    unsigned err = hbad ? RNNLM_DERR_HANDLE : (anybad ? RNNLM_DERR_VALUE : 0u);
#pragma unroll
    for (int c = 0; c < 3; ++c)
        if (w3[c] < 0 || w3[c] >= d.V) { err |= RNNLM_DERR_WORD; w3[c] = 0; }
    const int w1 = w3[0];
    const u64 h = mix64(d.seed ^ S ^ mix64((u64)w1 + 1));

    // history-cache probe: the linear-probe sequence from the key's position,
    // kProbeWin index records per round trip (one per lane); a record with the
    // key's hash and word before the first empty one is confirmed by an exact
    // comparison of the codes
    int hit = -1;
    unsigned base = (unsigned)(h & d.hi_mask);
    for (unsigned n = 0; n <= (d.hi_mask >> kProbeShift) && hit < 0; ++n) {
        const HcIdx r = d.hc_idx[(base + (lane & (kProbeWin - 1))) & d.hi_mask];
        const bool in = lane < kProbeWin;
        const u64 emp = __ballot(in && r.slot < 0);
        u64 cand = __ballot(in && r.slot >= 0 && r.hash == h && r.word == w1);
        if (emp) cand &= (emp & (~emp + 1ull)) - 1ull;
        for (; cand; cand &= cand - 1ull) {
            const int slot = __shfl(r.slot, __ffsll((unsigned long long)cand) - 1);
            const u64 *cc = d.hc_codes + (size_t)slot * CW;
            bool neq = false;
            if (d.qmode == RNNLM_Q_SIGN) {
                if (lane < CW) neq = cc[lane] != words[0];
            } else {
#pragma unroll
                for (int s = 0; s < kWordsPerLane; ++s) {
                    const int w = lane + 64 * s;
                    if (w < CW) neq |= cc[w] != words[s];
                }
            }
            if (__ballot(neq) == 0ull) { hit = slot; break; }
        }
        if (emp) break;
        base = (base + kProbeWin) & d.hi_mask;
    }

    // The GEMM's bf16 copy of the row, for a key the cache does not hold
    // (only such a key can become a GRU row; hit is wave-uniform).
    if (BF16 && hit < 0) {
        if (d.qmode == RNNLM_Q_SIGN) {
            uint16_t *hb = d.f_hbf + (size_t)i * d.LH;
#pragma unroll
            for (int u = 0; u < kSignWords; ++u)
                if (u < CW) hb[u * 64 + lane] = f32_to_bf16(rv[u]);
        } else {
            uint32_t *hb = reinterpret_cast<uint32_t *>(d.f_hbf + (size_t)i * d.LH);
            const float2 *v = reinterpret_cast<const float2 *>(rv);
#pragma unroll
            for (int s = 0; s < kWordsPerLane; ++s)
                if (lane + 64 * s < CW)
                    hb[lane + 64 * s] = (uint32_t)f32_to_bf16(v[s].x) | ((uint32_t)f32_to_bf16(v[s].y) << 16);
        }
    }

    // per-frame outputs
    u64 *out = d.f_codes + (size_t)i * CW;
    if (d.qmode == RNNLM_Q_SIGN) {
        if (lane < CW) out[lane] = words[0];
    } else {
#pragma unroll
        for (int s = 0; s < kWordsPerLane; ++s) {
            const int w = lane + 64 * s;
            if (w < CW) out[w] = words[s];
        }
    }
    if (lane == 0) {
        if (err) atomicOr(d.derr, err);
        HistRec hr;
        hr.hash = h;
        hr.slot = hit;
        hr.w1 = w3[0];
        d.f_hrec[i] = hr;
        if (f.h_hash) f.h_hash[i] = h;
    }
}

// SIGDIG: one block (4 waves) per history. The quantiser's integer work is
// the kernel's cost in this mode, so thread t takes code words t and t + 256
// (elements 4w..4w+3), four times as many lanes per history as one wave
// would give it. The key hash is a wrapping sum, so the four waves' partial
// sums combine in any order; the cache probe walks the same index records in
// every wave, and a candidate's codes are compared by all four.
constexpr int kSdWords = kMaxLH / 4 / 256;   // code words per thread of the longest vector

__device__ void hist_block_sigdig(const Dev &d, const FrameArgs &f, const DecadeTab &T, int i) {
    __shared__ u64 s_sum[4];
    __shared__ int s_flag[4];
    const int tid = threadIdx.x, lane = tid & 63, wv = wave_id();
    if (i >= f.n_hist) return;   // block-uniform
    int w3[3];
#pragma unroll
    for (int c = 0; c < 3; ++c) w3[c] = f.hist_words[(size_t)i * 3 + c];
    bool hbad = false;
    const float *x = hist_row(d, f, i, hbad);
    const int CW = d.CW;
    float4 v[kSdWords];
#pragma unroll
    for (int s = 0; s < kSdWords; ++s)
        v[s] = tid + 256 * s < CW ? ldg<float4>(x + 4 * (tid + 256 * s)) : make_float4(0.f, 0.f, 0.f, 0.f);
    if (d.wdtype == RNNLM_BF16) {   // the GEMM's bf16 copy of the row
        uint2 *hb = reinterpret_cast<uint2 *>(d.f_hbf + (size_t)i * d.LH);
#pragma unroll
        for (int s = 0; s < kSdWords; ++s)
            if (tid + 256 * s < CW) hb[tid + 256 * s] = pack_bf16x4(v[s]);
    }
    u64 words[kSdWords];
    bool bad = false;
    u64 hs = 0;
#pragma unroll
    for (int s = 0; s < kSdWords; ++s) {
        const int w = tid + 256 * s;
        words[s] = 0;
        if (w < CW) {
            words[s] = (u64)sigdig_code(v[s].x, d.qdigits, T, bad) |
                       ((u64)sigdig_code(v[s].y, d.qdigits, T, bad) << 16) |
                       ((u64)sigdig_code(v[s].z, d.qdigits, T, bad) << 32) |
                       ((u64)sigdig_code(v[s].w, d.qdigits, T, bad) << 48);
            hs += mix64(words[s] ^ ((u64)(w + 1) * kPhi));
        }
    }
    const u64 ws = wave_sum_u64(hs);
    const bool wbad = __ballot(bad) != 0ull;
    if (lane == 0) {
        s_sum[wv] = ws;
        s_flag[wv] = wbad ? 1 : 0;
    }
    __syncthreads();
    const u64 S = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    const bool anybad = (s_flag[0] | s_flag[1] | s_flag[2] | s_flag[3]) != 0;
    __syncthreads();   // s_flag is reused by the probe

    unsigned err = hbad ? RNNLM_DERR_HANDLE : (anybad ? RNNLM_DERR_VALUE : 0u);
#pragma unroll
    for (int c = 0; c < 3; ++c)
        if (w3[c] < 0 || w3[c] >= d.V) { err |= RNNLM_DERR_WORD; w3[c] = 0; }
    const int w1 = w3[0];
    const u64 h = mix64(d.seed ^ S ^ mix64((u64)w1 + 1));

    // history-cache probe in windows, as in hist_wave; every wave reads the
    // same records, so every branch below is uniform over the block
    int hit = -1;
    unsigned base = (unsigned)(h & d.hi_mask);
    for (unsigned n = 0; n <= (d.hi_mask >> kProbeShift) && hit < 0; ++n) {
        const HcIdx r = d.hc_idx[(base + (lane & (kProbeWin - 1))) & d.hi_mask];
        const bool in = lane < kProbeWin;
        const u64 emp = __ballot(in && r.slot < 0);
        u64 cand = __ballot(in && r.slot >= 0 && r.hash == h && r.word == w1);
        if (emp) cand &= (emp & (~emp + 1ull)) - 1ull;
        for (; cand; cand &= cand - 1ull) {
            const int slot = __shfl(r.slot, __ffsll((unsigned long long)cand) - 1);
            const u64 *cc = d.hc_codes + (size_t)slot * CW;
            bool neq = false;
#pragma unroll
            for (int s = 0; s < kSdWords; ++s) {
                const int w = tid + 256 * s;
                if (w < CW) neq |= cc[w] != words[s];
            }
            const bool wneq = __ballot(neq) != 0ull;
            if (lane == 0) s_flag[wv] = wneq ? 1 : 0;
            __syncthreads();
            const bool eq = (s_flag[0] | s_flag[1] | s_flag[2] | s_flag[3]) == 0;
            __syncthreads();
            if (eq) { hit = slot; break; }
        }
        if (emp) break;
        base = (base + kProbeWin) & d.hi_mask;
    }

    u64 *out = d.f_codes + (size_t)i * CW;
#pragma unroll
    for (int s = 0; s < kSdWords; ++s) {
        const int w = tid + 256 * s;
        if (w < CW) out[w] = words[s];
    }
    if (tid == 0) {
        if (err) atomicOr(d.derr, err);
        HistRec hr;
        hr.hash = h;
        hr.slot = hit;
        hr.w1 = w1;
        d.f_hrec[i] = hr;
        if (f.h_hash) f.h_hash[i] = h;
    }
}

// The frames of a launch (one per session) side by side: each role's blocks
// are split among the frames by the ranges in fb. MULTI = false (a single
// frame) reads everything at fixed argument offsets, so no argument load
// waits for another.
template <bool MULTI, bool BF16>
__global__ __launch_bounds__(256) void k_hist_key(Dev d0, FrameBlock fb, DecadeTab T) {
    const int b = blockIdx.x, n = MULTI ? fb.n : 1;
    const int hb = MULTI ? fb.hoff[n] : fb.hoff[1], qb = MULTI ? fb.qoff[n] : fb.qoff[1],
              sb = MULTI ? fb.soff[n] : fb.soff[1];
    int e, lb, role;
    if (b < hb) {
        e = MULTI ? entry_of(fb.hoff, n, b) : 0;
        lb = b - (MULTI ? fb.hoff[e] : 0);
        role = 0;
    } else if (b < hb + qb) {
        e = MULTI ? entry_of(fb.qoff, n, b - hb) : 0;
        lb = b - hb - (MULTI ? fb.qoff[e] : 0);
        role = 1;
    } else if (b < hb + qb + sb) {
        e = MULTI ? entry_of(fb.soff, n, b - hb - qb) : 0;
        lb = b - hb - qb - (MULTI ? fb.soff[e] : 0);
        role = 2;
    } else {
        e = MULTI ? b - hb - qb - sb : 0;
        lb = 0;
        role = 3;
    }
    const Dev d = MULTI ? session_view(d0, fb.sess[e]) : d0;
    const FrameArgs &f = fb.f[e];
    if (role == 0) {
        if (d.qmode == RNNLM_Q_SIGDIG) hist_block_sigdig(d, f, T, lb);   // one block per history
        else hist_wave<BF16>(d, f, lb * 4 + wave_id());                 // one wave per history
    }
    else if (role == 1) query_key(d, f, lb * blockDim.x + threadIdx.x);
    else if (role == 2) insert_staged(d, lb, fb.soff[e + 1] - fb.soff[e]);
    else fold_counts(d, fb.npart[e]);
}

// debug hook: quantise a flat array with the frame kernels' quantiser
__global__ __launch_bounds__(256) void k_debug_quantize(const float *x, long long n, int qmode, int k,
                                                        DecadeTab T, void *codes, int *err) {
    bool bad = false;
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (qmode == RNNLM_Q_SIGN) {
        // one wave per 64 elements, n a multiple of 64
        if (i < n) {
            float v = x[i];
            bad = nonfinite(v);
            u64 word = __ballot(v < 0.0f);
            if ((threadIdx.x & 63) == 0) reinterpret_cast<u64 *>(codes)[i >> 6] = word;
        }
    } else if (i < n) {
        if (qmode == RNNLM_Q_SIGDIG)
            reinterpret_cast<uint16_t *>(codes)[i] = (uint16_t)sigdig_code(x[i], k, T, bad);
        else
            reinterpret_cast<uint32_t *>(codes)[i] = exact_code(x[i], bad);
    }
    if (bad) atomicOr(err, RNNLM_DERR_VALUE);
}

// get_stats: block s folds session s's pending scoring counts
__global__ __launch_bounds__(256) void k_fold_stats(Dev d0, FoldParts fp) {
    __shared__ int s_red[4];
    __shared__ long long c[C_N];
    const Dev d = session_view(d0, blockIdx.x);
    const int npart = fp.npart[blockIdx.x];
    if (threadIdx.x < C_N) c[threadIdx.x] = d.ctr[threadIdx.x];
    __syncthreads();
    fold_partials(d, npart, c, s_red);
    if (threadIdx.x < C_N) d.ctr[threadIdx.x] = c[threadIdx.x];
}

__global__ void k_fill_u32(uint32_t *p, uint32_t v, long long n) {
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = v;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
void launch_fill_u32(void *p, uint32_t v, long long n, hipStream_t s) {
    if (n <= 0) return;
    long long blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    k_fill_u32<<<(unsigned)blocks, 256, 0, s>>>(reinterpret_cast<uint32_t *>(p), v, n);
}

void launch_fold_stats(const Dev &d, const FoldParts &fp, hipStream_t s) {
    k_fold_stats<<<d.sessions, 256, 0, s>>>(d, fp);
}

void launch_hist_key(const Dev &d, const FrameBlock &fb, const DecadeTab &T, hipStream_t s, Stamp ts) {
    const int n = fb.n;
    const unsigned grid = fb.hoff[n] + fb.qoff[n] + fb.soff[n] + n;
    if (d.wdtype == RNNLM_BF16) {
        if (n > 1) launch_k(k_hist_key<true, true>, grid, 256, s, ts, d, fb, T);
        else launch_k(k_hist_key<false, true>, grid, 256, s, ts, d, fb, T);
    } else {
        if (n > 1) launch_k(k_hist_key<true, false>, grid, 256, s, ts, d, fb, T);
        else launch_k(k_hist_key<false, false>, grid, 256, s, ts, d, fb, T);
    }
}
void launch_debug_quantize(const float *x, long long n, int qmode, int k, const DecadeTab &T,
                           void *codes, int *err, hipStream_t s) {
    long long blocks = (n + 255) / 256;
    k_debug_quantize<<<(unsigned)blocks, 256, 0, s>>>(x, n, qmode, k, T, codes, err);
}

}  // namespace rn
