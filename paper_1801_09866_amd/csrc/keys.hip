// History and query keys: quantise, hash, de-duplicate, probe and fill the
// two caches (Sec. 2.4 LM-query cache; Sec. 3 history cache of quantised
// history vectors). All decisions are integer-exact.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

__constant__ u64 kPow5[23] = {
    1ull, 5ull, 25ull, 125ull, 625ull, 3125ull, 15625ull, 78125ull, 390625ull, 1953125ull,
    9765625ull, 48828125ull, 244140625ull, 1220703125ull, 6103515625ull, 30517578125ull,
    152587890625ull, 762939453125ull, 3814697265625ull, 19073486328125ull, 95367431640625ull,
    476837158203125ull, 2384185791015625ull};
__constant__ uint32_t kPow10[4] = {1u, 10u, 100u, 1000u};

// k-significant-digit code of one fp32 element (Sec. 3 "rounding"), ties away
// from zero. Code = sign<<15 | (e+20)<<10 | m for +-m*10^(e-k+1), zero -> 0.
// |x| = M * 2^-s; the decade e = -j is found by comparing bit patterns with
// the exact decade boundaries, then m = floor(M*10^p/2^s + 1/2) with
// 10^p = 5^p * 2^p evaluated in 128-bit integers.
__device__ __forceinline__ uint32_t sigdig_code(float x, int k, const DecadeTab &T, bool &bad) {
    uint32_t b = __float_as_uint(x);
    uint32_t neg = b >> 31, mag = b & 0x7FFFFFFFu;
    if (mag > 0x3F800000u) { bad = true; return 0u; }   // |x| > 1, inf, nan
    if (mag < T.lo[20]) return 0u;                       // |x| < 1e-20
    int j = 0;
    while (mag < T.lo[j]) ++j;                           // 10^-j <= |x| < 10^(1-j)
    uint32_t ex = mag >> 23;                             // normal: |x| >= 1e-20
    u64 M = (u64)((mag & 0x7FFFFFu) | 0x800000u);
    int s = 150 - (int)ex;
    int p = k - 1 + j;
    int sh = s - p;                                      // >= 18 for |x| <= 1
    unsigned __int128 v = (unsigned __int128)M * kPow5[p] + ((unsigned __int128)1 << (sh - 1));
    uint32_t m = (uint32_t)(v >> sh);
    int e = -j;
    if (m == kPow10[k]) { m = kPow10[k - 1]; e += 1; }
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

// Quantise one vector of n elements into code words (see rnnlm.h for the
// per-mode layout); every thread of the block takes part. Returns the sum of
// mix64(word ^ (w+1)*phi) over the words this thread produced.
__device__ u64 quantise_vector(const float *x, int n, int qmode, int k, const DecadeTab &T,
                                    u64 *out, u64 *lds_copy, bool &bad) {
    const int tid = threadIdx.x, nt = blockDim.x;
    u64 hsum = 0;
    if (qmode == RNNLM_Q_SIGN) {
        const int lane = tid & 63, wv = tid >> 6, nw = nt >> 6;
        for (int w = wv; w < n / 64; w += nw) {
            float v = x[w * 64 + lane];
            bad |= nonfinite(v);
            u64 word = __ballot(v < 0.0f);
            if (lane == 0) {
                out[w] = word;
                if (lds_copy) lds_copy[w] = word;
                hsum += mix64(word ^ ((u64)(w + 1) * kPhi));
            }
        }
    } else if (qmode == RNNLM_Q_SIGDIG) {
        for (int w = tid; w < n / 4; w += nt) {
            float4 v = reinterpret_cast<const float4 *>(x)[w];
            u64 word = (u64)sigdig_code(v.x, k, T, bad) |
                            ((u64)sigdig_code(v.y, k, T, bad) << 16) |
                            ((u64)sigdig_code(v.z, k, T, bad) << 32) |
                            ((u64)sigdig_code(v.w, k, T, bad) << 48);
            out[w] = word;
            if (lds_copy) lds_copy[w] = word;
            hsum += mix64(word ^ ((u64)(w + 1) * kPhi));
        }
    } else {
        for (int w = tid; w < n / 2; w += nt) {
            float2 v = reinterpret_cast<const float2 *>(x)[w];
            u64 word = (u64)exact_code(v.x, bad) | ((u64)exact_code(v.y, bad) << 32);
            out[w] = word;
            if (lds_copy) lds_copy[w] = word;
            hsum += mix64(word ^ ((u64)(w + 1) * kPhi));
        }
    }
    return hsum;
}

// ---------------------------------------------------------------------------
// K1: one block per history: validate, quantise, hash, probe the history
// cache (exact code comparison), and enter the key into the frame table.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_hist_key(Dev d, FrameArgs f, DecadeTab T) {
    const int i = blockIdx.x, tid = threadIdx.x;
    __shared__ u64 s_codes[kMaxCW];
    __shared__ u64 s_red[4];
    __shared__ int s_flag[4];
    __shared__ int s_cand;
    __shared__ unsigned s_pos;

    bool bad = false;
    u64 hs = quantise_vector(f.hist_vec + (size_t)i * d.LH, d.LH, d.qmode, d.qdigits, T,
                                  d.f_codes + (size_t)i * d.CW, s_codes, bad);
    hs = wave_sum_u64(hs);
    int anybad = __syncthreads_or(bad ? 1 : 0);
    if ((tid & 63) == 0) s_red[tid >> 6] = hs;
    __syncthreads();

    u64 h = 0;
    int w1 = 0;
    if (tid == 0) {
        u64 S = s_red[0] + s_red[1] + s_red[2] + s_red[3];
        unsigned err = anybad ? RNNLM_DERR_VALUE : 0u;
        int w[3];
        for (int c = 0; c < 3; ++c) {
            w[c] = f.hist_words[(size_t)i * 3 + c];
            if (w[c] < 0 || w[c] >= d.V) { err |= RNNLM_DERR_WORD; w[c] = 0; }
            d.f_words[i * 3 + c] = w[c];
        }
        if (err) atomicOr(d.derr, err);
        w1 = w[0];
        h = mix64(d.seed ^ S ^ mix64((u64)w1 + 1));
        d.f_hhash[i] = h;
        if (f.h_hash) f.h_hash[i] = h;
        s_pos = (unsigned)(h & d.hi_mask);
        s_red[0] = h;
        s_flag[0] = w1;
    }
    __syncthreads();
    h = s_red[0];
    w1 = s_flag[0];

    // history-cache probe: walk the index until an empty slot; candidates with
    // equal hash and word are confirmed by comparing all code words
    int hit = -1;
    for (unsigned iter = 0; iter <= d.hi_mask; ++iter) {
        if (tid == 0) {
            int cand = -1;
            unsigned pos = s_pos;
            for (unsigned n = 0; n <= d.hi_mask; ++n) {
                int s = d.hc_islot[pos];
                if (s < 0) break;
                if (d.hc_ihash[pos] == h && d.hc_word[s] == w1) { cand = s; break; }
                pos = (pos + 1) & d.hi_mask;
            }
            s_pos = pos;
            s_cand = cand;
        }
        __syncthreads();
        int cand = s_cand;
        if (cand < 0) break;
        const u64 *cc = d.hc_codes + (size_t)cand * d.CW;
        int neq = 0;
        for (int w = tid; w < d.CW; w += blockDim.x) neq |= (cc[w] != s_codes[w]);
        neq = __syncthreads_or(neq);
        if (!neq) { hit = cand; break; }
        if (tid == 0) s_pos = (s_pos + 1) & d.hi_mask;
        __syncthreads();
    }

    if (tid == 0) {
        d.f_hcslot[i] = hit;
        // frame table: key -> lowest history index
        u64 key = h ? h : 1ull;
        unsigned pos = (unsigned)(h & d.ft_mask);
        for (unsigned n = 0; n <= d.ft_mask; ++n) {
            unsigned long long old = atomicCAS(&d.ft_hash[pos], 0ull, (u64)key);
            if (old == 0ull || old == key) { atomicMin(&d.ft_min[pos], i); break; }
            pos = (pos + 1) & d.ft_mask;
        }
        d.f_ftpos[i] = (int)pos;
    }
}

__device__ bool same_hist_key(const Dev &d, int a, int b) {
    if (d.f_words[a * 3] != d.f_words[b * 3]) return false;
    const u64 *ca = d.f_codes + (size_t)a * d.CW, *cb = d.f_codes + (size_t)b * d.CW;
    for (int w = 0; w < d.CW; ++w)
        if (ca[w] != cb[w]) return false;
    return true;
}

// exclusive scan of one int per thread over a 1024-thread block; returns the
// prefix and writes the block total to *total
__device__ int block_scan_1024(int v, int *s_tmp, int *total) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_tmp[wv] = x;
    __syncthreads();
    if (tid < 16) {
        int t = s_tmp[tid];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            int y = __shfl_up(t, o, 16);
            if (tid >= o) t += y;
        }
        s_tmp[16 + tid] = t;
    }
    __syncthreads();
    int base = wv ? s_tmp[16 + wv - 1] : 0;
    *total = s_tmp[31];
    __syncthreads();
    return base + x - v;
}

// ---------------------------------------------------------------------------
// K2: single block: history representatives, statuses, the GRU work list and
// history-cache admission (ascending index while below capacity).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_hist_plan(Dev d, FrameArgs f) {
    const int tid = threadIdx.x, n = f.n_hist;
    __shared__ int s_tmp[32];
    __shared__ int s_cnt[4];
    if (tid < 4) s_cnt[tid] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += 1024) {
        int m = d.ft_min[d.f_ftpos[i]];
        int rep = i;
        if (m != i) {
            if (same_hist_key(d, m, i)) rep = m;
            else {   // two keys share a 64-bit hash: find the first equal key
                for (int j = 0; j < i; ++j)
                    if (d.f_hhash[j] == d.f_hhash[i] && same_hist_key(d, j, i)) { rep = j; break; }
            }
        }
        d.f_hrep[i] = rep;
    }
    __syncthreads();
    const long long hc_size = d.ctr[C_HC_SIZE];
    int carry = 0;
    for (int c0 = 0; c0 < n; c0 += 1024) {
        int i = c0 + tid;
        int st = RNNLM_H_DUP;
        if (i < n) {
            int rep = d.f_hrep[i];
            st = d.f_hcslot[i] >= 0 ? RNNLM_HC_HIT : (rep == i ? RNNLM_H_REP : RNNLM_H_DUP);
        }
        int total;
        int r = block_scan_1024(i < n && st == RNNLM_H_REP ? 1 : 0, s_tmp, &total) + carry;
        if (i < n) {
            d.f_hstat[i] = st;
            if (st == RNNLM_HC_HIT) {
                int s = d.f_hcslot[i];
                d.f_hslot[i] = s;
                d.f_hptr[i] = (u64)(d.hc_val + (size_t)s * d.LH);
                atomicAdd(&s_cnt[0], 1);
            } else if (st == RNNLM_H_REP) {
                long long slot = hc_size + r;
                float *dst;
                if (slot < d.cap_hist) {
                    dst = d.hc_val + (size_t)slot * d.LH;
                    d.f_hslot[i] = (int)slot;
                    atomicAdd(&s_cnt[2], 1);
                } else {
                    dst = d.f_hval + (size_t)r * d.LH;
                    d.f_hslot[i] = -1;
                    atomicAdd(&s_cnt[3], 1);
                }
                d.f_rows[r] = i;
                d.f_rowdst[r] = (u64)dst;
                d.f_hptr[i] = (u64)dst;
            } else {
                atomicAdd(&s_cnt[1], 1);
            }
        }
        carry += total;
    }
    __syncthreads();
    for (int i = tid; i < n; i += 1024) {
        int st = d.f_hstat[i];
        int rep = d.f_hrep[i];
        if (st == RNNLM_H_DUP) {
            d.f_hslot[i] = d.f_hslot[rep];
            d.f_hptr[i] = d.f_hptr[rep];
        }
        if (f.h_status) f.h_status[i] = (uint8_t)st;
        if (f.h_rep) f.h_rep[i] = rep;
    }
    if (tid == 0) {
        d.ctr[C_FRAME_M] = carry;
        d.ctr[C_HC_SIZE] = hc_size + s_cnt[2];
        d.ctr[C_FRAMES] += 1;
        d.ctr[C_HISTS] += n;
        d.ctr[C_HIST_HITS] += s_cnt[0];
        d.ctr[C_HIST_DUPS] += s_cnt[1];
        d.ctr[C_GRU_ROWS] += carry;
        d.ctr[C_HIST_INS] += s_cnt[2];
        d.ctr[C_HIST_REJ] += s_cnt[3];
    }
}

// ---------------------------------------------------------------------------
// K3: per query: validate, build the key (history representative, MaxEnt
// context words, target), probe the score cache, enter the frame table.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_query_key(Dev d, FrameArgs f) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= f.n_query) return;
    unsigned err = 0;
    int i = f.q_hist[q];
    if (i < 0 || i >= f.n_hist) { err |= RNNLM_DERR_QHIST; i = 0; }
    int t = f.q_tgt[q];
    if (t < 0 || t >= d.V) { err |= RNNLM_DERR_WORD; t = 0; }
    if (err) atomicOr(d.derr, err);
    const int w2 = d.me_order >= 3 ? d.f_words[i * 3 + 1] : -1;
    const int w3 = d.me_order >= 4 ? d.f_words[i * 3 + 2] : -1;
    const int rh = d.f_hrep[i];
    d.f_qkey[q] = make_int4(rh, w2, w3, t);
    d.f_qhist[q] = i;

    int hit = -1;
    const int hs = d.f_hcslot[i];
    if (hs >= 0) {
        u64 sh = query_hash(hs, w2, w3, t);
        unsigned pos = (unsigned)(sh & d.si_mask);
        for (unsigned n = 0; n <= d.si_mask; ++n) {
            int s = d.sc_islot[pos];
            if (s < 0) break;
            if (d.sc_ihash[pos] == sh) {
                int4 k = d.sc_key[s];
                if (k.x == hs && k.y == w2 && k.z == w3 && k.w == t) { hit = s; break; }
            }
            pos = (pos + 1) & d.si_mask;
        }
    }
    d.f_qsc[q] = hit;

    u64 qh = query_hash(rh, w2, w3, t);
    u64 key = qh ? qh : 1ull;
    unsigned pos = (unsigned)(qh & d.qt_mask);
    for (unsigned n = 0; n <= d.qt_mask; ++n) {
        unsigned long long old = atomicCAS(&d.qt_hash[pos], 0ull, (u64)key);
        if (old == 0ull || old == key) { atomicMin(&d.qt_min[pos], q); break; }
        pos = (pos + 1) & d.qt_mask;
    }
    d.f_qtpos[q] = (int)pos;
}

__device__ __forceinline__ bool key_eq(int4 a, int4 b) {
    return a.x == b.x && a.y == b.y && a.z == b.z && a.w == b.w;
}

// K4: per query: representative (lowest index with the same key) and status.
__global__ __launch_bounds__(256) void k_query_resolve(Dev d, FrameArgs f) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= f.n_query) return;
    const int4 kq = d.f_qkey[q];
    int m = d.qt_min[d.f_qtpos[q]];
    int rep = q;
    if (m != q) {
        if (key_eq(d.f_qkey[m], kq)) rep = m;
        else {
            for (int j = 0; j < q; ++j)
                if (key_eq(d.f_qkey[j], kq)) { rep = j; break; }
        }
    }
    int st = d.f_qsc[q] >= 0 ? RNNLM_Q_SCORE_HIT : (rep < q ? RNNLM_Q_DUP : RNNLM_Q_COMPUTED);
    d.f_qrep[q] = rep;
    d.f_qstat[q] = st;
    d.f_qcand[q] = (st == RNNLM_Q_COMPUTED && d.f_hslot[d.f_qhist[q]] >= 0) ? 1 : 0;
    if (f.q_status) f.q_status[q] = (uint8_t)st;
    if (f.q_rep) f.q_rep[q] = rep;
}

// K5: single block: score-cache admission in ascending query index while
// below capacity; statistics.
__global__ __launch_bounds__(1024) void k_query_admit(Dev d, FrameArgs f) {
    const int tid = threadIdx.x, n = f.n_query;
    __shared__ int s_tmp[32];
    __shared__ int s_cnt[5];
    if (tid < 5) s_cnt[tid] = 0;
    __syncthreads();
    const long long sc_size = d.ctr[C_SC_SIZE];
    int carry = 0;
    for (int c0 = 0; c0 < n; c0 += 1024) {
        int q = c0 + tid;
        int cand = q < n ? d.f_qcand[q] : 0;
        int total;
        int r = block_scan_1024(cand, s_tmp, &total) + carry;
        if (q < n) {
            int st = d.f_qstat[q];
            atomicAdd(&s_cnt[st], 1);
            int id = -1;
            if (cand) {
                if (sc_size + r < d.cap_query) { id = (int)(sc_size + r); atomicAdd(&s_cnt[3], 1); }
                else atomicAdd(&s_cnt[4], 1);
            }
            d.f_qadmit[q] = id;
        }
        carry += total;
    }
    __syncthreads();
    if (tid == 0) {
        d.ctr[C_SC_SIZE] = sc_size + s_cnt[3];
        d.ctr[C_QUERIES] += n;
        d.ctr[C_COMPUTED] += s_cnt[RNNLM_Q_COMPUTED];
        d.ctr[C_QUERY_DUPS] += s_cnt[RNNLM_Q_DUP];
        d.ctr[C_SCORE_HITS] += s_cnt[RNNLM_Q_SCORE_HIT];
        d.ctr[C_SCORE_INS] += s_cnt[3];
        d.ctr[C_SCORE_REJ] += s_cnt[4];
    }
}

// ---------------------------------------------------------------------------
// K8: per history, after scoring: enter admitted keys into the history cache,
// copy h' to the caller's output, clear the frame table entries.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_hist_finish(Dev d, FrameArgs f) {
    const int i = blockIdx.x, tid = threadIdx.x;
    const int st = d.f_hstat[i];
    if (st == RNNLM_H_REP) {
        const int slot = d.f_hslot[i];
        if (slot >= 0) {
            const u64 *src = d.f_codes + (size_t)i * d.CW;
            u64 *dst = d.hc_codes + (size_t)slot * d.CW;
            for (int w = tid; w < d.CW; w += blockDim.x) dst[w] = src[w];
            if (tid == 0) {
                d.hc_word[slot] = d.f_words[i * 3];
                u64 h = d.f_hhash[i];
                unsigned pos = (unsigned)(h & d.hi_mask);
                for (unsigned n = 0; n <= d.hi_mask; ++n) {
                    if (atomicCAS(&d.hc_islot[pos], -1, slot) == -1) {
                        d.hc_ihash[pos] = h;
                        break;
                    }
                    pos = (pos + 1) & d.hi_mask;
                }
            }
        }
    }
    if (f.hnew) {
        const float4 *src = reinterpret_cast<const float4 *>(d.f_hptr[i]);
        float4 *dst = reinterpret_cast<float4 *>(f.hnew + (size_t)i * d.LH);
        for (int e = tid; e < d.LH / 4; e += blockDim.x) dst[e] = src[e];
    }
    if (tid == 0) {
        int pos = d.f_ftpos[i];
        d.ft_hash[pos] = 0ull;
        d.ft_min[pos] = 0x7FFFFFFF;
    }
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

void launch_hist_key(const Dev &d, const FrameArgs &f, const DecadeTab &T, hipStream_t s) {
    k_hist_key<<<f.n_hist, 256, 0, s>>>(d, f, T);
}
void launch_hist_plan(const Dev &d, const FrameArgs &f, hipStream_t s) {
    k_hist_plan<<<1, 1024, 0, s>>>(d, f);
}
void launch_query_key(const Dev &d, const FrameArgs &f, hipStream_t s) {
    k_query_key<<<(f.n_query + 255) / 256, 256, 0, s>>>(d, f);
}
void launch_query_resolve(const Dev &d, const FrameArgs &f, hipStream_t s) {
    k_query_resolve<<<(f.n_query + 255) / 256, 256, 0, s>>>(d, f);
}
void launch_query_admit(const Dev &d, const FrameArgs &f, hipStream_t s) {
    k_query_admit<<<1, 1024, 0, s>>>(d, f);
}
void launch_hist_finish(const Dev &d, const FrameArgs &f, hipStream_t s) {
    k_hist_finish<<<f.n_hist, 256, 0, s>>>(d, f);
}
void launch_debug_quantize(const float *x, long long n, int qmode, int k, const DecadeTab &T,
                           void *codes, int *err, hipStream_t s) {
    long long blocks = (n + 255) / 256;
    k_debug_quantize<<<(unsigned)blocks, 256, 0, s>>>(x, n, qmode, k, T, codes, err);
}

}  // namespace rn
