// Scoring and frame finish, one launch (blocks of 4 waves):
//   query waves (Sec. 2.2 NCE, Sec. 2.3 MaxEnt), one wave per query:
//     probe the LM-query cache (Sec. 2.4) if the history key was cached; on a
//     hit return the stored score, else
//       score = U_out[t] . h'_top + b_out[t] + sum_{n=2..N} maxent[slot_n]
//     The output row is read once, coalesced across the wave (16 B per lane
//     per step), and reduced with a fixed butterfly, so equal keys produce
//     equal bits. Admitted new keys are staged; the next frame's keys kernel
//     enters them into the table, so every probe of this frame sees the cache
//     as it was before the frame.
//   history waves, one per history record: admitted new history keys go into
//     the history-cache index (their h' is already in place), and h' is
//     copied to the caller's output.
// Admission order only matters when the frame's candidates could overflow
// the LM-query cache; then the last block to finish admits them in ascending
// query index.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

constexpr int kRowSteps = kMaxLH / 256;   // 16-byte fp32 steps per lane over the longest row
constexpr int kCodeSteps = kMaxCW / 64;   // code words per lane of the longest key

// staging slot e receives a new LM-query cache entry (hs = -1: slot unused)
__device__ __forceinline__ void stage_score(const Dev &d, long long e, int hs, int w2, int w3, int t, float s) {
    ScEnt en;
    en.hs = hs;
    en.w2 = w2;
    en.w3 = w3;
    en.t = t;
    en.val = s;
    en.pad[0] = en.pad[1] = en.pad[2] = 0;
    d.sc_stage[e] = en;
}

template <bool BF16, int RS>
__device__ __forceinline__ void score_query(const Dev &d, const FrameArgs &f, int q, int lane, bool near_cap,
                                            int *s_cnt) {
    const QRec rec = d.f_qrec[q];
    const int4 key = ldg<int4>(d.f_qwords + q);   // (w-1, w-2, w-3, target)
    const int w1 = key.x;
    const int t = key.w;
    const bool probe = rec.flags & QF_PROBE;   // wave-uniform: one query per wave
    // A query whose history key was cached first probes the LM cache (the
    // linear-probe sequence from the key's position, kProbeWin records at a
    // time, lane l reading record l of the window); only a miss then loads
    // the output row, the history row, the bias and the MaxEnt weights.
    // (Loading the rows alongside the probe was measured slower: the loads
    // wasted on hits cost more than the round trip they save on misses.)
    unsigned base = (unsigned)(query_hash((u64)rec.hs, key.y, key.z, t) & d.si_mask);
    ScEnt e = d.sc_tab[probe ? (base + (lane & (kProbeWin - 1))) & d.si_mask : 0];
    bool hit = false;
    float s = 0.0f;
    if (probe) {   // the first matching record before the first empty one
        for (unsigned k = 0; k <= (d.si_mask >> kProbeShift); ++k) {
            const bool in = lane < kProbeWin;
            const u64 stop = __ballot(in && (e.hs < 0 || (e.hs == rec.hs && e.w2 == key.y && e.w3 == key.z &&
                                                             e.t == t)));
            if (stop) {
                const int f = __ffsll((unsigned long long)stop) - 1;
                const int hs_f = __shfl(e.hs, f);
                const float v_f = __shfl(e.val, f);
                hit = hs_f >= 0;
                s = v_f;
                break;
            }
            base = (base + kProbeWin) & d.si_mask;
            e = d.sc_tab[(base + (lane & (kProbeWin - 1))) & d.si_mask];
        }
    }
    float acc = 0.0f, me = 0.0f;
    if (!hit) {
        // bias and MaxEnt weights: independent loads, issued with the rows
        float mw[3];
#pragma unroll
        for (int o = 2; o <= 4; ++o)
            mw[o - 2] = o <= d.me_order ? d.maxent[maxent_slot(o, w1, key.y, key.z, t, d.me_log2)] : 0.0f;
        const float bo = d.b_out[t];
        const float *h = reinterpret_cast<const float *>(rec.hptr);
        // The row loads are unconditional (a lane past the row reads its
        // start and its terms are zeroed in the sum): guarded loads become
        // separate blocks, after which the compiler waits for the first
        // step's data before it issues the next step's loads.
        if (!BF16) {   // the whole row in flight: 16 B per lane per 256 elements
            const float *u = reinterpret_cast<const float *>(d.U_out) + (size_t)t * d.H;
            float4 a[RS], b[RS];
#pragma unroll
            for (int st = 0; st < RS; ++st) {
                const int k = lane * 4 + st * 256;
                const int kc = k < d.H ? k : 0;
                a[st] = b[st] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (st < 4 || d.H > 1024) {   // wave-uniform: rows past 1024 elements only
                    a[st] = ldg<float4>(u + kc);
                    b[st] = ldg<float4>(h + kc);
                }
            }
            const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int st = 0; st < RS; ++st) {
                const bool in = lane * 4 + st * 256 < d.H;
                const float4 x = in ? a[st] : z4, y = in ? b[st] : z4;
                acc = fmaf(x.x, y.x, acc);
                acc = fmaf(x.y, y.y, acc);
                acc = fmaf(x.z, y.z, acc);
                acc = fmaf(x.w, y.w, acc);
            }
        } else {   // 8 bf16 weights per lane per 512 elements
            const uint16_t *u = reinterpret_cast<const uint16_t *>(d.U_out) + (size_t)t * d.H;
            uint4 a[RS / 2];
            float4 b0[RS / 2], b1[RS / 2];
#pragma unroll
            for (int st = 0; st < RS / 2; ++st) {
                const int k = lane * 8 + st * 512;
                const int kc = k < d.H ? k : 0;
                a[st] = make_uint4(0u, 0u, 0u, 0u);
                b0[st] = b1[st] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (st < 2 || d.H > 1024) {   // wave-uniform: rows past 1024 elements only
                    a[st] = ldg<uint4>(u + kc);
                    b0[st] = ldg<float4>(h + kc);
                    b1[st] = ldg<float4>(h + kc + 4);
                }
            }
#pragma unroll
            for (int st = 0; st < RS / 2; ++st) {
                if (lane * 8 + st * 512 >= d.H) {   // terms past the row are zero
                    a[st] = make_uint4(0u, 0u, 0u, 0u);
                    b0[st] = b1[st] = make_float4(0.f, 0.f, 0.f, 0.f);
                }
                acc = fmaf(__uint_as_float(a[st].x << 16), b0[st].x, acc);
                acc = fmaf(__uint_as_float(a[st].x & 0xFFFF0000u), b0[st].y, acc);
                acc = fmaf(__uint_as_float(a[st].y << 16), b0[st].z, acc);
                acc = fmaf(__uint_as_float(a[st].y & 0xFFFF0000u), b0[st].w, acc);
                acc = fmaf(__uint_as_float(a[st].z << 16), b1[st].x, acc);
                acc = fmaf(__uint_as_float(a[st].z & 0xFFFF0000u), b1[st].y, acc);
                acc = fmaf(__uint_as_float(a[st].w << 16), b1[st].z, acc);
                acc = fmaf(__uint_as_float(a[st].w & 0xFFFF0000u), b1[st].w, acc);
            }
        }
        me = bo;   // the bias, then orders 2..N in turn
        if (d.me_order >= 2) me += mw[0];
        if (d.me_order >= 3) me += mw[1];
        if (d.me_order >= 4) me += mw[2];
    }
    if (!hit) s = wave_sum(acc) + me;
    if (lane == 0) {
        const int st = hit ? RNNLM_Q_SCORE_HIT : (rec.flags & 3);
        f.scores[q] = s;
        if (f.q_status) f.q_status[q] = (uint8_t)st;
        atomicAdd(&s_cnt[st], 1);
        const bool cand = !hit && (rec.flags & QF_CAND);
        if (near_cap) {
            d.f_qcand[q] = cand ? 1 : 0;
        } else if (rec.flags & QF_CAND) {   // own staging slot: entry, or unused on a hit
            stage_score(d, rec.flags >> 6, cand ? rec.hs : -1, key.y, key.z, t, s);
            if (cand) atomicAdd(&s_cnt[3], 1);
        }
    }
}

template <int RS, int CS>
__device__ __forceinline__ void finish_history(const Dev &d, const FrameArgs &f, int i, int lane) {
    // one round of loads: status, slot after the frame, where h' lives, and
    // the key's codes (needed if the key enters the cache)
    const int st = d.f_hstat[i];
    const int slot = d.f_hslot[i];
    const float4 *src = reinterpret_cast<const float4 *>(d.f_hptr[i]);
    const bool enter = st == RNNLM_H_REP && slot >= 0;   // wave-uniform
    u64 code[CS];
    if (enter) {
#pragma unroll
        for (int c = 0; c < CS; ++c)
            if (lane + 64 * c < d.CW) code[c] = d.f_codes[(size_t)i * d.CW + lane + 64 * c];
    }
    // then the h' row, in flight while an admitted key enters the index
    float4 v[RS];
    if (f.hnew) {
#pragma unroll
        for (int k = 0; k < RS; ++k)
            if (lane + 64 * k < d.LH / 4) v[k] = ldg<float4>(src + lane + 64 * k);
    }
    if (enter) {
        u64 *dst = d.hc_codes + (size_t)slot * d.CW;
#pragma unroll
        for (int c = 0; c < CS; ++c)
            if (lane + 64 * c < d.CW) dst[lane + 64 * c] = code[c];
        if (lane == 0) {
            const HistRec hr = d.f_hrec[i];
            unsigned pos = (unsigned)(hr.hash & d.hi_mask);
            for (unsigned n = 0; n <= d.hi_mask; ++n) {
                HcIdx *r = d.hc_idx + pos;
                if (atomicCAS(&r->slot, -1, slot) == -1) {
                    r->hash = hr.hash;
                    r->word = hr.w1;
                    break;
                }
                pos = (pos + 1) & d.hi_mask;
            }
        }
    }
    if (f.hnew) {
        float4 *dst = reinterpret_cast<float4 *>(f.hnew + (size_t)i * d.LH);
#pragma unroll
        for (int k = 0; k < RS; ++k)
            if (lane + 64 * k < d.LH / 4) dst[lane + 64 * k] = v[k];
    }
}

// exclusive scan over a 256-thread block
__device__ int scan256(int v, int *s_tmp, int *total) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_tmp[wv] = x;
    __syncthreads();
    int base = 0;
    for (int k = 0; k < wv; ++k) base += s_tmp[k];
    *total = s_tmp[0] + s_tmp[1] + s_tmp[2] + s_tmp[3];
    __syncthreads();
    return base + x - v;
}

// ordered admission for a frame whose candidates could overflow the cache:
// ascending query index while the cache has room (run by the last block)
__device__ void admit_in_order(const Dev &d, const FrameArgs &f, int *s_tmp) {
    const long long size0 = d.ctr[C_SC_SIZE];
    int carry = 0, ins = 0, rej = 0;
    __shared__ int s_ins, s_rej;
    if (threadIdx.x == 0) s_ins = s_rej = 0;
    __syncthreads();
    for (int c0 = 0; c0 < f.n_query; c0 += 256) {
        const int q = c0 + threadIdx.x;
        const int cand = q < f.n_query ? d.f_qcand[q] : 0;
        int total;
        const int rank = scan256(cand, s_tmp, &total) + carry;
        if (cand) {
            if (size0 + rank < d.cap_query) {
                const QRec rec = d.f_qrec[q];
                const int4 key = d.f_qwords[q];
                stage_score(d, rank, rec.hs, key.y, key.z, key.w, f.scores[q]);
                ++ins;
            } else {
                ++rej;
            }
        }
        carry += total;
    }
    if (ins) atomicAdd(&s_ins, ins);
    if (rej) atomicAdd(&s_rej, rej);
    __syncthreads();
    if (threadIdx.x == 0) {   // the only writer of these counters in this frame
        d.ctr[C_SCORE_INS] += s_ins;
        d.ctr[C_SCORE_REJ] += s_rej;
        d.ctr[C_SC_SIZE] += s_ins;
        d.ctr[C_STAGED] = s_ins;   // admitted entries occupy staging slots 0 .. s_ins-1
    }
}

// Each frame of the launch owns a contiguous range of blocks: its query
// blocks, then its history blocks. MULTI = false: one frame, whose range is
// the whole grid (everything at fixed argument offsets).
template <bool BF16, bool MULTI, int RS, int CS>
__global__ __launch_bounds__(256) void k_score_finish(Dev d0, FrameBlock fb) {
    __shared__ int s_cnt[4];
    __shared__ int s_tmp[8];
    __shared__ int s_last;
    const int e = MULTI ? entry_of(fb.boff, fb.n, blockIdx.x) : 0;
    const int b = MULTI ? (int)blockIdx.x - fb.boff[e] : (int)blockIdx.x;   // block within the frame
    const int nblk = MULTI ? fb.boff[e + 1] - fb.boff[e] : (int)gridDim.x;
    const int qblocks = fb.qblk[e];
    const Dev d = MULTI ? session_view(d0, fb.sess[e]) : d0;
    const FrameArgs &f = fb.f[e];
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const bool near_cap = d.ctr[C_NEAR_CAP] != 0;
    if (tid < 4) s_cnt[tid] = 0;
    __syncthreads();
    if (b < qblocks) {
        const int q = b * 4 + w;
        if (q < f.n_query) score_query<BF16, RS>(d, f, q, lane, near_cap, s_cnt);
    } else {
        const int i = (b - qblocks) * 4 + w;
        if (i < f.n_hist) finish_history<RS, CS>(d, f, i, lane);
    }
    __syncthreads();
    if (tid == 0 && b < qblocks)   // folded into the counters by the next keys kernel
        d.f_part[b] = make_int4(s_cnt[RNNLM_Q_COMPUTED], s_cnt[RNNLM_Q_DUP], s_cnt[RNNLM_Q_SCORE_HIT], s_cnt[3]);
    if (!near_cap) return;   // uniform over the frame's blocks
    // the frame's last block to finish admits its candidates in order
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd((unsigned long long *)&d.ctr[C_DONE], 1ull) == (unsigned long long)(nblk - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    admit_in_order(d, f, s_tmp);
    if (tid == 0) d.ctr[C_DONE] = 0;
}

template <int RS, int CS>
static void launch_sf(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts) {
    const int nb = fb.boff[fb.n];
    const bool multi = fb.n > 1;
    if (d.wdtype == RNNLM_BF16) {
        if (multi) launch_k(k_score_finish<true, true, RS, CS>, nb, 256, s, ts, d, fb);
        else launch_k(k_score_finish<true, false, RS, CS>, nb, 256, s, ts, d, fb);
    } else {
        if (multi) launch_k(k_score_finish<false, true, RS, CS>, nb, 256, s, ts, d, fb);
        else launch_k(k_score_finish<false, false, RS, CS>, nb, 256, s, ts, d, fb);
    }
}

// Register arrays sized to the model: with rows of at most 1024 elements and
// keys of at most 256 code words a wave holds half the row registers and a
// quarter of the code registers of the longest case, and eight waves fit per
// SIMD instead of six or seven.
void launch_score_finish(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts) {
    const bool short_row = d.LH <= 1024, short_key = d.CW <= 256;
    if (short_row && short_key) launch_sf<4, 4>(d, fb, s, ts);
    else if (short_row) launch_sf<4, kCodeSteps>(d, fb, s, ts);
    else if (short_key) launch_sf<kRowSteps, 4>(d, fb, s, ts);
    else launch_sf<kRowSteps, kCodeSteps>(d, fb, s, ts);
}

}  // namespace rn
