// Frame planner: one 1024-thread block decides everything about a frame that
// needs the whole frame at once (Sec. 2.4 query de-duplication; Sec. 3 history
// de-duplication on quantised keys), using LDS hash tables:
//   histories: representative (lowest index with an equal key), status
//              (HC_HIT / H_REP / H_DUP), the GRU work list, and history-cache
//              admission in ascending index while below capacity;
//   queries:   representative, whether the key may enter the LM-query cache
//              (ranked in query order), and the scorer's record. The LM-query
//              cache itself is probed by the scorer.
// History keys meet in an LDS hash table on their 64-bit key hash, and a
// table match is confirmed by comparing codes, so a collision can only cost
// time. Equal query keys always share a history representative, so queries
// are bucketed by representative (an LDS counting sort) and compared exactly
// within their bucket: no hashing at all.
// Memory discipline: every input is loaded in one round of independent,
// coalesced loads; the middle of the kernel is LDS work (plus a load for each
// rare duplicate check); all results are stored at the end. This keeps the
// block to about one memory round trip.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

constexpr int PT = 1024;                           // threads
constexpr int HR = kPlanMaxHist / PT;              // histories per thread at most
constexpr int QR = kPlanMaxQuery / PT;             // queries per thread at most
constexpr int TAB_BYTES = 3 * kPlanMaxQuery * 4;    // 96 KB: history table, then query keys
static_assert(4 * kPlanMaxHist * 12 <= TAB_BYTES, "history table does not fit");

__device__ bool same_hist_key(const Dev &d, int a, int b) {
    if (d.f_words[a * 3] != d.f_words[b * 3]) return false;
    const u64 *ca = d.f_codes + (size_t)a * d.CW, *cb = d.f_codes + (size_t)b * d.CW;
    for (int w = 0; w < d.CW; ++w)
        if (ca[w] != cb[w]) return false;
    return true;
}

// exclusive scan of one int per thread across the block; *total = block sum
__device__ int block_scan(int v, int *s_tmp, int *total) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_tmp[wv] = x;
    __syncthreads();
    if (tid < 16) {
        int t = s_tmp[tid];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const int y = __shfl_up(t, o, 16);
            if (tid >= o) t += y;
        }
        s_tmp[16 + tid] = t;
    }
    __syncthreads();
    const int base = wv ? s_tmp[16 + wv - 1] : 0;
    *total = s_tmp[31];
    __syncthreads();
    return base + x - v;
}

// wave-aggregated increment of an LDS counter by the number of lanes with p
__device__ __forceinline__ void count_lanes(int *ctr, bool p) {
    const int k = __popcll(__ballot(p));
    if ((threadIdx.x & 63) == 0 && k) atomicAdd(ctr, k);
}

__global__ __launch_bounds__(PT) void k_frame_plan(Dev d, FrameArgs f, int npart) {
    __shared__ __align__(16) unsigned char s_tab[TAB_BYTES];
    __shared__ int s_rep[kPlanMaxHist];   // representative | status << 16
    __shared__ int s_hsa[kPlanMaxHist];   // cache slot after the frame (-1: not cached)
    __shared__ int s_loc[kPlanMaxHist];   // where h' lives: slot >= 0, or -(work row + 1)
    __shared__ int s_row[kPlanMaxHist];   // GRU work row of a new key (-1 otherwise)
    __shared__ int s_bcnt[kPlanMaxHist];  // queries per representative, then bucket offsets
    __shared__ unsigned short s_bq[kPlanMaxQuery];   // queries grouped by representative
    __shared__ long long c[C_N];          // the counters, read once and written back once
    __shared__ int s_tmp[32];
    __shared__ int s_cnt[8];

    const int tid = threadIdx.x, n = f.n_hist, nq = f.n_query;
    const int RQ = (nq + PT - 1) / PT;    // active query rounds (block-uniform)

    // ---------------- one round of independent loads ----------------
    long long ctr_v = 0;
    if (tid < C_N) ctr_v = d.ctr[tid];
    int4 part = make_int4(0, 0, 0, 0);
    for (int b = tid; b < npart; b += PT) {
        const int4 p = d.f_part[b];
        part.x += p.x; part.y += p.y; part.z += p.z; part.w += p.w;
    }
    u64 h_hash[HR];
    int h_slot[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = min(tid + r * PT, n - 1);   // clamped: no divergent loads
        h_hash[r] = d.f_hhash[i];
        h_slot[r] = d.f_hcslot[i];
    }
    int4 qk[QR];
    int qw1[QR];
    const int qlast = nq > 0 ? nq - 1 : 0;
#pragma unroll
    for (int r = 0; r < QR; ++r) {   // clamped, unconditional: idle rounds all read one element
        const int q = min(tid + r * PT, qlast);
        qk[r] = d.f_qkey[q];
        qw1[r] = d.f_qw1[q];
    }

    // counters and last frame's scoring counts
    if (tid < C_N) c[tid] = ctr_v;
    if (tid < 8) s_cnt[tid] = 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        part.x += __shfl_xor(part.x, o, 64);
        part.y += __shfl_xor(part.y, o, 64);
        part.z += __shfl_xor(part.z, o, 64);
        part.w += __shfl_xor(part.w, o, 64);
    }
    __syncthreads();
    if ((tid & 63) == 0 && npart) {
        atomicAdd(&s_cnt[4], part.x);
        atomicAdd(&s_cnt[5], part.y);
        atomicAdd(&s_cnt[6], part.z);
        atomicAdd(&s_cnt[7], part.w);
    }

    // ---------------- histories ----------------
    int HT = 64;
    while (HT < 4 * n) HT <<= 1;   // load <= 1/4: short probe chains
    u64 *hkey = reinterpret_cast<u64 *>(s_tab);
    int *hmin = reinterpret_cast<int *>(s_tab + HT * 8);
    for (int e = tid; e < HT; e += PT) {
        hkey[e] = 0ull;
        hmin[e] = 0x7FFFFFFF;
    }
    __syncthreads();
    if (tid == 0) {
        c[C_COMPUTED] += s_cnt[4];
        c[C_QUERY_DUPS] += s_cnt[5];
        c[C_SCORE_HITS] += s_cnt[6];
        c[C_SCORE_INS] += s_cnt[7];
        c[C_SC_SIZE] += s_cnt[7];
    }
    unsigned hpos[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        if (i < n) {
            const u64 h = h_hash[r];
            const u64 key = h ? h : 1ull;
            unsigned pos = (unsigned)(h & (HT - 1));
            for (int k = 0; k < HT; ++k) {
                const u64 old = atomicCAS(&hkey[pos], 0ull, key);
                if (old == 0ull || old == key) { atomicMin(&hmin[pos], i); break; }
                pos = (pos + 1) & (HT - 1);
            }
            hpos[r] = pos;
        }
    }
    __syncthreads();
    int h_rep[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        h_rep[r] = i;
        if (i < n) {
            const int m = hmin[hpos[r]];
            if (m != i) {
                if (same_hist_key(d, m, i)) h_rep[r] = m;
                else {   // two keys share a table key: find the first equal key
                    for (int j = 0; j < i; ++j)
                        if (d.f_hhash[j] == h_hash[r] && same_hist_key(d, j, i)) { h_rep[r] = j; break; }
                }
            }
        }
    }
    // statuses, GRU work rows, history-cache admission (ascending index)
    const long long hc_size = c[C_HC_SIZE];
    int carry = 0;
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        if (r * PT >= n) break;   // block-uniform
        const int i = tid + r * PT;
        const bool live = i < n;
        int st = RNNLM_H_DUP;
        if (live) st = h_slot[r] >= 0 ? RNNLM_HC_HIT : (h_rep[r] == i ? RNNLM_H_REP : RNNLM_H_DUP);
        int total;
        const int row = block_scan(live && st == RNNLM_H_REP ? 1 : 0, s_tmp, &total) + carry;
        const bool adm = live && st == RNNLM_H_REP && hc_size + row < d.cap_hist;
        if (live) {
            s_rep[i] = h_rep[r] | (st << 16);
            s_row[i] = st == RNNLM_H_REP ? row : -1;
            if (st == RNNLM_HC_HIT) {
                s_hsa[i] = h_slot[r];
                s_loc[i] = h_slot[r];
            } else if (st == RNNLM_H_REP) {
                s_hsa[i] = adm ? (int)(hc_size + row) : -1;
                s_loc[i] = adm ? (int)(hc_size + row) : -(row + 1);
            }
        }
        count_lanes(&s_cnt[0], live && st == RNNLM_HC_HIT);
        count_lanes(&s_cnt[1], live && st == RNNLM_H_DUP);
        count_lanes(&s_cnt[2], adm);
        count_lanes(&s_cnt[3], live && st == RNNLM_H_REP && !adm);
        carry += total;
    }
    __syncthreads();
    // duplicates share their representative's h' and cache slot
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        if (i < n && (s_rep[i] >> 16) == RNNLM_H_DUP) {
            s_hsa[i] = s_hsa[h_rep[r]];
            s_loc[i] = s_loc[h_rep[r]];
        }
    }
    if (tid == 0) {
        c[C_FRAME_M] = carry;
        c[C_HC_SIZE] = hc_size + s_cnt[2];
        c[C_FRAMES] += 1;
        c[C_HISTS] += n;
        c[C_HIST_HITS] += s_cnt[0];
        c[C_HIST_DUPS] += s_cnt[1];
        c[C_GRU_ROWS] += carry;
        c[C_HIST_INS] += s_cnt[2];
        c[C_HIST_REJ] += s_cnt[3];
        c[C_QUERIES] += nq;
        c[C_STAGED] = 0;   // the keys kernel has entered last frame's admitted scores
        c[C_NEAR_CAP] = 0;
    }

    // ---------------- queries ----------------
    if (RQ > 0) {
        int *s_qt = reinterpret_cast<int *>(s_tab);          // target
        int *s_qw2 = s_qt + kPlanMaxQuery;                    // key context words
        int *s_qw3 = s_qw2 + kPlanMaxQuery;
        for (int e = tid; e < n; e += PT) s_bcnt[e] = 0;
        __syncthreads();   // history table dead; duplicates' fix-up ordered
        // count the queries of each representative; the count's old value is
        // the query's place in its bucket
        int slot[QR];
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) {
                s_qt[q] = qk[r].w;
                s_qw2[q] = qk[r].y;
                s_qw3[q] = qk[r].z;
                slot[r] = atomicAdd(&s_bcnt[s_rep[qk[r].x] & 0xFFFF], 1);
            }
        }
        __syncthreads();
        // bucket offsets: exclusive scan of the counts in representative order
        int carry2 = 0;
        for (int c0 = 0; c0 < n; c0 += PT) {
            const int e = c0 + tid;
            const int v = e < n ? s_bcnt[e] : 0;
            int total;
            const int off = block_scan(v, s_tmp, &total) + carry2;
            if (e < n) s_bcnt[e] = off;
            carry2 += total;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) s_bq[s_bcnt[s_rep[qk[r].x] & 0xFFFF] + slot[r]] = (unsigned short)q;
        }
        __syncthreads();
        // one thread per bucket: representative = lowest query index with the
        // same (context, target) among the bucket's queries. The bucket's keys
        // are read once; each query's representative then replaces its target
        // in s_qt (only this thread touches the bucket's entries).
        constexpr int KB = 8;    // bucket entries held in registers
        for (int hr = tid; hr < n; hr += PT) {
            const int b0 = s_bcnt[hr], b1 = hr + 1 < n ? s_bcnt[hr + 1] : nq;
            const int k = b1 - b0;
            if (k == 0) continue;
            if (k <= KB) {
                int bq[KB], bt[KB], b2[KB], b3[KB];
#pragma unroll
                for (int j = 0; j < KB; ++j) {
                    if (j < k) {
                        bq[j] = s_bq[b0 + j];
                        bt[j] = s_qt[bq[j]];
                        b2[j] = s_qw2[bq[j]];
                        b3[j] = s_qw3[bq[j]];
                    }
                }
#pragma unroll
                for (int j = 0; j < KB; ++j) {
                    if (j < k) {
                        int rep = bq[j];
#pragma unroll
                        for (int l = 0; l < KB; ++l)
                            if (l < k && bq[l] < rep && bt[l] == bt[j] && b2[l] == b2[j] && b3[l] == b3[j]) rep = bq[l];
                        s_qt[bq[j]] = rep;   // own entries only; keys were read above
                    }
                }
            } else {   // a large bucket, in LDS: sort it by query index, then resolve
                       // from the back, so each write lands on an entry no later
                       // comparison reads
                for (int j = 1; j < k; ++j) {
                    const unsigned short v = s_bq[b0 + j];
                    int l = j - 1;
                    while (l >= 0 && s_bq[b0 + l] > v) {
                        s_bq[b0 + l + 1] = s_bq[b0 + l];
                        --l;
                    }
                    s_bq[b0 + l + 1] = v;
                }
                for (int j = k - 1; j >= 0; --j) {
                    const int qj = s_bq[b0 + j];
                    int rep = qj;
                    for (int l = 0; l < j; ++l) {
                        const int ql = s_bq[b0 + l];
                        if (s_qt[ql] == s_qt[qj] && s_qw2[ql] == s_qw2[qj] && s_qw3[ql] == s_qw3[qj]) { rep = ql; break; }
                    }
                    s_qt[qj] = rep;
                }
            }
        }
        __syncthreads();
        const long long sc_size = c[C_SC_SIZE];
        int qcarry = 0;
        int qrep[QR];
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            if (r >= RQ) break;   // block-uniform
            const int q = tid + r * PT;
            int rep = q;
            bool cand = false;
            if (q < nq) {
                rep = s_qt[q];
                cand = rep == q && s_hsa[qk[r].x] >= 0;   // may enter the LM-query cache
            }
            int total;
            const int rank = block_scan(cand ? 1 : 0, s_tmp, &total) + qcarry;
            qrep[r] = rep | (cand ? (rank << 16) : (int)0x80000000);   // rep, rank < 2^15
            qcarry += total;
        }
        // scorer records
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) {
                const int i = qk[r].x;
                const int rep = qrep[r] & 0xFFFF;
                const bool cand = qrep[r] >= 0;
                const int loc = s_loc[i];
                const float *base = loc >= 0 ? d.hc_val + (size_t)loc * d.LH : d.f_hval + (size_t)(-loc - 1) * d.LH;
                QRec rec;
                rec.hptr = (u64)(base + (size_t)(d.L - 1) * d.H);
                rec.t = qk[r].w;
                rec.flags = (rep < q ? RNNLM_Q_DUP : RNNLM_Q_COMPUTED) | (cand ? QF_CAND : 0) |
                            ((s_rep[i] >> 16) == RNNLM_HC_HIT ? QF_PROBE : 0) | (cand ? (qrep[r] >> 16) << 6 : 0);
                rec.hs = s_hsa[i];
                rec.w1 = qw1[r];
                rec.w2 = qk[r].y;
                rec.w3 = qk[r].z;
                d.f_qrec[q] = rec;
                if (f.q_rep) f.q_rep[q] = rep;
            }
        }
        if (tid == 0) {
            // admission is order-independent unless the candidates could overflow the cache
            const bool near = sc_size + qcarry > d.cap_query;
            c[C_NEAR_CAP] = near ? 1 : 0;
            c[C_STAGED] = near ? 0 : qcarry;   // staging slots the scorer fills
        }
    }

    // ---------------- per-history results ----------------
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        if (i < n) {
            const int st = s_rep[i] >> 16;
            const int loc = s_loc[i];
            const float *hp = loc >= 0 ? d.hc_val + (size_t)loc * d.LH : d.f_hval + (size_t)(-loc - 1) * d.LH;
            d.f_hstat[i] = st;
            d.f_hslot[i] = s_hsa[i];
            d.f_hptr[i] = (u64)hp;
            if (st == RNNLM_H_REP) {
                const int row = s_row[i];
                d.f_rows[row] = i;
                d.f_rowdst[row] = (u64)hp;
            }
            if (f.h_status) f.h_status[i] = (uint8_t)st;
            if (f.h_rep) f.h_rep[i] = h_rep[r];
        }
    }
    __syncthreads();
    if (tid < C_N) d.ctr[tid] = c[tid];
}

void launch_frame_plan(const Dev &d, const FrameArgs &f, int npart, hipStream_t s) {
    k_frame_plan<<<1, PT, 0, s>>>(d, f, npart);
}

}  // namespace rn
