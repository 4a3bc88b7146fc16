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
// time. Query keys meet in a second table on a 32-bit fingerprint, again
// confirmed by an exact key comparison.
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
constexpr int TAB_BYTES = 124 * 1024;              // both hash tables
constexpr int HW = kPlanMaxHist / 64;              // history flag words
constexpr int QW = kPlanMaxQuery / 64;             // query flag words
// worst case: history table at load 1/2 and the query table at load <= 8/9
static_assert(2 * kPlanMaxHist * 12 + (kPlanMaxQuery + kPlanMaxQuery / 8) * 8 <= TAB_BYTES,
              "hash tables do not fit");
static_assert(QW <= 128, "flag prefix covers two words per lane");

__device__ bool same_hist_key(const Dev &d, int a, int b) {
    if (d.f_words[a * 3] != d.f_words[b * 3]) return false;
    const u64 *ca = d.f_codes + (size_t)a * d.CW, *cb = d.f_codes + (size_t)b * d.CW;
    for (int w = 0; w < d.CW; ++w)
        if (ca[w] != cb[w]) return false;
    return true;
}

// wave-aggregated increment of an LDS counter by the number of lanes with p
__device__ __forceinline__ void count_lanes(int *ctr, bool p) {
    const int k = __popcll(__ballot(p));
    if ((threadIdx.x & 63) == 0 && k) atomicAdd(ctr, k);
}

// Ranks from flag words: element e (e = r * PT + 64 * wave + lane) sets bit
// lane of word e / 64 with a wave ballot; one wave then turns the words' bit
// counts into an exclusive prefix (two words per lane), so the rank of e is
// pre[e / 64] + the set bits below it in its word. Returns the total (in
// every lane of the calling wave).
__device__ int flag_prefix(const u64 *words, int *pre, int nw) {
    const int lane = threadIdx.x & 63;
    const int w0 = 2 * lane, w1 = w0 + 1;
    const int c0 = w0 < nw ? __popcll(words[w0]) : 0, c1 = w1 < nw ? __popcll(words[w1]) : 0;
    int x = c0 + c1;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    const int ex = x - c0 - c1;
    if (w0 < nw) pre[w0] = ex;
    if (w1 < nw) pre[w1] = ex + c0;
    return __shfl(x, 63, 64);
}

__device__ __forceinline__ int flag_rank(const u64 *words, const int *pre, int e) {
    const int lane = e & 63;
    return pre[e >> 6] + __popcll(words[e >> 6] & ((1ull << lane) - 1ull));
}

// In-frame placement hash of a query key (history representative, context
// words, target): the key is folded into 64 bits (injective on realistic
// ranges, and any collision is caught by the exact check) and mixed once.
__device__ __forceinline__ u64 frame_query_hash(int rep, int w2, int w3, int t) {
    const u64 x = (((u64)(uint32_t)(t + 1) << 32) | (uint32_t)(w2 + 2)) + (u64)(uint32_t)(w3 + 2) * kPhi +
                  (u64)(uint32_t)rep * 0xD6E8FEB86659FD93ull;
    return mix64(x);
}

// block e plans entry e of the frame block (its session's frame); MULTI =
// false: one frame, at fixed argument offsets
template <bool MULTI>
__global__ __launch_bounds__(PT) void k_frame_plan(Dev d0, FrameBlock fb) {
    const int e = MULTI ? (int)blockIdx.x : 0;
    const Dev d = MULTI ? session_view(d0, fb.sess[e]) : d0;
    const FrameArgs &f = fb.f[e];
    __shared__ __align__(16) unsigned char s_tab[TAB_BYTES];
    __shared__ int s_rep[kPlanMaxHist];   // representative | status << 16
    __shared__ int s_hsa[kPlanMaxHist];   // cache slot after the frame (-1: not cached)
    __shared__ int s_loc[kPlanMaxHist];   // where h' lives: slot >= 0, or -(work row + 1)
    __shared__ int s_row[kPlanMaxHist];   // GRU work row of a new key (-1 otherwise)
    __shared__ u64 s_hflag[HW], s_qflag[QW];
    __shared__ int s_hpre[HW], s_qpre[QW];
    __shared__ long long c[C_N];          // the counters, read once and written back once
    __shared__ int s_cnt[4];
    __shared__ int s_tot;

    const int tid = threadIdx.x, n = f.n_hist, nq = f.n_query;
    const int RQ = (nq + PT - 1) / PT;    // active query rounds (block-uniform)

    // ---------------- one round of independent loads ----------------
    long long ctr_v = 0;
    if (tid < C_N) ctr_v = d.ctr[tid];
    u64 h_hash[HR];
    const float *h_src[HR];   // each history's vector (its row, or its handle)
    int h_slot[HR], h_w1[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = min(tid + r * PT, n - 1);   // clamped: no divergent loads
        h_hash[r] = d.f_hhash[i];
        h_slot[r] = d.f_hcslot[i];
        h_w1[r] = d.f_words[i * 3];
        bool unused = false;   // the keys kernel reports bad handles
        h_src[r] = hist_row(d, f, i, unused);
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

    // ---------------- both tables cleared while the loads are in flight ----
    // history table: 64-bit key hash + lowest index per slot (load <= 1/4 when
    // both tables fit that way, else 1/2); query table: 32-bit fingerprint +
    // lowest index per slot, in the rest
    int HT = 64;
    while (HT < 4 * n) HT <<= 1;
    if (HT * 12 + 12 * nq > TAB_BYTES) HT >>= 1;
    const int TQ = min((TAB_BYTES - HT * 12) / 8, max(64, 4 * nq));
    u64 *hkey = reinterpret_cast<u64 *>(s_tab);
    int *hmin = reinterpret_cast<int *>(s_tab + HT * 8);
    unsigned *qfp = reinterpret_cast<unsigned *>(s_tab + HT * 12);
    int *qmin = reinterpret_cast<int *>(s_tab + HT * 12 + TQ * 4);
    for (int e = tid; e < HT; e += PT) {
        hkey[e] = 0ull;
        hmin[e] = 0x7FFFFFFF;
    }
    if (RQ > 0) {
        for (int e = tid; e < TQ; e += PT) {
            qfp[e] = 0u;
            qmin[e] = 0x7FFFFFFF;
        }
    }
    if (tid < C_N) c[tid] = ctr_v;   // the previous frame's scoring counts are already folded in
    if (tid < 4) s_cnt[tid] = 0;
    __syncthreads();

    // ---------------- histories ----------------
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
    // statuses; the GRU work row of a new key is its rank among the frame's
    // new keys (ascending index), and keys enter the history cache in that
    // order while it has room
    int h_st[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        if (r * PT >= n) break;   // block-uniform
        const int i = tid + r * PT;
        const bool live = i < n;
        h_st[r] = !live ? RNNLM_H_DUP : h_slot[r] >= 0 ? RNNLM_HC_HIT : (h_rep[r] == i ? RNNLM_H_REP : RNNLM_H_DUP);
        const u64 b = __ballot(live && h_st[r] == RNNLM_H_REP);
        if ((tid & 63) == 0) s_hflag[i >> 6] = b;
    }
    __syncthreads();
    if (tid < 64) {
        const int tot = flag_prefix(s_hflag, s_hpre, (n + 63) >> 6);
        if (tid == 0) s_tot = tot;
    }
    __syncthreads();
    const long long hc_size = c[C_HC_SIZE];
    const int M = s_tot;
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        if (r * PT >= n) break;   // block-uniform
        const int i = tid + r * PT;
        const bool live = i < n;
        const int st = h_st[r];
        const int row = live && st == RNNLM_H_REP ? flag_rank(s_hflag, s_hpre, i) : -1;
        const bool adm = row >= 0 && hc_size + row < d.cap_hist;
        if (live) {
            s_rep[i] = h_rep[r] | (st << 16);
            s_row[i] = row;
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
    }
    __syncthreads();
    // duplicates share their representative's h' and cache slot
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        if (i < n && h_st[r] == RNNLM_H_DUP) {
            s_hsa[i] = s_hsa[h_rep[r]];
            s_loc[i] = s_loc[h_rep[r]];
        }
    }
    if (tid == 0) {
        const long long room = d.cap_hist > hc_size ? d.cap_hist - hc_size : 0;
        const int ins = (int)(M < room ? M : room);
        c[C_FRAME_M] = M;
        c[C_HC_SIZE] = hc_size + ins;
        c[C_FRAMES] += 1;
        c[C_HISTS] += n;
        c[C_HIST_HITS] += s_cnt[0];
        c[C_HIST_DUPS] += s_cnt[1];
        c[C_GRU_ROWS] += M;
        c[C_HIST_INS] += ins;
        c[C_HIST_REJ] += M - ins;
        c[C_QUERIES] += nq;
        c[C_STAGED] = 0;   // the keys kernel has entered last frame's admitted scores
        c[C_NEAR_CAP] = 0;
    }

    // ---------------- queries ----------------
    // Query keys meet on a 32-bit fingerprint; each slot keeps the lowest
    // query index that reached it, and a match is confirmed against that
    // query's exact key (on a fingerprint collision the query scans the
    // earlier queries itself, which stays exact).
    if (RQ > 0) {
        int qrh[QR];          // the query's history representative
        unsigned qpos[QR];
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) {
                qrh[r] = s_rep[qk[r].x] & 0xFFFF;
                const u64 h = frame_query_hash(qrh[r], qk[r].y, qk[r].z, qk[r].w);
                const unsigned fp = (unsigned)(h >> 32) | 1u;
                unsigned pos = (unsigned)(((h & 0xFFFFFFFFull) * (u64)TQ) >> 32);
                for (int k = 0; k < TQ; ++k) {
                    const unsigned old = atomicCAS(&qfp[pos], 0u, fp);
                    if (old == 0u || old == fp) { atomicMin(&qmin[pos], q); break; }
                    if (++pos == (unsigned)TQ) pos = 0;
                }
                qpos[r] = pos;
            }
        }
        __syncthreads();   // also orders the duplicates' fix-up
        int qrepv[QR];
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            qrepv[r] = q;
            if (r < RQ && q < nq) {
                const int m = qmin[qpos[r]];
                if (m != q) {
                    const int4 km = d.f_qkey[m];
                    if ((s_rep[km.x] & 0xFFFF) == qrh[r] && km.y == qk[r].y && km.z == qk[r].z && km.w == qk[r].w) {
                        qrepv[r] = m;
                    } else {
                        for (int j = 0; j < q; ++j) {
                            const int4 kj = d.f_qkey[j];
                            if ((s_rep[kj.x] & 0xFFFF) == qrh[r] && kj.y == qk[r].y && kj.z == qk[r].z &&
                                kj.w == qk[r].w) {
                                qrepv[r] = j;
                                break;
                            }
                        }
                    }
                }
            }
        }
        // a new key whose history is (or will be) cached may enter the
        // LM-query cache; candidates are ranked in query order
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            if (r >= RQ) break;   // block-uniform
            const int q = tid + r * PT;
            const bool cand = q < nq && qrepv[r] == q && s_hsa[qk[r].x] >= 0;
            const u64 b = __ballot(cand);
            if ((tid & 63) == 0) s_qflag[q >> 6] = b;
        }
        __syncthreads();
        if (tid < 64) {
            const int tot = flag_prefix(s_qflag, s_qpre, (nq + 63) >> 6);
            if (tid == 0) s_tot = tot;
        }
        __syncthreads();
        const int ncand = s_tot;
        const long long sc_size = c[C_SC_SIZE];
        // scorer records
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) {
                const int i = qk[r].x;
                const int rep = qrepv[r];
                const bool cand = (s_qflag[q >> 6] >> (q & 63)) & 1ull;
                const int rank = cand ? flag_rank(s_qflag, s_qpre, q) : 0;
                const int loc = s_loc[i];
                const float *base = loc >= 0 ? d.hc_val + (size_t)loc * d.LH : d.f_hval + (size_t)(-loc - 1) * d.LH;
                QRec rec;
                rec.hptr = (u64)(base + (size_t)(d.L - 1) * d.H);
                rec.t = qk[r].w;
                rec.flags = (rep < q ? RNNLM_Q_DUP : RNNLM_Q_COMPUTED) | (cand ? QF_CAND : 0) |
                            ((s_rep[i] >> 16) == RNNLM_HC_HIT ? QF_PROBE : 0) | (cand ? rank << 6 : 0);
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
            const bool near = sc_size + ncand > d.cap_query;
            c[C_NEAR_CAP] = near ? 1 : 0;
            c[C_STAGED] = near ? 0 : ncand;   // staging slots the scorer fills
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
                d.f_roww[row] = h_w1[r];
                d.f_rowh[row] = (u64)h_src[r];
                d.f_rowdst[row] = (u64)hp;
            }
            if (f.h_status) f.h_status[i] = (uint8_t)st;
            if (f.h_rep) f.h_rep[i] = h_rep[r];
        }
    }
    __syncthreads();
    if (tid < C_N) d.ctr[tid] = c[tid];
}

void launch_frame_plan(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts) {
    if (fb.n > 1) launch_k(k_frame_plan<true>, fb.n, PT, s, ts, d, fb);
    else launch_k(k_frame_plan<false>, 1, PT, s, ts, d, fb);
}

}  // namespace rn
