// Frame planner: one 1024-thread block decides everything about a frame that
// needs the whole frame at once (Sec. 2.4 query de-duplication; Sec. 3 history
// de-duplication on quantised keys), using LDS hash tables:
//   histories: representative (lowest index with an equal key), status
//              (HC_HIT / H_REP / H_DUP), the GRU work list, and history-cache
//              admission in ascending index while below capacity;
//   queries:   representative, whether the key may enter the LM-query cache
//              (ranked in query order), and the scorer's record. The LM-query
//              cache itself is probed by the scorer.
// Equal keys are found by a slot race rather than by probing: every key
// lowers its slot of a table to (fingerprint, index) with one atomic min;
// after a barrier it reads the slot back. The smallest fingerprint at a slot
// keeps it, with its lowest index; the other keys at that slot race again in
// a smaller table at a position drawn from their fingerprint; the few left
// after the last table settle in a small probed table, and any left over
// from that resolve by an exact scan. Every round is
// branch-free and ends with one barrier, so the cost is a few short LDS
// rounds instead of probe chains of dependent atomics. A settled key's
// representative is confirmed by an exact key comparison, so a fingerprint
// collision can only cost time.
// Queries are placed on their history's key hash rather than on its
// representative, so both tables fill in the same rounds; the exact check
// then compares representatives.
// Memory discipline: every input is loaded in one round of independent,
// coalesced loads, and the query keys are kept in LDS when they fit; the
// middle of the kernel is LDS work (plus loads for the rare key comparisons
// of duplicate histories). Per-history results are stored as soon as they
// are final, so they drain while the queries are planned.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace rn {

constexpr int PT = 1024;                           // threads
constexpr int HR_MAX = kPlanMaxHist / PT;          // histories per thread at most
constexpr int QR_MAX = kPlanMaxQuery / PT;         // queries per thread at most
constexpr int TAB_BYTES = 124 * 1024;              // race tables and staged query keys
constexpr int HW = kPlanMaxHist / 64;              // history flag words
constexpr int QW = kPlanMaxQuery / 64;             // query flag words
constexpr int KR = 4;                              // race rounds (tables per kind)
constexpr int HIB = 11, QIB = 13;                  // index bits in a history / query slot
constexpr int OVF = 128;                           // overflow table slots per kind
static_assert(kPlanMaxHist <= (1 << HIB) && kPlanMaxQuery <= (1 << QIB), "slot index fields too narrow");
static_assert(QW <= 128, "flag prefix covers two words per lane");
static_assert(kPlanMaxHist <= 65536, "representatives are packed in 16 bits");

// Slots of the race tables of one kind: table k has max(64, S0 / 4^k) slots.
__host__ __device__ constexpr int race_slots(int s0) {
    int t = 0;
    for (int k = 0; k < KR; ++k) t += (s0 >> (2 * k)) > 64 ? (s0 >> (2 * k)) : 64;
    return t;
}
__host__ __device__ constexpr int pow2_at_least(int x) {
    int p = 64;
    while (p < x) p <<= 1;
    return p;
}
// worst case: both first tables at load <= 1/2, query keys not staged
static_assert(4 * (race_slots(pow2_at_least(2 * kPlanMaxHist)) + race_slots(pow2_at_least(2 * kPlanMaxQuery))) <=
                  TAB_BYTES,
              "race tables do not fit");

// odd multipliers that place a key hash's low word in the tables after the first
__device__ __forceinline__ unsigned race_mult(int k) {
    return k == 1 ? 0x9E3779B1u : k == 2 ? 0x85EBCA77u : 0xC2B2AE3Du;
}

// Race tables of one kind: slot offset and position shift of each table.
struct Race {
    int off[KR], sh[KR];
};
__device__ __forceinline__ Race race_layout(int s0, int &base) {
    Race R;
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int sz = max(64, s0 >> (2 * k));
        R.off[k] = base;
        R.sh[k] = __clz(sz) + 1;   // 32 - log2(sz)
        base += sz;
    }
    return R;
}

__device__ bool same_hist_key(const Dev &d, int a, int b) {
    if (d.f_hrec[a].w1 != d.f_hrec[b].w1) return false;
    const u64 *ca = d.f_codes + (size_t)a * d.CW, *cb = d.f_codes + (size_t)b * d.CW;
    for (int w = 0; w < d.CW; w += 4) {   // four independent loads per side per step
        u64 x = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int j = min(w + k, d.CW - 1);
            x |= ca[j] ^ cb[j];
        }
        if (x) return false;
    }
    return true;
}

// wave-aggregated increment of an LDS counter by the number of lanes with p
__device__ __forceinline__ void count_lanes(int *ctr, bool p) {
    const int k = __popcll(__ballot(p));
    if ((threadIdx.x & 63) == 0 && k) atomicAdd(ctr, k);
}

// Inclusive sum over the 64 lanes of a wave (all lanes active), with DPP
// moves: shifts by 1, 2, 4 and 8 within each row of 16 lanes, then the last
// lane of row 0 is added to row 1 and row 3 gets row 2's, then lane 31 (rows 0
// and 1 in full) is added to rows 2 and 3.
__device__ __forceinline__ int wave_incl_sum(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);    // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);    // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);    // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);    // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);   // row_bcast:15 into rows 1, 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);   // row_bcast:31 into rows 2, 3
    return x;
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
    const int x = wave_incl_sum(c0 + c1);
    const int ex = x - c0 - c1;
    if (w0 < nw) pre[w0] = ex;
    if (w1 < nw) pre[w1] = ex + c0;
    return __builtin_amdgcn_readlane(x, 63);
}

__device__ __forceinline__ int flag_rank(const u64 *words, const int *pre, int e) {
    const int lane = e & 63;
    return pre[e >> 6] + __popcll(words[e >> 6] & ((1ull << lane) - 1ull));
}

// Insert value v (fingerprint above `ib` index bits) of a key whose hash has
// low word lo into an overflow table of OVF slots (empty: all ones): a slot
// holding the same fingerprint keeps the lower index. Returns the slot, or
// OVF when the table is full.
__device__ __forceinline__ unsigned overflow_insert(uint32_t *t, uint32_t lo, uint32_t v, int ib) {
    unsigned pos = lo & (OVF - 1);
    for (int k = 0; k < OVF; ++k) {
        const uint32_t old = atomicCAS(&t[pos], 0xFFFFFFFFu, v);
        if (old == 0xFFFFFFFFu) return pos;
        if ((old >> ib) == (v >> ib)) {
            atomicMin(&t[pos], v);
            return pos;
        }
        pos = (pos + 1) & (OVF - 1);
    }
    return OVF;
}

// In-frame placement hash of a query key: its history's key hash (folded to
// 32 bits), context words and target, mixed once. Equal keys hash equally;
// the exact check catches every collision.
__device__ __forceinline__ u64 frame_query_hash(unsigned hh, int w2, int w3, int t) {
    const u64 x = (((u64)hh << 32) | (uint32_t)(t + 1)) + (u64)(uint32_t)(w2 + 2) * kPhi +
                  (u64)(uint32_t)(w3 + 2) * 0xD6E8FEB86659FD93ull;
    return mix64(x);
}

// block e plans entry e of the frame block (its session's frame); MULTI =
// false: one frame, at fixed argument offsets. HR, QR: histories and queries
// per thread, sized by the host to the block's largest frame, so that no
// thread loads, keeps or steps over rounds no frame of the launch has (a
// Large frame of 2048 queries needs 2 of the 8 query rounds; 15-20% less
// planner time than always sizing for the maxima).
template <bool MULTI, int HR, int QR>
__global__ __launch_bounds__(PT) void k_frame_plan(Dev d0, FrameBlock fb) {
    const int e = MULTI ? (int)blockIdx.x : 0;
    const Dev d = MULTI ? session_view(d0, fb.sess[e]) : d0;
    const FrameArgs &f = fb.f[e];
    __shared__ __align__(16) unsigned char s_tab[TAB_BYTES];
    __shared__ unsigned s_hh[kPlanMaxHist];  // folded key hash of each history
    __shared__ int s_rep[kPlanMaxHist];      // representative | status << 16
    __shared__ int s_hsa[kPlanMaxHist];      // cache slot after the frame (-1: not cached)
    __shared__ int s_loc[kPlanMaxHist];      // where h' lives: slot >= 0, or -(work row + 1)
    __shared__ u64 s_hflag[HW], s_qflag[QW];
    __shared__ int s_hpre[HW], s_qpre[QW];
    __shared__ long long c[C_N];             // the counters, read once and written back once
    __shared__ int s_cnt[2];
    __shared__ int s_htot, s_qtot;
    __shared__ int s_more[3];          // race rounds: some key lost in round k (k mod 3)
    __shared__ uint32_t s_ovf[2 * OVF];  // keys still racing after the last table: histories, then queries

    const int tid = threadIdx.x, lane = tid & 63, n = f.n_hist, nq = f.n_query;
    const int RQ = (nq + PT - 1) / PT;    // active query rounds (block-uniform)

    // ---------------- one round of independent loads ----------------
    // clamped, unconditional loads: no branch between the argument loads and
    // these, and idle elements all read one in-bounds element
    const long long ctr_v = ldg<long long>(d.ctr + min(tid, C_N - 1));
    const int hlast = n > 0 ? n - 1 : 0;
    u64 h_hash[HR], h_hp[HR];
    int h_slot[HR], h_w1[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = min(tid + r * PT, hlast);
        const HistRec hr = d.f_hrec[i];   // one 16-byte load per history
        h_hash[r] = hr.hash;
        h_slot[r] = hr.slot;
        h_w1[r] = hr.w1;
    }
    int4 qk[QR];
    const int qlast = nq > 0 ? nq - 1 : 0;
#pragma unroll
    for (int r = 0; r < QR; ++r) {
        const int q = min(tid + r * PT, qlast);
        qk[r] = d.f_qkey[q];
    }
#pragma unroll
    for (int r = 0; r < HR; ++r)   // handles are checked where they are used
        h_hp[r] = f.hist_ptr ? f.hist_ptr[min(tid + r * PT, hlast)] : 0;

    // ---------------- race tables (block-uniform sizes) ----------------
    // first tables at load <= 1/4, else the query one, then the history one,
    // at load <= 1/2; query keys are staged in LDS when they still fit
    int S0 = pow2_at_least(4 * n), Q0 = pow2_at_least(4 * nq);
    if (4 * (race_slots(S0) + race_slots(Q0)) > TAB_BYTES) Q0 >>= 1;
    if (4 * (race_slots(S0) + race_slots(Q0)) > TAB_BYTES) S0 >>= 1;
    const bool stage = 16 * nq + 4 * (race_slots(S0) + race_slots(Q0)) <= TAB_BYTES;
    const int qk_bytes = stage ? 16 * nq : 0;
    int4 *s_qk = reinterpret_cast<int4 *>(s_tab);
    uint32_t *tab = reinterpret_cast<uint32_t *>(s_tab + qk_bytes);
    int tab_slots = 0;
    const Race HRc = race_layout(S0, tab_slots);
    const Race QRc = race_layout(RQ > 0 ? Q0 : 0, tab_slots);
    if (tid < 2 * OVF) s_ovf[tid] = 0xFFFFFFFFu;
    for (int k = tid; k < tab_slots / 4; k += PT)   // slot counts are multiples of 64
        reinterpret_cast<uint4 *>(tab)[k] = make_uint4(0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu);
    if (tid < 2) s_cnt[tid] = 0;
    if (tid == 0) s_more[0] = 0;
    // the loads have landed: keep what other threads read
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        if (i < n) s_hh[i] = (unsigned)(h_hash[r] ^ (h_hash[r] >> 32));
    }
    if (stage) {
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            const int q = tid + r * PT;
            if (r < RQ && q < nq) s_qk[q] = qk[r];
        }
    }
    if (tid < C_N) c[tid] = ctr_v;   // the previous frame's scoring counts are already folded in
    __syncthreads();

    // ---------------- both races ----------------
    // slot value: fingerprint bits (the key hash's high word) above the
    // index, so a smaller value wins; every table is addressed by the hash's
    // low word (table k through its own multiplier), so equal keys always
    // move together while keys that share a fingerprint part at each table
    uint32_t hv[HR], hlo[HR], hpos[HR], qv[QR], qlo[QR], qpos[QR];
    unsigned hpend = 0, qpend = 0;   // bit r: element of round r still racing
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        const int i = tid + r * PT;
        hv[r] = ((uint32_t)(h_hash[r] >> 32) & ~((1u << HIB) - 1)) | (uint32_t)i;
        hlo[r] = (uint32_t)h_hash[r];
        hpos[r] = hlo[r] >> HRc.sh[0];
        if (i < n) {
            atomicMin(&tab[HRc.off[0] + hpos[r]], hv[r]);
            hpend |= 1u << r;
        }
    }
#pragma unroll
    for (int r = 0; r < QR; ++r) {
        const int q = tid + r * PT;
        qv[r] = 0;
        qlo[r] = 0;
        qpos[r] = 0;
        if (r < RQ) {
            const u64 h = frame_query_hash(s_hh[qk[r].x], qk[r].y, qk[r].z, qk[r].w);
            qv[r] = ((uint32_t)(h >> 32) & ~((1u << QIB) - 1)) | (uint32_t)q;
            qlo[r] = (uint32_t)h;
            qpos[r] = qlo[r] >> QRc.sh[0];
            if (q < nq) {
                atomicMin(&tab[QRc.off[0] + qpos[r]], qv[r]);
                qpend |= 1u << r;
            }
        }
    }
    __syncthreads();
    int hmin[HR], qmin[QR];
#pragma unroll
    for (int r = 0; r < HR; ++r) hmin[r] = tid + r * PT;
#pragma unroll
    for (int r = 0; r < QR; ++r) qmin[r] = tid + r * PT;
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const bool more = k + 1 < KR;
        bool lost = false;
#pragma unroll
        for (int r = 0; r < HR; ++r) {
            if (r * PT >= n) break;   // block-uniform
            const uint32_t got = tab[HRc.off[k] + hpos[r]];
            const bool pend = (hpend >> r) & 1u;
            const bool win = pend && (got >> HIB) == (hv[r] >> HIB);
            hmin[r] = win ? (int)(got & ((1u << HIB) - 1)) : hmin[r];
            const bool lose = pend && !win;
            if (win) hpend &= ~(1u << r);
            if (more) {
                hpos[r] = (hlo[r] * race_mult(k + 1)) >> HRc.sh[more ? k + 1 : k];
                if (lose) atomicMin(&tab[HRc.off[more ? k + 1 : k] + hpos[r]], hv[r]);
            }
            lost |= lose;
        }
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            if (r >= RQ) break;   // block-uniform
            const uint32_t got = tab[QRc.off[k] + qpos[r]];
            const bool pend = (qpend >> r) & 1u;
            const bool win = pend && (got >> QIB) == (qv[r] >> QIB);
            qmin[r] = win ? (int)(got & ((1u << QIB) - 1)) : qmin[r];
            const bool lose = pend && !win;
            if (win) qpend &= ~(1u << r);
            if (more) {
                qpos[r] = (qlo[r] * race_mult(k + 1)) >> QRc.sh[more ? k + 1 : k];
                if (lose) atomicMin(&tab[QRc.off[more ? k + 1 : k] + qpos[r]], qv[r]);
            }
            lost |= lose;
        }
        if (__any(lost) && (tid & 63) == 0) s_more[k % 3] = 1;
        if (tid == 0) s_more[(k + 1) % 3] = 0;
        __syncthreads();
        if (!s_more[k % 3]) break;   // block-uniform: nobody lost
        if (more) continue;
        // Keys still racing after the last table (rare): open addressing in
        // a small table of their own (compare-and-swap probing; few keys,
        // short chains), where a fingerprint again keeps its lowest index.
        // A key that finds no slot stays racing and takes the exact scan.
        unsigned hop[HR], qop[QR];
#pragma unroll
        for (int r = 0; r < HR; ++r) {
            hop[r] = OVF;
            if ((hpend >> r) & 1u) hop[r] = overflow_insert(s_ovf, hlo[r], hv[r], HIB);
        }
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            qop[r] = OVF;
            if (r < RQ && ((qpend >> r) & 1u)) qop[r] = overflow_insert(s_ovf + OVF, qlo[r], qv[r], QIB);
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < HR; ++r)
            if (hop[r] < OVF) {
                hmin[r] = (int)(s_ovf[hop[r]] & ((1u << HIB) - 1));
                hpend &= ~(1u << r);
            }
#pragma unroll
        for (int r = 0; r < QR; ++r)
            if (qop[r] < OVF) {
                qmin[r] = (int)(s_ovf[OVF + qop[r]] & ((1u << QIB) - 1));
                qpend &= ~(1u << r);
            }
    }

    // ---------------- history representatives and statuses ----------------
    int h_rep[HR], h_st[HR];
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        if (r * PT >= n) break;   // block-uniform
        const int i = tid + r * PT;
        const bool live = i < n;
        h_rep[r] = i;
        h_st[r] = RNNLM_H_DUP;
        bool scan = false;   // still racing after the last table, or a settled representative of another key
        if (live) {
            const int m = (hpend >> r) & 1u ? -1 : hmin[r];
            if (m != i) {
                if (m >= 0 && same_hist_key(d, m, i)) h_rep[r] = m;
                else scan = true;
            }
        }
        // the first equal key, searched by the whole wave 64 indices at a time
        for (u64 todo = __ballot(scan); todo; todo &= todo - 1) {
            const int src = __ffsll((unsigned long long)todo) - 1;
            const int is = __shfl(i, src);
            const u64 hs = ((u64)(uint32_t)__shfl((int)(h_hash[r] >> 32), src) << 32) |
                           (uint32_t)__shfl((int)(uint32_t)h_hash[r], src);
            int found = is;
            for (int j0 = 0; j0 < is; j0 += 64) {
                const int j = j0 + lane;
                const bool eq = j < is && d.f_hrec[min(j, hlast)].hash == hs && same_hist_key(d, j, is);
                const u64 b = __ballot(eq);
                if (b) {
                    found = j0 + __ffsll((unsigned long long)b) - 1;
                    break;
                }
            }
            if (lane == src) h_rep[r] = found;
        }
        if (live) {
            h_st[r] = h_slot[r] >= 0 ? RNNLM_HC_HIT : (h_rep[r] == i ? RNNLM_H_REP : RNNLM_H_DUP);
            s_rep[i] = h_rep[r] | (h_st[r] << 16);
            if (h_st[r] == RNNLM_HC_HIT) s_hsa[i] = h_slot[r];
        }
        const u64 b = __ballot(live && h_st[r] == RNNLM_H_REP);
        if ((tid & 63) == 0) s_hflag[i >> 6] = b;
    }
    __syncthreads();

    // ---------------- GRU rows (one wave) and query representatives --------
    if (tid < 64) {
        const int tot = flag_prefix(s_hflag, s_hpre, (n + 63) >> 6);
        if (tid == 0) s_htot = tot;
    }
    // two queries have equal keys when their histories have the same
    // representative and their words agree
    auto same_query = [&](const int4 a, const int4 b) {
        return ((s_rep[a.x] ^ s_rep[b.x]) & 0xFFFF) == 0 && a.y == b.y && a.z == b.z && a.w == b.w;
    };
    int qrepv[QR];
    if (RQ > 0) {
        int4 km[QR];
        const int qlim = nq - 1;   // qmin of an idle element can name a missing query
        if (stage) {
#pragma unroll
            for (int r = 0; r < QR; ++r)
                if (r < RQ) km[r] = s_qk[min(qmin[r], qlim)];
        } else {
#pragma unroll
            for (int r = 0; r < QR; ++r)
                if (r < RQ) km[r] = ldg<int4>(d.f_qkey + min(qmin[r], qlim));
        }
#pragma unroll
        for (int r = 0; r < QR; ++r) {
            if (r >= RQ) break;   // block-uniform
            const int q = tid + r * PT;
            qrepv[r] = q;
            const bool pend = (qpend >> r) & 1u;
            bool scan = false;   // still racing, or a settled representative of another key
            if (q < nq && (pend || qmin[r] != q)) {
                if (!pend && same_query(km[r], qk[r])) qrepv[r] = qmin[r];
                else scan = true;
            }
            // the first equal key, searched by the whole wave 64 indices at a time
            for (u64 todo = __ballot(scan); todo; todo &= todo - 1) {
                const int src = __ffsll((unsigned long long)todo) - 1;
                const int qs = __shfl(q, src);
                const int4 ks = make_int4(__shfl(qk[r].x, src), __shfl(qk[r].y, src), __shfl(qk[r].z, src),
                                          __shfl(qk[r].w, src));
                int found = qs;
                for (int j0 = 0; j0 < qs; j0 += 64) {
                    const int j = min(j0 + lane, qlim);
                    const int4 kj = stage ? s_qk[j] : ldg<int4>(d.f_qkey + j);
                    const u64 b = __ballot(j0 + lane < qs && same_query(kj, ks));
                    if (b) {
                        found = j0 + __ffsll((unsigned long long)b) - 1;
                        break;
                    }
                }
                if (lane == src) qrepv[r] = found;
            }
        }
    }
    __syncthreads();

    // ---------------- placements and per-history results ----------------
    // Where history h's h' goes: a cache hit keeps its slot; a new key's GRU
    // row is its rank among the frame's new keys (ascending index), and it
    // enters the history cache in that order while there is room; a
    // duplicate shares its representative's.
    const long long hc_size = c[C_HC_SIZE];
    auto place = [&](int h, int &hsa, int &loc, int &row) {
        int sr = s_rep[h];
        if ((sr >> 16) == RNNLM_H_DUP) {
            h = sr & 0xFFFF;
            sr = s_rep[h];
        }
        row = -1;
        if ((sr >> 16) == RNNLM_HC_HIT) {
            hsa = loc = s_hsa[h];
        } else {
            row = flag_rank(s_hflag, s_hpre, h);
            const bool adm = hc_size + row < d.cap_hist;
            hsa = adm ? (int)(hc_size + row) : -1;
            loc = adm ? hsa : -(row + 1);
        }
    };
#pragma unroll
    for (int r = 0; r < HR; ++r) {
        if (r * PT >= n) break;   // block-uniform
        const int i = tid + r * PT;
        const bool live = i < n;
        if (live) {
            const int st = h_st[r];
            int hsa, loc, row;
            place(i, hsa, loc, row);
            s_hsa[i] = hsa;
            s_loc[i] = loc;
            const float *hp = loc >= 0 ? d.hc_val + (size_t)loc * d.LH : d.f_hval + (size_t)(-loc - 1) * d.LH;
            d.f_hstat[i] = st;
            d.f_hslot[i] = hsa;
            d.f_hptr[i] = (u64)hp;
            if (st == RNNLM_H_REP) {
                const float *src = f.hist_ptr ? handle_row(d, h_hp[r]) : f.hist_vec + (size_t)i * d.LH;
                d.f_roww[row] = h_w1[r];
                d.f_rowh[row] = (u64)src;
                d.f_rowdst[row] = (u64)hp;
                if (d.wdtype == RNNLM_BF16) d.f_rowhb[row] = (u64)(d.f_hbf + (size_t)i * d.LH);
            }
            if (f.h_status) f.h_status[i] = (uint8_t)st;
            if (f.h_rep) f.h_rep[i] = h_rep[r];
        }
        count_lanes(&s_cnt[0], live && h_st[r] == RNNLM_HC_HIT);
        count_lanes(&s_cnt[1], live && h_st[r] == RNNLM_H_DUP);
    }
    // a new key whose history is (or will be) cached may enter the LM-query
    // cache; candidates are ranked in query order. When the history cache
    // has room for all of the frame's new keys, every history is cached.
    const bool all_cached = hc_size + s_htot <= d.cap_hist;   // block-uniform
#pragma unroll
    for (int r = 0; r < QR; ++r) {
        if (r >= RQ) break;   // block-uniform
        const int q = tid + r * PT;
        bool cand = false;
        if (q < nq && qrepv[r] == q) {
            cand = true;
            if (!all_cached) {
                int hsa, loc, row;
                place(qk[r].x, hsa, loc, row);
                cand = hsa >= 0;
            }
        }
        const u64 b = __ballot(cand);
        if ((tid & 63) == 0) s_qflag[q >> 6] = b;
    }
    __syncthreads();

    if (tid == 0) {
        const int M = s_htot;
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

    // ---------------- query ranks (one wave) and scorer records -------------
    if (RQ > 0) {
        if (tid < 64) {
            const int tot = flag_prefix(s_qflag, s_qpre, (nq + 63) >> 6);
            if (tid == 0) s_qtot = tot;
        }
        __syncthreads();
        const long long sc_size = c[C_SC_SIZE];
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
                rec.flags = (rep < q ? RNNLM_Q_DUP : RNNLM_Q_COMPUTED) | (cand ? QF_CAND : 0) |
                            ((s_rep[i] >> 16) == RNNLM_HC_HIT ? QF_PROBE : 0) | (cand ? rank << 6 : 0);
                rec.hs = s_hsa[i];
                d.f_qrec[q] = rec;
                if (f.q_rep) f.q_rep[q] = rep;
            }
        }
        if (tid == 0) {
            // admission is order-independent unless the candidates could overflow the cache
            const int ncand = s_qtot;
            const bool near = sc_size + ncand > d.cap_query;
            c[C_NEAR_CAP] = near ? 1 : 0;
            c[C_STAGED] = near ? 0 : ncand;   // staging slots the scorer fills
        }
    }
    // only lane 0 of wave 0 changes the counters after they are read in: the
    // wave writes them back once it is done, without waiting for the others
    __builtin_amdgcn_wave_barrier();
    if (tid < C_N) d.ctr[tid] = c[tid];
}

template <bool MULTI, int HR>
static void launch_plan_q(const Dev &d, const FrameBlock &fb, int qr, hipStream_t s, Stamp ts) {
    switch (qr) {
        case 1: launch_k(k_frame_plan<MULTI, HR, 1>, fb.n, PT, s, ts, d, fb); break;
        case 2: launch_k(k_frame_plan<MULTI, HR, 2>, fb.n, PT, s, ts, d, fb); break;
        case 4: launch_k(k_frame_plan<MULTI, HR, 4>, fb.n, PT, s, ts, d, fb); break;
        default: launch_k(k_frame_plan<MULTI, HR, QR_MAX>, fb.n, PT, s, ts, d, fb); break;
    }
}

void launch_frame_plan(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts) {
    // per-thread rounds sized to the block's largest frame
    int mh = 0, mq = 0;
    for (int e = 0; e < fb.n; ++e) {
        mh = std::max(mh, fb.f[e].n_hist);
        mq = std::max(mq, fb.f[e].n_query);
    }
    const int hr = mh <= PT ? 1 : HR_MAX;
    const int qr = mq <= PT ? 1 : mq <= 2 * PT ? 2 : mq <= 4 * PT ? 4 : QR_MAX;
    if (fb.n > 1) {
        if (hr == 1) launch_plan_q<true, 1>(d, fb, qr, s, ts);
        else launch_plan_q<true, HR_MAX>(d, fb, qr, s, ts);
    } else {
        if (hr == 1) launch_plan_q<false, 1>(d, fb, qr, s, ts);
        else launch_plan_q<false, HR_MAX>(d, fb, qr, s, ts);
    }
}

}  // namespace rn
