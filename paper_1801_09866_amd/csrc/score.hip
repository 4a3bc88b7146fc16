// Query scoring (Sec. 2.2 NCE, Sec. 2.3 MaxEnt): one wave per query.
//   score = U_out[t] . h'_top + b_out[t] + sum_{n=2..N} maxent[slot_n]
// The output row is read once, coalesced across the wave (16 B per lane per
// step), and reduced with a fixed butterfly, so every query with the same key
// produces the same bits. Stored scores are returned for cache hits, and new
// admitted keys are entered into the LM-query cache.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

template <bool BF16>
__global__ __launch_bounds__(256) void k_score(Dev d, FrameArgs f) {
    const int q = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (q >= f.n_query) return;
    const int st = d.f_qstat[q];
    const int4 key = d.f_qkey[q];
    const int i = d.f_qhist[q], t = key.w;
    float s;
    if (st == RNNLM_Q_SCORE_HIT) {
        s = d.sc_val[d.f_qsc[q]];
    } else {
        const float *h = reinterpret_cast<const float *>(d.f_hptr[i]) + (size_t)(d.L - 1) * d.H;
        float acc = 0.0f;
        if (!BF16) {
            const float *u = reinterpret_cast<const float *>(d.U_out) + (size_t)t * d.H;
            for (int e = lane * 4; e < d.H; e += 256) {
                const float4 a = *reinterpret_cast<const float4 *>(u + e);
                const float4 b = *reinterpret_cast<const float4 *>(h + e);
                acc = fmaf(a.x, b.x, acc);
                acc = fmaf(a.y, b.y, acc);
                acc = fmaf(a.z, b.z, acc);
                acc = fmaf(a.w, b.w, acc);
            }
        } else {
            const uint16_t *u = reinterpret_cast<const uint16_t *>(d.U_out) + (size_t)t * d.H;
            for (int e = lane * 8; e < d.H; e += 512) {
                const uint4 a = *reinterpret_cast<const uint4 *>(u + e);
                const float4 b0 = *reinterpret_cast<const float4 *>(h + e);
                const float4 b1 = *reinterpret_cast<const float4 *>(h + e + 4);
                acc = fmaf(__uint_as_float(a.x << 16), b0.x, acc);
                acc = fmaf(__uint_as_float(a.x & 0xFFFF0000u), b0.y, acc);
                acc = fmaf(__uint_as_float(a.y << 16), b0.z, acc);
                acc = fmaf(__uint_as_float(a.y & 0xFFFF0000u), b0.w, acc);
                acc = fmaf(__uint_as_float(a.z << 16), b1.x, acc);
                acc = fmaf(__uint_as_float(a.z & 0xFFFF0000u), b1.y, acc);
                acc = fmaf(__uint_as_float(a.w << 16), b1.z, acc);
                acc = fmaf(__uint_as_float(a.w & 0xFFFF0000u), b1.w, acc);
            }
        }
        s = wave_sum(acc);
        s += d.b_out[t];
        const int w1 = d.f_words[i * 3], w2 = d.f_words[i * 3 + 1], w3 = d.f_words[i * 3 + 2];
        for (int o = 2; o <= d.me_order; ++o) s += d.maxent[maxent_slot(o, w1, w2, w3, t, d.me_log2)];
    }
    if (lane == 0) {
        f.scores[q] = s;
        const int id = d.f_qadmit[q];
        if (id >= 0) {
            const int hs = d.f_hslot[i];
            d.sc_key[id] = make_int4(hs, key.y, key.z, t);
            d.sc_val[id] = s;
            const u64 sh = query_hash(hs, key.y, key.z, t);
            unsigned pos = (unsigned)(sh & d.si_mask);
            for (unsigned n = 0; n <= d.si_mask; ++n) {
                if (atomicCAS(&d.sc_islot[pos], -1, id) == -1) {
                    d.sc_ihash[pos] = sh;
                    break;
                }
                pos = (pos + 1) & d.si_mask;
            }
        }
        const int tp = d.f_qtpos[q];
        d.qt_hash[tp] = 0ull;
        d.qt_min[tp] = 0x7FFFFFFF;
    }
}

void launch_score(const Dev &d, const FrameArgs &f, hipStream_t s) {
    const int blocks = (f.n_query + 3) / 4;
    if (d.wdtype == RNNLM_BF16)
        k_score<true><<<blocks, 256, 0, s>>>(d, f);
    else
        k_score<false><<<blocks, 256, 0, s>>>(d, f);
}

}  // namespace rn
