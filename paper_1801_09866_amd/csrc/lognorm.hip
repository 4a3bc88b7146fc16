// Full-vocabulary log normaliser (Sec. 2.2: the normalisation over V that
// NCE lets the decoder skip), used to measure NCE self-normalisation:
//   logZ_i = log sum_v exp(U_out[v] . h_i + b_out[v] [+ MaxEnt_i(v)]),
// where the optional MaxEnt term (Sec. 2.3) adds, for every word v, the
// hashed n-gram weights of v after history i's context words.
// Pass 1: an fp32 MFMA GEMM over vocabulary tiles; each block keeps all n <=
// 256 rows of h and 128 vocabulary rows, and its epilogue reduces its logits
// to a (max, sum exp(. - max)) pair per row. No logit reaches HBM.
// Pass 2: per row, a fixed-shape tree combines the pairs of all tiles.
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

namespace rn {

typedef float f4_t __attribute__((ext_vector_type(4)));

// A block takes all n <= 256 rows and LN_NC x 16 vocabulary rows; 8 waves of
// 32 rows each. 13 column tiles (208 rows) leave 962 vocabulary tiles at
// V = 200,000: under two rounds over the 256 CUs, with little idle tail.
// K advances 16 at a time through double-buffered LDS (32 at a time measured
// slower: more registers live across the barrier). LDS rows are 24 floats:
// with 20 the fragment reads (16 rows, 16 bytes each) conflict in the banks.
constexpr int LN_BM = 256, LN_NC = 13, LN_BN = 16 * LN_NC, LN_BK = 16, LN_LD = LN_BK + 8;
static_assert(LN_BK == 16 && LN_BM == 256 && LN_BN > 128 && LN_BN <= 256,
              "loaders: 4 threads x 4 k per row, rows tid / 4 + 128 j");

int lognorm_tiles(int V) { return (V + LN_BN - 1) / LN_BN; }
static_assert(kStaticMaxV == kStaticMaxTiles * LN_BN, "static normaliser limit");

__global__ __launch_bounds__(512) void k_lognorm_gemm(Dev d, const float *h, const int32_t *words, int n) {
    __shared__ float As[2][LN_BM][LN_LD];
    __shared__ float Bs[2][LN_BN][LN_LD];
    __shared__ u64 s_g[LN_BM][3];   // MaxEnt: per row and order 2..4, the hash of its context words
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int tile = blockIdx.x, v0 = tile * LN_BN;
    const int H = d.H, V = d.V;
    const float *U = reinterpret_cast<const float *>(d.U_out);

    // Rows past n (A) or past V (B) read row 0, always in bounds and finite;
    // their products only reach output rows that are not written and logits
    // the epilogue masks, so no select sits between a load and its use (a
    // select right after the load would make every K step wait for memory).
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    // A rows lr and lr + 128; B rows lr and, where the tile has it, lr + 128.
    // Named registers: loop-carried arrays of these end up in scratch.
    const int rb1 = lr + 128;
    const bool b_last = rb1 < LN_BN;
    auto arow = [&](int r) { return h + (size_t)(r < n ? r : 0) * H + lk; };
    auto brow = [&](int r) { return U + (size_t)(r < LN_BN && v0 + r < V ? v0 + r : 0) * H + lk; };
    const float *pa0 = arow(lr), *pa1 = arow(lr + 128);
    const float *pb0 = brow(lr), *pb1 = brow(rb1);
    auto ld = [](const float *p) { return *reinterpret_cast<const float4 *>(p); };
    float4 a0 = ld(pa0), a1 = ld(pa1);
    float4 b0 = ld(pb0), b1 = ld(pb1);
    auto stage = [&](int buf) {
        *reinterpret_cast<float4 *>(&As[buf][lr][lk]) = a0;
        *reinterpret_cast<float4 *>(&As[buf][lr + 128][lk]) = a1;
        *reinterpret_cast<float4 *>(&Bs[buf][lr][lk]) = b0;
        if (b_last) *reinterpret_cast<float4 *>(&Bs[buf][rb1][lk]) = b1;
    };
    if (words && tid < LN_BM) {   // while the first K slice is in flight
        int wv[3];
        unsigned err = 0;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            wv[c] = tid < n ? words[tid * 3 + c] : 0;
            if (wv[c] < 0 || wv[c] >= V) { err = RNNLM_DERR_WORD; wv[c] = 0; }
        }
        for (int o = 2; o <= d.me_order; ++o) s_g[tid][o - 2] = maxent_prefix(o, wv[0], wv[1], wv[2]);
        if (err && tile == 0) atomicOr(d.derr, err);
    }
    stage(0);
    __syncthreads();

    f4_t acc[2][LN_NC];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < LN_NC; ++b) acc[a][b] = f4_t{0, 0, 0, 0};

    const int fr = lane & 15, fk = 4 * (lane >> 4);
    const int nk = H / LN_BK;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;   // block-uniform
        if (more) {   // next K slice in flight while this one multiplies
            const int k0 = (kt + 1) * LN_BK;
            a0 = ld(pa0 + k0);
            a1 = ld(pa1 + k0);
            b0 = ld(pb0 + k0);
            b1 = ld(pb1 + k0);
        }
#pragma unroll
        for (int hk = 0; hk < LN_BK; hk += 16) {
            float4 a[2];
#pragma unroll
            for (int r = 0; r < 2; ++r) a[r] = *reinterpret_cast<const float4 *>(&As[buf][w * 32 + r * 16 + fr][hk + fk]);
            // one B fragment at a time: 8 MFMAs per LDS read keeps few registers live
#pragma unroll
            for (int c = 0; c < LN_NC; ++c) {
                const float4 b = *reinterpret_cast<const float4 *>(&Bs[buf][c * 16 + fr][hk + fk]);
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r].x, b.x, acc[r][c], 0, 0, 0);
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r].y, b.y, acc[r][c], 0, 0, 0);
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r].z, b.z, acc[r][c], 0, 0, 0);
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r].w, b.w, acc[r][c], 0, 0, 0);
                }
            }
        }
        if (more) stage(buf ^ 1);
        __syncthreads();
    }

    // epilogue: logits of this lane's columns, then per-row (max, sum exp)
    float bias[LN_NC];
    bool valid[LN_NC];
#pragma unroll
    for (int c = 0; c < LN_NC; ++c) {
        const int v = v0 + c * 16 + fr;
        valid[c] = v < V;
        bias[c] = valid[c] ? d.b_out[v] : 0.0f;
    }
    const int NT = gridDim.x;
    const uint64_t me_mask = (1ull << d.me_log2) - 1;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = w * 32 + r * 16 + 4 * (lane >> 4) + e;
            float lg[LN_NC];
#pragma unroll
            for (int c = 0; c < LN_NC; ++c) lg[c] = acc[r][c][e] + bias[c];
            if (words) {   // this row's n-gram weights of every column word, gathered together
                for (int o = 2; o <= d.me_order; ++o) {
                    const u64 g = s_g[row][o - 2];
                    float me[LN_NC];
#pragma unroll
                    for (int c = 0; c < LN_NC; ++c) {
                        const int v = v0 + c * 16 + fr;
                        me[c] = d.maxent[mix64(g ^ (u64)(valid[c] ? v + 1 : 1)) & me_mask];
                    }
#pragma unroll
                    for (int c = 0; c < LN_NC; ++c) lg[c] += me[c];
                }
            }
            float m = -INFINITY;
#pragma unroll
            for (int c = 0; c < LN_NC; ++c)
                if (valid[c]) m = fmaxf(m, lg[c]);
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
            float sum = 0.0f;
#pragma unroll
            for (int c = 0; c < LN_NC; ++c)
                if (valid[c]) sum += expf(lg[c] - m);
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) sum += __shfl_xor(sum, o, 64);
            if (fr == 0 && row < n) d.ln_part[(size_t)row * NT + tile] = make_float2(m, sum);
        }
    }
}

__device__ __forceinline__ float2 lse_combine(float2 a, float2 b) {
    const float M = fmaxf(a.x, b.x);
    if (M == -INFINITY) return make_float2(-INFINITY, 0.0f);
    return make_float2(M, a.y * expf(a.x - M) + b.y * expf(b.x - M));
}

__global__ __launch_bounds__(256) void k_lognorm_combine(Dev d, int NT, float *logz) {
    __shared__ float2 s[256];
    const int row = blockIdx.x, tid = threadIdx.x;
    float2 acc = make_float2(-INFINITY, 0.0f);
    for (int t = tid; t < NT; t += 256) acc = lse_combine(acc, d.ln_part[(size_t)row * NT + t]);
    s[tid] = acc;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) s[tid] = lse_combine(s[tid], s[tid + o]);
        __syncthreads();
    }
    if (tid == 0) logz[row] = s[0].x + logf(s[0].y);
}

// The normaliser's partial pairs for callers that cannot allocate: a
// file-scope device array, one per GPU, held until the process ends. Host
// code reaches it only through the address hipGetSymbolAddress returns for
// the current device (looked up once per device and kept).
constexpr size_t kStaticPartBytes = size_t(256) * kStaticMaxTiles * sizeof(float2);
static __device__ __align__(256) float2 scratch[kStaticPartBytes / sizeof(float2)];

hipError_t lognorm_static_scratch(float2 **ptr) {
    static std::mutex mu;
    static float2 *by_dev[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!by_dev[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        by_dev[dev] = static_cast<float2 *>(p);
    }
    *ptr = by_dev[dev];
    return hipSuccess;
}

void launch_lognorm_gemm(const Dev &d, const float *h, const int32_t *words, int n, hipStream_t s, Stamp ts) {
    launch_k(k_lognorm_gemm, lognorm_tiles(d.V), 512, s, ts, d, h, words, n);
}

void launch_lognorm_combine(const Dev &d, int n, float *logz, hipStream_t s, Stamp ts) {
    launch_k(k_lognorm_combine, n, 256, s, ts, d, lognorm_tiles(d.V), logz);
}

}  // namespace rn
