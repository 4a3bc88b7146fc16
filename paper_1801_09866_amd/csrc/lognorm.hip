// Full-vocabulary log normaliser (Sec. 2.2: the normalisation over V that
// NCE lets the decoder skip), used to measure NCE self-normalisation:
//   logZ_i = log sum_v exp(U_out[v] . h_i + b_out[v]).
// Pass 1: an fp32 MFMA GEMM over vocabulary tiles; each block keeps all n <=
// 256 rows of h and 128 vocabulary rows, and its epilogue reduces its logits
// to a (max, sum exp(. - max)) pair per row. No logit reaches HBM.
// Pass 2: per row, a fixed-shape tree combines the pairs of all tiles.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

typedef float f4_t __attribute__((ext_vector_type(4)));

constexpr int LN_BM = 256, LN_BN = 128, LN_BK = 16, LN_LD = LN_BK + 4;

int lognorm_tiles(int V) { return (V + LN_BN - 1) / LN_BN; }

__global__ __launch_bounds__(512) void k_lognorm_gemm(Dev d, const float *h, int n) {
    __shared__ float As[2][LN_BM][LN_LD];
    __shared__ float Bs[2][LN_BN][LN_LD];
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int tile = blockIdx.x, v0 = tile * LN_BN;
    const int H = d.H, V = d.V;
    const float *U = reinterpret_cast<const float *>(d.U_out);

    // A: 256 rows x 16 k = 1024 float4, two per thread; B: 128 x 16 = 512, one
    const int a_r0 = tid >> 2, a_r1 = a_r0 + 128, a_k = (tid & 3) * 4;
    const int b_r = tid >> 2, b_k = (tid & 3) * 4;
    const bool a_ok0 = a_r0 < n, a_ok1 = a_r1 < n, b_ok = v0 + b_r < V;
    const float *ap0 = h + (size_t)(a_ok0 ? a_r0 : 0) * H + a_k;
    const float *ap1 = h + (size_t)(a_ok1 ? a_r1 : 0) * H + a_k;
    const float *bp = U + (size_t)(b_ok ? v0 + b_r : 0) * H + b_k;
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);

    float4 ra0, ra1, rb;
    auto load = [&](int k0) {
        ra0 = a_ok0 ? *reinterpret_cast<const float4 *>(ap0 + k0) : zero;
        ra1 = a_ok1 ? *reinterpret_cast<const float4 *>(ap1 + k0) : zero;
        rb = b_ok ? *reinterpret_cast<const float4 *>(bp + k0) : zero;
    };
    auto store = [&](int buf) {
        *reinterpret_cast<float4 *>(&As[buf][a_r0][a_k]) = ra0;
        *reinterpret_cast<float4 *>(&As[buf][a_r1][a_k]) = ra1;
        *reinterpret_cast<float4 *>(&Bs[buf][b_r][b_k]) = rb;
    };

    f4_t acc[2][8];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 8; ++b) acc[a][b] = f4_t{0, 0, 0, 0};

    const int fr = lane & 15, fk = 4 * (lane >> 4);
    const int nk = H / LN_BK;
    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * LN_BK);
        float4 a[2], b[8];
#pragma unroll
        for (int r = 0; r < 2; ++r) a[r] = *reinterpret_cast<const float4 *>(&As[buf][w * 32 + r * 16 + fr][fk]);
#pragma unroll
        for (int c = 0; c < 8; ++c) b[c] = *reinterpret_cast<const float4 *>(&Bs[buf][c * 16 + fr][fk]);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const float av[4] = {a[r].x, a[r].y, a[r].z, a[r].w};
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const float bv[4] = {b[c].x, b[c].y, b[c].z, b[c].w};
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s], bv[s], acc[r][c], 0, 0, 0);
            }
        }
        if (kt + 1 < nk) store(buf ^ 1);
        __syncthreads();
    }

    // epilogue: logits of this lane's columns, then per-row (max, sum exp)
    float bias[8];
    bool valid[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int v = v0 + c * 16 + fr;
        valid[c] = v < V;
        bias[c] = valid[c] ? d.b_out[v] : 0.0f;
    }
    const int NT = gridDim.x;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float m = -INFINITY;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                if (valid[c]) m = fmaxf(m, acc[r][c][e] + bias[c]);
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
            float sum = 0.0f;
#pragma unroll
            for (int c = 0; c < 8; ++c)
                if (valid[c]) sum += expf(acc[r][c][e] + bias[c] - m);
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) sum += __shfl_xor(sum, o, 64);
            const int row = w * 32 + r * 16 + 4 * (lane >> 4) + e;
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

void launch_lognorm_gemm(const Dev &d, const float *h, int n, hipStream_t s, Stamp ts) {
    launch_k(k_lognorm_gemm, lognorm_tiles(d.V), 512, s, ts, d, h, n);
}

void launch_lognorm_combine(const Dev &d, int n, float *logz, hipStream_t s, Stamp ts) {
    launch_k(k_lognorm_combine, n, 256, s, ts, d, lognorm_tiles(d.V), logz);
}

}  // namespace rn
