// GRU step for the frame's unique history keys (Sec. 2.1), one launch per
// layer. One MFMA GEMM produces all gate pre-activations of a row block:
//   rows:     A = [x ; h]  gathered per work-list row (x = embedding of the
//             input word for the first layer, the lower layer's h' above it;
//             h = that layer's slice of the history vector)
//   columns:  packed weights [3H][Kx + H] = [W_ih | W_hh] per gate row.
// The reset and update gates accumulate over all of K. The candidate keeps its
// input part (k < Kx) and recurrent part (k >= Kx) in separate accumulators,
// because the reset gate scales only the recurrent part:
//   r = sigmoid(a_r), z = sigmoid(a_z), n = tanh(a_nx + b_n + r * a_nh),
//   h' = (1 - z) * n + z * h.
// The epilogue is fused: no gate pre-activation ever reaches HBM.
#include "common.hpp"
#include "kernels.hpp"

namespace rn {

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));

constexpr int G_BM = 64;    // work-list rows per block
constexpr int G_BJ = 32;    // hidden units per block (x 3 gates)
constexpr int G_THREADS = 512;

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }

// block -> (row tile, unit tile); blocks are dealt to the 8 XCDs round-robin,
// so give every XCD its own set of unit tiles: each XCD then streams only
// 1/8 of the weights, which stay resident in its L2.
__device__ __forceinline__ void gru_tile_of(int b, int NJ, int &mt, int &jt) {
    if ((NJ & 7) == 0) {
        const int xcd = b & 7, idx = b >> 3, per = NJ >> 3;
        mt = idx / per;
        jt = xcd + 8 * (idx % per);
    } else {
        mt = b / NJ;
        jt = b % NJ;
    }
}

struct RowSrc {
    const void *x;      // start of this row's x part (fp32, or bf16 embedding)
    const float *h;     // start of this row's h part
    bool x_bf16;
    bool valid;
};

__device__ __forceinline__ RowSrc row_source(const Dev &d, const FrameArgs &f, int layer, int m, int M) {
    RowSrc r;
    r.valid = m < M;
    r.x_bf16 = false;
    r.x = nullptr;
    r.h = nullptr;
    if (!r.valid) return r;
    const int i = d.f_rows[m];
    r.h = f.hist_vec + (size_t)i * d.LH + (size_t)layer * d.H;
    if (layer == 0) {
        const int w = d.f_words[i * 3];
        if (d.wdtype == RNNLM_BF16) {
            r.x = reinterpret_cast<const uint16_t *>(d.emb) + (size_t)w * d.E;
            r.x_bf16 = true;
        } else {
            r.x = reinterpret_cast<const float *>(d.emb) + (size_t)w * d.E;
        }
    } else {
        r.x = reinterpret_cast<const float *>(d.f_rowdst[m]) + (size_t)(layer - 1) * d.H;
    }
    return r;
}

__device__ __forceinline__ void gru_epilogue(const Dev &d, const FrameArgs &f, int layer, int M, int m0,
                                             int j0, int rb, int ub, const f4_t &ar, const f4_t &az,
                                             const f4_t &anx, const f4_t &anh) {
    const int lane = threadIdx.x & 63;
    const int j = j0 + ub * 16 + (lane & 15);
    const float *b = d.b_ih[layer];
    const float br = b[j], bz = b[d.H + j], bn = b[2 * d.H + j];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int m = m0 + rb * 16 + 4 * (lane >> 4) + e;
        if (m < M) {
            const int i = d.f_rows[m];
            const float hprev = f.hist_vec[(size_t)i * d.LH + (size_t)layer * d.H + j];
            const float r = sigmoidf_(ar[e] + br);
            const float z = sigmoidf_(az[e] + bz);
            const float n = tanhf(anx[e] + bn + r * anh[e]);
            float *dst = reinterpret_cast<float *>(d.f_rowdst[m]) + (size_t)layer * d.H + j;
            *dst = (1.0f - z) * n + z * hprev;
        }
    }
}

// ------------------------------- fp32 -------------------------------------
constexpr int F_BK = 32;
constexpr int F_LDA = F_BK + 4;   // padded LDS row (floats)

__global__ __launch_bounds__(G_THREADS) void k_gru_f32(Dev d, FrameArgs f, int layer) {
    const int M = (int)d.ctr[C_FRAME_M];
    const int NJ = d.H / G_BJ;
    int mt, jt;
    gru_tile_of(blockIdx.x, NJ, mt, jt);
    const int m0 = mt * G_BM, j0 = jt * G_BJ;
    if (m0 >= M) return;

    __shared__ float As[2][G_BM][F_LDA];
    __shared__ float Bs[2][3 * G_BJ][F_LDA];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const float *Wp = reinterpret_cast<const float *>(d.Wp[layer]);

    // A loader: row tid/8, 4 consecutive k at (tid%8)*4
    const int a_row = tid >> 3, a_k = (tid & 7) * 4;
    const RowSrc src = row_source(d, f, layer, m0 + a_row, M);
    // B loader: rows (gate, unit) tid/8 and tid/8 + 64
    const int b_k = (tid & 7) * 4;
    const int b_r0 = tid >> 3, b_r1 = b_r0 + 64;
    const float *bp0 = Wp + (size_t)((b_r0 / G_BJ) * d.H + j0 + (b_r0 % G_BJ)) * K + b_k;
    const float *bp1 = Wp + (size_t)((b_r1 / G_BJ) * d.H + j0 + (b_r1 % G_BJ)) * K + b_k;
    const bool has_b1 = b_r1 < 3 * G_BJ;

    float4 ra, rb0, rb1;
    auto load = [&](int k0) {
        const int k = k0 + a_k;
        if (!src.valid) ra = make_float4(0.f, 0.f, 0.f, 0.f);
        else if (k < Kx) ra = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(src.x) + k);
        else ra = *reinterpret_cast<const float4 *>(src.h + (k - Kx));
        rb0 = *reinterpret_cast<const float4 *>(bp0 + k0);
        if (has_b1) rb1 = *reinterpret_cast<const float4 *>(bp1 + k0);
    };
    auto store = [&](int buf) {
        *reinterpret_cast<float4 *>(&As[buf][a_row][a_k]) = ra;
        *reinterpret_cast<float4 *>(&Bs[buf][b_r0][b_k]) = rb0;
        if (has_b1) *reinterpret_cast<float4 *>(&Bs[buf][b_r1][b_k]) = rb1;
    };

    f4_t ar = {0, 0, 0, 0}, az = ar, anx = ar, anh = ar;
    const int rb = w & 3, ub = w >> 2;
    const int fr = lane & 15, fk = 4 * (lane >> 4);

    const int nk = K / F_BK;
    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * F_BK);
        const bool xphase = kt * F_BK < Kx;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const float4 a = *reinterpret_cast<const float4 *>(&As[buf][rb * 16 + fr][hh * 16 + fk]);
            const float4 br = *reinterpret_cast<const float4 *>(&Bs[buf][0 * G_BJ + ub * 16 + fr][hh * 16 + fk]);
            const float4 bz = *reinterpret_cast<const float4 *>(&Bs[buf][1 * G_BJ + ub * 16 + fr][hh * 16 + fk]);
            const float4 bn = *reinterpret_cast<const float4 *>(&Bs[buf][2 * G_BJ + ub * 16 + fr][hh * 16 + fk]);
            const float av[4] = {a.x, a.y, a.z, a.w};
            const float rv[4] = {br.x, br.y, br.z, br.w};
            const float zv[4] = {bz.x, bz.y, bz.z, bz.w};
            const float nv[4] = {bn.x, bn.y, bn.z, bn.w};
            if (xphase) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    ar = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], rv[c], ar, 0, 0, 0);
                    az = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], zv[c], az, 0, 0, 0);
                    anx = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], nv[c], anx, 0, 0, 0);
                }
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    ar = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], rv[c], ar, 0, 0, 0);
                    az = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], zv[c], az, 0, 0, 0);
                    anh = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], nv[c], anh, 0, 0, 0);
                }
            }
        }
        if (kt + 1 < nk) store(buf ^ 1);
        __syncthreads();
    }
    gru_epilogue(d, f, layer, M, m0, j0, rb, ub, ar, az, anx, anh);
}

// ------------------------------- bf16 -------------------------------------
constexpr int H_BK = 64;
constexpr int H_LDA = H_BK + 8;   // padded LDS row (bf16 elements)

__device__ __forceinline__ uint4 pack_bf16x8(float4 a, float4 b) {
    uint4 r;
    r.x = (uint32_t)f32_to_bf16(a.x) | ((uint32_t)f32_to_bf16(a.y) << 16);
    r.y = (uint32_t)f32_to_bf16(a.z) | ((uint32_t)f32_to_bf16(a.w) << 16);
    r.z = (uint32_t)f32_to_bf16(b.x) | ((uint32_t)f32_to_bf16(b.y) << 16);
    r.w = (uint32_t)f32_to_bf16(b.z) | ((uint32_t)f32_to_bf16(b.w) << 16);
    return r;
}

__global__ __launch_bounds__(G_THREADS) void k_gru_bf16(Dev d, FrameArgs f, int layer) {
    const int M = (int)d.ctr[C_FRAME_M];
    const int NJ = d.H / G_BJ;
    int mt, jt;
    gru_tile_of(blockIdx.x, NJ, mt, jt);
    const int m0 = mt * G_BM, j0 = jt * G_BJ;
    if (m0 >= M) return;

    __shared__ uint16_t As[2][G_BM][H_LDA];
    __shared__ uint16_t Bs[2][3 * G_BJ][H_LDA];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const uint16_t *Wp = reinterpret_cast<const uint16_t *>(d.Wp[layer]);

    const int a_row = tid >> 3, a_k = (tid & 7) * 8;
    const RowSrc src = row_source(d, f, layer, m0 + a_row, M);
    const int b_k = (tid & 7) * 8;
    const int b_r0 = tid >> 3, b_r1 = b_r0 + 64;
    const uint16_t *bp0 = Wp + (size_t)((b_r0 / G_BJ) * d.H + j0 + (b_r0 % G_BJ)) * K + b_k;
    const uint16_t *bp1 = Wp + (size_t)((b_r1 / G_BJ) * d.H + j0 + (b_r1 % G_BJ)) * K + b_k;
    const bool has_b1 = b_r1 < 3 * G_BJ;

    uint4 ra, rb0, rb1;
    auto load = [&](int k0) {
        const int k = k0 + a_k;
        if (!src.valid) {
            ra = make_uint4(0, 0, 0, 0);
        } else if (k < Kx) {
            if (src.x_bf16) {
                ra = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(src.x) + k);
            } else {
                const float *p = reinterpret_cast<const float *>(src.x) + k;
                ra = pack_bf16x8(*reinterpret_cast<const float4 *>(p), *reinterpret_cast<const float4 *>(p + 4));
            }
        } else {
            const float *p = src.h + (k - Kx);
            ra = pack_bf16x8(*reinterpret_cast<const float4 *>(p), *reinterpret_cast<const float4 *>(p + 4));
        }
        rb0 = *reinterpret_cast<const uint4 *>(bp0 + k0);
        if (has_b1) rb1 = *reinterpret_cast<const uint4 *>(bp1 + k0);
    };
    auto store = [&](int buf) {
        *reinterpret_cast<uint4 *>(&As[buf][a_row][a_k]) = ra;
        *reinterpret_cast<uint4 *>(&Bs[buf][b_r0][b_k]) = rb0;
        if (has_b1) *reinterpret_cast<uint4 *>(&Bs[buf][b_r1][b_k]) = rb1;
    };

    f4_t ar = {0, 0, 0, 0}, az = ar, anx = ar, anh = ar;
    const int rb = w & 3, ub = w >> 2;
    const int fr = lane & 15, fk = 8 * (lane >> 4);

    const int nk = K / H_BK;
    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * H_BK);
        const bool xphase = kt * H_BK < Kx;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const bf8_t a = *reinterpret_cast<const bf8_t *>(&As[buf][rb * 16 + fr][hh * 32 + fk]);
            const bf8_t br = *reinterpret_cast<const bf8_t *>(&Bs[buf][0 * G_BJ + ub * 16 + fr][hh * 32 + fk]);
            const bf8_t bz = *reinterpret_cast<const bf8_t *>(&Bs[buf][1 * G_BJ + ub * 16 + fr][hh * 32 + fk]);
            const bf8_t bn = *reinterpret_cast<const bf8_t *>(&Bs[buf][2 * G_BJ + ub * 16 + fr][hh * 32 + fk]);
            ar = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, br, ar, 0, 0, 0);
            az = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bz, az, 0, 0, 0);
            if (xphase) anx = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bn, anx, 0, 0, 0);
            else anh = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bn, anh, 0, 0, 0);
        }
        if (kt + 1 < nk) store(buf ^ 1);
        __syncthreads();
    }
    gru_epilogue(d, f, layer, M, m0, j0, rb, ub, ar, az, anx, anh);
}

// --------------------------- weight packing -------------------------------
__global__ void k_pack_layer(const void *W_ih, const void *W_hh, void *dst, int rows, int Kx, int H,
                             int elem) {
    const int K = Kx + H;
    const long long n = (long long)rows * K;
    for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (long long)gridDim.x * blockDim.x) {
        const long long r = e / K;
        const int k = (int)(e % K);
        if (elem == 4) {
            const float v = k < Kx ? reinterpret_cast<const float *>(W_ih)[r * Kx + k]
                                   : reinterpret_cast<const float *>(W_hh)[r * H + (k - Kx)];
            reinterpret_cast<float *>(dst)[e] = v;
        } else {
            const uint16_t v = k < Kx ? reinterpret_cast<const uint16_t *>(W_ih)[r * Kx + k]
                                      : reinterpret_cast<const uint16_t *>(W_hh)[r * H + (k - Kx)];
            reinterpret_cast<uint16_t *>(dst)[e] = v;
        }
    }
}

void launch_pack_layer(const Dev &d, int layer, const void *W_ih, const void *W_hh, void *dst,
                       hipStream_t s) {
    const int Kx = layer == 0 ? d.E : d.H;
    k_pack_layer<<<2048, 256, 0, s>>>(W_ih, W_hh, dst, 3 * d.H, Kx, d.H,
                                       d.wdtype == RNNLM_BF16 ? 2 : 4);
}

void launch_gru_layer(const Dev &d, const FrameArgs &f, int layer, int max_rows, hipStream_t s) {
    if (max_rows <= 0) return;
    const int NJ = d.H / G_BJ;
    const int NM = (max_rows + G_BM - 1) / G_BM;
    int blocks = NM * NJ;
    if ((NJ & 7) == 0) blocks = ((blocks + 7) / 8) * 8;   // whole rounds over the XCDs
    if (d.wdtype == RNNLM_BF16)
        k_gru_bf16<<<blocks, G_THREADS, 0, s>>>(d, f, layer);
    else
        k_gru_f32<<<blocks, G_THREADS, 0, s>>>(d, f, layer);
}

}  // namespace rn
