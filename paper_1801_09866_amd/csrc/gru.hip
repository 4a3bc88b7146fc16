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
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace rn {

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));

constexpr int G_THREADS = 512;

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }


struct RowSrc {
    const void *x;      // start of this row's x part (fp32, or bf16 embedding)
    const float *h;     // start of this row's h part
    bool x_bf16;
    bool valid;
};

// The GRU rows of all the launch's frames back to back: entry e's rows are
// [moff[e], moff[e+1]), and their work lists live in its session's scratch
// (sofs[e] bytes after session 0's).
struct Rows {
    int n;
    int moff[kMaxSessions + 1];
    long long sofs[kMaxSessions];
};

// sessions of the launch's frames (the GRU needs no other frame argument)
struct SessList {
    int n;
    int sess[kMaxSessions];
};

// The planner's GRU row count of each of the launch's frames, issued as the
// kernel's first loads (entries past the frame count load frame 0's and are
// not used), so that waiting for them waits for nothing issued later.
struct RowCounts {
    long long c[kMaxSessions];
};

__device__ __forceinline__ RowCounts load_row_counts(const Dev &d, const SessList &sl) {
    RowCounts rc;
#pragma unroll
    for (int e = 0; e < kMaxSessions; ++e) {
        const int ee = e < sl.n ? e : 0;
        rc.c[e] = ldg<long long>(shift_ptr(d.ctr, (long long)sl.sess[ee] * d.sess_stride) + C_FRAME_M);
    }
    return rc;
}

__device__ __forceinline__ Rows make_rows(const Dev &d, const SessList &sl, const RowCounts &rc) {
    Rows R;
    R.n = sl.n;
#pragma unroll
    for (int e = 0; e < kMaxSessions; ++e) R.sofs[e] = (long long)sl.sess[e < sl.n ? e : 0] * d.sess_stride;
    R.moff[0] = 0;
#pragma unroll
    for (int e = 0; e < kMaxSessions; ++e)
        R.moff[e + 1] = R.moff[e] + (e < sl.n ? __builtin_amdgcn_readfirstlane((int)rc.c[e]) : 0);
    return R;
}

// element `m` (a row of the whole launch) of a per-session work-list array
template <class T>
__device__ __forceinline__ T row_at(const Rows &R, T *arr, int m) {
    if (R.n == 1) return shift_ptr(arr, R.sofs[0])[m];   // one frame (a scalar branch)
    long long o = R.sofs[0];
    int base = 0;
#pragma unroll
    for (int e = 1; e < kMaxSessions; ++e)   // unrolled selects: no indexed private arrays
        if (e < R.n && m >= R.moff[e]) {
            o = R.sofs[e];
            base = R.moff[e];
        }
    return shift_ptr(arr, o)[m - base];
}

__device__ __forceinline__ RowSrc row_source(const Dev &d, const Rows &R, int layer, int m, int M) {
    RowSrc r;
    r.valid = m < M;
    r.x_bf16 = false;
    r.x = nullptr;
    r.h = nullptr;
    if (!r.valid) return r;
    r.h = reinterpret_cast<const float *>(row_at(R, d.f_rowh, m)) + (size_t)layer * d.H;
    if (layer == 0) {
        const int w = row_at(R, d.f_roww, m);
        if (d.wdtype == RNNLM_BF16) {
            r.x = reinterpret_cast<const uint16_t *>(d.emb) + (size_t)w * d.E;
            r.x_bf16 = true;
        } else {
            r.x = reinterpret_cast<const float *>(d.emb) + (size_t)w * d.E;
        }
    } else {
        r.x = reinterpret_cast<const float *>(row_at(R, d.f_rowdst, m)) + (size_t)(layer - 1) * d.H;
    }
    return r;
}

__device__ __forceinline__ uint4 pack_bf16x8(float4 a, float4 b) {
    uint4 r;
    r.x = (uint32_t)f32_to_bf16(a.x) | ((uint32_t)f32_to_bf16(a.y) << 16);
    r.y = (uint32_t)f32_to_bf16(a.z) | ((uint32_t)f32_to_bf16(a.w) << 16);
    r.z = (uint32_t)f32_to_bf16(b.x) | ((uint32_t)f32_to_bf16(b.y) << 16);
    r.w = (uint32_t)f32_to_bf16(b.z) | ((uint32_t)f32_to_bf16(b.w) << 16);
    return r;
}

// One LDS buffer serves every path.
constexpr int G_LDS_FLOATS = 35840;   // 140 KB

// ------------------------ narrow path (few rows) ---------------------------
// A frame with few new keys is bound by reading the weights once and by
// memory latency, not by FLOPs. Every block owns 4 hidden units for all rows,
// so all 256 CUs share the weight stream (each XCD its own contiguous 1/8,
// which stays in its L2). One 16 x 16 MFMA tile holds the block's 12 gate
// columns (r, z, n of 4 units; 4 columns padding) for 16 rows; the 8 waves
// split K, each keeping an input-part and a recurrent-part accumulator per
// row tile (the candidate gate needs them apart), and issue all of a pass's
// operand loads at once. The partial tiles meet in LDS in a fixed order, and
// one thread per (row, unit) applies the gates with operands it loaded before
// the K loop.
constexpr int N_MAXROWS = 32;   // rows handled by the narrow path at most
constexpr int N_TILES = N_MAXROWS / 16;
template <bool BF16W>
constexpr int n_pass() { return BF16W ? 8 : 12; }   // steps whose operands are loaded together

// One K step of one gate tile from 16 bytes of operands per lane: fp32
// takes 4 k per lane (four 16x16x4 MFMAs over the float4's components), bf16
// takes 8 (one 16x16x32 MFMA).
__device__ __forceinline__ f4_t nw_mfma(float4 a, float4 b, f4_t c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
}
__device__ __forceinline__ f4_t nw_mfma(uint4 a, uint4 b, f4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8_t, a), __builtin_bit_cast(bf8_t, b), c, 0, 0, 0);
}

// Operands of the narrow path that do not depend on the frame's row count.
// The kernel issues these loads as it starts, so that they are in flight
// while the planner's row count comes back: the epilogue biases and the row
// lists of the launch's first frame for rows 0..31 (read at indices clamped to
// the lists' length; used only when that frame is the launch's only one, and
// an entry only once its row is known to be below the count). The operand
// rows they point at are then one round trip from the kernel's start instead
// of two.
template <bool BF16W>
struct NarrowPre {
    float br, bz, bn;
    u64 rowh[N_TILES], rowd[N_TILES];   // A rows: history source, destination (the layer below's h')
    int roww[N_TILES];                  // A rows: input word (first layer)
    u64 edst, ehsrc;                    // epilogue row: destination and history source
};

template <bool BF16W>
__device__ __forceinline__ void narrow_preload(const Dev &d, const SessList &sl, int layer, int g,
                                               NarrowPre<BF16W> &p) {
    const int tid = threadIdx.x, col = tid & 15;
    // a fixed set of loads, none behind a branch
    const int j = 4 * g + (tid & 3);
    const float *bb = d.bl;
    p.br = ldg<float>(bb + j);
    p.bz = ldg<float>(bb + d.H + j);
    p.bn = ldg<float>(bb + 2 * d.H + j);
    // the row lists of the launch's first frame (used when it is the only one)
    const long long o = (long long)sl.sess[0] * d.sess_stride;
    const int last = d.max_hist - 1;
#pragma unroll
    for (int t = 0; t < N_TILES; ++t) {
        const int m = min(16 * t + col, last);
        p.rowh[t] = ldg<u64>(shift_ptr(d.f_rowh, o) + m);
        p.rowd[t] = ldg<u64>(shift_ptr(d.f_rowdst, o) + m);
        p.roww[t] = ldg<int>(shift_ptr(d.f_roww, o) + m);
    }
    const int me = min(min(tid >> 2, N_MAXROWS - 1), last);
    p.edst = ldg<u64>(shift_ptr(d.f_rowdst, o) + me);
    p.ehsrc = ldg<u64>(shift_ptr(d.f_rowh, o) + me);
}

template <bool BF16W, bool USE_PRE, int NT>
__device__ __forceinline__ void gru_narrow(const Dev &d, const Rows &R, int layer, int M, float *smem, int g,
                                           const NarrowPre<BF16W> &pre) {
    using T = typename std::conditional<BF16W, uint4, float4>::type;
    using E = typename std::conditional<BF16W, uint16_t, float>::type;
    constexpr int KS = BF16W ? 32 : 16;   // k per step
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H, K = Kx + d.H;
    const int nsteps = K / KS;
    const int s0 = (w * nsteps) / 8, s1 = ((w + 1) * nsteps) / 8;   // scalars
    const int col = lane & 15, kq = (KS / 4) * (lane >> 4);
    // columns 12..15 of the tile are padding: they repeat gate 0's weights, and
    // the epilogue never reads them (an MFMA output column depends only on
    // its own B column)
    const int gate = col >> 2, j0 = 4 * g;
    const E *wrow = reinterpret_cast<const E *>(d.Wl) + (size_t)((gate < 3 ? gate : 0) * d.H + j0 + (col & 3)) * K + kq;
    const int nt = (M + 15) >> 4;         // row tiles (block-uniform)
    const bool pre_rows = USE_PRE && R.n == 1;   // block-uniform

    // epilogue operands of thread (row m, unit u), loaded before the K loop
    const int em = tid >> 2, eu = tid & 3;
    const bool eth = em < M;
    float ebr = 0.f, ebz = 0.f, ebn = 0.f, ehp = 0.f;
    float *edst = nullptr;
    if (eth) {
        const int j = j0 + eu;
        if (USE_PRE) {
            ebr = pre.br;
            ebz = pre.bz;
            ebn = pre.bn;
        } else {
            const float *bb = d.bl;
            ebr = bb[j];
            ebz = bb[d.H + j];
            ebn = bb[2 * d.H + j];
        }
        const u64 dp = pre_rows ? pre.edst : (u64)row_at(R, d.f_rowdst, em);
        const u64 hp = pre_rows ? pre.ehsrc : (u64)row_at(R, d.f_rowh, em);
        edst = reinterpret_cast<float *>(dp) + (size_t)layer * d.H + j;
        ehp = reinterpret_cast<const float *>(hp)[(size_t)layer * d.H + j];
    }
    constexpr int PASS = n_pass<BF16W>();   // a wave has 6 bf16 steps at K = 1536
    T b[PASS];
    RowSrc src[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int m = 16 * t + col;
        if (pre_rows) {
            RowSrc &r = src[t];
            r.valid = m < M;
            r.x_bf16 = false;
            r.x = nullptr;
            r.h = nullptr;
            if (r.valid) {
                r.h = reinterpret_cast<const float *>(pre.rowh[t]) + (size_t)layer * d.H;
                if (layer == 0) {
                    const size_t wd = (size_t)(unsigned)pre.roww[t];
                    r.x_bf16 = d.wdtype == RNNLM_BF16;
                    r.x = r.x_bf16 ? (const void *)(reinterpret_cast<const uint16_t *>(d.emb) + wd * d.E)
                                   : (const void *)(reinterpret_cast<const float *>(d.emb) + wd * d.E);
                } else {
                    r.x = reinterpret_cast<const float *>(pre.rowd[t]) + (size_t)(layer - 1) * d.H;
                }
            }
        } else {
            src[t] = row_source(d, R, layer, m, M);
        }
    }

    auto loadA = [&](const RowSrc &rs, int k) -> T {
        if (!rs.valid) return T{0, 0, 0, 0};
        if (!BF16W) {
            const float *p = k < Kx ? reinterpret_cast<const float *>(rs.x) + k : rs.h + (k - Kx);
            return __builtin_bit_cast(T, ldg<float4>(p));
        }
        if (k < Kx && rs.x_bf16)
            return __builtin_bit_cast(T, ldg<uint4>(reinterpret_cast<const uint16_t *>(rs.x) + k));
        const float *p = k < Kx ? reinterpret_cast<const float *>(rs.x) + k : rs.h + (k - Kx);
        return __builtin_bit_cast(T, pack_bf16x8(ldg<float4>(p), ldg<float4>(p + 4)));
    };

    f4_t accx[NT], acch[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) accx[t] = acch[t] = f4_t{0, 0, 0, 0};
    for (int p0 = s0; p0 < s1; p0 += PASS) {
        T a[NT][PASS];
#pragma unroll
        for (int c = 0; c < PASS; ++c) {
            const int st = p0 + c;
            if (st < s1) {   // wave-uniform
                const int k = st * KS;
                b[c] = ldg<T>(wrow + k);
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (t < nt) a[t][c] = loadA(src[t], k + kq);
            }
        }
#pragma unroll
        for (int c = 0; c < PASS; ++c) {
            const int st = p0 + c;
            if (st < s1) {
                const bool xp = st * KS < Kx;   // wave-uniform
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    if (t < nt) {
                        if (xp) accx[t] = nw_mfma(a[t][c], b[c], accx[t]);
                        else acch[t] = nw_mfma(a[t][c], b[c], acch[t]);
                    }
                }
            }
        }
    }
    // partial tiles to LDS: [wave][tile][part][lane][4]
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t < nt) {
            float *px = smem + ((size_t)((w * NT + t) * 2 + 0) * 64 + lane) * 4;
            float *ph = smem + ((size_t)((w * NT + t) * 2 + 1) * 64 + lane) * 4;
            *reinterpret_cast<float4 *>(px) = make_float4(accx[t][0], accx[t][1], accx[t][2], accx[t][3]);
            *reinterpret_cast<float4 *>(ph) = make_float4(acch[t][0], acch[t][1], acch[t][2], acch[t][3]);
        }
    }
    __syncthreads();
    if (eth) {
        // D[row][col] sits in lane 16 * (row / 4) + col, element row % 4
        const int t = em >> 4, i = em & 15, e = i & 3, lb = 16 * (i >> 2);
        float xr = 0.f, xz = 0.f, xn = 0.f, hr = 0.f, hz = 0.f, hn = 0.f;
        for (int v = 0; v < 8; ++v) {   // fixed order: equal inputs give equal bits
            const float *px = smem + (size_t)((v * NT + t) * 2 + 0) * 256 + e;
            const float *ph = smem + (size_t)((v * NT + t) * 2 + 1) * 256 + e;
            xr += px[(lb + eu) * 4];
            xz += px[(lb + 4 + eu) * 4];
            xn += px[(lb + 8 + eu) * 4];
            hr += ph[(lb + eu) * 4];
            hz += ph[(lb + 4 + eu) * 4];
            hn += ph[(lb + 8 + eu) * 4];
        }
        const float r = sigmoidf_(xr + hr + ebr);
        const float z = sigmoidf_(xz + hz + ebz);
        const float n = tanhf(xn + ebn + r * hn);
        *edst = (1.0f - z) * n + z * ehp;
    }
}

// -------------------- tiled path (more than 32 rows): fp32 ------------------
// Tiles of BM = 16 * RB rows x 16 hidden units (48 weight rows: the units'
// reset, update and candidate rows). The row-tile height follows the row
// count: R row tiles per unit tile, with R chosen so that R x (H / 16) tiles
// make about one tile per CU, so any M up to 128 * R rows is split into R
// nearly equal row tiles (16-row granularity) and the CUs stay evenly loaded
// (at H = 1024: four row tiles of at most 128 rows for M <= 512).
// The block's 8 waves form 2 row groups x 4 K quarters: wave w takes the row
// blocks rb = g, g + 2, ... (g = w / 4) and k = 16 (w % 4) .. + 15 of every
// 64-wide K step. Waves w and w + 4 share a SIMD, so every SIMD carries the
// same MFMA work whatever RB is, even when the two groups' row-block counts
// differ. The four K quarters' partial sums meet in LDS in a fixed order, two
// row blocks at a time, and each thread applies the gates to one output.
constexpr int KS_TU = 16;            // hidden units per tile
constexpr int KS_RBMAX = 8;          // 16-row blocks per tile at most
constexpr int KS_BK = 64;            // K step
constexpr int KS_LDA = KS_BK + 8;    // padded LDS row (floats): 288 B, no bank conflicts for the fragment reads
constexpr int KS_BROWS = 3 * KS_TU;  // weight rows per tile
constexpr int KS_OPER = 2 * (16 * KS_RBMAX + KS_BROWS) * KS_LDA;   // two operand buffers (floats)
constexpr int KS_PTRS = KS_OPER;     // per tile row: destination, history source, input source (u64 each)
constexpr int KS_HPREV = KS_PTRS + 16 * KS_RBMAX * 6;   // per tile row: h of the tile's 16 units
static_assert(KS_HPREV + 16 * KS_RBMAX * KS_TU <= G_LDS_FLOATS, "fp32 tiles exceed the LDS buffer");
static_assert(2 * 4 * 3 * 4 * 64 * 4 <= KS_OPER, "partial sums exceed the operand buffers");

typedef float (*KsLds)[16 * KS_RBMAX + KS_BROWS][KS_LDA];

// row tiles of the fp32 tiled path for M rows
__device__ __forceinline__ int ks_row_tiles(const Dev &d, int M) {
    const int NU = d.H / KS_TU;
    const int R0 = max(1, 256 / NU);
    return R0 * ((M + 128 * R0 - 1) / (128 * R0));
}

// The register stage of one K step: NPA A rows and two B rows per thread.
template <int NPA>
struct KsStage {
    float4 a[NPA], b0, b1;
};

// Every thread issues the same loads, none behind a branch (a pass past the
// tile re-reads its last row, and every thread loads a second B row), so
// that the wait for one stage never has to cover the next one as well.
template <int RB>
__device__ __forceinline__ void ks_load(KsStage<(16 * RB + 31) / 32> &S, const u64 *ptrs, int a_r, int a_k, int k0,
                                        int Kx, const float *bp0, const float *bp1) {
    constexpr int BM = 16 * RB, NPA = (BM + 31) / 32;
    const bool xp = k0 < Kx;   // uniform: a K step lies wholly in the input part or the history part
#pragma unroll
    for (int p = 0; p < NPA; ++p) {
        const int row = min(a_r + 32 * p, BM - 1);
        const float *src = reinterpret_cast<const float *>(ptrs[3 * row + (xp ? 2 : 1)]);
        S.a[p] = ldg<float4>(src + (xp ? k0 : k0 - Kx) + a_k);
    }
    S.b0 = ldg<float4>(bp0 + k0);
    S.b1 = ldg<float4>(bp1 + k0);
}

template <int RB>
__device__ __forceinline__ void ks_store(const KsStage<(16 * RB + 31) / 32> &S, KsLds As, int buf, int a_r, int a_k,
                                         bool has_b1) {
    constexpr int BM = 16 * RB, NPA = (BM + 31) / 32;
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (a_r + 32 * p < BM) *reinterpret_cast<float4 *>(&As[buf][a_r + 32 * p][a_k]) = S.a[p];
    *reinterpret_cast<float4 *>(&As[buf][BM + a_r][a_k]) = S.b0;
    if (has_b1) *reinterpret_cast<float4 *>(&As[buf][BM + 32 + a_r][a_k]) = S.b1;
}

// One K step of a wave of row group G: its row blocks G, G + 2, ... x
// (reset, update, candidate) over its 16 k of the step, four per MFMA. NG:
// the candidate gate's accumulator (2: input part, 3: history part). mid()
// is where the caller stores the next step's operands into the other LDS
// buffer: after the first k's MFMAs for row group 0, before any MFMA for row
// group 1, so that the stores of the two waves sharing a SIMD drain while the
// other wave's MFMAs run, rather than all between the last MFMA and the
// barrier (6-8% faster loops than storing after the MFMAs, and another 2-3%
// from staggering the two groups).
template <int RB, int G, int NG, class MID>
__device__ __forceinline__ void ks_step(f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], KsLds As, int buf,
                                        int rl, int kc, MID mid) {
    constexpr int NRB = (RB - G + 1) / 2;   // 0 for the second group of a one-block tile
    if constexpr (NRB == 0) {
        mid();
        return;
    }
    float4 a[NRB > 0 ? NRB : 1], b[3];
#pragma unroll
    for (int g = 0; g < 3; ++g) b[g] = *reinterpret_cast<const float4 *>(&As[buf][16 * RB + 16 * g + rl][kc]);
#pragma unroll
    for (int i = 0; i < NRB; ++i) a[i] = *reinterpret_cast<const float4 *>(&As[buf][16 * (G + 2 * i) + rl][kc]);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        if (c == (G == 0 ? 1 : 0)) mid();
#pragma unroll
        for (int i = 0; i < NRB; ++i) {
            acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[0][c], acc[i][0], 0, 0, 0);
            acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[1][c], acc[i][1], 0, 0, 0);
            acc[i][NG] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[2][c], acc[i][NG], 0, 0, 0);
        }
    }
}

// What the epilogue of a tile needs besides the partial sums.
struct KsEpi {
    const u64 *ptrs;     // per tile row: destination first (0 past M), then the sources
    const float *hprev;  // per tile row: h of the tile's units
    float br, bz, bn;    // this thread's unit's biases
    int j;               // this thread's unit
    size_t lofs;         // this layer's offset in a destination row
};

// The end of a tile, for the wave of row group G and K quarter q = w % 4,
// which holds NRB row blocks' four accumulators (reset, update, candidate
// input part, candidate history part). In one LDS round each wave stores the
// partial sums of the blocks it does not finish, [group][block][other
// quarter][part][lane], over the operand buffers; wave q then finishes its
// group's block q (when it has one): the four quarters' partials are added
// in quarter order (the same fixed order whichever wave finishes), and each
// lane applies the gates to its four rows of one unit. NP: u64 pointers per
// tile row (the destination first; with 5, the fifth is where the bf16 copy
// of h' goes for the next layer, or 0).
template <int RB, int G, int NP>
__device__ __forceinline__ void ks_gates(const f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], float *smem,
                                         const KsEpi &ep, int w, int lane, int tid) {
    constexpr int NRB = (RB - G + 1) / 2;
    static_assert(NRB <= 4, "a group has at most four row blocks");
    f4_t *red = reinterpret_cast<f4_t *>(smem);
    const int q = w & 3;   // wave-uniform
    // slot of block i's partial from quarter qq (qq != i), part g
    auto slot = [](int i, int qq, int g) { return ((G * 4 + i) * 3 + (qq - (qq > i))) * 4 + g; };
#pragma unroll
    for (int i = 0; i < NRB; ++i)
        if (i != q)
#pragma unroll
            for (int g = 0; g < 4; ++g) red[slot(i, q, g) * 64 + lane] = acc[i][g];
    __syncthreads();
    (void)tid;
    if (q >= NRB) return;   // wave-uniform: no block q in this group
    // the wave's own partial of block q, picked by a branch per quarter so
    // that the accumulators are only ever indexed by constants
    f4_t sum[4];
    auto finish = [&](auto QQc) {
        constexpr int QQ = decltype(QQc)::value;
        if constexpr (QQ < NRB) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                sum[g] = QQ == 0 ? acc[QQ][g] : red[slot(QQ, 0, g) * 64 + lane];
#pragma unroll
                for (int qq = 1; qq < 4; ++qq) sum[g] += qq == QQ ? acc[QQ][g] : red[slot(QQ, qq, g) * 64 + lane];
            }
        }
    };
    switch (q) {
        case 0: finish(std::integral_constant<int, 0>()); break;
        case 1: finish(std::integral_constant<int, 1>()); break;
        case 2: finish(std::integral_constant<int, 2>()); break;
        default: finish(std::integral_constant<int, 3>()); break;
    }
    // D[row][col] sits in lane 16 * (row / 4) + col, element row % 4
    const int eu = lane & 15;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int row = 16 * (G + 2 * q) + 4 * (lane >> 4) + e;
        const u64 dp = ep.ptrs[NP * row];
        if (dp) {
            const float rr = sigmoidf_(sum[0][e] + ep.br);
            const float z = sigmoidf_(sum[1][e] + ep.bz);
            const float n = tanhf(sum[2][e] + ep.bn + rr * sum[3][e]);
            const float hn = (1.0f - z) * n + z * ep.hprev[row * KS_TU + eu];
            reinterpret_cast<float *>(dp)[ep.lofs + ep.j] = hn;
            if constexpr (NP == 5) {
                const u64 xp = ep.ptrs[NP * row + 4];
                if (xp) reinterpret_cast<uint16_t *>(xp)[ep.j] = f32_to_bf16(hn);
            }
        }
    }
}

// The K loop, the partial sums and the gates, as run by a wave of row group
// G (wave-uniform). Every wave runs the same barriers whatever its group.
template <int RB, int G>
__device__ __forceinline__ void ks_waves(KsLds As, float *smem, const KsEpi &ep, int a_r, int a_k, int Kx, int nk,
                                         const float *bp0, const float *bp1, bool has_b1, int w, int lane, int tid) {
    constexpr int NPA = (16 * RB + 31) / 32;
    constexpr int NRB = (RB - G + 1) / 2;
    f4_t acc[NRB > 0 ? NRB : 1][4];   // [row block G + 2 i][reset, update, candidate input part, candidate history part]
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[i][g] = f4_t{0, 0, 0, 0};
    const int rl = lane & 15, kc = 16 * (w & 3) + 4 * (lane >> 4);
    // two register stages: the loads of step s + 2 are issued while step s
    // multiplies; S0 carries the odd steps and S1 the even ones from step 2
    // on, and LDS buffer s & 1 holds step s (step 0 is in LDS already)
    KsStage<NPA> S0, S1;
    ks_load<RB>(S0, ep.ptrs, a_r, a_k, KS_BK, Kx, bp0, bp1);
    ks_load<RB>(S1, ep.ptrs, a_r, a_k, min(2, nk - 1) * KS_BK, Kx, bp0, bp1);
    // step kt: multiply LDS buffer kt & 1; store the stage holding step kt + 1
    // into the other buffer (during the MFMAs: every wave passed the previous
    // step's barrier, so nobody reads that buffer any more) and load step
    // kt + 3 into it (S0 holds the odd steps, S1 the even ones); NG: the
    // candidate gate's accumulator. The input part's steps come first, then
    // the history part's, each in a loop of its own, so that no branch
    // between MFMAs picks the accumulator.
    auto step = [&](int kt, auto NGc, auto PARc) {
        constexpr int NG = decltype(NGc)::value, PAR = decltype(PARc)::value;
        KsStage<NPA> &St = PAR == 0 ? S0 : S1;
        ks_step<RB, G, NG>(acc, As, PAR, rl, kc, [&] {
            if (kt + 1 < nk) ks_store<RB>(St, As, 1 - PAR, a_r, a_k, has_b1);
        });
        // past the last step the stage re-reads the last step (unused), so
        // that every step issues the same loads and the waits stay exact
        ks_load<RB>(St, ep.ptrs, a_r, a_k, min(kt + 3, nk - 1) * KS_BK, Kx, bp0, bp1);
        __syncthreads();
    };
    using X = std::integral_constant<int, 2>;
    using Hh = std::integral_constant<int, 3>;
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    const int nx = Kx / KS_BK;
    int kt = 0;
    for (; kt + 1 < nx; kt += 2) {
        step(kt, X(), P0());
        step(kt + 1, X(), P1());
    }
    if (kt < nx) step(kt++, X(), P0());
    if (kt & 1) step(kt++, Hh(), P1());
    for (; kt + 1 < nk; kt += 2) {
        step(kt, Hh(), P0());
        step(kt + 1, Hh(), P1());
    }
    if (kt < nk) step(kt, Hh(), P0());
    ks_gates<RB, G, 3>(acc, smem, ep, w, lane, tid);
}

template <int RB>
__device__ __forceinline__ void gru_ks_f32(const Dev &d, const Rows &R, int layer, int M, float *smem, int tile, int NR) {
    constexpr int BM = 16 * RB;
    constexpr int NPA = (BM + 31) / 32;   // A rows per loading thread
    const int NU = d.H / KS_TU;
    int rt, ut;
    if ((NU & 7) == 0) {   // every XCD keeps its own unit tiles (and their weights in its L2)
        const int xcd = tile & 7, idx = tile >> 3, per = NU >> 3;
        rt = idx / per;
        ut = xcd + 8 * (idx % per);
    } else {
        rt = tile / NU;
        ut = tile % NU;
    }
    const int m0 = rt * BM, j0 = ut * KS_TU;
    if (rt >= NR || m0 >= M) return;   // block-uniform

    KsLds As = reinterpret_cast<KsLds>(smem);               // rows 0..BM-1: A, then the 48 B rows
    u64 *ptrs = reinterpret_cast<u64 *>(smem + KS_PTRS);   // [BM][3]; the sources point at this layer's part
    float *hprev = smem + KS_HPREV;                         // [BM][16]

    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const float *Wp = reinterpret_cast<const float *>(d.Wl);

    // the tile's row pointers: destination (0 past M), history source and
    // input source; rows past M read row M - 1 (their products only reach
    // rows the epilogue skips, and no select sits between a load and its use)
    if (tid < BM) {
        const int m = min(m0 + tid, M - 1);
        const RowSrc src = row_source(d, R, layer, m, M);
        ptrs[3 * tid] = m0 + tid < M ? (u64)row_at(R, d.f_rowdst, m) : 0;
        ptrs[3 * tid + 1] = (u64)src.h;
        ptrs[3 * tid + 2] = (u64)src.x;
    }
    __syncthreads();
    // A loader: rows tid/16 + 32 p, 4 consecutive k at 4 (tid % 16). B
    // loader: weight rows tid/16 (and tid/16 + 32 for tid < 256): gate
    // row / 16, unit row % 16
    const int a_r = tid >> 4, a_k = (tid & 15) * 4;
    const float *bp0 = Wp + (size_t)((a_r >> 4) * d.H + j0 + (a_r & 15)) * K + a_k;
    const float *bp1 = Wp + (size_t)(2 * d.H + j0 + (a_r & 15)) * K + a_k;
    const bool has_b1 = tid < 256;   // wave-uniform

    // step 0 into LDS, with the epilogue's h (the tile's 16 units of each
    // row's history): thread (row i, unit u) for rows i = tid/16 + 32 p
    const int hi = tid >> 4, hu = tid & 15;
    float hv[NPA];
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (hi + 32 * p < BM) hv[p] = reinterpret_cast<const float *>(ptrs[3 * (hi + 32 * p) + 1])[j0 + hu];
    KsEpi ep;
    ep.ptrs = ptrs;
    ep.hprev = hprev;
    ep.j = j0 + hu;
    ep.br = d.bl[ep.j];
    ep.bz = d.bl[d.H + ep.j];
    ep.bn = d.bl[2 * d.H + ep.j];
    ep.lofs = (size_t)layer * d.H;
    {
        KsStage<NPA> S;
        ks_load<RB>(S, ptrs, a_r, a_k, 0, Kx, bp0, bp1);
        ks_store<RB>(S, As, 0, a_r, a_k, has_b1);
    }
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (hi + 32 * p < BM) hprev[(hi + 32 * p) * KS_TU + hu] = hv[p];
    __syncthreads();
    const int nk = K / KS_BK;   // >= 2: E, H are multiples of 64
    if (w < 4) ks_waves<RB, 0>(As, smem, ep, a_r, a_k, Kx, nk, bp0, bp1, has_b1, w, lane, tid);
    else ks_waves<RB, 1>(As, smem, ep, a_r, a_k, Kx, nk, bp0, bp1, has_b1, w, lane, tid);
    __syncthreads();   // LDS is reused by the next tile
}

// start of row m of a per-session per-row array of `stride` elements
template <class T>
__device__ __forceinline__ T *row_ptr(const Rows &R, T *arr, int m, size_t stride) {
    long long o = R.sofs[0];
    int base = 0;
    if (R.n > 1) {   // uniform
#pragma unroll
        for (int e = 1; e < kMaxSessions; ++e)
            if (e < R.n && m >= R.moff[e]) {
                o = R.sofs[e];
                base = R.moff[e];
            }
    }
    return shift_ptr(arr, o) + (size_t)(m - base) * stride;
}

// Many rows (more than one 16-unit tile per CU): fp32 tiles of 16 RB rows x
// 64 hidden units (192 weight rows), 32-k steps (128 bytes per operand row;
// E and H are multiples of 64, so a step lies wholly in one part). Wave
// w = 4 g + uq takes row blocks g, g + 2, ... and units 16 uq .. + 15 over the
// whole step: per row block and gate, two float4 fragments of 16 k, four
// 16x16x4 MFMAs each, and no partial sums to exchange. Each step carries
// twice the MFMA work of a 16-unit tile's step, with a quarter of the tiles
// (12-13% faster at 2048-16384 rows; at most 512 rows, where 16-unit tiles
// make one per CU, 64-unit tiles would leave each wave a single row block).
constexpr int KF_TU = 64;                                  // hidden units per tile
constexpr int KF_BROWS = 3 * KF_TU;                        // weight rows per tile
constexpr int KF_BK = 32;                                  // K step (floats)
constexpr int KF_LDA = 40;                                 // LDS row (floats): 128 bytes of operands, 32 of padding
constexpr int KF_ROWS = 16 * KS_RBMAX + KF_BROWS;
constexpr int KF_OPER = 2 * KF_ROWS * KF_LDA;              // two operand buffers (floats)
constexpr int KF_PTRS = KF_OPER;                           // per tile row: destination, history source, input source
constexpr int KF_HPREV = KF_PTRS + 16 * KS_RBMAX * 6;      // per tile row: h of the tile's 64 units
static_assert(KF_HPREV + 16 * KS_RBMAX * KF_TU <= G_LDS_FLOATS, "64-unit fp32 tiles exceed the LDS buffer");

typedef float (*KfLds)[KF_ROWS][KF_LDA];

__device__ __forceinline__ int kf_row_tiles(const Dev &d, int M) {
    const int NU = d.H / KF_TU;
    const int R0 = max(1, 256 / NU);
    return R0 * ((M + 128 * R0 - 1) / (128 * R0));
}

// A thread's share of one K step: 16-byte chunk t % 8 of A rows t / 8 and
// t / 8 + 64 and of weight rows t / 8, t / 8 + 64, t / 8 + 128 (gate 0, 1, 2
// of unit t / 8).
struct KfStage {
    float4 a0, a1, b0, b1, b2;
};

template <int RB>
__device__ __forceinline__ void kf_load(KfStage &S, const u64 *ptrs, int a_r, int a_c4, int k0, int Kx,
                                        const float *bp, size_t bstride) {
    constexpr int BM = 16 * RB;
    const bool xp = k0 < Kx;   // uniform
    const int ko = (xp ? k0 : k0 - Kx) + a_c4;
    const int r0 = min(a_r, BM - 1), r1 = min(a_r + 64, BM - 1);
    S.a0 = ldg<float4>(reinterpret_cast<const float *>(ptrs[3 * r0 + (xp ? 2 : 1)]) + ko);
    S.a1 = ldg<float4>(reinterpret_cast<const float *>(ptrs[3 * r1 + (xp ? 2 : 1)]) + ko);
    S.b0 = ldg<float4>(bp + k0);
    S.b1 = ldg<float4>(bp + bstride + k0);
    S.b2 = ldg<float4>(bp + 2 * bstride + k0);
}

template <int RB>
__device__ __forceinline__ void kf_store(const KfStage &S, KfLds As, int buf, int a_r, int a_c4) {
    constexpr int BM = 16 * RB;
    if (a_r < BM) *reinterpret_cast<float4 *>(&As[buf][a_r][a_c4]) = S.a0;
    if (a_r + 64 < BM) *reinterpret_cast<float4 *>(&As[buf][a_r + 64][a_c4]) = S.a1;
    *reinterpret_cast<float4 *>(&As[buf][BM + a_r][a_c4]) = S.b0;
    *reinterpret_cast<float4 *>(&As[buf][BM + 64 + a_r][a_c4]) = S.b1;
    *reinterpret_cast<float4 *>(&As[buf][BM + 128 + a_r][a_c4]) = S.b2;
}

// One K step of a wave of row group G and unit quarter uq. mid() runs after
// the first row block's MFMAs (before them with one row block).
template <int RB, int G, int NG, class MID>
__device__ __forceinline__ void kf_step(f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], KfLds As,
                                        int buf, int rl, int kc, int uq, MID mid) {
    constexpr int NRB = (RB - G + 1) / 2;
    if constexpr (NRB == 0) {
        mid();
        return;
    }
    // the step's two 16-k halves one after the other: seven fragments live at a time
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        float4 b[3], a[NRB > 0 ? NRB : 1];
#pragma unroll
        for (int q = 0; q < 3; ++q)
            b[q] = *reinterpret_cast<const float4 *>(&As[buf][16 * RB + 64 * q + 16 * uq + rl][kc + 16 * h]);
#pragma unroll
        for (int i = 0; i < NRB; ++i) a[i] = *reinterpret_cast<const float4 *>(&As[buf][16 * (G + 2 * i) + rl][kc + 16 * h]);
#pragma unroll
        for (int i = 0; i < NRB; ++i) {
            if (h == 0 && (i == 1 || NRB == 1)) mid();
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[0][c], acc[i][0], 0, 0, 0);
                acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[1][c], acc[i][1], 0, 0, 0);
                acc[i][NG] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][c], b[2][c], acc[i][NG], 0, 0, 0);
            }
        }
    }
}

template <int RB, int G>
__device__ __forceinline__ void kf_gates(const f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4],
                                         const KsEpi &ep, int uq, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    const int eu = lane & 15;
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        // D[row][col] sits in lane 16 * (row / 4) + col, element row % 4
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = 16 * (G + 2 * i) + 4 * (lane >> 4) + e;
            const u64 dp = ep.ptrs[3 * row];
            if (dp) {
                const float rr = sigmoidf_(acc[i][0][e] + ep.br);
                const float z = sigmoidf_(acc[i][1][e] + ep.bz);
                const float n = tanhf(acc[i][2][e] + ep.bn + rr * acc[i][3][e]);
                const float hn = (1.0f - z) * n + z * ep.hprev[row * KF_TU + 16 * uq + eu];
                reinterpret_cast<float *>(dp)[ep.lofs + ep.j] = hn;
            }
        }
    }
}

template <int RB, int G>
__device__ __forceinline__ void kf_waves(KfLds As, const KsEpi &ep, int a_r, int a_c4, int Kx, int K, const float *bp,
                                         size_t bstride, int w, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    f4_t acc[NRB > 0 ? NRB : 1][4];   // [row block G + 2 i][reset, update, candidate input part, history part]
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = f4_t{0, 0, 0, 0};
    const int uq = w & 3;
    const int rl = lane & 15, kc = 4 * (lane >> 4);
    const int nk = K / KF_BK, nx = Kx / KF_BK;   // nx >= 2
    KfStage S0, S1;
    kf_load<RB>(S0, ep.ptrs, a_r, a_c4, KF_BK, Kx, bp, bstride);
    kf_load<RB>(S1, ep.ptrs, a_r, a_c4, 2 * KF_BK, Kx, bp, bstride);
    auto step = [&](int kt, auto NGc, auto PARc) {
        constexpr int NG = decltype(NGc)::value, PAR = decltype(PARc)::value;
        KfStage &St = PAR == 0 ? S0 : S1;
        kf_step<RB, G, NG>(acc, As, PAR, rl, kc, uq, [&] {
            if (kt + 1 < nk) kf_store<RB>(St, As, 1 - PAR, a_r, a_c4);
        });
        // past the last step the stage re-reads the last step (unused)
        kf_load<RB>(St, ep.ptrs, a_r, a_c4, min(kt + 3, nk - 1) * KF_BK, Kx, bp, bstride);
        __syncthreads();
    };
    using X = std::integral_constant<int, 2>;
    using Hh = std::integral_constant<int, 3>;
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    int kt = 0;
    for (; kt + 1 < nx; kt += 2) {
        step(kt, X(), P0());
        step(kt + 1, X(), P1());
    }
    if (kt < nx) step(kt++, X(), P0());
    if (kt & 1) step(kt++, Hh(), P1());
    for (; kt + 1 < nk; kt += 2) {
        step(kt, Hh(), P0());
        step(kt + 1, Hh(), P1());
    }
    if (kt < nk) step(kt, Hh(), P0());
    kf_gates<RB, G>(acc, ep, uq, lane);
}

template <int RB>
__device__ __forceinline__ void gru_kf_f32(const Dev &d, const Rows &R, int layer, int M, float *smem, int tile,
                                           int NR) {
    constexpr int BM = 16 * RB;
    const int NU = d.H / KF_TU;
    int rt, ut;
    if ((NU & 7) == 0) {   // every XCD keeps its own unit tiles
        const int xcd = tile & 7, idx = tile >> 3, per = NU >> 3;
        rt = idx / per;
        ut = xcd + 8 * (idx % per);
    } else {
        rt = tile / NU;
        ut = tile % NU;
    }
    const int m0 = rt * BM, j0 = ut * KF_TU;
    if (rt >= NR || m0 >= M) return;   // block-uniform

    KfLds As = reinterpret_cast<KfLds>(smem);
    u64 *ptrs = reinterpret_cast<u64 *>(smem + KF_PTRS);   // [BM][3]
    float *hprev = smem + KF_HPREV;                         // [BM][64]
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const float *Wp = reinterpret_cast<const float *>(d.Wl);
    // the tile's row pointers, as for the 16-unit tiles
    if (tid < BM) {
        const int m = min(m0 + tid, M - 1);
        const RowSrc src = row_source(d, R, layer, m, M);
        ptrs[3 * tid] = m0 + tid < M ? (u64)row_at(R, d.f_rowdst, m) : 0;
        ptrs[3 * tid + 1] = (u64)src.h;
        ptrs[3 * tid + 2] = (u64)src.x;
    }
    __syncthreads();
    // loaders: rows tid / 8 (+ 64), chunk tid % 8 of 4 floats; weight rows
    // j0 + tid / 8 of each gate
    const int a_r = tid >> 3, a_c4 = (tid & 7) * 4;
    const float *bp = Wp + (size_t)(j0 + a_r) * K + a_c4;
    const size_t bstride = (size_t)d.H * K;
    // step 0 into LDS, with the epilogue's h: thread (row tid / 64 + 8 p, unit tid % 64)
    const int hi = tid >> 6, hu = tid & 63;
    float hv[2 * RB];
#pragma unroll
    for (int p = 0; p < 2 * RB; ++p) hv[p] = reinterpret_cast<const float *>(ptrs[3 * (hi + 8 * p) + 1])[j0 + hu];
    KsEpi ep;
    ep.ptrs = ptrs;
    ep.hprev = hprev;
    ep.j = j0 + 16 * (w & 3) + (lane & 15);
    ep.br = d.bl[ep.j];
    ep.bz = d.bl[d.H + ep.j];
    ep.bn = d.bl[2 * d.H + ep.j];
    ep.lofs = (size_t)layer * d.H;
    {
        KfStage S;
        kf_load<RB>(S, ptrs, a_r, a_c4, 0, Kx, bp, bstride);
        kf_store<RB>(S, As, 0, a_r, a_c4);
    }
#pragma unroll
    for (int p = 0; p < 2 * RB; ++p) hprev[(hi + 8 * p) * KF_TU + hu] = hv[p];
    __syncthreads();
    if (w < 4) kf_waves<RB, 0>(As, ep, a_r, a_c4, Kx, K, bp, bstride, w, lane);
    else kf_waves<RB, 1>(As, ep, a_r, a_c4, Kx, K, bp, bstride, w, lane);
    __syncthreads();   // LDS is reused by the next tile
}

// ---------------- tiled path (33 rows and more): bf16, 16-unit tiles --------
// For few rows, while 32-unit tiles would be at most two row blocks high
// (at H = 1024, 256 rows): their eight row tiles per unit tile pad such row
// counts to whole row blocks and take twice the K steps, and these tiles
// measured 1-8 us faster per launch at 33-256 rows. The fp32 tile's shape
// and schedule (16 RB rows x 16 hidden units, 8 waves as
// 2 row groups x 4 K quarters, double-buffered LDS, loads three steps ahead)
// with bf16 operands: the history rows were rounded once per frame by the
// keys kernel, and the second layer's input is the bf16 copy of the first
// layer's h' that its tiles' epilogue writes. A step is 128 k, i.e. the same
// 256 bytes per operand row as an fp32 step, so the LDS layout and every LDS
// address are the fp32 tile's; a wave's quarter is 32 k, one 16 x 16 x 32 MFMA
// per row block and gate part. A step may straddle the input / history
// boundary or reach past K (E and H are multiples of 64): each 8-k chunk is
// loaded from its own part (clamped inside K), and a wave's quarter, which
// lies wholly in one part (or past K), feeds zeros to the candidate gate's
// other accumulator (or to every product).
constexpr int KSB_BK = 128;                               // K step (bf16 elements)
constexpr int KSB_PTRS = KS_OPER;                         // per tile row: dst, h fp32, h bf16, x bf16, x copy dst
constexpr int KSB_HPREV = KSB_PTRS + 16 * KS_RBMAX * 10;  // per tile row: h of the tile's 16 units
static_assert(KSB_HPREV + 16 * KS_RBMAX * KS_TU <= G_LDS_FLOATS, "bf16 tiles exceed the LDS buffer");

template <int NPA>
struct KsbStage {
    uint4 a[NPA], b0, b1;
};

// Every thread issues the same loads, none behind a branch: a chunk past K
// re-reads the last chunk inside K (its products are zeroed), rows past the
// tile re-read its last row. bp0, bp1: the starts of the thread's weight rows.
template <int RB>
__device__ __forceinline__ void ksb_load(KsbStage<(16 * RB + 31) / 32> &S, const u64 *ptrs, int a_r, int a_k, int k0,
                                         int Kx, int K, const uint16_t *bp0, const uint16_t *bp1) {
    constexpr int BM = 16 * RB, NPA = (BM + 31) / 32;
    const int k = min(k0 + a_k, K - 8);
    const bool xp = k < Kx;
#pragma unroll
    for (int p = 0; p < NPA; ++p) {
        const int row = min(a_r + 32 * p, BM - 1);
        const uint16_t *src = reinterpret_cast<const uint16_t *>(ptrs[5 * row + (xp ? 3 : 2)]);
        S.a[p] = ldg<uint4>(src + (xp ? k : k - Kx));
    }
    S.b0 = ldg<uint4>(bp0 + k);
    S.b1 = ldg<uint4>(bp1 + k);
}

template <int RB>
__device__ __forceinline__ void ksb_store(const KsbStage<(16 * RB + 31) / 32> &S, KsLds As, int buf, int a_r, int a_c,
                                          bool has_b1) {
    constexpr int BM = 16 * RB, NPA = (BM + 31) / 32;
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (a_r + 32 * p < BM) *reinterpret_cast<uint4 *>(&As[buf][a_r + 32 * p][a_c]) = S.a[p];
    *reinterpret_cast<uint4 *>(&As[buf][BM + a_r][a_c]) = S.b0;
    if (has_b1) *reinterpret_cast<uint4 *>(&As[buf][BM + 32 + a_r][a_c]) = S.b1;
}

// One K step of a wave of row group G: its row blocks G, G + 2, ... x
// (reset, update, candidate input part, candidate history part) over its 32 k
// of the step. live: the quarter lies inside K; xp: in the input part. mid()
// runs after the first row block's MFMAs (before them with one row block), as
// in the fp32 step.
template <int RB, int G, class MID>
__device__ __forceinline__ void ksb_step(f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], KsLds As,
                                         int buf, int rl, int kc, bool live, bool xp, MID mid) {
    constexpr int NRB = (RB - G + 1) / 2;
    if constexpr (NRB == 0) {
        mid();
        return;
    }
    const uint4 z = make_uint4(0, 0, 0, 0);
    uint4 g[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) g[q] = *reinterpret_cast<const uint4 *>(&As[buf][16 * RB + 16 * q + rl][kc]);
    bf8_t b[4];
    b[0] = __builtin_bit_cast(bf8_t, g[0]);
    b[1] = __builtin_bit_cast(bf8_t, g[1]);
    b[2] = __builtin_bit_cast(bf8_t, xp ? g[2] : z);
    b[3] = __builtin_bit_cast(bf8_t, xp ? z : g[2]);
    bf8_t a[NRB > 0 ? NRB : 1];
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        const uint4 v = *reinterpret_cast<const uint4 *>(&As[buf][16 * (G + 2 * i) + rl][kc]);
        a[i] = __builtin_bit_cast(bf8_t, live ? v : z);
    }
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        if (i == 1 || (NRB == 1 && i == 0)) mid();
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[q], acc[i][q], 0, 0, 0);
    }
}

template <int RB, int G>
__device__ __forceinline__ void ksb_waves(KsLds As, float *smem, const KsEpi &ep, int a_r, int a_k, int a_c, int Kx,
                                          int K, const uint16_t *bp0, const uint16_t *bp1, bool has_b1, int w,
                                          int lane, int tid) {
    constexpr int NPA = (16 * RB + 31) / 32;
    constexpr int NRB = (RB - G + 1) / 2;
    f4_t acc[NRB > 0 ? NRB : 1][4];   // [row block G + 2 i][reset, update, candidate input part, history part]
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = f4_t{0, 0, 0, 0};
    const int rl = lane & 15, kc = 16 * (w & 3) + 4 * (lane >> 4);   // kc in floats: bf16 k = 32 (w % 4) + 8 (lane / 16)
    const int ns = (K + KSB_BK - 1) / KSB_BK;                         // >= 1
    // two register stages as in the fp32 tile: S0 carries the odd steps and
    // S1 the even ones from step 2 on; LDS buffer s & 1 holds step s
    KsbStage<NPA> S0, S1;
    ksb_load<RB>(S0, ep.ptrs, a_r, a_k, min(1, ns - 1) * KSB_BK, Kx, K, bp0, bp1);
    ksb_load<RB>(S1, ep.ptrs, a_r, a_k, min(2, ns - 1) * KSB_BK, Kx, K, bp0, bp1);
    auto step = [&](int st, auto PARc) {
        constexpr int PAR = decltype(PARc)::value;
        const int kq = st * KSB_BK + 32 * (w & 3);   // wave-uniform
        KsbStage<NPA> &St = PAR == 0 ? S0 : S1;
        ksb_step<RB, G>(acc, As, PAR, rl, kc, kq < K, kq < Kx, [&] {
            if (st + 1 < ns) ksb_store<RB>(St, As, 1 - PAR, a_r, a_c, has_b1);
        });
        // past the last step the stage re-reads the last step (unused), so
        // that every step issues the same loads and the waits stay exact
        ksb_load<RB>(St, ep.ptrs, a_r, a_k, min(st + 3, ns - 1) * KSB_BK, Kx, K, bp0, bp1);
        __syncthreads();
    };
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    int st = 0;
    for (; st + 1 < ns; st += 2) {
        step(st, P0());
        step(st + 1, P1());
    }
    if (st < ns) step(st, P0());
    ks_gates<RB, G, 5>(acc, smem, ep, w, lane, tid);
}

template <int RB>
__device__ __forceinline__ void gru_ks_bf16(const Dev &d, const Rows &R, int layer, int M, float *smem, int tile,
                                            int NR) {
    constexpr int BM = 16 * RB;
    constexpr int NPA = (BM + 31) / 32;
    const int NU = d.H / KS_TU;
    int rt, ut;
    if ((NU & 7) == 0) {   // every XCD keeps its own unit tiles (and their weights in its L2)
        const int xcd = tile & 7, idx = tile >> 3, per = NU >> 3;
        rt = idx / per;
        ut = xcd + 8 * (idx % per);
    } else {
        rt = tile / NU;
        ut = tile % NU;
    }
    const int m0 = rt * BM, j0 = ut * KS_TU;
    if (rt >= NR || m0 >= M) return;   // block-uniform

    KsLds As = reinterpret_cast<KsLds>(smem);
    u64 *ptrs = reinterpret_cast<u64 *>(smem + KSB_PTRS);   // [BM][5]
    float *hprev = smem + KSB_HPREV;                         // [BM][16]

    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const uint16_t *Wp = reinterpret_cast<const uint16_t *>(d.Wl);

    // the tile's row pointers (rows past M read row M - 1: their products
    // only reach rows the epilogue skips): destination, fp32 h (this layer's
    // part), bf16 h (this layer's part), bf16 x (embedding row, or the bf16
    // copy of the first layer's h'), and where the first layer's tiles put
    // that copy when there is a second layer
    if (tid < BM) {
        const int m = min(m0 + tid, M - 1);
        const bool live = m0 + tid < M;
        ptrs[5 * tid] = live ? row_at(R, d.f_rowdst, m) : 0;
        ptrs[5 * tid + 1] = row_at(R, d.f_rowh, m) + (u64)layer * d.H * 4;
        ptrs[5 * tid + 2] = row_at(R, d.f_rowhb, m) + (u64)layer * d.H * 2;
        ptrs[5 * tid + 3] = layer == 0 ? (u64)(reinterpret_cast<const uint16_t *>(d.emb) +
                                               (size_t)(unsigned)row_at(R, d.f_roww, m) * d.E)
                                       : (u64)row_ptr(R, d.f_xbf, m, d.H);
        ptrs[5 * tid + 4] = live && layer == 0 && d.L == 2 ? (u64)row_ptr(R, d.f_xbf, m, d.H) : 0;
    }
    __syncthreads();
    // A loader: rows tid/16 + 32 p, 8 consecutive k at 8 (tid % 16). B
    // loader: weight rows tid/16 (and tid/16 + 32 for tid < 256): gate
    // row / 16, unit row % 16. a_c: the chunk's LDS column in floats.
    const int a_r = tid >> 4, a_k = (tid & 15) * 8, a_c = (tid & 15) * 4;
    const uint16_t *bp0 = Wp + (size_t)((a_r >> 4) * d.H + j0 + (a_r & 15)) * K;   // row starts: the loads add k
    const uint16_t *bp1 = Wp + (size_t)(2 * d.H + j0 + (a_r & 15)) * K;
    const bool has_b1 = tid < 256;   // wave-uniform

    // step 0 into LDS, with the epilogue's fp32 h (the tile's 16 units of each
    // row's history): thread (row i, unit u) for rows i = tid/16 + 32 p
    const int hi = tid >> 4, hu = tid & 15;
    float hv[NPA];
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (hi + 32 * p < BM) hv[p] = reinterpret_cast<const float *>(ptrs[5 * (hi + 32 * p) + 1])[j0 + hu];
    KsEpi ep;
    ep.ptrs = ptrs;
    ep.hprev = hprev;
    ep.j = j0 + hu;
    ep.br = d.bl[ep.j];
    ep.bz = d.bl[d.H + ep.j];
    ep.bn = d.bl[2 * d.H + ep.j];
    ep.lofs = (size_t)layer * d.H;
    {
        KsbStage<NPA> S;
        ksb_load<RB>(S, ptrs, a_r, a_k, 0, Kx, K, bp0, bp1);
        ksb_store<RB>(S, As, 0, a_r, a_c, has_b1);
    }
#pragma unroll
    for (int p = 0; p < NPA; ++p)
        if (hi + 32 * p < BM) hprev[(hi + 32 * p) * KS_TU + hu] = hv[p];
    __syncthreads();
    if (w < 4) ksb_waves<RB, 0>(As, smem, ep, a_r, a_k, a_c, Kx, K, bp0, bp1, has_b1, w, lane, tid);
    else ksb_waves<RB, 1>(As, smem, ep, a_r, a_k, a_c, Kx, K, bp0, bp1, has_b1, w, lane, tid);
    __syncthreads();   // LDS is reused by the next tile
}

// --------------- tiled path (more rows): bf16, 32- and 64-unit tiles --------
// 16 RB rows x 32 hidden units (96 weight rows) per tile, 64-k steps (128
// bytes per operand row), double-buffered LDS and two register stages as in
// the fp32 tile. E and H are multiples of 64, so a step lies wholly in the
// input part or the history part. The 8 waves are 2 row groups x 2 unit
// halves x 2 K halves: wave w = 4 g + 2 uh + kh takes row blocks g, g + 2,
// ..., units 16 uh .. 16 uh + 15 of the tile and k = 32 kh .. 32 kh + 31 of
// each step, one 16 x 16 x 32 MFMA per row block and gate. Waves w and w + 4
// (one of each row group) share a SIMD. The history rows were rounded to
// bf16 once per frame by the keys kernel, and the second layer's input is the
// bf16 copy of the first layer's h' that its tiles' epilogue writes. Twice as
// wide as the fp32 tile: a bf16 step's MFMAs are short, so each tile's fixed
// cost (row pointers, first steps, gates) and each step's LDS round are
// spread over twice the MFMA work, with half as many tiles.
constexpr int KW_TU = 32;                                  // hidden units per tile
constexpr int KW_BROWS = 3 * KW_TU;                        // weight rows per tile
constexpr int KW_BK = 64;                                  // K step (bf16 elements)
constexpr int KW_LDA = 40;                                 // LDS row (floats): 128 bytes of operands, 32 of padding
constexpr int KW_ROWS = 16 * KS_RBMAX + KW_BROWS;
constexpr int KW_OPER = 2 * KW_ROWS * KW_LDA;              // two operand buffers (floats)
constexpr int KW_PTRS = KW_OPER;                           // per tile row: dst, h fp32, h bf16, x bf16, x copy dst
constexpr int KW_HPREV = KW_PTRS + 16 * KS_RBMAX * 10;     // per tile row: h of the tile's 32 units
static_assert(KW_HPREV + 16 * KS_RBMAX * KW_TU <= G_LDS_FLOATS, "wide bf16 tiles exceed the LDS buffer");
static_assert(2 * 2 * 4 * 4 * 64 * 4 <= KW_OPER, "partial sums exceed the operand buffers");

typedef float (*KwLds)[KW_ROWS][KW_LDA];

// row tiles of the wide bf16 path for M rows (about one tile per CU)
__device__ __forceinline__ int kw_row_tiles(const Dev &d, int M) {
    const int NU = d.H / KW_TU;
    const int R0 = max(1, 256 / NU);
    return R0 * ((M + 128 * R0 - 1) / (128 * R0));
}

// A thread's share of one K step: 16-byte chunk t % 8 of A rows t / 8 and
// t / 8 + 64 and of weight rows t / 8 and t / 8 + 64 (the second weight row
// for t < 256 only: a tile has 96).
struct KwStage {
    uint4 a0, a1, b0, b1;
};

// Every thread issues the same loads: rows past the tile re-read its last
// row, and a thread with no second weight row re-reads its first. bp0, bp1:
// the thread's chunk of its weight rows at k = 0.
template <int RB>
__device__ __forceinline__ void kw_load(KwStage &S, const u64 *ptrs, int a_r, int a_c8, int k0, int Kx,
                                        const uint16_t *bp0, const uint16_t *bp1) {
    constexpr int BM = 16 * RB;
    const bool xp = k0 < Kx;   // uniform: a step lies wholly in one part
    const int ko = (xp ? k0 : k0 - Kx) + a_c8;
    const int r0 = min(a_r, BM - 1), r1 = min(a_r + 64, BM - 1);
    S.a0 = ldg<uint4>(reinterpret_cast<const uint16_t *>(ptrs[5 * r0 + (xp ? 3 : 2)]) + ko);
    S.a1 = ldg<uint4>(reinterpret_cast<const uint16_t *>(ptrs[5 * r1 + (xp ? 3 : 2)]) + ko);
    S.b0 = ldg<uint4>(bp0 + k0);
    S.b1 = ldg<uint4>(bp1 + k0);
}

template <int RB>
__device__ __forceinline__ void kw_store(const KwStage &S, KwLds As, int buf, int a_r, int a_cf, bool has_b1) {
    constexpr int BM = 16 * RB;
    if (a_r < BM) *reinterpret_cast<uint4 *>(&As[buf][a_r][a_cf]) = S.a0;
    if (a_r + 64 < BM) *reinterpret_cast<uint4 *>(&As[buf][a_r + 64][a_cf]) = S.a1;
    *reinterpret_cast<uint4 *>(&As[buf][BM + a_r][a_cf]) = S.b0;
    if (has_b1) *reinterpret_cast<uint4 *>(&As[buf][BM + 64 + a_r][a_cf]) = S.b1;
}

// One K step of a wave of row group G and unit half uh: its row blocks G, G +
// 2, ... x (reset, update, candidate) over its 32 k of the step. NG: the
// candidate gate's accumulator (2: input part, 3: history part). mid() runs
// after the first row block's MFMAs (before them with one row block).
template <int RB, int G, int NG, class MID>
__device__ __forceinline__ void kw_step(f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], KwLds As,
                                        int buf, int rl, int kc, int uh, MID mid) {
    constexpr int NRB = (RB - G + 1) / 2;
    if constexpr (NRB == 0) {
        mid();
        return;
    }
    bf8_t b[3];
#pragma unroll
    for (int q = 0; q < 3; ++q)
        b[q] = __builtin_bit_cast(bf8_t, *reinterpret_cast<const uint4 *>(&As[buf][16 * RB + 32 * q + 16 * uh + rl][kc]));
    bf8_t a[NRB > 0 ? NRB : 1];
#pragma unroll
    for (int i = 0; i < NRB; ++i)
        a[i] = __builtin_bit_cast(bf8_t, *reinterpret_cast<const uint4 *>(&As[buf][16 * (G + 2 * i) + rl][kc]));
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        if (i == 1 || NRB == 1) mid();
        acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[0], acc[i][0], 0, 0, 0);
        acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[1], acc[i][1], 0, 0, 0);
        acc[i][NG] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[2], acc[i][NG], 0, 0, 0);
    }
}

// The end of a wide tile, for the wave of row group G, unit half uh and K
// half kh. Each wave stores the partial sums of the row blocks the other K
// half finishes ([group][unit half][block][part][lane], over the operand
// buffers); after one barrier the wave of K half i % 2 finishes block i: its
// partial plus the other half's (two terms, so the sum is the same whichever
// wave adds them), and each lane applies the gates to its four rows of one
// unit.
template <int RB, int G>
__device__ __forceinline__ void kw_gates(const f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4],
                                         float *smem, const KsEpi &ep, int uh, int kh, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    static_assert(NRB <= 4, "a group has at most four row blocks");
    f4_t *red = reinterpret_cast<f4_t *>(smem);
    auto slot = [&](int i, int g) { return (((G * 2 + uh) * 4 + i) * 4 + g) * 64 + lane; };
#pragma unroll
    for (int i = 0; i < NRB; ++i)
        if ((i & 1) != kh)
#pragma unroll
            for (int g = 0; g < 4; ++g) red[slot(i, g)] = acc[i][g];
    __syncthreads();
    const int eu = lane & 15;
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        if ((i & 1) != kh) continue;   // wave-uniform
        f4_t sum[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) sum[g] = acc[i][g] + red[slot(i, g)];
        // D[row][col] sits in lane 16 * (row / 4) + col, element row % 4
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = 16 * (G + 2 * i) + 4 * (lane >> 4) + e;
            const u64 dp = ep.ptrs[5 * row];
            if (dp) {
                const float rr = sigmoidf_(sum[0][e] + ep.br);
                const float z = sigmoidf_(sum[1][e] + ep.bz);
                const float n = tanhf(sum[2][e] + ep.bn + rr * sum[3][e]);
                const float hn = (1.0f - z) * n + z * ep.hprev[row * KW_TU + 16 * uh + eu];
                reinterpret_cast<float *>(dp)[ep.lofs + ep.j] = hn;
                const u64 xp = ep.ptrs[5 * row + 4];
                if (xp) reinterpret_cast<uint16_t *>(xp)[ep.j] = f32_to_bf16(hn);
            }
        }
    }
}

template <int RB, int G>
__device__ __forceinline__ void kw_waves(KwLds As, float *smem, const KsEpi &ep, int a_r, int a_c8, int a_cf,
                                         int Kx, int K, const uint16_t *bp0, const uint16_t *bp1, bool has_b1,
                                         int w, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    f4_t acc[NRB > 0 ? NRB : 1][4];   // [row block G + 2 i][reset, update, candidate input part, history part]
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = f4_t{0, 0, 0, 0};
    const int uh = (w >> 1) & 1, kh = w & 1;
    const int rl = lane & 15, kc = 16 * kh + 4 * (lane >> 4);   // kc in floats: bf16 k = 32 kh + 8 (lane / 16)
    const int nk = K / KW_BK, nx = Kx / KW_BK;                    // nk >= 2
    // S0 carries the odd steps and S1 the even ones from step 2 on; LDS
    // buffer s & 1 holds step s (step 0 is in LDS already)
    KwStage S0, S1;
    kw_load<RB>(S0, ep.ptrs, a_r, a_c8, KW_BK, Kx, bp0, bp1);
    kw_load<RB>(S1, ep.ptrs, a_r, a_c8, min(2, nk - 1) * KW_BK, Kx, bp0, bp1);
    auto step = [&](int kt, auto NGc, auto PARc) {
        constexpr int NG = decltype(NGc)::value, PAR = decltype(PARc)::value;
        KwStage &St = PAR == 0 ? S0 : S1;
        kw_step<RB, G, NG>(acc, As, PAR, rl, kc, uh, [&] {
            if (kt + 1 < nk) kw_store<RB>(St, As, 1 - PAR, a_r, a_cf, has_b1);
        });
        // past the last step the stage re-reads the last step (unused)
        kw_load<RB>(St, ep.ptrs, a_r, a_c8, min(kt + 3, nk - 1) * KW_BK, Kx, bp0, bp1);
        __syncthreads();
    };
    using X = std::integral_constant<int, 2>;
    using Hh = std::integral_constant<int, 3>;
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    int kt = 0;
    for (; kt + 1 < nx; kt += 2) {
        step(kt, X(), P0());
        step(kt + 1, X(), P1());
    }
    if (kt < nx) step(kt++, X(), P0());
    if (kt & 1) step(kt++, Hh(), P1());
    for (; kt + 1 < nk; kt += 2) {
        step(kt, Hh(), P0());
        step(kt + 1, Hh(), P1());
    }
    if (kt < nk) step(kt, Hh(), P0());
    kw_gates<RB, G>(acc, smem, ep, uh, kh, lane);
}

template <int RB>
__device__ __forceinline__ void gru_kw_bf16(const Dev &d, const Rows &R, int layer, int M, float *smem, int tile,
                                            int NR) {
    constexpr int BM = 16 * RB;
    const int NU = d.H / KW_TU;
    int rt, ut;
    if ((NU & 7) == 0) {   // every XCD keeps its own unit tiles (and their weights in its L2)
        const int xcd = tile & 7, idx = tile >> 3, per = NU >> 3;
        rt = idx / per;
        ut = xcd + 8 * (idx % per);
    } else {
        rt = tile / NU;
        ut = tile % NU;
    }
    const int m0 = rt * BM, j0 = ut * KW_TU;
    if (rt >= NR || m0 >= M) return;   // block-uniform

    KwLds As = reinterpret_cast<KwLds>(smem);
    u64 *ptrs = reinterpret_cast<u64 *>(smem + KW_PTRS);   // [BM][5]
    float *hprev = smem + KW_HPREV;                         // [BM][32]

    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const uint16_t *Wp = reinterpret_cast<const uint16_t *>(d.Wl);

    // the tile's row pointers (rows past M read row M - 1: their products
    // only reach rows the epilogue skips): destination, fp32 h (this layer's
    // part), bf16 h (this layer's part), bf16 x (embedding row, or the bf16
    // copy of the first layer's h'), and where the first layer's tiles put
    // that copy when there is a second layer
    if (tid < BM) {
        const int m = min(m0 + tid, M - 1);
        const bool live = m0 + tid < M;
        ptrs[5 * tid] = live ? row_at(R, d.f_rowdst, m) : 0;
        ptrs[5 * tid + 1] = row_at(R, d.f_rowh, m) + (u64)layer * d.H * 4;
        ptrs[5 * tid + 2] = row_at(R, d.f_rowhb, m) + (u64)layer * d.H * 2;
        ptrs[5 * tid + 3] = layer == 0 ? (u64)(reinterpret_cast<const uint16_t *>(d.emb) +
                                               (size_t)(unsigned)row_at(R, d.f_roww, m) * d.E)
                                       : (u64)row_ptr(R, d.f_xbf, m, d.H);
        ptrs[5 * tid + 4] = live && layer == 0 && d.L == 2 ? (u64)row_ptr(R, d.f_xbf, m, d.H) : 0;
    }
    __syncthreads();
    // loaders: rows tid / 8 (+ 64), chunk tid % 8 (8 bf16 = 4 floats of an
    // LDS row); weight row b of the tile is gate b / 32, unit b % 32
    const int a_r = tid >> 3, a_c8 = (tid & 7) * 8, a_cf = (tid & 7) * 4;
    const bool has_b1 = tid < 256;   // wave-uniform
    const uint16_t *bp0 = Wp + (size_t)((a_r >> 5) * d.H + j0 + (a_r & 31)) * K + a_c8;
    const uint16_t *bp1 = has_b1 ? Wp + (size_t)(2 * d.H + j0 + a_r) * K + a_c8 : bp0;

    // step 0 into LDS, with the epilogue's fp32 h (the tile's 32 units of
    // each row's history): thread (row tid / 32 + 16 p, unit tid % 32)
    const int hi = tid >> 5, hu = tid & 31;
    float hv[RB];
#pragma unroll
    for (int p = 0; p < RB; ++p) hv[p] = reinterpret_cast<const float *>(ptrs[5 * (hi + 16 * p) + 1])[j0 + hu];
    KsEpi ep;
    ep.ptrs = ptrs;
    ep.hprev = hprev;
    ep.j = j0 + 16 * ((w >> 1) & 1) + (lane & 15);
    ep.br = d.bl[ep.j];
    ep.bz = d.bl[d.H + ep.j];
    ep.bn = d.bl[2 * d.H + ep.j];
    ep.lofs = (size_t)layer * d.H;
    {
        KwStage S;
        kw_load<RB>(S, ptrs, a_r, a_c8, 0, Kx, bp0, bp1);
        kw_store<RB>(S, As, 0, a_r, a_cf, has_b1);
    }
#pragma unroll
    for (int p = 0; p < RB; ++p) hprev[(hi + 16 * p) * KW_TU + hu] = hv[p];
    __syncthreads();
    if (w < 4) kw_waves<RB, 0>(As, smem, ep, a_r, a_c8, a_cf, Kx, K, bp0, bp1, has_b1, w, lane);
    else kw_waves<RB, 1>(As, smem, ep, a_r, a_c8, a_cf, Kx, K, bp0, bp1, has_b1, w, lane);
    __syncthreads();   // LDS is reused by the next tile
}

// Many rows (more than one 32-unit tile per CU): tiles of 16 RB rows x 64
// hidden units (192 weight rows), 64-k steps, the same loaders and LDS rows.
// Wave w = 4 g + uq takes row blocks g, g + 2, ... and units 16 uq .. + 15
// over the whole step (two 16 x 16 x 32 MFMAs per row block and gate), so the
// gates need no partial sums from other waves. Half as many tiles again, each
// with twice the MFMA work per step: 13-25% faster than 32-unit tiles at
// 2048-16384 rows, but slower while 32-unit tiles still make one per CU
// (their LDS traffic per MFMA is lower).
constexpr int KQ_TU = 64;
constexpr int KQ_BROWS = 3 * KQ_TU;
constexpr int KQ_ROWS = 16 * KS_RBMAX + KQ_BROWS;
constexpr int KQ_OPER = 2 * KQ_ROWS * KW_LDA;
constexpr int KQ_PTRS = KQ_OPER;
constexpr int KQ_HPREV = KQ_PTRS + 16 * KS_RBMAX * 10;
static_assert(KQ_HPREV + 16 * KS_RBMAX * KQ_TU <= G_LDS_FLOATS, "64-unit bf16 tiles exceed the LDS buffer");
typedef float (*KqLds)[KQ_ROWS][KW_LDA];

__device__ __forceinline__ int kq_row_tiles(const Dev &d, int M) {
    const int NU = d.H / KQ_TU;
    const int R0 = max(1, 256 / NU);
    return R0 * ((M + 128 * R0 - 1) / (128 * R0));
}

// A thread's share of one K step: 16-byte chunk t % 8 of A rows t / 8 and
// t / 8 + 64 and of weight rows t / 8, t / 8 + 64, t / 8 + 128 (gate 0, 1, 2
// of unit t / 8).
struct KqStage {
    uint4 a0, a1, b0, b1, b2;
};

template <int RB>
__device__ __forceinline__ void kq_load(KqStage &S, const u64 *ptrs, int a_r, int a_c8, int k0, int Kx,
                                        const uint16_t *bp, size_t bstride) {
    constexpr int BM = 16 * RB;
    const bool xp = k0 < Kx;
    const int ko = (xp ? k0 : k0 - Kx) + a_c8;
    const int r0 = min(a_r, BM - 1), r1 = min(a_r + 64, BM - 1);
    S.a0 = ldg<uint4>(reinterpret_cast<const uint16_t *>(ptrs[5 * r0 + (xp ? 3 : 2)]) + ko);
    S.a1 = ldg<uint4>(reinterpret_cast<const uint16_t *>(ptrs[5 * r1 + (xp ? 3 : 2)]) + ko);
    S.b0 = ldg<uint4>(bp + k0);
    S.b1 = ldg<uint4>(bp + bstride + k0);
    S.b2 = ldg<uint4>(bp + 2 * bstride + k0);
}

template <int RB>
__device__ __forceinline__ void kq_store(const KqStage &S, KqLds As, int buf, int a_r, int a_cf) {
    constexpr int BM = 16 * RB;
    if (a_r < BM) *reinterpret_cast<uint4 *>(&As[buf][a_r][a_cf]) = S.a0;
    if (a_r + 64 < BM) *reinterpret_cast<uint4 *>(&As[buf][a_r + 64][a_cf]) = S.a1;
    *reinterpret_cast<uint4 *>(&As[buf][BM + a_r][a_cf]) = S.b0;
    *reinterpret_cast<uint4 *>(&As[buf][BM + 64 + a_r][a_cf]) = S.b1;
    *reinterpret_cast<uint4 *>(&As[buf][BM + 128 + a_r][a_cf]) = S.b2;
}

template <int RB, int G, int NG, class MID>
__device__ __forceinline__ void kq_step(f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4], KqLds As,
                                        int buf, int rl, int kc, int uq, MID mid) {
    constexpr int NRB = (RB - G + 1) / 2;
    if constexpr (NRB == 0) {
        mid();
        return;
    }
    bf8_t b[2][3];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int q = 0; q < 3; ++q)
            b[h][q] = __builtin_bit_cast(
                bf8_t, *reinterpret_cast<const uint4 *>(&As[buf][16 * RB + 64 * q + 16 * uq + rl][kc + 16 * h]));
    bf8_t a[NRB > 0 ? NRB : 1][2];
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h)
            a[i][h] = __builtin_bit_cast(bf8_t, *reinterpret_cast<const uint4 *>(&As[buf][16 * (G + 2 * i) + rl][kc + 16 * h]));
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
        if (i == 1 || NRB == 1) mid();
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i][h], b[h][0], acc[i][0], 0, 0, 0);
            acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i][h], b[h][1], acc[i][1], 0, 0, 0);
            acc[i][NG] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i][h], b[h][2], acc[i][NG], 0, 0, 0);
        }
    }
}

template <int RB, int G>
__device__ __forceinline__ void kq_gates(const f4_t (&acc)[(RB - G + 1) / 2 > 0 ? (RB - G + 1) / 2 : 1][4],
                                         const KsEpi &ep, int uq, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    const int eu = lane & 15;
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = 16 * (G + 2 * i) + 4 * (lane >> 4) + e;
            const u64 dp = ep.ptrs[5 * row];
            if (dp) {
                const float rr = sigmoidf_(acc[i][0][e] + ep.br);
                const float z = sigmoidf_(acc[i][1][e] + ep.bz);
                const float n = tanhf(acc[i][2][e] + ep.bn + rr * acc[i][3][e]);
                const float hn = (1.0f - z) * n + z * ep.hprev[row * KQ_TU + 16 * uq + eu];
                reinterpret_cast<float *>(dp)[ep.lofs + ep.j] = hn;
                const u64 xp = ep.ptrs[5 * row + 4];
                if (xp) reinterpret_cast<uint16_t *>(xp)[ep.j] = f32_to_bf16(hn);
            }
        }
    }
}

template <int RB, int G>
__device__ __forceinline__ void kq_waves(KqLds As, const KsEpi &ep, int a_r, int a_c8, int a_cf, int Kx, int K,
                                         const uint16_t *bp, size_t bstride, int w, int lane) {
    constexpr int NRB = (RB - G + 1) / 2;
    f4_t acc[NRB > 0 ? NRB : 1][4];
#pragma unroll
    for (int i = 0; i < NRB; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][q] = f4_t{0, 0, 0, 0};
    const int uq = w & 3;
    const int rl = lane & 15, kc = 4 * (lane >> 4);
    const int nk = K / KW_BK, nx = Kx / KW_BK;
    KqStage S0, S1;
    kq_load<RB>(S0, ep.ptrs, a_r, a_c8, KW_BK, Kx, bp, bstride);
    kq_load<RB>(S1, ep.ptrs, a_r, a_c8, min(2, nk - 1) * KW_BK, Kx, bp, bstride);
    auto step = [&](int kt, auto NGc, auto PARc) {
        constexpr int NG = decltype(NGc)::value, PAR = decltype(PARc)::value;
        KqStage &St = PAR == 0 ? S0 : S1;
        kq_step<RB, G, NG>(acc, As, PAR, rl, kc, uq, [&] {
            if (kt + 1 < nk) kq_store<RB>(St, As, 1 - PAR, a_r, a_cf);
        });
        kq_load<RB>(St, ep.ptrs, a_r, a_c8, min(kt + 3, nk - 1) * KW_BK, Kx, bp, bstride);
        __syncthreads();
    };
    using X = std::integral_constant<int, 2>;
    using Hh = std::integral_constant<int, 3>;
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    int kt = 0;
    for (; kt + 1 < nx; kt += 2) {
        step(kt, X(), P0());
        step(kt + 1, X(), P1());
    }
    if (kt < nx) step(kt++, X(), P0());
    if (kt & 1) step(kt++, Hh(), P1());
    for (; kt + 1 < nk; kt += 2) {
        step(kt, Hh(), P0());
        step(kt + 1, Hh(), P1());
    }
    if (kt < nk) step(kt, Hh(), P0());
    kq_gates<RB, G>(acc, ep, uq, lane);
}

template <int RB>
__device__ __forceinline__ void gru_kq_bf16(const Dev &d, const Rows &R, int layer, int M, float *smem, int tile,
                                            int NR) {
    constexpr int BM = 16 * RB;
    const int NU = d.H / KQ_TU;
    int rt, ut;
    if ((NU & 7) == 0) {   // every XCD keeps its own unit tiles
        const int xcd = tile & 7, idx = tile >> 3, per = NU >> 3;
        rt = idx / per;
        ut = xcd + 8 * (idx % per);
    } else {
        rt = tile / NU;
        ut = tile % NU;
    }
    const int m0 = rt * BM, j0 = ut * KQ_TU;
    if (rt >= NR || m0 >= M) return;

    KqLds As = reinterpret_cast<KqLds>(smem);
    u64 *ptrs = reinterpret_cast<u64 *>(smem + KQ_PTRS);
    float *hprev = smem + KQ_HPREV;
    const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
    const int Kx = layer == 0 ? d.E : d.H;
    const int K = Kx + d.H;
    const uint16_t *Wp = reinterpret_cast<const uint16_t *>(d.Wl);
    // the tile's row pointers, as for the 32-unit tiles
    if (tid < BM) {
        const int m = min(m0 + tid, M - 1);
        const bool live = m0 + tid < M;
        ptrs[5 * tid] = live ? row_at(R, d.f_rowdst, m) : 0;
        ptrs[5 * tid + 1] = row_at(R, d.f_rowh, m) + (u64)layer * d.H * 4;
        ptrs[5 * tid + 2] = row_at(R, d.f_rowhb, m) + (u64)layer * d.H * 2;
        ptrs[5 * tid + 3] = layer == 0 ? (u64)(reinterpret_cast<const uint16_t *>(d.emb) +
                                               (size_t)(unsigned)row_at(R, d.f_roww, m) * d.E)
                                       : (u64)row_ptr(R, d.f_xbf, m, d.H);
        ptrs[5 * tid + 4] = live && layer == 0 && d.L == 2 ? (u64)row_ptr(R, d.f_xbf, m, d.H) : 0;
    }
    __syncthreads();
    // weight rows a_r, a_r + 64, a_r + 128 of the tile: gate 0, 1, 2 of unit a_r
    const int a_r = tid >> 3, a_c8 = (tid & 7) * 8, a_cf = (tid & 7) * 4;
    const uint16_t *bp = Wp + (size_t)(j0 + a_r) * K + a_c8;
    const size_t bstride = (size_t)d.H * K;
    // step 0 into LDS, with the epilogue's fp32 h: thread (row tid / 64 + 8 p,
    // unit tid % 64)
    const int hi = tid >> 6, hu = tid & 63;
    float hv[2 * RB];
#pragma unroll
    for (int p = 0; p < 2 * RB; ++p) hv[p] = reinterpret_cast<const float *>(ptrs[5 * (hi + 8 * p) + 1])[j0 + hu];
    KsEpi ep;
    ep.ptrs = ptrs;
    ep.hprev = hprev;
    ep.j = j0 + 16 * (w & 3) + (lane & 15);
    ep.br = d.bl[ep.j];
    ep.bz = d.bl[d.H + ep.j];
    ep.bn = d.bl[2 * d.H + ep.j];
    ep.lofs = (size_t)layer * d.H;
    {
        KqStage S;
        kq_load<RB>(S, ptrs, a_r, a_c8, 0, Kx, bp, bstride);
        kq_store<RB>(S, As, 0, a_r, a_cf);
    }
#pragma unroll
    for (int p = 0; p < 2 * RB; ++p) hprev[(hi + 8 * p) * KQ_TU + hu] = hv[p];
    __syncthreads();
    if (w < 4) kq_waves<RB, 0>(As, ep, a_r, a_c8, a_cf, Kx, K, bp, bstride, w, lane);
    else kq_waves<RB, 1>(As, ep, a_r, a_c8, a_cf, Kx, K, bp, bstride, w, lane);
    __syncthreads();
}

// One launch per layer; the device-side row count picks the path.
static_assert(8 * N_TILES * 2 * 256 <= G_LDS_FLOATS, "narrow partial tiles exceed the LDS buffer");

// ONE: the launch scores a single frame (the host knows), so the row lists
// need no per-frame selection and the narrow path's operands can be loaded
// before the row count is known.
template <bool BF16W, bool ONE>
__global__ __launch_bounds__(G_THREADS) void k_gru(Dev d, SessList sl, int layer) {
    __shared__ __align__(16) float smem[G_LDS_FLOATS];
    // the narrow path's unit group of a block index: each XCD its own contiguous share
    const int NB = d.H / 4;
    const int by_xcd = ((NB & 7) == 0) & ((int)gridDim.x >= NB);   // arithmetic, not a branch
    auto group = [&](int t) { return t + by_xcd * ((t & 7) * (NB >> 3) + (t >> 3) - t); };
    NarrowPre<BF16W> pre;
    Rows R;
    if (ONE) {
        // every block loads one group's operands (a block past the groups the last one's, unused)
        narrow_preload<BF16W>(d, sl, layer, min(group(blockIdx.x), NB - 1), pre);
        const long long c = ldg<long long>(shift_ptr(d.ctr, (long long)sl.sess[0] * d.sess_stride) + C_FRAME_M);
        // The row count takes a dependence on the preloaded values, times a
        // zero the compiler cannot see (a launch of one frame has sl.n = 1).
        // Without a use ahead of the branch on the count, the compiler moves
        // these loads into the narrow path, behind the count's round trip;
        // with it, the count and the operands arrive in the same round trip.
        const u64 mix = pre.rowh[0] ^ pre.rowd[0] ^ pre.edst ^ pre.ehsrc ^ (u64)(unsigned)pre.roww[0] ^
                        (u64)(__float_as_uint(pre.br) ^ __float_as_uint(pre.bz) ^ __float_as_uint(pre.bn));
        const int dep = __builtin_amdgcn_readfirstlane((int)(mix ^ (mix >> 32))) * (sl.n - 1);
        R.n = 1;
        R.sofs[0] = (long long)sl.sess[0] * d.sess_stride;
#pragma unroll
        for (int e = 1; e < kMaxSessions; ++e) R.sofs[e] = R.sofs[0];
        R.moff[0] = 0;
#pragma unroll
        for (int e = 1; e <= kMaxSessions; ++e) R.moff[e] = (int)c + dep;
    } else {
        R = make_rows(d, sl, load_row_counts(d, sl));
    }
    const int M = R.moff[kMaxSessions];   // rows of all the launch's frames
    if (M <= 0) return;
    if (ONE && M <= 16) {             // few rows: every CU streams its share of the weights
        if ((int)blockIdx.x < NB) gru_narrow<BF16W, true, 1>(d, R, layer, M, smem, group(blockIdx.x), pre);
        for (int t = blockIdx.x + gridDim.x; t < NB; t += gridDim.x) {
            __syncthreads();
            gru_narrow<BF16W, false, 1>(d, R, layer, M, smem, group(t), pre);
        }
    } else if (M <= N_MAXROWS) {      // the same, one or two row tiles
        for (int t = blockIdx.x; t < NB; t += gridDim.x) {
            __syncthreads();
            gru_narrow<BF16W, false, N_TILES>(d, R, layer, M, smem, group(t), pre);
        }
    } else if constexpr (BF16W) {
        const int NU = d.H / KW_TU;
        const int NRw = kw_row_tiles(d, M);
        if ((M + 15) / 16 <= 2 * NRw) {   // 32-unit tiles would be 1 or 2 row blocks high: (16 RB) x 16-unit tiles
            const int NR = ks_row_tiles(d, M);
            const int RB = __builtin_amdgcn_readfirstlane(((M + 15) / 16 + NR - 1) / NR);
            const int ntiles = NR * (d.H / KS_TU);
            for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
                switch (RB) {
                    case 1: gru_ks_bf16<1>(d, R, layer, M, smem, t, NR); break;
                    case 2: gru_ks_bf16<2>(d, R, layer, M, smem, t, NR); break;
                    case 3: gru_ks_bf16<3>(d, R, layer, M, smem, t, NR); break;
                    case 4: gru_ks_bf16<4>(d, R, layer, M, smem, t, NR); break;
                    case 5: gru_ks_bf16<5>(d, R, layer, M, smem, t, NR); break;
                    case 6: gru_ks_bf16<6>(d, R, layer, M, smem, t, NR); break;
                    case 7: gru_ks_bf16<7>(d, R, layer, M, smem, t, NR); break;
                    default: gru_ks_bf16<8>(d, R, layer, M, smem, t, NR); break;
                }
            }
            return;
        }
        if (M > 128 * max(1, 256 / NU)) {   // (16 RB) x 64-unit tiles
            const int NR = kq_row_tiles(d, M);
            const int RB = __builtin_amdgcn_readfirstlane(((M + 15) / 16 + NR - 1) / NR);
            const int ntiles = NR * (d.H / KQ_TU);
            for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
                switch (RB) {
                    case 1: gru_kq_bf16<1>(d, R, layer, M, smem, t, NR); break;
                    case 2: gru_kq_bf16<2>(d, R, layer, M, smem, t, NR); break;
                    case 3: gru_kq_bf16<3>(d, R, layer, M, smem, t, NR); break;
                    case 4: gru_kq_bf16<4>(d, R, layer, M, smem, t, NR); break;
                    case 5: gru_kq_bf16<5>(d, R, layer, M, smem, t, NR); break;
                    case 6: gru_kq_bf16<6>(d, R, layer, M, smem, t, NR); break;
                    case 7: gru_kq_bf16<7>(d, R, layer, M, smem, t, NR); break;
                    default: gru_kq_bf16<8>(d, R, layer, M, smem, t, NR); break;
                }
            }
            return;
        }
        // (16 RB) x 32-unit tiles, K split over the waves
        const int NR = NRw;
        const int RB = __builtin_amdgcn_readfirstlane(((M + 15) / 16 + NR - 1) / NR);
        const int ntiles = NR * (d.H / KW_TU);
        for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
            switch (RB) {
                case 1: gru_kw_bf16<1>(d, R, layer, M, smem, t, NR); break;
                case 2: gru_kw_bf16<2>(d, R, layer, M, smem, t, NR); break;
                case 3: gru_kw_bf16<3>(d, R, layer, M, smem, t, NR); break;
                case 4: gru_kw_bf16<4>(d, R, layer, M, smem, t, NR); break;
                case 5: gru_kw_bf16<5>(d, R, layer, M, smem, t, NR); break;
                case 6: gru_kw_bf16<6>(d, R, layer, M, smem, t, NR); break;
                case 7: gru_kw_bf16<7>(d, R, layer, M, smem, t, NR); break;
                default: gru_kw_bf16<8>(d, R, layer, M, smem, t, NR); break;
            }
        }
    } else {
        if (M > 128 * max(1, 256 / (d.H / KS_TU))) {   // fp32: (16 RB) x 64-unit tiles
            const int NR = kf_row_tiles(d, M);
            const int RB = __builtin_amdgcn_readfirstlane(((M + 15) / 16 + NR - 1) / NR);
            const int ntiles = NR * (d.H / KF_TU);
            for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
                switch (RB) {
                    case 1: gru_kf_f32<1>(d, R, layer, M, smem, t, NR); break;
                    case 2: gru_kf_f32<2>(d, R, layer, M, smem, t, NR); break;
                    case 3: gru_kf_f32<3>(d, R, layer, M, smem, t, NR); break;
                    case 4: gru_kf_f32<4>(d, R, layer, M, smem, t, NR); break;
                    case 5: gru_kf_f32<5>(d, R, layer, M, smem, t, NR); break;
                    case 6: gru_kf_f32<6>(d, R, layer, M, smem, t, NR); break;
                    case 7: gru_kf_f32<7>(d, R, layer, M, smem, t, NR); break;
                    default: gru_kf_f32<8>(d, R, layer, M, smem, t, NR); break;
                }
            }
            return;
        }
        // fp32: (16 RB) x 16-unit tiles, K split over the waves
        const int NR = ks_row_tiles(d, M);
        const int RB = __builtin_amdgcn_readfirstlane(((M + 15) / 16 + NR - 1) / NR);
        const int ntiles = NR * (d.H / KS_TU);
        for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
            switch (RB) {
                case 1: gru_ks_f32<1>(d, R, layer, M, smem, t, NR); break;
                case 2: gru_ks_f32<2>(d, R, layer, M, smem, t, NR); break;
                case 3: gru_ks_f32<3>(d, R, layer, M, smem, t, NR); break;
                case 4: gru_ks_f32<4>(d, R, layer, M, smem, t, NR); break;
                case 5: gru_ks_f32<5>(d, R, layer, M, smem, t, NR); break;
                case 6: gru_ks_f32<6>(d, R, layer, M, smem, t, NR); break;
                case 7: gru_ks_f32<7>(d, R, layer, M, smem, t, NR); break;
                default: gru_ks_f32<8>(d, R, layer, M, smem, t, NR); break;
            }
        }
    }
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

void launch_gru_layer(const Dev &d0, const FrameBlock &fb, int layer, int max_rows, hipStream_t s, Stamp ts) {
    if (max_rows <= 0) return;
    Dev d = d0;
    d.Wl = d0.Wp[layer];
    d.bl = d0.b_ih[layer];
    SessList sl;
    sl.n = fb.n;
    for (int e = 0; e < kMaxSessions; ++e) sl.sess[e] = e < fb.n ? fb.sess[e] : 0;
    // one block per CU (the LDS buffer allows no more); blocks loop over tiles
    const int blocks = 256;
    if (d.wdtype == RNNLM_BF16) {
        if (fb.n == 1) launch_k(k_gru<true, true>, blocks, G_THREADS, s, ts, d, sl, layer);
        else launch_k(k_gru<true, false>, blocks, G_THREADS, s, ts, d, sl, layer);
    } else {
        if (fb.n == 1) launch_k(k_gru<false, true>, blocks, G_THREADS, s, ts, d, sl, layer);
        else launch_k(k_gru<false, false>, blocks, G_THREADS, s, ts, d, sl, layer);
    }
}

}  // namespace rn
