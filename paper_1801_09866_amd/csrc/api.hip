// C ABI (include/rnnlm.h): configuration checks, workspace carve-up, weight
// packing, and the per-frame launch sequence.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "common.hpp"
#include "kernels.hpp"

#define RNNLM_API extern "C" __attribute__((visibility("default")))

struct rnnlm_t {
    rnnlm_config cfg;
    rn::Dev dev;
    unsigned host_derr;   // sticky device error as last read by rnnlm_get_stats
    // per session: scoring blocks of its last frame whose counts are not
    // folded yet, and a bound on the scores that frame staged for the cache
    int pending_parts[rn::kMaxSessions] = {};
    int staged_max[rn::kMaxSessions] = {};
    // optional per-stage timing (rnnlm_profile)
    uint32_t prof_mask = 0;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> prof_pool;   // created events
    std::vector<int> prof_stage;                                 // stage of each used pair
    size_t prof_used = 0;
};

namespace {

// Hands out a start/stop event pair for one stage's launches when that stage
// is timed; the kernels' own dispatch packets take the timestamps.
struct StageTimer {
    rn::Stamp ts;
    StageTimer(rnnlm_t *ctx, int stage) {
        if (!(ctx->prof_mask & (1u << stage))) return;
        if (ctx->prof_used == ctx->prof_pool.size()) {
            hipEvent_t a, b;
            if (hipEventCreate(&a) != hipSuccess) return;
            if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
            ctx->prof_pool.emplace_back(a, b);
        }
        auto &pr = ctx->prof_pool[ctx->prof_used++];
        ctx->prof_stage.push_back(stage);
        ts.start = pr.first;
        ts.stop = pr.second;
    }
    // stamps for kernel k of a stage of n kernels
    rn::Stamp part(int k, int n) const {
        rn::Stamp p;
        if (k == 0) p.start = ts.start;
        if (k == n - 1) p.stop = ts.stop;
        return p;
    }
};

}  // namespace

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(RNNLM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- exact decimal decade boundaries (smallest fp32 >= 10^-j) ----------
typedef unsigned __int128 u128;

// true iff the positive fp32 with bit pattern b is >= 10^-j
bool ge_pow10_neg(uint32_t b, int j) {
    const uint32_t ex = b >> 23;
    const uint64_t M = ex ? ((b & 0x7FFFFFu) | 0x800000u) : (b & 0x7FFFFFu);
    const int s = ex ? 150 - (int)ex : 149;   // value = M * 2^-s
    if (s <= 0) return true;
    if (s >= 127) return false;               // < 2^-103, far below 1e-20
    u128 p = 1;
    for (int i = 0; i < j; ++i) p *= 10;
    return (u128)M * p >= ((u128)1 << s);
}

rn::DecadeTab make_decades() {
    rn::DecadeTab t;
    for (int j = 0; j <= 20; ++j) {
        float approx = 1.0f;
        for (int i = 0; i < j; ++i) approx /= 10.0f;
        uint32_t b;
        memcpy(&b, &approx, 4);
        while (!ge_pow10_neg(b, j)) ++b;
        while (b > 0 && ge_pow10_neg(b - 1, j)) --b;
        t.lo[j] = b;
    }
    return t;
}

const rn::DecadeTab &decades() {
    static rn::DecadeTab t;
    static std::once_flag once;
    std::call_once(once, [] { t = make_decades(); });
    return t;
}

uint32_t pow2_at_least(long long n) {
    uint32_t p = 16;
    while ((long long)p < n) p <<= 1;
    return p;
}

int sessions_of(const rnnlm_config &c) { return c.sessions > 0 ? c.sessions : 1; }

int code_words(const rnnlm_config &c) {
    const int LH = c.L * c.H;
    return c.qmode == RNNLM_Q_SIGN ? LH / 64 : (c.qmode == RNNLM_Q_SIGDIG ? LH / 4 : LH / 2);
}

int check_config(const rnnlm_config *c) {
    if (!c) return fail(RNNLM_EINVAL, "null config");
    if (c->V < 1 || c->V > (1 << 30)) return fail(RNNLM_EINVAL, "V out of range");
    if (c->E < 64 || c->E % 64) return fail(RNNLM_EINVAL, "E must be a positive multiple of 64");
    if (c->H < 64 || c->H % 64) return fail(RNNLM_EINVAL, "H must be a positive multiple of 64");
    if (c->L < 1 || c->L > 2) return fail(RNNLM_EINVAL, "L must be 1 or 2");
    if (c->L * c->H > rn::kMaxLH) return fail(RNNLM_EINVAL, "L*H must be <= %d", rn::kMaxLH);
    if (c->wdtype != RNNLM_F32 && c->wdtype != RNNLM_BF16) return fail(RNNLM_EINVAL, "bad wdtype");
    if (c->maxent_log2 < 1 || c->maxent_log2 > 30) return fail(RNNLM_EINVAL, "maxent_log2 out of range");
    if (c->maxent_order < 1 || c->maxent_order > 4) return fail(RNNLM_EINVAL, "maxent_order must be 1..4");
    if (c->qmode < RNNLM_Q_EXACT || c->qmode > RNNLM_Q_SIGDIG) return fail(RNNLM_EINVAL, "bad qmode");
    if (c->qmode == RNNLM_Q_SIGDIG && (c->qdigits < 1 || c->qdigits > 3))
        return fail(RNNLM_EINVAL, "qdigits must be 1..3");
    if (c->max_hist < 1 || c->max_hist > rn::kPlanMaxHist)
        return fail(RNNLM_EINVAL, "max_hist must be 1..%d", rn::kPlanMaxHist);
    if (c->max_query < 0 || c->max_query > rn::kPlanMaxQuery)
        return fail(RNNLM_EINVAL, "max_query must be 0..%d", rn::kPlanMaxQuery);
    if (c->cap_hist < 0 || c->cap_hist > (1LL << 28)) return fail(RNNLM_EINVAL, "cap_hist out of range");
    if (c->cap_query < 0 || c->cap_query > (1LL << 29)) return fail(RNNLM_EINVAL, "cap_query out of range");
    if (c->sessions < 0 || c->sessions > rn::kMaxSessions)
        return fail(RNNLM_EINVAL, "sessions must be 0..%d (0 means 1)", rn::kMaxSessions);
    return RNNLM_OK;
}

// Sequential carve-up of the workspace; with base == nullptr it only sizes.
struct Carver {
    char *base;
    size_t off = 0;
    template <class T>
    T *take(size_t count) {
        off = (off + 255) & ~(size_t)255;
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

struct Extents {
    uint32_t HI, SI;   // open-addressing table sizes (load <= 1/2)
};

Extents extents(const rnnlm_config &c) {
    Extents e;
    e.HI = pow2_at_least(2 * c.cap_hist);
    e.SI = pow2_at_least(2 * c.cap_query);
    return e;
}

// Lay out every device buffer; returns total bytes. Pointers are filled when
// base != nullptr. packed[l] receives the packed weight buffer of layer l.
size_t layout(const rnnlm_config &c, char *base, rn::Dev &d, void **packed) {
    Carver cv{base};
    const Extents x = extents(c);
    const int LH = c.L * c.H, CW = code_words(c);
    const size_t welem = c.wdtype == RNNLM_BF16 ? 2 : 4;
    for (int l = 0; l < 2; ++l) {
        packed[l] = nullptr;
        if (l < c.L) {
            const size_t Kx = l == 0 ? c.E : c.H;
            packed[l] = cv.take<char>((size_t)3 * c.H * (Kx + c.H) * welem);
        }
    }
    d.ln_part = cv.take<float2>((size_t)256 * rn::lognorm_tiles(c.V));
    // one session's state; sessions 1.. repeat it sess_stride bytes apart
    const size_t mh = c.max_hist, mq = c.max_query > 0 ? c.max_query : 1;
    const size_t ch = c.cap_hist > 0 ? c.cap_hist : 1;
    cv.off = (cv.off + 255) & ~(size_t)255;
    const size_t s0 = cv.off;
    d.hc_idx = cv.take<rn::HcIdx>(x.HI);
    d.hc_codes = cv.take<unsigned long long>(ch * CW);
    d.hc_val = cv.take<float>(ch * LH);
    d.sc_tab = cv.take<rn::ScEnt>(x.SI);
    d.sc_stage = cv.take<rn::ScEnt>(mq);
    d.ctr = cv.take<long long>(rn::C_N);
    d.derr = cv.take<unsigned>(1);
    d.f_codes = cv.take<unsigned long long>(mh * CW);
    d.f_hrec = cv.take<rn::HistRec>(mh);
    d.f_hstat = cv.take<int>(mh);
    d.f_hslot = cv.take<int>(mh);
    d.f_hptr = cv.take<unsigned long long>(mh);
    d.f_roww = cv.take<int>(mh);
    d.f_rowh = cv.take<unsigned long long>(mh);
    d.f_rowdst = cv.take<unsigned long long>(mh);
    d.f_hval = cv.take<float>(mh * LH);
    const bool bf = c.wdtype == RNNLM_BF16;
    d.f_hbf = cv.take<uint16_t>(bf ? mh * LH : 8);
    d.f_rowhb = cv.take<unsigned long long>(mh);
    d.f_xbf = cv.take<uint16_t>(bf && c.L == 2 ? mh * c.H : 8);
    d.f_qkey = cv.take<int4>(mq);
    d.f_qwords = cv.take<int4>(mq);
    d.f_qrec = cv.take<rn::QRec>(mq);
    d.f_qcand = cv.take<int>(mq);
    d.f_part = cv.take<int4>((mq + 3) / 4);
    const size_t stride = ((cv.off - s0) + 255) & ~(size_t)255;
    d.sessions = sessions_of(c);
    d.sess_stride = (long long)stride;
    return s0 + stride * d.sessions;
}

// Empty caches (index slot / entry key = -1) and zero counters, with fill
// kernels rather than memsets so the sequence can live in a captured graph.
void reset_state(const rn::Dev &d, const Extents &x, hipStream_t s) {
    for (int k = 0; k < d.sessions; ++k) {
        const long long o = k * d.sess_stride;
        auto at = [o](void *p) { return static_cast<void *>(static_cast<char *>(p) + o); };
        rn::launch_fill_u32(at(d.hc_idx), 0xFFFFFFFFu, (long long)x.HI * sizeof(rn::HcIdx) / 4, s);
        rn::launch_fill_u32(at(d.sc_tab), 0xFFFFFFFFu, (long long)x.SI * sizeof(rn::ScEnt) / 4, s);
        rn::launch_fill_u32(at(d.ctr), 0u, 2LL * rn::C_N, s);
        rn::launch_fill_u32(at(d.derr), 0u, 1, s);
    }
}

}  // namespace

RNNLM_API const char *rnnlm_last_error(void) { return g_err.c_str(); }

RNNLM_API int rnnlm_workspace_size(const rnnlm_config *cfg, size_t *bytes) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!bytes) return fail(RNNLM_EINVAL, "null bytes");
    rn::Dev d;
    void *packed[2];
    *bytes = layout(*cfg, nullptr, d, packed);
    return RNNLM_OK;
}

RNNLM_API int rnnlm_create(const rnnlm_config *cfg, const rnnlm_weights *w, void *workspace,
                           size_t ws_bytes, void *stream, rnnlm_t **out) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!w || !workspace || !out) return fail(RNNLM_EINVAL, "null weights, workspace or out");
    if (reinterpret_cast<uintptr_t>(workspace) & 255) return fail(RNNLM_EINVAL, "workspace not 256-byte aligned");
    if (!w->emb || !w->U_out || !w->b_out) return fail(RNNLM_EINVAL, "null emb, U_out or b_out");
    if (cfg->maxent_order >= 2 && !w->maxent) return fail(RNNLM_EINVAL, "null maxent table");
    for (int l = 0; l < cfg->L; ++l)
        if (!w->W_ih[l] || !w->W_hh[l] || !w->b_ih[l]) return fail(RNNLM_EINVAL, "null GRU weights of layer %d", l);
    rn::Dev d;
    memset(&d, 0, sizeof d);
    void *packed[2];
    const size_t need = layout(*cfg, reinterpret_cast<char *>(workspace), d, packed);
    if (ws_bytes < need) return fail(RNNLM_ENOMEM, "workspace has %zu bytes, needs %zu", ws_bytes, need);
    const Extents x = extents(*cfg);
    d.V = cfg->V; d.E = cfg->E; d.H = cfg->H; d.L = cfg->L; d.LH = cfg->L * cfg->H;
    d.wdtype = cfg->wdtype; d.me_log2 = cfg->maxent_log2; d.me_order = cfg->maxent_order;
    d.qmode = cfg->qmode; d.qdigits = cfg->qmode == RNNLM_Q_SIGDIG ? cfg->qdigits : 0;
    d.max_hist = cfg->max_hist; d.max_query = cfg->max_query; d.CW = code_words(*cfg);
    d.cap_hist = cfg->cap_hist; d.cap_query = cfg->cap_query; d.seed = cfg->seed;
    d.hi_mask = x.HI - 1; d.si_mask = x.SI - 1;
    d.emb = w->emb; d.U_out = w->U_out; d.b_out = w->b_out; d.maxent = w->maxent;
    for (int l = 0; l < 2; ++l) {
        d.Wp[l] = packed[l];
        d.b_ih[l] = l < cfg->L ? w->b_ih[l] : nullptr;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    for (int l = 0; l < cfg->L; ++l) rn::launch_pack_layer(d, l, w->W_ih[l], w->W_hh[l], packed[l], s);
    reset_state(d, x, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "rnnlm_create launch");
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "rnnlm_create sync");
    (void)decades();
    rnnlm_t *ctx = new (std::nothrow) rnnlm_t;
    if (!ctx) return fail(RNNLM_ENOMEM, "host allocation failed");
    ctx->cfg = *cfg;
    ctx->dev = d;
    ctx->host_derr = 0;
    *out = ctx;
    return RNNLM_OK;
}

// Host checks of one frame; fills f. Returns RNNLM_OK, or 1 for an empty frame.
static int frame_args(const rnnlm_config &c, const rnnlm_frame *fr, const rnnlm_out *out, rn::FrameArgs &f) {
    if (!fr || !out) return fail(RNNLM_EINVAL, "null frame or out");
    if (fr->n_hist < 0 || fr->n_hist > c.max_hist) return fail(RNNLM_EINVAL, "n_hist %d outside [0, %d]", fr->n_hist, c.max_hist);
    if (fr->n_query < 0 || fr->n_query > c.max_query) return fail(RNNLM_EINVAL, "n_query %d outside [0, %d]", fr->n_query, c.max_query);
    if (fr->n_query > 0 && fr->n_hist == 0) return fail(RNNLM_EINVAL, "queries without histories");
    if (fr->n_hist > 0 && ((!fr->hist_vec && !fr->hist_ptr) || !fr->hist_words)) return fail(RNNLM_EINVAL, "null history arrays");
    if (fr->n_query > 0 && (!fr->q_hist || !fr->q_tgt || !out->scores)) return fail(RNNLM_EINVAL, "null query arrays or scores");
    if (fr->n_hist == 0) return 1;
    if (!fr->hist_ptr && (reinterpret_cast<uintptr_t>(fr->hist_vec) & 15)) return fail(RNNLM_EINVAL, "hist_vec must be 16-byte aligned");
    if (out->hnew && (reinterpret_cast<uintptr_t>(out->hnew) & 15)) return fail(RNNLM_EINVAL, "hnew must be 16-byte aligned");
    f.n_hist = fr->n_hist; f.n_query = fr->n_query;
    f.hist_vec = fr->hist_vec; f.hist_ptr = reinterpret_cast<const rn::u64 *>(fr->hist_ptr);
    f.hist_words = fr->hist_words; f.q_hist = fr->q_hist; f.q_tgt = fr->q_tgt;
    f.scores = out->scores; f.hnew = out->hnew; f.q_status = out->q_status; f.h_status = out->h_status;
    f.q_rep = out->q_rep; f.h_rep = out->h_rep; f.h_hash = reinterpret_cast<rn::u64 *>(out->h_hash);
    return RNNLM_OK;
}

RNNLM_API int rnnlm_score_frames(rnnlm_t *ctx, const rnnlm_frame *frames, const rnnlm_out *outs, int32_t n,
                                 void *stream) {
    if (!ctx) return fail(RNNLM_EINVAL, "null context");
    if (n < 0 || n > ctx->dev.sessions) return fail(RNNLM_EINVAL, "%d frames for %d sessions", n, ctx->dev.sessions);
    if (n > 0 && (!frames || !outs)) return fail(RNNLM_EINVAL, "null frames or outs");
    if (ctx->host_derr) return fail(RNNLM_EDEVICE, "sticky device error 0x%x; call rnnlm_cache_reset", ctx->host_derr);
    const rnnlm_config &c = ctx->cfg;
    rn::FrameBlock fb;
    memset(&fb, 0, sizeof fb);
    int maxh = 0;
    for (int k = 0; k < n; ++k) {   // frame k belongs to session k; empty frames take no part
        rn::FrameArgs f;
        const int rc = frame_args(c, frames + k, outs + k, f);
        if (rc < 0) return rc;
        if (rc == 1) continue;
        const int e = fb.n++;
        fb.f[e] = f;
        fb.sess[e] = k;
        fb.npart[e] = ctx->pending_parts[k];
        // key blocks: one per history for k significant digits, else one per 4 histories
        fb.hoff[e + 1] = fb.hoff[e] + (c.qmode == RNNLM_Q_SIGDIG ? f.n_hist : (f.n_hist + 3) / 4);
        fb.qoff[e + 1] = fb.qoff[e] + (f.n_query + 255) / 256;
        fb.soff[e + 1] = fb.soff[e] + (ctx->staged_max[k] + 255) / 256;
        fb.qblk[e] = (f.n_query + 3) / 4;
        fb.boff[e + 1] = fb.boff[e] + fb.qblk[e] + (f.n_hist + 3) / 4;
        maxh += f.n_hist;
    }
    if (fb.n == 0) return RNNLM_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int s0 = fb.sess[0];   // the launches see the context from entry 0's session
    const rn::Dev d = rn::session_view(ctx->dev, s0);
    int sess_abs[rn::kMaxSessions];
    for (int e = 0; e < fb.n; ++e) {
        sess_abs[e] = fb.sess[e];
        fb.sess[e] -= s0;
    }
    rn::launch_hist_key(d, fb, decades(), s, StageTimer(ctx, 0).ts);
    rn::launch_frame_plan(d, fb, s, StageTimer(ctx, 1).ts);
    {
        const StageTimer t(ctx, 2);
        for (int l = 0; l < c.L; ++l) rn::launch_gru_layer(d, fb, l, maxh, s, t.part(l, c.L));
    }
    rn::launch_score_finish(d, fb, s, StageTimer(ctx, 3).ts);
    for (int e = 0; e < fb.n; ++e) {
        ctx->pending_parts[sess_abs[e]] = (fb.f[e].n_query + 3) / 4;
        ctx->staged_max[sess_abs[e]] = fb.f[e].n_query;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "rnnlm_score_frames launch");
    return RNNLM_OK;
}

RNNLM_API int rnnlm_score_frame(rnnlm_t *ctx, const rnnlm_frame *fr, const rnnlm_out *out, void *stream) {
    if (!ctx || !fr || !out) return fail(RNNLM_EINVAL, "null context, frame or out");
    return rnnlm_score_frames(ctx, fr, out, 1, stream);
}

RNNLM_API int rnnlm_cache_reset(rnnlm_t *ctx, void *stream) {
    if (!ctx) return fail(RNNLM_EINVAL, "null context");
    reset_state(ctx->dev, extents(ctx->cfg), reinterpret_cast<hipStream_t>(stream));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "rnnlm_cache_reset launch");
    ctx->host_derr = 0;
    for (int k = 0; k < rn::kMaxSessions; ++k) ctx->pending_parts[k] = ctx->staged_max[k] = 0;
    return RNNLM_OK;
}

static int log_normalizer(rnnlm_t *ctx, const float *h_top, const int32_t *words, int32_t n, float *logz,
                          void *stream, const char *name) {
    if (!ctx) return fail(RNNLM_EINVAL, "null context");
    if (n < 0 || n > ctx->cfg.max_hist) return fail(RNNLM_EINVAL, "n %d outside [0, %d]", n, ctx->cfg.max_hist);
    if (n == 0) return RNNLM_OK;
    if (!h_top || !logz) return fail(RNNLM_EINVAL, "null h_top or logz");
    if (reinterpret_cast<uintptr_t>(h_top) & 15) return fail(RNNLM_EINVAL, "h_top must be 16-byte aligned");
    if (ctx->cfg.wdtype != RNNLM_F32) return fail(RNNLM_EINVAL, "the normaliser needs fp32 output weights");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    for (int r0 = 0; r0 < n; r0 += 256) {
        const int nr = n - r0 < 256 ? n - r0 : 256;
        const float *hb = h_top + (size_t)r0 * ctx->cfg.H;
        rn::launch_lognorm_gemm(ctx->dev, hb, words ? words + (size_t)r0 * 3 : nullptr, nr, s, StageTimer(ctx, 8).ts);
        rn::launch_lognorm_combine(ctx->dev, nr, logz + r0, s, StageTimer(ctx, 9).ts);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, name);
    return RNNLM_OK;
}

RNNLM_API int rnnlm_log_normalizer(rnnlm_t *ctx, const float *h_top, int32_t n, float *logz, void *stream) {
    return log_normalizer(ctx, h_top, nullptr, n, logz, stream, "rnnlm_log_normalizer launch");
}

RNNLM_API int rnnlm_log_normalizer_maxent(rnnlm_t *ctx, const float *h_top, const int32_t *words, int32_t n,
                                          float *logz, void *stream) {
    if (n > 0 && !words) return fail(RNNLM_EINVAL, "null words");
    return log_normalizer(ctx, h_top, words, n, logz, stream, "rnnlm_log_normalizer_maxent launch");
}

RNNLM_API int rnnlm_log_normalizer_static(const float *U_out, const float *b_out, int32_t V, int32_t H,
                                          const float *h_top, int32_t n, float *logz, void *stream) {
    if (V < 1 || rn::lognorm_tiles(V) > rn::kStaticMaxTiles)
        return fail(RNNLM_EINVAL, "V %d outside [1, %d]: the static scratch holds %d vocabulary tiles", V,
                    rn::kStaticMaxV, rn::kStaticMaxTiles);
    if (H < 64 || H % 64 || H > rn::kMaxLH) return fail(RNNLM_EINVAL, "H must be a multiple of 64 in [64, %d]", rn::kMaxLH);
    if (n < 0) return fail(RNNLM_EINVAL, "n %d < 0", n);
    if (n == 0) return RNNLM_OK;
    if (!U_out || !b_out || !h_top || !logz) return fail(RNNLM_EINVAL, "null U_out, b_out, h_top or logz");
    if ((reinterpret_cast<uintptr_t>(h_top) | reinterpret_cast<uintptr_t>(U_out)) & 15)
        return fail(RNNLM_EINVAL, "h_top and U_out must be 16-byte aligned");
    float2 *part = nullptr;
    hipError_t e = rn::lognorm_static_scratch(&part);
    if (e != hipSuccess) return hip_fail(e, "rnnlm_log_normalizer_static scratch");
    rn::Dev d;
    memset(&d, 0, sizeof d);
    d.V = V; d.H = H; d.U_out = U_out; d.b_out = b_out;
    d.me_log2 = 1; d.me_order = 1;   // no MaxEnt terms
    d.ln_part = part;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    for (int r0 = 0; r0 < n; r0 += 256) {   // each chunk's pairs are combined before the next overwrites them
        const int nr = n - r0 < 256 ? n - r0 : 256;
        rn::launch_lognorm_gemm(d, h_top + (size_t)r0 * H, nullptr, nr, s);
        rn::launch_lognorm_combine(d, nr, logz + r0, s);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "rnnlm_log_normalizer_static launch");
    return RNNLM_OK;
}

// Fold every session's pending scoring counts, then read all counters and
// error words (synchronises).
static int read_counters(rnnlm_t *ctx, long long (*c)[rn::C_N], unsigned *derr, hipStream_t s) {
    const rn::Dev &d = ctx->dev;
    rn::FoldParts fp;
    for (int k = 0; k < rn::kMaxSessions; ++k) {
        fp.npart[k] = ctx->pending_parts[k];
        ctx->pending_parts[k] = 0;
    }
    rn::launch_fold_stats(d, fp, s);
    hipError_t e = hipGetLastError();
    for (int k = 0; k < d.sessions && e == hipSuccess; ++k) {
        const char *base = reinterpret_cast<const char *>(d.ctr) + k * d.sess_stride;
        e = hipMemcpyAsync(c[k], base, sizeof c[k], hipMemcpyDeviceToHost, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(derr + k, reinterpret_cast<const char *>(d.derr) + k * d.sess_stride, sizeof(unsigned),
                               hipMemcpyDeviceToHost, s);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "rnnlm_get_stats");
    return RNNLM_OK;
}

static void fill_stats(rnnlm_stats *st, const long long *c, unsigned derr) {
    st->frames += c[rn::C_FRAMES]; st->queries += c[rn::C_QUERIES]; st->score_hits += c[rn::C_SCORE_HITS];
    st->query_dups += c[rn::C_QUERY_DUPS]; st->computed += c[rn::C_COMPUTED]; st->hists += c[rn::C_HISTS];
    st->hist_hits += c[rn::C_HIST_HITS]; st->hist_dups += c[rn::C_HIST_DUPS]; st->gru_rows += c[rn::C_GRU_ROWS];
    st->hist_inserted += c[rn::C_HIST_INS]; st->hist_rejected += c[rn::C_HIST_REJ];
    st->score_inserted += c[rn::C_SCORE_INS]; st->score_rejected += c[rn::C_SCORE_REJ];
    st->hist_cache_size += c[rn::C_HC_SIZE]; st->score_cache_size += c[rn::C_SC_SIZE];
    st->device_error |= (int32_t)derr;
}

static int stats_of(rnnlm_t *ctx, int session, rnnlm_stats *st, void *stream) {
    long long c[rn::kMaxSessions][rn::C_N];
    unsigned derr[rn::kMaxSessions] = {};
    const int rc = read_counters(ctx, c, derr, reinterpret_cast<hipStream_t>(stream));
    if (rc) return rc;
    memset(st, 0, sizeof *st);
    unsigned all = 0;
    for (int k = 0; k < ctx->dev.sessions; ++k) {
        all |= derr[k];
        if (session < 0 || session == k) fill_stats(st, c[k], derr[k]);
    }
    if (all) {   // sticky for the whole context
        ctx->host_derr = all;
        return fail(RNNLM_EDEVICE, "device error bits 0x%x", all);
    }
    return RNNLM_OK;
}

RNNLM_API int rnnlm_get_stats(rnnlm_t *ctx, rnnlm_stats *st, void *stream) {
    if (!ctx || !st) return fail(RNNLM_EINVAL, "null context or stats");
    return stats_of(ctx, -1, st, stream);
}

RNNLM_API int rnnlm_get_session_stats(rnnlm_t *ctx, int32_t session, rnnlm_stats *st, void *stream) {
    if (!ctx || !st) return fail(RNNLM_EINVAL, "null context or stats");
    if (session < 0 || session >= ctx->dev.sessions) return fail(RNNLM_EINVAL, "session %d outside [0, %d)", session, ctx->dev.sessions);
    return stats_of(ctx, session, st, stream);
}

RNNLM_API int rnnlm_debug_quantize(int32_t qmode, int32_t qdigits, const float *x, int64_t n, void *codes,
                                   int32_t *err, void *stream) {
    if (qmode < RNNLM_Q_EXACT || qmode > RNNLM_Q_SIGDIG) return fail(RNNLM_EINVAL, "bad qmode");
    if (qmode == RNNLM_Q_SIGDIG && (qdigits < 1 || qdigits > 3)) return fail(RNNLM_EINVAL, "qdigits must be 1..3");
    if (n < 0 || n > (1LL << 34)) return fail(RNNLM_EINVAL, "n outside [0, 2^34]");
    if (qmode == RNNLM_Q_SIGN && n % 64) return fail(RNNLM_EINVAL, "sign codes need n to be a multiple of 64");
    if (n == 0) return RNNLM_OK;
    if (!x || !codes || !err) return fail(RNNLM_EINVAL, "null pointer");
    rn::launch_debug_quantize(x, n, qmode, qdigits, decades(), codes, reinterpret_cast<int *>(err),
                              reinterpret_cast<hipStream_t>(stream));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "rnnlm_debug_quantize launch");
    return RNNLM_OK;
}

static void profile_release(rnnlm_t *ctx) {
    for (auto &pr : ctx->prof_pool) {
        (void)hipEventDestroy(pr.first);
        (void)hipEventDestroy(pr.second);
    }
    ctx->prof_pool.clear();
    ctx->prof_stage.clear();
    ctx->prof_used = 0;
}

RNNLM_API int rnnlm_profile(rnnlm_t *ctx, uint32_t stage_mask) {
    if (!ctx) return fail(RNNLM_EINVAL, "null context");
    if (stage_mask >> RNNLM_NSTAGES) return fail(RNNLM_EINVAL, "bad stage mask");
    if (stage_mask == 0) {
        profile_release(ctx);
    } else {
        ctx->prof_stage.clear();
        ctx->prof_used = 0;
    }
    ctx->prof_mask = stage_mask;
    return RNNLM_OK;
}

RNNLM_API int rnnlm_profile_read(rnnlm_t *ctx, double *ms, int64_t *launches) {
    if (!ctx || !ms || !launches) return fail(RNNLM_EINVAL, "null argument");
    for (int i = 0; i < RNNLM_NSTAGES; ++i) { ms[i] = 0.0; launches[i] = 0; }
    for (size_t k = 0; k < ctx->prof_used; ++k) {
        auto &pr = ctx->prof_pool[k];
        hipError_t e = hipEventSynchronize(pr.second);
        if (e != hipSuccess) return hip_fail(e, "rnnlm_profile_read");
        float t = 0.0f;
        e = hipEventElapsedTime(&t, pr.first, pr.second);
        if (e != hipSuccess) return hip_fail(e, "rnnlm_profile_read elapsed");
        ms[ctx->prof_stage[k]] += t;
        launches[ctx->prof_stage[k]] += 1;
    }
    return RNNLM_OK;
}

RNNLM_API void rnnlm_destroy(rnnlm_t *ctx) {
    if (!ctx) return;
    profile_release(ctx);
    delete ctx;
}
