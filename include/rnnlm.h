/*
 * rnnlm.h -- C ABI of a frame-wise RNNLM query scorer for AMD MI355X (gfx950).
 *
 * Method: Lee, Park, Kim, Lee, "Accelerating recurrent neural network language
 * model based online speech recognition system", arXiv 1801.09866.
 *
 * A decoder emits, per decoding frame, LM queries = (history, next word). The
 * library scores a whole frame per call (the paper's frame-wise batching,
 * Sec. 4): each history vector is quantised (Sec. 3: exact, sign only, or k
 * significant digits), keyed together with the word fed to the GRU, and
 * de-duplicated against the frame and a GPU-resident history cache (Sec. 3,
 * Fig. 2); each query is keyed by its history key, MaxEnt context words and
 * target word and de-duplicated against the frame and an LM-query cache
 * (Sec. 2.4, Fig. 1). Every history key not cached runs one GRU step
 * (Sec. 2.1); every query not cached gets the unnormalised NCE score of its
 * target word (Sec. 2.2) plus hashed n-gram MaxEnt weights (Sec. 2.3).
 *
 * Memory: every pointer argument is DEVICE memory owned by the caller unless
 * stated otherwise. Weights are borrowed and must outlive the context. The
 * library allocates no device memory of its own: packed weights, caches and
 * per-frame scratch live in the caller's workspace (rnnlm_workspace_size).
 * The context object itself is a small host allocation. The one exception is
 * a 4 MiB static device array per GPU, the scratch of the allocation-free
 * rnnlm_log_normalizer_static.
 *
 * Streams: `stream` arguments are hipStream_t values passed as void* (NULL =
 * the default stream). All work is enqueued on that stream and nothing blocks
 * the host, except rnnlm_create (which synchronises once) and rnnlm_get_stats.
 * A context is used by one host thread at a time; calls on one context must be
 * ordered on one stream.
 *
 * Errors: functions return RNNLM_OK (0) or a negative code and never throw.
 * Host-checkable problems (null pointers, sizes above the configured maxima,
 * bad config) return RNNLM_EINVAL before enqueueing anything. Problems only
 * the device can see (a word id outside [0, V), a query's history index
 * outside the frame, a non-finite history element, or |x| > 1 under decimal
 * rounding) set bits of a sticky device flag; the offending ids are clamped so
 * no access leaves its buffer, and that frame's outputs are unspecified.
 * rnnlm_get_stats reports the flag and returns RNNLM_EDEVICE; afterwards
 * rnnlm_score_frame returns RNNLM_EDEVICE until rnnlm_cache_reset clears it.
 * rnnlm_last_error() returns a message for the calling thread's last failure.
 */
#ifndef RNNLM_H
#define RNNLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { RNNLM_OK = 0, RNNLM_EINVAL = -1, RNNLM_ENOMEM = -2, RNNLM_EHIP = -3, RNNLM_EDEVICE = -4 };

/* History quantisation (Sec. 3, Table 1): EXACT keeps the fp32 bits (-0 = +0);
 * SIGN keeps only x < 0 per element; SIGDIG rounds to `qdigits` (1..3)
 * significant decimal digits, ties away from zero, elements in [-1, 1]. */
enum { RNNLM_Q_EXACT = 0, RNNLM_Q_SIGN = 1, RNNLM_Q_SIGDIG = 2 };
/* Weight precision: fp32, or bf16 embedding / GRU / output weights with fp32
 * accumulation (biases and MaxEnt weights stay fp32). */
enum { RNNLM_F32 = 0, RNNLM_BF16 = 1 };
/* Per-history status (the history cache of Sec. 3, Fig. 2): key cached before
 * this frame (HC_HIT); first of its key in the frame, GRU computed (H_REP);
 * later copy of a key in the frame (H_DUP). */
enum { RNNLM_H_REP = 0, RNNLM_H_DUP = 1, RNNLM_HC_HIT = 2 };
/* Per-query status (the LM-query cache of Sec. 2.4, Fig. 1): score computed
 * (COMPUTED); copy of an earlier query of the frame with the same key
 * (Q_DUP); stored score returned (SCORE_HIT). */
enum { RNNLM_Q_COMPUTED = 0, RNNLM_Q_DUP = 1, RNNLM_Q_SCORE_HIT = 2 };
/* Sticky device error bits, for input the method cannot key or score (an id
 * outside the vocabulary, a value outside the quantiser's domain of Sec. 3,
 * a query naming no history of its frame; HANDLE: a null or misaligned
 * history handle). */
enum { RNNLM_DERR_WORD = 1, RNNLM_DERR_QHIST = 2, RNNLM_DERR_VALUE = 4, RNNLM_DERR_HANDLE = 8 };

typedef struct rnnlm_t rnnlm_t;   /* opaque */

typedef struct {
    int32_t V;             /* vocabulary size; word 0 is the sentence start */
    int32_t E;             /* embedding width; multiple of 64 */
    int32_t H;             /* GRU width; multiple of 64 */
    int32_t L;             /* stacked GRU layers, 1 or 2 */
    int32_t wdtype;        /* RNNLM_F32 or RNNLM_BF16 */
    int32_t maxent_log2;   /* MaxEnt table has 2^maxent_log2 weights, 1..30 */
    int32_t maxent_order;  /* n-gram orders 2..maxent_order are summed (1..4; 1 = none) */
    int32_t qmode;         /* RNNLM_Q_* */
    int32_t qdigits;       /* significant digits for RNNLM_Q_SIGDIG, 1..3 */
    int32_t max_hist;      /* largest n_hist of any frame, 1..2048 */
    int32_t max_query;     /* largest n_query of any frame, 0..8192 */
    int32_t sessions;      /* independent decode sessions, 1..8 (0 means 1): each has its own caches and
                            * statistics, and rnnlm_score_frames scores one frame of each per call */
    int64_t cap_hist;      /* history-cache entries per session (admission stops when full) */
    int64_t cap_query;     /* LM-query cache entries per session */
    uint64_t seed;         /* seed of the history-key hash */
} rnnlm_config;

typedef struct {
    const void *emb;       /* [V][E], wdtype */
    const void *W_ih[2];   /* layer l: [3H][Kx], Kx = E (l = 0) or H; gate blocks (reset, update, candidate); wdtype */
    const void *W_hh[2];   /* layer l: [3H][H], same gate blocks; wdtype */
    const float *b_ih[2];  /* layer l: [3H] fp32; the recurrent bias is zero */
    const void *U_out;     /* [V][H] NCE output rows, wdtype */
    const float *b_out;    /* [V] fp32 */
    const float *maxent;   /* [2^maxent_log2] fp32 */
} rnnlm_weights;

typedef struct {
    int32_t n_hist;             /* history records in this frame, <= max_hist */
    int32_t n_query;            /* queries in this frame, <= max_query */
    const float *hist_vec;      /* [n_hist][L*H] fp32, layer-major concatenation of the layer states */
    const int32_t *hist_words;  /* [n_hist][3]: (w-1, w-2, w-3); w-1 is the GRU input word; BOS = 0 pads */
    const int32_t *q_hist;      /* [n_query] index into this frame's histories */
    const int32_t *q_tgt;       /* [n_query] target word */
    /* Optional history handles, for closing the decode loop without copies
     * (a hypothesis extended in frame t has as history the h' of frame t):
     * [n_hist] device addresses, each of one history's L*H fp32 row, for
     * instance a row of an earlier frame's hnew output. When non-NULL,
     * hist_vec is not read and may be NULL. Each address must be 16-byte
     * aligned and point at L*H readable floats that are not written while
     * the frame runs; a NULL or misaligned one sets RNNLM_DERR_HANDLE (a
     * placeholder row is read instead). */
    const uint64_t *hist_ptr;
} rnnlm_frame;

typedef struct {
    float *scores;      /* [n_query] fp32 log-domain scores (required when n_query > 0) */
    float *hnew;        /* [n_hist][L*H] GRU outputs per history record (nullable) */
    uint8_t *q_status;  /* [n_query] RNNLM_Q_* (nullable) */
    int32_t *q_rep;     /* [n_query] lowest query index with the same key (nullable) */
    uint8_t *h_status;  /* [n_hist] RNNLM_H_* (nullable) */
    int32_t *h_rep;     /* [n_hist] lowest history index with the same key (nullable) */
    uint64_t *h_hash;   /* [n_hist] 64-bit hash of the history key (nullable) */
} rnnlm_out;

typedef struct {
    int64_t frames, queries, score_hits, query_dups, computed;
    int64_t hists, hist_hits, hist_dups, gru_rows;
    int64_t hist_inserted, hist_rejected, score_inserted, score_rejected;
    int64_t hist_cache_size, score_cache_size;
    int32_t device_error;  /* RNNLM_DERR_* bits */
    int32_t pad;
} rnnlm_stats;

/* Bytes of device workspace a context with this config needs (256-byte
 * aligned base required). Returns RNNLM_EINVAL for an invalid config. */
int rnnlm_workspace_size(const rnnlm_config *cfg, size_t *bytes);

/* Bind weights (device pointers, borrowed), carve up `workspace` (device,
 * caller-owned, >= rnnlm_workspace_size bytes), pack the GRU weights, and
 * empty both caches. Synchronises `stream` once. *out receives the context. */
int rnnlm_create(const rnnlm_config *cfg, const rnnlm_weights *w, void *workspace,
                 size_t ws_bytes, void *stream, rnnlm_t **out);

/* Score one frame (Sec. 2.4 + Sec. 3 + Sec. 4): quantise, key and de-duplicate
 * the histories and queries, run the GRU for uncached history keys, score the
 * uncached queries, fill `out`, then admit the frame's new keys to the caches
 * in ascending index while capacity lasts (a query's score is only admitted
 * when its history key is cached). Asynchronous on `stream`. Only this call's
 * kernels read the frame's inputs (and, through hist_ptr, the rows it names):
 * once they have completed in stream order, the caller may reuse those
 * buffers, e.g. as the target of the next frame's host-to-device copy. The
 * call only enqueues kernels (no allocation, memset or synchronisation), so
 * a sequence of frames may be captured into a HIP graph and replayed from
 * the same cache state (stage timing off). */
int rnnlm_score_frame(rnnlm_t *ctx, const rnnlm_frame *frame, const rnnlm_out *out, void *stream);

/* A block of independent frames in one set of launches (Sec. 4 batches a
 * frame's queries into one transfer; this batches frames of independent
 * decoders into one launch): frames[k] (host array of n <= sessions) is the
 * next frame of session k, scored against session k's caches exactly as
 * rnnlm_score_frame would, with its outputs in outs[k]. Empty frames take no
 * part. Sessions share the weights and the launches; with n = 1 this is
 * rnnlm_score_frame on session 0. Errors as rnnlm_score_frame (a host check
 * failing for any frame enqueues nothing). */
int rnnlm_score_frames(rnnlm_t *ctx, const rnnlm_frame *frames, const rnnlm_out *outs, int32_t n, void *stream);

/* Empty both caches of every session -- the LM-query cache (Sec. 2.4, Fig. 1)
 * and the history cache (Sec. 3, Fig. 2), for instance between utterances --
 * zero the statistics and clear the sticky device flag. Asynchronous on
 * `stream` (fill kernels, no memset); returns RNNLM_EINVAL for a null
 * context. */
int rnnlm_cache_reset(rnnlm_t *ctx, void *stream);

/* Full-vocabulary log normaliser (the computation NCE avoids, Sec. 2.2):
 * logz[i] = log sum_v exp(U_out[v] . h_top[i] + b_out[v]) for i < n.
 * h_top: [n][H] fp32 device; logz: [n] fp32 device; n <= max_hist. */
int rnnlm_log_normalizer(rnnlm_t *ctx, const float *h_top, int32_t n, float *logz, void *stream);

/* The same normaliser over the full model output: every word's logit also
 * gets its hashed n-gram MaxEnt weights (Sec. 2.3) after history i's context,
 *   logz[i] = log sum_v exp(U_out[v] . h_top[i] + b_out[v]
 *                           + sum_{o=2..N} maxent[slot_o(words[i], v)]),
 * with the slots the scores use. words: [n][3] int32 device, (w-1, w-2, w-3)
 * of each history (the word of the GRU step that made h_top[i] is w-1 of the
 * next step, so pass the context of the queries to be normalised). A word
 * outside [0, V) sets RNNLM_DERR_WORD and is read as 0. Other arguments and
 * errors as rnnlm_log_normalizer. */
int rnnlm_log_normalizer_maxent(rnnlm_t *ctx, const float *h_top, const int32_t *words, int32_t n, float *logz,
                                void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * normaliser of rnnlm_log_normalizer without a context or workspace,
 *   logz[i] = log sum_v exp(U_out[v] . h_top[i] + b_out[v]),  i < n,
 * computed by the same kernels. U_out: [V][H] fp32, b_out: [V] fp32, h_top:
 * [n][H] fp32, logz: [n] fp32, all device memory owned by the caller; h_top
 * and U_out 16-byte aligned; H a multiple of 64, at most 2048; any n >= 0.
 * The partial (max, sum) pairs live in a static device array of the library
 * (4 MiB, one per GPU, held until the process ends), so V is at most 425,984;
 * a larger V, a bad H or a null pointer returns RNNLM_EINVAL before anything
 * is enqueued. The call allocates nothing and issues no memset: two kernel
 * launches per 256 rows on `stream`. Calls that overlap on one GPU (other
 * streams, other host threads) share that array and race; order them. */
int rnnlm_log_normalizer_static(const float *U_out, const float *b_out, int32_t V, int32_t H,
                                const float *h_top, int32_t n, float *logz, void *stream);

/* Copy the device statistics, summed over all sessions, into *stats (host
 * memory); synchronises `stream`. The counts are those Table 1 of Sec. 3
 * compares across history compressions (unique LM queries = computed, GRU
 * rows) and the two caches' hits and sizes (Sec. 2.4, Sec. 3). Returns
 * RNNLM_EDEVICE if the sticky device flag of any session is set
 * (device_error: the OR of all sessions' bits). */
int rnnlm_get_stats(rnnlm_t *ctx, rnnlm_stats *stats, void *stream);

/* The same for one session (0 <= session < sessions); a device error in any
 * session still returns RNNLM_EDEVICE. */
int rnnlm_get_session_stats(rnnlm_t *ctx, int32_t session, rnnlm_stats *stats, void *stream);

/* Test hook: quantise n fp32 elements x with the library's own kernel
 * (the history compression of Sec. 3: sign only, or k significant digits).
 * codes: EXACT -> uint32[n]; SIGDIG -> uint16[n]; SIGN -> uint64[n/64]
 * (n a multiple of 64; element i is bit i%64 of word i/64). err: one device
 * int32 that receives RNNLM_DERR_VALUE if an element was out of domain
 * (it is OR-ed, so clear it first). */
int rnnlm_debug_quantize(int32_t qmode, int32_t qdigits, const float *x, int64_t n,
                         void *codes, int32_t *err, void *stream);

/* Benchmark hook: per-stage kernel timing. Stages (bit i of stage_mask):
 * 0 history keys, 1 frame plan (de-duplication, cache probes, admission),
 * 2 GRU GEMM (all layers), 3 scoring and frame finish, 8 normaliser GEMM,
 * 9 normaliser combine. A timed stage's kernels are launched with a HIP
 * start/stop event pair that their dispatch packets stamp (hipExtLaunchKernel),
 * so a stage's time runs from the start of its first kernel to the end of its
 * last and excludes the gaps between stages. stage_mask = 0 turns timing off
 * and releases the events. The events are host-side HIP objects; no device
 * memory is allocated. */
enum { RNNLM_NSTAGES = 10 };
int rnnlm_profile(rnnlm_t *ctx, uint32_t stage_mask);

/* Sum of kernel time (ms) and number of timed launches per stage since the
 * last rnnlm_profile call; synchronises on the recorded events (host arrays
 * of RNNLM_NSTAGES entries). */
int rnnlm_profile_read(rnnlm_t *ctx, double *ms, int64_t *launches);

/* Release the host-side context (the workspace stays the caller's). */
void rnnlm_destroy(rnnlm_t *ctx);

/* Message describing the calling thread's most recent failure ("" if none). */
const char *rnnlm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* RNNLM_H */
