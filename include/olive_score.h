/*
 * olive_score.h -- C ABI of the fused per-position scoring library (gfx950).
 *
 * The method trains a student on teacher continuations of its own prefixes: each
 * packed sequence is a student prefix followed by a teacher continuation, split at
 * a per-sequence cut point (Sec. 3.1, Alg. 1). This library scores such a batch in
 * one pass over the vocabulary, for a student model S and optionally a teacher
 * model T that share one vocabulary of V tokens:
 *
 *   z_X[t, v]  = s_X * sum_k h_X[t, k] * W_X[k, v]          (vocabulary projection)
 *   lse_X[t]   = log sum_v exp(z_X[t, v])                    (full-vocabulary normaliser)
 *   logp_X[t]  = z_X[t, y_t] - lse_X[t]                      (log-prob of the realised
 *                token; Eq. 1's loss is minus its sum over the continuation)
 *   kl[t]      = sum_v p_T[t, v] (log p_T[t, v] - log p_S[t, v])
 *                (KL(teacher || student), the divergence distillation minimises, Sec. 6,
 *                 reported only inside the selected region, exactly +0.0 elsewhere)
 *   argmax_X[t]= lowest v attaining max_v z_X[t, v]          (greedy token; the K = 1
 *                case of the top-K overlap statistic of Sec. 4.1)
 *   ce[b]      = - sum over scored t of sequence b of logp_S[t]   (Eq. 1, per sequence)
 *
 * s_X is the logit scale (1/temperature; the paper trains at temperature 1.0,
 * App. A, Table 3). Positions are pre-shifted: hidden row t scores targets[t].
 *
 * Conventions for every call:
 *   - All pointers named as device pointers must be device (HBM) memory on the
 *     current HIP device; host pointers are marked "host".
 *   - Calls that take a stream are asynchronous on it (0 = the null stream): they
 *     only validate host-visible arguments and enqueue kernels. The caller keeps
 *     every input and output alive until the stream has finished.
 *   - The scoring and backward calls record no memset and never synchronise, so a
 *     call may be captured into a HIP graph and replayed: a replay repeats the
 *     captured call on whatever the captured buffers then hold (the host-side
 *     arguments: shapes, region, output set and span count, are those of the capture;
 *     OLIVE_FLAG_KERNEL_TIMING's events are re-recorded into the captured slot).
 *   - No call allocates device memory except olive_score_init; every workspace is
 *     owned by the context and sized at init.
 *   - A context is not safe for concurrent use from several host threads or for
 *     overlapping calls on different streams.
 *   - Functions return an olive_status and never throw or abort.
 */
#ifndef OLIVE_SCORE_H
#define OLIVE_SCORE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct olive_score_ctx olive_score_ctx; /* opaque */

typedef enum {
    OLIVE_OK = 0,
    OLIVE_E_NULL = 1,        /* a required pointer is NULL */
    OLIVE_E_SHAPE = 2,       /* a size is <= 0, or exceeds what the context was built for */
    OLIVE_E_DTYPE = 3,       /* unknown dtype or weight layout */
    OLIVE_E_RANGE = 4,       /* a value is out of range (logit scale not finite and > 0, region) */
    OLIVE_E_HIP = 5,         /* a HIP runtime call failed */
    OLIVE_E_NOMEM = 6,       /* device allocation failed at init */
    OLIVE_E_UNSUPPORTED = 7, /* valid but not supported by this library (see each field) */
    OLIVE_E_LIMIT = 8        /* beyond the fixed limits of olive_kl_masked_static */
} olive_status;

typedef enum { OLIVE_F32 = 0, OLIVE_BF16 = 1 } olive_dtype;   /* of h and W; accumulate fp32 */

typedef enum {
    OLIVE_W_DV = 0,  /* W given as [d][V] row-major (the workloads' layout): init repacks it */
    OLIVE_W_VD = 1   /* W given as [V][d] row-major (an nn.Linear weight): borrowed, no copy */
} olive_wlayout;

typedef enum {
    OLIVE_REGION_TEACHER = 0, /* local t >= cut: the teacher continuation, Eq. 1's scored tokens */
    OLIVE_REGION_STUDENT = 1, /* local t <  cut: the student prefix (OPD scores these, Sec. 1) */
    OLIVE_REGION_ALL = 2,     /* every valid position */
    OLIVE_REGION_SPANS = 3    /* the scored spans given to olive_score_batch_spans: the
                                 teacher's actions of a multi-turn rollout (Sec. 3.2) */
} olive_region;

/* Fixed at init. */
typedef struct {
    int64_t vocab;              /* V >= 1, shared by both models, V < 2^31 */
    int32_t d_student;          /* hidden width of S, in [1, 12288] */
    int32_t d_teacher;          /* hidden width of T in [1, 12288], or 0 for student-only */
    int32_t dtype;              /* olive_dtype of h and W */
    int32_t w_layout;           /* olive_wlayout of the weights passed to init */
    float logit_scale_student;  /* s_S, finite and > 0 (1.0 = temperature 1) */
    float logit_scale_teacher;  /* s_T, finite and > 0; ignored for student-only */
    int64_t max_positions;      /* largest packed batch T a call may pass, >= 1, < 2^31 */
    int32_t max_seqs;           /* largest number of sequences B a call may pass, >= 1 */
    int32_t flags;              /* bit set of OLIVE_FLAG_* (0 = defaults) */
} olive_score_desc;

/* Force the generic fp32-FMA kernel even where the bf16 MFMA kernel applies. The
 * MFMA kernel applies to bf16 contexts whose hidden widths are multiples of 64, with
 * V >= 256 and 16-byte aligned weight and hidden-state buffers; every other case runs
 * the generic kernel, which returns the same outputs more slowly. */
#define OLIVE_FLAG_SIMPLE_KERNEL 1
/* Record HIP events around the vocabulary-scoring kernel of every call (for
 * olive_score_kernel_times); costs two event records per call. */
#define OLIVE_FLAG_KERNEL_TIMING 2
/* Reserve the workspace of the top-K statistics (olive_score_outputs' topk_* and
 * kl_topk fields). Needs a bf16 teacher context on which the MFMA kernel applies and
 * 512 <= V <= 2^23 (else init returns E_UNSUPPORTED). The workspace holds about
 * max_positions x 6.7 KB of device memory. */
#define OLIVE_FLAG_TOPK 4
/* Reserve the workspace of olive_score_backward. Needs a bf16 context on which the
 * MFMA kernel applies (else init returns E_UNSUPPORTED). The workspace holds about
 * 2 V min(max_positions, 8192) + 2 d_S V + 8 max_positions bytes of device memory, plus
 * 4 (V / 256 + 2) min(max_positions, 8192) bytes (3.1 GB for V = 151936, d_S = 2048 and
 * 8192 or more positions). */
#define OLIVE_FLAG_BACKWARD 8
/* Score with the 256 x 128 two-model MFMA kernel instead of the 256 x 256 one. Without
 * this flag a bf16 context on which the MFMA kernel applies keeps K-blocked copies of its
 * weights and a panel buffer for the hidden rows of a call (2 (V rounded up to 256 +
 * max_positions rounded up to 256) (d_S + d_T) bytes of device memory, d_T = 0 for a
 * student-only context: 1.9 GB + 0.4 GB for V = 151936, d_S + d_T = 6144 and 32768
 * positions), and its student-only calls, calls with one KL direction (kl or kl_reverse,
 * not both) and no top-K output, and olive_score_backward's student passes (the
 * cross-entropy alone in one sweep that forms its own normalisers, else the normaliser
 * pass) run the 256 x 256 kernel. That kernel forms KL's cross term with the softmax weights of the
 * divergence's first distribution (p_T for kl, p_S for kl_reverse) held in fp16 and
 * normalised by their own sum (Sec. 6's KL; the weights' rounding moves a KL value by at
 * most 2^-11 (1 - 2^-11)^-1 times the mean absolute deviation of the logit difference
 * under that distribution, which is at most 2 (KL + TV)); every other output is formed
 * as in the 256 x 128 kernel. */
#define OLIVE_FLAG_NARROW_TILE 16

/* One packed batch of stitched sequences (Sec. 3.1: x, y_1..k, continuation). */
typedef struct {
    int32_t num_seqs;            /* B >= 1 (<= desc.max_seqs) */
    int32_t region;              /* olive_region selecting where kl and ce are taken */
    int64_t total_positions;     /* T = cu_seqlens[B] (host copy of it), 0 < T <= max_positions */
    const int32_t *cu_seqlens;   /* device [B+1]: cu[0] = 0, nondecreasing, cu[B] = T */
    const int32_t *cut;          /* device [B]: local cut index in [0, len_b] */
    const int32_t *valid_len;    /* device [B] or NULL (= len_b): positions t >= valid_len_b
                                    (past an end-of-sequence) are not scored; in [0, len_b] */
    const int32_t *targets;      /* device [T]: realised token of each position, in [0, V) */
    const void *h_student;       /* device [T][d_student] row-major, desc.dtype */
    const void *h_teacher;       /* device [T][d_teacher] row-major, or NULL (student only) */
} olive_batch;

/*
 * Create a scoring context for one pair of projection weights.
 *   out        host: receives the context (NULL on failure).
 *   desc       host: sizes, dtype, layout, scales (copied).
 *   w_student  device: W_S in desc.w_layout ([d_S][V] or [V][d_S]).
 *   w_teacher  device: W_T likewise, or NULL when desc.d_teacher == 0.
 *   hip_stream the stream the repack runs on; init synchronises it before returning.
 * With OLIVE_W_DV the context owns a repacked [V][d] copy of each weight; with
 * OLIVE_W_VD it borrows the caller's buffers, which must outlive the context.
 * Errors: E_NULL, E_SHAPE, E_DTYPE, E_RANGE, E_NOMEM, E_HIP.
 */
olive_status olive_score_init(olive_score_ctx **out, const olive_score_desc *desc,
                              const void *w_student, const void *w_teacher, void *hip_stream);

/*
 * Per-position log-probs and greedy tokens of both models (Eq. 1's summands, at
 * every valid position, prefix and continuation alike).
 *   logp_student  device [T] fp32: logp_S, 0 at positions past the valid length.
 *   logp_teacher  device [T] fp32 or NULL; must be NULL on a student-only context
 *                 or when b->h_teacher is NULL.
 *   argmax_student, argmax_teacher  device [T] int32 or NULL: greedy token, -1 past
 *                 the valid length.
 * Errors: E_NULL, E_SHAPE, E_RANGE, E_UNSUPPORTED, E_HIP. Content errors found on the
 * device (a target outside [0, V), a cut or valid length outside [0, len_b], a
 * decreasing cu_seqlens) set the context's device error word (olive_score_last_error)
 * and make the affected outputs NaN.
 */
olive_status olive_token_logprobs(olive_score_ctx *ctx, const olive_batch *b,
                                  float *logp_student, float *logp_teacher,
                                  int32_t *argmax_student, int32_t *argmax_teacher,
                                  void *hip_stream);

/*
 * The fused scoring of both models in one pass: masked KL(teacher || student) per
 * position, the counts, and optionally every output of olive_token_logprobs and
 * Eq. 1's per-sequence loss. Needs a teacher context and b->h_teacher.
 *   kl          device [T] fp32: KL in the region, exactly +0.0 elsewhere.
 *   counts      device [2] int64 or NULL: counts[0] = positions in the region and
 *               valid (scored), counts[1] = valid positions.
 *   logp_*, argmax_*  as in olive_token_logprobs, each may be NULL.
 *   ce_per_seq  device [B] fp32 or NULL: minus the sum of logp_S over the scored
 *               positions of each sequence (0 for an empty region).
 * Errors: as olive_token_logprobs, plus E_UNSUPPORTED on a student-only context.
 */
olive_status olive_kl_masked(olive_score_ctx *ctx, const olive_batch *b, float *kl,
                             int64_t *counts, float *logp_student, float *logp_teacher,
                             int32_t *argmax_student, int32_t *argmax_teacher,
                             float *ce_per_seq, void *hip_stream);

/* Score only the region's positions: log-probs and greedy tokens outside the region
 * get the fixed values of positions past the valid length (0 and -1), and the
 * vocabulary pass covers the scored positions only, so its cost scales with the
 * scored count instead of the valid count (Eq. 1 needs the region alone). */
#define OLIVE_OUT_REGION_ONLY 1

/*
 * Output set of olive_score_batch. Every pointer may be NULL (that output is not
 * formed); at least one must be set. Device buffers, caller-owned, as in
 * olive_kl_masked.
 */
typedef struct {
    int32_t size;                /* host: sizeof(olive_score_outputs) (checked) */
    int32_t flags;               /* bit set of OLIVE_OUT_* (0 = defaults) */
    float *kl;                   /* [T] fp32: KL(teacher || student) in the region, +0.0
                                    elsewhere (the divergence distillation minimises, Sec. 6) */
    float *kl_reverse;           /* [T] fp32: KL(student || teacher), masked the same way (the
                                    per-token objective of on-policy distillation, Sec. 1) */
    int64_t *counts;             /* [2] int64: scored (region and valid) and valid positions */
    float *logp_student;         /* [T] fp32, as in olive_token_logprobs */
    float *logp_teacher;         /* [T] fp32 */
    int32_t *argmax_student;     /* [T] int32 */
    int32_t *argmax_teacher;     /* [T] int32 */
    float *ce_per_seq;           /* [B] fp32: Eq. 1's loss per sequence */
    /* Top-K statistics, K = 16 (need OLIVE_FLAG_TOPK at init and a teacher). TopK_X is
     * the set of model X's 16 largest logits, larger value first and the lower
     * vocabulary index first among equal values. At scored positions: */
    float *topk_overlap;         /* [T] fp32: |TopK_S & TopK_T| / 16 (Sec. 4.1's top-K
                                    overlap ratio), +0.0 at other valid positions */
    float *kl_topk;              /* [T] fp32: sum over v in TopK_T of
                                    p_T(v) (log p_T(v) - log p_S(v)) with the full-vocabulary
                                    normalisers: the top-16 approximation of KL(teacher ||
                                    student) (App. A, Table 3), +0.0 elsewhere */
    int32_t *topk_student;       /* [T][16] int32: TopK_S in rank order, -1 elsewhere */
    int32_t *topk_teacher;       /* [T][16] int32: TopK_T in rank order, -1 elsewhere */
    /* Appended field: a caller built against the layout without it passes the smaller
     * size (offsetof(olive_score_outputs, jsd)) and is served as before. */
    float *jsd;                  /* [T] fp32: the Jensen-Shannon divergence
                                    1/2 KL(p_S || m) + 1/2 KL(p_T || m), m = (p_S + p_T) / 2,
                                    in the region, +0.0 elsewhere: the symmetric companion
                                    of the reverse KL of on-policy distillation (Sec. 1).
                                    Formed by a second pass over the vocabulary for the
                                    scored positions; needs the MFMA path (E_UNSUPPORTED
                                    otherwise) */
} olive_score_outputs;

/*
 * Scored spans of a multi-turn batch (Sec. 3.2): the student's turns and every
 * environment observation stay in the context, only the teacher's actions are
 * scored. Spans are local, half-open [start, end), per sequence increasing and
 * disjoint, 0 <= start <= end <= len_b; a position is scored when it lies in one
 * of its sequence's spans and before the sequence's valid length.
 */
typedef struct {
    int32_t size;                /* host: sizeof(olive_spans) (checked) */
    int32_t num_spans;           /* S >= 0: spans over the whole batch */
    const int32_t *span_offsets; /* device [B+1]: sequence b's spans are entries
                                    [off[b], off[b+1]); off[0] = 0, nondecreasing, off[B] = S */
    const int32_t *spans;        /* device [S][2]: (start, end) pairs; may be NULL when S = 0 */
} olive_spans;

/*
 * Every per-position output of one batch in one fused pass over the vocabulary:
 * olive_kl_masked's outputs plus the reverse KL and the top-K statistics (and, in a
 * second pass over the scored positions, the Jensen-Shannon divergence). Teacher
 * outputs (kl, kl_reverse, jsd, logp_teacher, argmax_teacher and every top-K output)
 * need a teacher context and b->h_teacher. Malformed sequences give NaN (top-K indices -1)
 * as for the other outputs.
 * Errors: E_NULL (out, or every output pointer, NULL), E_RANGE (out->size wrong or
 * unknown flags), E_UNSUPPORTED (a top-K output without OLIVE_FLAG_TOPK at init, a
 * top-K output or jsd where the MFMA kernel does not apply, e.g. hidden states that
 * are not 16-byte aligned), and as olive_kl_masked.
 */
olive_status olive_score_batch(olive_score_ctx *ctx, const olive_batch *b,
                               const olive_score_outputs *out, void *hip_stream);

/*
 * olive_score_batch with a span region: b->region must be OLIVE_REGION_SPANS and
 * b->cut may be NULL (it is not read). kl, kl_reverse and ce_per_seq are taken over
 * the spans; log-probs and greedy tokens at every valid position as usual.
 * Errors: as olive_score_batch, plus E_NULL (spans, or its arrays while S > 0),
 * E_RANGE (spans->size wrong, S < 0, or b->region not OLIVE_REGION_SPANS). Malformed
 * offsets or spans found on the device set bit 16 of the device error word and make
 * the affected sequences' outputs NaN (all of them for bad offsets).
 */
olive_status olive_score_batch_spans(olive_score_ctx *ctx, const olive_batch *b,
                                     const olive_spans *spans, const olive_score_outputs *out,
                                     void *hip_stream);

/*
 * Gradient outputs of olive_score_backward. L = w_ce * sum_b CE_b (Eq. 1's loss, summed
 * over the sequences) + w_kl * sum over the region's positions of KL(p_T || p_S): the
 * student's update step on the masked CE loss (the update of Alg. 1, Eq. 1, Sec. 3.1),
 * with an optional distillation term. Device buffers, caller-owned, overwritten.
 */
typedef struct {
    int32_t size;                /* host: sizeof(olive_grad_outputs) (checked) */
    int32_t flags;               /* 0 or OLIVE_GRAD_REUSE_FORWARD */
    float w_ce;                  /* weight of the CE sum, finite */
    float w_kl;                  /* weight of the KL sum, finite; 0 leaves the teacher out
                                    (its hidden states may then be NULL) */
    float *grad_h_student;       /* [T][d_S] fp32 or NULL: dL/dh_S, +0.0 at positions
                                    outside the region or past the valid length */
    float *grad_w_student;       /* fp32 or NULL: dL/dW_S in the context's weight layout,
                                    [d_S][V] (OLIVE_W_DV) or [V][d_S] (OLIVE_W_VD) */
    int64_t *counts;             /* [2] int64 or NULL: scored and valid positions */
} olive_grad_outputs;

/* olive_grad_outputs.flags: take the log-normalisers (lse_S, and lse_T when w_kl != 0)
 * from the last forward call on this context (olive_score_batch, _spans, olive_kl_masked,
 * olive_token_logprobs) instead of recomputing them, which saves one MFMA pass over the
 * student's (and teacher's) vocabulary. That call must have run on the MFMA path with
 * the same batch: the same sizes, region, spans and device pointers, holding the same
 * data (the caller's part: contents are not compared), and must be ordered before the
 * backward (the same stream, or the caller's synchronisation). Otherwise, or after a
 * backward without this flag has replaced the normalisers, or when w_kl != 0 and that
 * call scored the student only, the backward returns E_RANGE. */
#define OLIVE_GRAD_REUSE_FORWARD 1

/*
 * Backward pass of the student's loss: dL/dh_S and dL/dW_S for the scaled logits
 * z_S = s_S h_S W_S. Per scored position the logit gradient is
 * w_ce (p_S - onehot(y)) + w_kl (p_S - p_T); it is formed in one fused pass over the
 * vocabulary (recomputing the student's logits, and the teacher's when w_kl != 0, from
 * the forward normalisers; for the cross-entropy alone without reused normalisers on a
 * context with the 256 x 256 kernel, the same pass forms the normalisers and stores the
 * weights exp(s_S z - m) of each vocabulary tile, m its running max, in fp16 (2^15
 * scaled), which one more pass over the stored values rescales) and held
 * in bf16 (round to nearest even) as the operand of the two products
 * dL/dh = s_S g W^T and dL/dW = s_S h^T g, which accumulate in fp32.
 * spans: NULL, or the scored spans when b->region is OLIVE_REGION_SPANS.
 * Errors: E_NULL (g, or both gradient pointers, NULL; a required batch pointer NULL),
 * E_RANGE (g->size or flags wrong, OLIVE_GRAD_REUSE_FORWARD without a matching forward
 * call, a weight not finite, region / spans as for
 * olive_score_batch_spans), E_UNSUPPORTED (no OLIVE_FLAG_BACKWARD at init; w_kl != 0
 * without a teacher; hidden states not 16-byte aligned), E_SHAPE as olive_kl_masked.
 * Content errors on the device set the error word as in the forward calls and make
 * the gradients of the affected rows (and so dL/dW) NaN.
 */
olive_status olive_score_backward(olive_score_ctx *ctx, const olive_batch *b,
                                  const olive_spans *spans, const olive_grad_outputs *g,
                                  void *hip_stream);
/* With OLIVE_GRAD_REUSE_FORWARD the backward is the logit-gradient pass and the two
 * products only: a training step's forward call supplies the normalisers. */

/*
 * olive_kl_masked without a context, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the call allocates nothing. Its per-call workspace lives in a fixed
 * device array of 24 MiB that the library holds on each GPU it runs on until the process
 * ends; the weights are read in place.
 *   desc       host: as for olive_score_init, with w_layout = OLIVE_W_VD (the weights are
 *              borrowed, not repacked), a teacher (d_teacher > 0), flags 0 or
 *              OLIVE_FLAG_SIMPLE_KERNEL (else E_UNSUPPORTED), and the limits
 *              max_positions <= 8192, max_seqs <= 256, vocab <= 262144 (else E_LIMIT).
 *   w_student, w_teacher  device: [V][d_S] and [V][d_T] row-major, desc.dtype.
 *   b and every output as in olive_kl_masked (the same values, within the same
 *   acceptance bars: the kernels are those of olive_kl_masked).
 * Every call on one GPU uses that GPU's one array and leaves its contents behind (each
 * call writes what it reads, nothing needs clearing): calls that overlap on one GPU
 * (several streams or host threads) race and must not be issued. The device error word
 * is not reported: content errors make the affected outputs NaN as in olive_kl_masked.
 * Each call first forms the weight-row norms that bound the rounding of the exact
 * greedy decisions (one read of both weight matrices).
 * Errors: E_NULL, E_DTYPE, E_SHAPE, E_RANGE, E_UNSUPPORTED, E_LIMIT, E_HIP, and the
 * checks of olive_kl_masked on the batch.
 */
olive_status olive_kl_masked_static(const olive_score_desc *desc, const void *w_student,
                                    const void *w_teacher, const olive_batch *b, float *kl,
                                    int64_t *counts, float *logp_student, float *logp_teacher,
                                    int32_t *argmax_student, int32_t *argmax_teacher,
                                    float *ce_per_seq, void *hip_stream);

/* Release a context and everything it owns (NULL is accepted). Synchronises the device. */
olive_status olive_score_free(olive_score_ctx *ctx);

/* A static, NUL-terminated description of a status code (never NULL). */
const char *olive_status_string(olive_status s);

/*
 * Read and clear the context's device error word (synchronises the device).
 *   device_code host: receives a bit set, 0 when no content error occurred:
 *   1 = target out of [0, V), 2 = cut out of [0, len], 4 = valid_len out of [0, len],
 *   8 = cu_seqlens not nondecreasing from 0 or cu[B] != T, 16 = span offsets or spans
 *   malformed (olive_score_batch_spans).
 */
olive_status olive_score_last_error(olive_score_ctx *ctx, int32_t *device_code);

/*
 * Diagnostics of the last scoring call (synchronises the device).
 *   out host [6] int64: [0] vocabulary splits used, [1] rows whose greedy token was
 *   re-decided from exact logits (bf16 products summed in fp64) because the gap between
 *   their two largest fp32 logits was at most 2^-14 max(1, |s max|); every such row of
 *   the call is re-decided (the list holds max_positions rows),
 *   [2] kernel id (0 = MFMA bf16 256 x 128, 1 = generic, 2 = MFMA bf16 256 x 256),
 *   [3] persistent workgroups launched,
 *   [4] (position, model) pairs whose top-K set needed a filter pass over the
 *   vocabulary, [5] pairs of those that needed an exhaustive exact scan (more than
 *   256 near-tied candidates); [4] and [5] are 0 without top-K outputs.
 */
olive_status olive_score_last_stats(olive_score_ctx *ctx, int64_t *out);

/*
 * Durations of the vocabulary-scoring kernel (the fused projection + softmax pass)
 * of the last n calls, oldest first, from events recorded on the call's stream
 * (synchronises the device). Needs OLIVE_FLAG_KERNEL_TIMING at init.
 *   out host [n] fp32: milliseconds; n in [1, 64] and at most the number of calls
 *   made since init. Errors: E_NULL, E_RANGE (n out of range), E_UNSUPPORTED (no
 *   timing flag), E_HIP.
 */
olive_status olive_score_kernel_times(olive_score_ctx *ctx, float *out, int32_t n);

#ifdef __cplusplus
}
#endif

#endif /* OLIVE_SCORE_H */
