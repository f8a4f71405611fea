// Host side of the C ABI declared in include/olive_score.h: argument validation,
// workspace ownership, and the per-call launch sequence
//   prep -> rowmap -> score (MFMA or generic) -> combine -> [fixup] -> [top-K] -> [ce].
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstddef>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "olive_internal.hpp"

using namespace olive;

// Scratch of olive_kl_masked_static (one copy per GPU, held until the process ends). In
// host code this name is a host-side stand-in, not a device address: each GPU's copy is
// reached through the address hipGetSymbolAddress returns for it.
constexpr size_t kStaticScratchBytes = (size_t)24 << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

struct olive_score_ctx {
    olive_score_desc desc;
    int device = 0;
    int n_cu = 0;
    const void *ws = nullptr, *wt = nullptr;   // [V][d] weights used by the kernels
    void *ws_own = nullptr, *wt_own = nullptr; // repacked copies (OLIVE_W_DV)
    uint32_t *rowmap = nullptr;
    int32_t *seqbuf = nullptr;
    Sched *sched = nullptr;
    float *part = nullptr;
    int64_t pstride = 0;
    float *logp_tmp = nullptr;
    float *lse_buf = nullptr;                   // [P][2] normalisers for the JSD pass
    int32_t *flagged = nullptr;
    int flag_cap = 0;                           // rows the near-tie list holds: max_positions
    int fx_window = 0;                          // generic path: flagged rows per window
    void *fx_scratch = nullptr;
    float *wn_s = nullptr, *wn_t = nullptr;     // weight-row L2 norms (rounding bounds)
    float wmax_s = 0.f, wmax_t = 0.f;           // their maxima
    const float *wmax_dev = nullptr;            // or the maxima in device memory
    int32_t *err = nullptr;
    void *tk_buf = nullptr;                     // top-K workspace (OLIVE_FLAG_TOPK)
    TopkWork tkw = {};
    void *fx_buf = nullptr;                     // greedy re-decision queue (MFMA path)
    FilterQueue fxq = {};
    // backward workspace (OLIVE_FLAG_BACKWARD)
    bool bw = false;
    int bw_chunk = 0;                           // scored rows per logit-gradient chunk
    int64_t bw_vp = 0;                          // V rounded up to 64
    float *bw_lse = nullptr;                    // [P][2]
    uint16_t *bw_wt = nullptr;                  // W_S^T panels [bw_vp/64][d_S][64] bf16
    uint16_t *bw_dzt = nullptr;                 // panels [bw_vp/64][chunk][64]
    uint16_t *bw_hrt = nullptr;                 // [d_S][chunk]
    float *bw_mref = nullptr;                   // [vocabulary tiles][chunk], then gy [chunk]
                                                // and yrow [chunk] (int32)
    // Normalisers of the last forward call on the MFMA path and the batch they belong
    // to, for a backward on that batch (OLIVE_GRAD_REUSE_FORWARD). Scored rows take the
    // same compacted index in every pass (scored-first compaction), so the forward's
    // rows [0, n_scored) are the backward's.
    const float *fwd_lse = nullptr;             // bw_lse, or the top-K workspace's
    bool fwd_lse_ok = false, fwd_lse_t = false; // valid; holds lse_T too
    olive_batch fwd_batch = {};
    bool fwd_spans = false;
    olive_spans fwd_sp = {};
    // 256 x 256 kernel (forward KL calls with a teacher on the MFMA path): K-blocked
    // panels of both weights (made at init) and of a call's compacted hidden rows
    bool wide = false;
    uint16_t *wp_s = nullptr, *wp_t = nullptr;  // [d/32][wp_rows][32]
    uint16_t *hp_s = nullptr, *hp_t = nullptr;  // [d/32][hp_rows][32]
    int64_t wp_rows = 0, hp_rows = 0;
    bool bf16 = false, has_t = false, mfma_ok = false, topk = false;
    int last_kernel = -1, last_grid = 0;
    bool timing = false;
    hipEvent_t ev[2][64] = {};     // start / end of the scoring kernel, ring of 64 calls
    int64_t n_calls = 0;
};

namespace {

// Flagged rows the generic path's exact re-decision takes per window (its scratch holds
// one window's per-chunk winners); the windows cover every row a call can flag.
constexpr int kFixupWindowRows = 8192;

void release(olive_score_ctx *c) {
    if (!c) return;
    for (int k = 0; k < 2; ++k)
        for (int i = 0; i < 64; ++i)
            if (c->ev[k][i]) (void)hipEventDestroy(c->ev[k][i]);
    void *ptrs[] = {c->ws_own, c->wt_own, c->rowmap, c->seqbuf, c->sched, c->part,
                    c->logp_tmp, c->lse_buf, c->flagged, c->fx_scratch, c->wn_s, c->wn_t, c->err,
                    c->tk_buf, c->fx_buf, c->bw_lse, c->bw_wt, c->bw_dzt, c->bw_hrt, c->bw_mref,
                    c->wp_s, c->wp_t, c->hp_s, c->hp_t};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
    delete c;
}

bool finite_positive(float x) { return std::isfinite(x) && x > 0.f; }

// Host checks of a descriptor (init and the no-allocation entry point).
olive_status check_desc(const olive_score_desc &d) {
    if (d.dtype != OLIVE_F32 && d.dtype != OLIVE_BF16) return OLIVE_E_DTYPE;
    if (d.w_layout != OLIVE_W_DV && d.w_layout != OLIVE_W_VD) return OLIVE_E_DTYPE;
    if (d.vocab < 1 || d.vocab >= (int64_t)1 << 31) return OLIVE_E_SHAPE;
    if (d.d_student < 1 || d.d_teacher < 0) return OLIVE_E_SHAPE;
    if (d.max_positions < 1 || d.max_positions >= ((int64_t)1 << 31) - 1) return OLIVE_E_SHAPE;
    if (d.max_seqs < 1) return OLIVE_E_SHAPE;
    if (d.d_student > 12288 || d.d_teacher > 12288) return OLIVE_E_UNSUPPORTED;
    if (!finite_positive(d.logit_scale_student)) return OLIVE_E_RANGE;
    if (d.d_teacher > 0 && !finite_positive(d.logit_scale_teacher)) return OLIVE_E_RANGE;
    if (d.flags & ~(OLIVE_FLAG_SIMPLE_KERNEL | OLIVE_FLAG_KERNEL_TIMING | OLIVE_FLAG_TOPK |
                    OLIVE_FLAG_BACKWARD | OLIVE_FLAG_NARROW_TILE))
        return OLIVE_E_RANGE;
    return OLIVE_OK;
}

// Whether the bf16 MFMA kernel applies to a context of this descriptor and weights.
bool mfma_applies(const olive_score_desc &d, const void *w_student, const void *w_teacher) {
    const bool has_t = d.d_teacher > 0;
    return d.dtype == OLIVE_BF16 && (d.d_student % 64 == 0) && (d.d_teacher % 64 == 0) &&
           d.vocab >= 256 && !(d.flags & OLIVE_FLAG_SIMPLE_KERNEL) &&
           (d.w_layout == OLIVE_W_DV ||      // borrowed weights: 16-byte rows
            (((uintptr_t)w_student & 15) == 0 && (!has_t || ((uintptr_t)w_teacher & 15) == 0)));
}

// The batch (and spans) a call was given are those of the recorded forward call: the same
// sizes, region and device pointers.
bool same_batch(const olive_score_ctx *c, const olive_batch *b, const olive_spans *sp) {
    const olive_batch &f = c->fwd_batch;
    if (f.num_seqs != b->num_seqs || f.region != b->region ||
        f.total_positions != b->total_positions || f.cu_seqlens != b->cu_seqlens ||
        f.cut != b->cut || f.valid_len != b->valid_len || f.targets != b->targets ||
        f.h_student != b->h_student || f.h_teacher != b->h_teacher)
        return false;
    if (c->fwd_spans != (sp != nullptr)) return false;
    return !sp || (c->fwd_sp.num_spans == sp->num_spans &&
                   c->fwd_sp.span_offsets == sp->span_offsets && c->fwd_sp.spans == sp->spans);
}

template <typename T>
olive_status dev_alloc(T **p, size_t bytes) {
    *p = nullptr;
    if (bytes == 0) bytes = 16;
    if (hipMalloc((void **)p, bytes) != hipSuccess) { *p = nullptr; return OLIVE_E_NOMEM; }
    return OLIVE_OK;
}

olive_status check_hip(hipError_t e) { return e == hipSuccess ? OLIVE_OK : OLIVE_E_HIP; }

constexpr int64_t kBackwardChunk = 8192;   // scored rows per logit-gradient chunk

// W_S^T in K-blocked panels [bw_vp/64][d_S][64] (zeros past V), from the [V][d_S]
// weights the kernels use; the gradient panels' columns past V are zeroed once (no
// pass writes them).
olive_status backward_init(olive_score_ctx *c, hipStream_t st) {
    const int64_t V = c->desc.vocab, ds = c->desc.d_student;
    bool ok = launch_panel_t(c->ws, V, (int)ds, c->bw_vp, c->bw_wt, st) == hipSuccess &&
              hipMemsetAsync(c->bw_dzt, 0, (size_t)c->bw_chunk * c->bw_vp * 2, st) ==
                  hipSuccess &&
              hipStreamSynchronize(st) == hipSuccess;
    return ok ? OLIVE_OK : OLIVE_E_HIP;
}

// Top-K lists need two splits at least (16 listed entries) and at most 1024
// vocabulary tiles per split (the 16-bit row ordinal of a list key).
int topk_min_splits(int n_vtiles) {
    const int s = (n_vtiles + 1023) / 1024;
    return s > 2 ? s : 2;
}

// The scoring of one batch, shared by every scoring entry point.
olive_status run(olive_score_ctx *ctx, const olive_batch *b, const olive_spans *spans,
                 float *kl, float *kl_rev, int64_t *counts, float *logp_s, float *logp_t,
                 int32_t *am_s, int32_t *am_t, float *ce, hipStream_t st,
                 bool region_only = false, TopkOut tk = TopkOut{}, float *jsd = nullptr) {
    const olive_score_desc &d = ctx->desc;
    if (!b->cu_seqlens || !b->targets || !b->h_student) return OLIVE_E_NULL;
    if (!spans && !b->cut) return OLIVE_E_NULL;
    if (b->num_seqs < 1 || b->num_seqs > d.max_seqs) return OLIVE_E_SHAPE;
    if (b->total_positions < 1 || b->total_positions > d.max_positions) return OLIVE_E_SHAPE;
    if (spans) {
        if (b->region != OLIVE_REGION_SPANS) return OLIVE_E_RANGE;
        if (spans->size != (int32_t)sizeof(olive_spans) || spans->num_spans < 0)
            return OLIVE_E_RANGE;
        if (!spans->span_offsets || (spans->num_spans > 0 && !spans->spans)) return OLIVE_E_NULL;
    } else if (b->region < OLIVE_REGION_TEACHER || b->region > OLIVE_REGION_ALL) {
        return OLIVE_E_RANGE;
    }
    const bool topk = tk.any();
    if (topk && !ctx->topk) return OLIVE_E_UNSUPPORTED;
    const bool want_t = kl || kl_rev || jsd || logp_t || am_t || topk;
    if (want_t && (!ctx->has_t || !b->h_teacher)) return OLIVE_E_UNSUPPORTED;
    const bool has_t = want_t;
    const int64_t T = b->total_positions;
    const int64_t V = d.vocab;
    const int n_vtiles = (int)((V + 255) / 256);
    // The MFMA kernel streams hidden rows with 16-byte DMAs: it needs 16-byte aligned
    // hidden-state buffers; others take the generic kernel.
    const bool mfma = ctx->mfma_ok && ((uintptr_t)b->h_student & 15) == 0 &&
                      (!has_t || ((uintptr_t)b->h_teacher & 15) == 0);
    if (topk && !mfma) return OLIVE_E_UNSUPPORTED;   // the top-K lists come from the MFMA pass
    if (jsd && !mfma) return OLIVE_E_UNSUPPORTED;    // the JSD pass is an MFMA pass
    // The 256 x 256 kernel takes student-only calls and calls with one KL direction; both
    // directions at once and the top-K lists need both models' logits side by side (the
    // 256 x 128 kernel).
    const bool wide = mfma && ctx->wide && !(kl && kl_rev) && !topk;
    const bool wide_rev = wide && kl_rev;
    float *logp_tmp = (ce && !logp_s) ? ctx->logp_tmp : nullptr;
    // normalisers kept for a backward on this batch (MFMA path, backward contexts), and
    // read by the top-K stages and the JSD pass
    float *lse_out = topk ? ctx->tkw.lse
                          : ((mfma && ctx->bw) ? ctx->bw_lse : (jsd ? ctx->lse_buf : nullptr));
    ctx->fwd_lse_ok = false;

    olive_status s;
    int grid = 0;
    int fixed_splits = 1;
    int64_t max_units = 0;
    if (mfma) {
        grid = ctx->n_cu;
    } else {
        int64_t pt = (T + SIMPLE_BT - 1) / SIMPLE_BT;
        int64_t want = (2048 + pt - 1) / pt;
        int lim = n_vtiles < MAX_SPLITS ? n_vtiles : MAX_SPLITS;
        fixed_splits = (int)(want < 1 ? 1 : (want > lim ? lim : want));
        max_units = pt * fixed_splits;
    }
    s = check_hip(launch_prep(*b, spans, region_only, V, ctx->seqbuf, ctx->sched, ctx->err, counts,
                              wide ? WIDE_BT : (mfma ? MFMA_BT : SIMPLE_BT), mfma ? 0 : 1,
                              n_vtiles, grid,
                              fixed_splits, topk ? topk_min_splits(n_vtiles) : 1, st));
    if (s) return s;
    s = check_hip(launch_rowmap(*b, spans, region_only, V, ctx->seqbuf, ctx->sched, ctx->rowmap,
                                ctx->err,
                                logp_s,
                                has_t ? logp_t : nullptr, am_s, has_t ? am_t : nullptr,
                                has_t ? kl : nullptr, has_t ? kl_rev : nullptr,
                                has_t ? jsd : nullptr, logp_tmp, tk, st));
    if (s) return s;

    ScoreArgs a;
    a.hs = b->h_student;
    a.ht = has_t ? b->h_teacher : nullptr;
    a.ws = ctx->ws;
    a.wt = has_t ? ctx->wt : nullptr;
    a.rowmap = ctx->rowmap;
    a.sched = ctx->sched;
    a.part = ctx->part;
    a.pstride = ctx->pstride;
    a.V = (int32_t)V;
    a.ds = d.d_student;
    a.dt = has_t ? d.d_teacher : 0;
    a.n_vtiles = n_vtiles;
    a.sS = d.logit_scale_student;
    a.sT = has_t ? d.logit_scale_teacher : 1.f;
    a.cS = a.sS * 1.4426950408889634f;
    a.cT = a.sT * 1.4426950408889634f;
    a.wmax_s = ctx->wmax_s;
    a.wmax_t = ctx->wmax_t;
    a.wmax_dev = ctx->wmax_dev;
    a.wps = ctx->wp_s;
    a.wpt = has_t ? ctx->wp_t : nullptr;
    a.hps = ctx->hp_s;
    a.hpt = has_t ? ctx->hp_t : nullptr;
    a.vpad = ctx->wp_rows;
    a.prow = ctx->hp_rows;
    a.wide = wide ? (wide_rev ? 2 : 1) : 0;
    const bool same_scale = has_t && (a.sS == a.sT);

    if (wide) {
        // the call's compacted hidden rows into panels (zero past them, to the tile end)
        s = check_hip(launch_panel_h(b->h_student, d.d_student, ctx->rowmap, ctx->sched,
                                     ctx->hp_rows, ctx->hp_s, st));
        if (!s && has_t)
            s = check_hip(launch_panel_h(b->h_teacher, d.d_teacher, ctx->rowmap, ctx->sched,
                                         ctx->hp_rows, ctx->hp_t, st));
        if (s) return s;
    }
    const int slot = (int)(ctx->n_calls % 64);
    if (ctx->timing && hipEventRecord(ctx->ev[0][slot], st) != hipSuccess) return OLIVE_E_HIP;
    if (wide)
        s = check_hip(launch_score_wide(a, same_scale, has_t, wide_rev, grid, st));
    else if (mfma)
        s = check_hip(launch_score_mfma(a, has_t, same_scale, has_t && kl_rev, topk, grid, st));
    else
        s = check_hip(launch_score_simple(a, ctx->bf16, has_t, max_units, st));
    if (s) return s;
    if (ctx->timing && hipEventRecord(ctx->ev[1][slot], st) != hipSuccess) return OLIVE_E_HIP;
    ctx->n_calls++;
    ctx->last_kernel = wide ? 2 : (mfma ? 0 : 1);
    ctx->last_grid = mfma ? grid : (int)max_units;

    int32_t *flagged = (am_s || (has_t && am_t)) ? ctx->flagged : nullptr;
    s = check_hip(launch_combine(a, ctx->bf16, has_t, same_scale, b->targets, ctx->err, logp_s,
                                 has_t ? logp_t : nullptr, am_s, has_t ? am_t : nullptr,
                                 has_t ? kl : nullptr, has_t ? kl_rev : nullptr, logp_tmp,
                                 lse_out, flagged, ctx->flag_cap, T, st));
    if (s) return s;
    if (mfma && ctx->bw && lse_out) {
        ctx->fwd_lse = lse_out;
        ctx->fwd_lse_ok = true;
        ctx->fwd_lse_t = has_t;
        ctx->fwd_batch = *b;
        ctx->fwd_spans = spans != nullptr;
        if (spans) ctx->fwd_sp = *spans;
    }
    if (flagged) {
        if (mfma)
            s = check_hip(launch_argmax_fix(a, flagged, ctx->flag_cap, ctx->fxq, am_s,
                                            has_t ? am_t : nullptr, st));
        else
            // windows over the flagged list: at most one entry per compacted row
            for (int64_t f0 = 0; f0 < T && !s; f0 += ctx->fx_window)
                s = check_hip(launch_fixup_impl(a, ctx->bf16, flagged, (int)f0, ctx->fx_window,
                                                ctx->fx_scratch, ctx->wn_s, ctx->wn_t, am_s,
                                                has_t ? am_t : nullptr, st));
        if (s) return s;
    }
    if (topk) {
        s = check_hip(launch_topk(a, ctx->tkw, tk, T, st));
        if (s) return s;
    }
    if (jsd) {
        // second pass over the scored rows (compacted first), from the normalisers
        JsdArgs z;
        z.lse = lse_out;
        s = check_hip(launch_score_jsd(a, z, grid, st));
        if (s) return s;
        s = check_hip(launch_jsd_combine(a, jsd, grid, T, st));
        if (s) return s;
    }
    if (ce) {
        s = check_hip(launch_ce(*b, spans, ctx->seqbuf, ctx->sched,
                                logp_s ? logp_s : ctx->logp_tmp, ce, st));
        if (s) return s;
    }
    return OLIVE_OK;
}

// The backward pass: forward normalisers of the scored rows (region-only forward),
// then per chunk of scored rows the logit gradient and the two products.
olive_status run_backward(olive_score_ctx *ctx, const olive_batch *b, const olive_spans *spans,
                          const olive_grad_outputs *go, hipStream_t st) {
    const olive_score_desc &d = ctx->desc;
    if (!b->cu_seqlens || !b->targets || !b->h_student) return OLIVE_E_NULL;
    if (!spans && !b->cut) return OLIVE_E_NULL;
    if (b->num_seqs < 1 || b->num_seqs > d.max_seqs) return OLIVE_E_SHAPE;
    if (b->total_positions < 1 || b->total_positions > d.max_positions) return OLIVE_E_SHAPE;
    if (spans) {
        if (b->region != OLIVE_REGION_SPANS) return OLIVE_E_RANGE;
        if (spans->size != (int32_t)sizeof(olive_spans) || spans->num_spans < 0)
            return OLIVE_E_RANGE;
        if (!spans->span_offsets || (spans->num_spans > 0 && !spans->spans)) return OLIVE_E_NULL;
    } else if (b->region < OLIVE_REGION_TEACHER || b->region > OLIVE_REGION_ALL) {
        return OLIVE_E_RANGE;
    }
    const bool has_t = go->w_kl != 0.f;
    if (has_t && (!ctx->has_t || !b->h_teacher)) return OLIVE_E_UNSUPPORTED;
    if (((uintptr_t)b->h_student & 15) != 0 || (has_t && ((uintptr_t)b->h_teacher & 15) != 0))
        return OLIVE_E_UNSUPPORTED;
    const bool reuse = (go->flags & OLIVE_GRAD_REUSE_FORWARD) != 0;
    if (reuse && !(ctx->fwd_lse_ok && (!has_t || ctx->fwd_lse_t) && same_batch(ctx, b, spans)))
        return OLIVE_E_RANGE;
    const int64_t T = b->total_positions;
    const int64_t V = d.vocab;
    const int n_vtiles = (int)((V + 255) / 256);
    const int grid = ctx->n_cu;
    // The row compaction and schedule, for position tiles of tile_rows: the normaliser
    // pass runs the 256 x 256 kernel where the context keeps its panels, the gradient
    // passes take 128-row tiles.
    auto schedule = [&](int tile_rows) {
        olive_status e = check_hip(launch_prep(*b, spans, true, V, ctx->seqbuf, ctx->sched,
                                               ctx->err, go->counts, tile_rows, 0, n_vtiles,
                                               grid, 1, 1, st));
        if (!e)
            e = check_hip(launch_rowmap(*b, spans, true, V, ctx->seqbuf, ctx->sched, ctx->rowmap,
                                        ctx->err, nullptr, nullptr, nullptr, nullptr, nullptr,
                                        nullptr, nullptr, nullptr, TopkOut{}, st));
        return e;
    };
    const bool wide = !reuse && ctx->wide;
    const int ch = ctx->bw_chunk;
    // The cross-entropy's logit gradient runs on the 256 x 256 kernel where the context
    // keeps its panels. Chunks start at multiples of 8192 rows (or at 0), so at tile
    // boundaries of the panels. Without a forward call's normalisers that pass forms
    // them itself (one sweep of the student instead of two): it stores each tile's
    // weights relative to the running max, and a rescale follows once the chunk's
    // normalisers are known.
    const bool wide_dz = ctx->wide && !has_t && (ch % WIDE_BT == 0 || T <= ch);
    const bool online = wide && wide_dz;
    olive_status s = schedule(wide && !online ? WIDE_BT : MFMA_BT);
    if (s) return s;
    ScoreArgs a;
    a.hs = b->h_student;
    a.ht = has_t ? b->h_teacher : nullptr;
    a.ws = ctx->ws;
    a.wt = has_t ? ctx->wt : nullptr;
    a.rowmap = ctx->rowmap;
    a.sched = ctx->sched;
    a.part = ctx->part;
    a.pstride = ctx->pstride;
    a.V = (int32_t)V;
    a.ds = d.d_student;
    a.dt = has_t ? d.d_teacher : 0;
    a.n_vtiles = n_vtiles;
    a.sS = d.logit_scale_student;
    a.sT = has_t ? d.logit_scale_teacher : 1.f;
    a.cS = a.sS * 1.4426950408889634f;
    a.cT = a.sT * 1.4426950408889634f;
    a.wmax_s = ctx->wmax_s;
    a.wmax_t = ctx->wmax_t;
    a.wmax_dev = ctx->wmax_dev;
    const bool same_scale = has_t && (a.sS == a.sT);
    a.wps = ctx->wp_s;
    a.wpt = has_t ? ctx->wp_t : nullptr;
    a.hps = ctx->hp_s;
    a.hpt = has_t ? ctx->hp_t : nullptr;
    a.vpad = ctx->wp_rows;
    a.prow = ctx->hp_rows;
    a.wide = wide ? 1 : 0;
    const float *lse = ctx->fwd_lse;
    if (online) {
        // the chunk passes write the normalisers; they replace a forward call's for reuse
        ctx->fwd_lse_ok = false;
        lse = ctx->bw_lse;
    } else if (!reuse) {
        // the forward normalisers of the scored rows; they replace a forward call's for
        // reuse (always, wherever that call's are kept: one rule for every output set)
        ctx->fwd_lse_ok = false;
        if (wide) {
            s = check_hip(launch_panel_h(b->h_student, d.d_student, ctx->rowmap, ctx->sched,
                                         ctx->hp_rows, ctx->hp_s, st));
            if (!s && has_t)
                s = check_hip(launch_panel_h(b->h_teacher, d.d_teacher, ctx->rowmap,
                                             ctx->sched, ctx->hp_rows, ctx->hp_t, st));
            if (!s) s = check_hip(launch_score_wide(a, same_scale, has_t, false, grid, st));
        } else {
            s = check_hip(launch_score_mfma(a, has_t, same_scale, false, false, grid, st));
        }
        if (s) return s;
        s = check_hip(launch_combine(a, true, has_t, same_scale, b->targets, ctx->err, nullptr,
                                     nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                     ctx->bw_lse, nullptr, 0, T, st));
        if (s) return s;
        lse = ctx->bw_lse;
        if (wide) {
            // the gradient passes' 128-row position tiles
            s = schedule(MFMA_BT);
            if (s) return s;
            a.wide = 0;
        }
    }
    const int ds = d.d_student;
    if (go->grad_h_student) {
        s = check_hip(launch_fill(go->grad_h_student, T * ds, st));
        if (s) return s;
    }
    // the hidden-row panels of every scored row (built by the normaliser pass, or here
    // when there was none)
    if (wide_dz && (!wide || online)) {
        s = check_hip(launch_panel_h(b->h_student, d.d_student, ctx->rowmap, ctx->sched,
                                     ctx->hp_rows, ctx->hp_s, st));
        if (s) return s;
    }
    // scored rows <= T: chunks past the call's positions are never launched (those past
    // the scored count, known only on the device, exit at once)
    for (int64_t c0 = 0; c0 < T; c0 += ch) {
        DzArgs z;
        z.c0 = (int)c0;
        z.chunk = ch;
        z.vp = ctx->bw_vp;
        z.lse = lse;
        z.targets = b->targets;
        z.w_ce = go->w_ce;
        z.w_kl = go->w_kl;
        z.dz_t = ctx->bw_dzt;
        z.mref = ctx->bw_mref;
        z.gy = ctx->bw_mref + (int64_t)((V + 255) / 256) * ch;
        z.yrow = (int32_t *)(z.gy + ch);
        if (wide_dz) {
            ScoreArgs aw = a;
            aw.wps = ctx->wp_s;
            aw.hps = (const char *)ctx->hp_s + c0 * 64;   // panel row c0 (32 bf16 per row)
            aw.vpad = ctx->wp_rows;
            aw.prow = ctx->hp_rows;
            if (online) {
                s = check_hip(launch_score_wide_dz_online(aw, z, grid, st));
                if (!s) s = check_hip(launch_dz_lse(a, z, grid, ctx->bw_lse, ctx->err, st));
                if (!s) s = check_hip(launch_dz_rescale(a, z, ctx->bw_lse, st));
            } else {
                s = check_hip(launch_score_wide_dz(aw, z, grid, st));
            }
        } else {
            s = check_hip(launch_score_dz(a, z, has_t, grid, st));
        }
        if (s) return s;
        if (go->grad_w_student) {
            s = check_hip(launch_zero_tail(ctx->bw_dzt, ctx->bw_vp, ch, ctx->sched, (int)c0, st));
            if (s) return s;
            s = check_hip(launch_gather_t(b->h_student, ds, ctx->rowmap, ctx->sched, (int)c0, ch,
                                          ch, ctx->bw_hrt, st));
            if (s) return s;
            GemmArgs g = {};
            // dz_t panels [vp/64][chunk][64]: rows v, K = scored rows, read transposed
            g.A = (const char *)ctx->bw_dzt;
            g.a_panels = (int)(ctx->bw_vp / 64);
            g.a_prows = ch;
            g.B = (const char *)ctx->bw_hrt;        // [d_S][chunk]
            g.ldb = (int64_t)ch * 2;
            g.bkstep = 128;
            g.M = (int)V;
            g.N = ds;
            g.k_dev = &ctx->sched->t_valid;
            g.k_off = (int)c0;
            g.k_cap = ch;
            g.C = go->grad_w_student;
            const bool dv = d.w_layout == OLIVE_W_DV;
            g.trans_out = dv;                       // [d_S][V]: C[k][v]
            g.ldc = dv ? V : ds;
            g.alpha = a.sS;
            g.accumulate = c0 > 0;
            s = check_hip(launch_gemm(g, grid, st));
            if (s) return s;
        }
        if (go->grad_h_student) {
            GemmArgs g = {};
            // K-blocked panels: one K step of either operand is a contiguous block
            g.A = (const char *)ctx->bw_wt;         // W_S^T [vp/64][d_S][64]: rows k, K = v
            g.lda = 128;
            g.akstep = (int64_t)ds * 128;
            g.B = (const char *)ctx->bw_dzt;        // [vp/64][chunk][64]
            g.ldb = 128;
            g.bkstep = (int64_t)ch * 128;
            g.M = ds;
            g.K = (int)ctx->bw_vp;
            g.n_dev = &ctx->sched->t_valid;
            g.n_off = (int)c0;
            g.n_cap = ch;
            g.C = go->grad_h_student;               // row of scored row n: rowmap[c0 + n]
            g.ldc = ds;
            g.rowmap = ctx->rowmap;
            g.rowmap_off = (int)c0;
            g.trans_out = true;
            g.alpha = a.sS;
            g.accumulate = false;
            // d_S / 256 x rows / 128 tiles rarely fill the grid: halve K over two units
            // (the rows of dL/dh were zero-filled above)
            g.ksplit = 2;
            s = check_hip(launch_gemm(g, grid, st));
            if (s) return s;
        }
    }
    return OLIVE_OK;
}

// ---------------------------------------------------------------------------------
// Scratch of olive_kl_masked_static: one fixed device array per GPU, so that the call
// allocates nothing. Limits: positions, sequences and vocabulary of a call.
constexpr int64_t kStaticMaxPositions = 8192;
constexpr int32_t kStaticMaxSeqs = 256;
constexpr int64_t kStaticMaxVocab = 262144;
constexpr int kStaticFxWindow = 512;              // generic path: flagged rows per window

struct StaticDevice {
    bool ready = false;
    char *base = nullptr;      // this device's copy of `scratch`
    int n_cu = 0;
};
constexpr int kStaticDevices = 64;
StaticDevice g_static[kStaticDevices];
std::mutex g_static_mu;

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Once per device, with that device current: the address of its copy of the scratch
// array and its compute-unit count.
olive_status static_setup(int dev, StaticDevice **out) {
    if (dev < 0 || dev >= kStaticDevices) return OLIVE_E_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_static_mu);
    StaticDevice &s = g_static[dev];
    if (!s.ready) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return OLIVE_E_HIP;
        int n_cu = 0;
        if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) !=
                hipSuccess || n_cu < 1)
            return OLIVE_E_HIP;
        s.base = (char *)p;
        s.n_cu = n_cu;
        s.ready = true;
    }
    *out = &s;
    return OLIVE_OK;
}

// Lays the per-call workspace of a context out in a device's scratch array (the limits'
// sizes); false when it would not fit.
bool static_carve(olive_score_ctx *c, char *base) {
    const int64_t P = kStaticMaxPositions;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *p = base + off;
        off += align256(bytes);
        return p;
    };
    c->sched = (Sched *)take(sizeof(Sched));
    c->err = (int32_t *)take(sizeof(int32_t));
    c->wmax_dev = (const float *)take(2 * sizeof(float));
    c->seqbuf = (int32_t *)take((size_t)seqbuf_entries(kStaticMaxSeqs) * sizeof(int32_t));
    c->rowmap = (uint32_t *)take((size_t)P * sizeof(uint32_t));
    c->pstride = (P + 255) / 256 * 256;
    c->part = (float *)take((size_t)NFIELDS * MAX_SPLITS * c->pstride * sizeof(float));
    c->logp_tmp = (float *)take((size_t)P * sizeof(float));
    c->flag_cap = (int)P;
    c->flagged = (int32_t *)take((size_t)4 * P * sizeof(int32_t));
    c->fx_buf = take(filter_queue_bytes(P, FX_CCAP));
    c->fx_window = kStaticFxWindow;
    c->fx_scratch = take((size_t)kStaticFxWindow * fixup_chunks(kStaticMaxVocab) * 2 *
                         fixup_result_bytes());
    c->wn_s = (float *)take((size_t)kStaticMaxVocab * sizeof(float));
    c->wn_t = (float *)take((size_t)kStaticMaxVocab * sizeof(float));
    if (off > kStaticScratchBytes) return false;
    c->fxq = filter_queue_carve(c->fx_buf, c->flag_cap, FX_CCAP, &c->sched->n_fxq[0],
                                &c->sched->n_fx_fb);
    c->fxq.smask = &c->sched->fx_smask[0];
    return true;
}

}  // namespace

extern "C" {

olive_status olive_kl_masked_static(const olive_score_desc *desc, const void *w_student,
                                    const void *w_teacher, const olive_batch *b, float *kl,
                                    int64_t *counts, float *logp_student, float *logp_teacher,
                                    int32_t *argmax_student, int32_t *argmax_teacher,
                                    float *ce_per_seq, void *hip_stream) {
    if (!desc || !b || !kl) return OLIVE_E_NULL;
    const olive_score_desc &d = *desc;
    if (olive_status e = check_desc(d)) return e;
    // borrowed [V][d] weights only (a repacked copy would need memory); no per-context
    // options (timing, top-K, backward workspaces)
    if (d.w_layout != OLIVE_W_VD || (d.flags & ~OLIVE_FLAG_SIMPLE_KERNEL) || d.d_teacher == 0)
        return OLIVE_E_UNSUPPORTED;
    if (!w_student || !w_teacher) return OLIVE_E_NULL;
    if (d.max_positions > kStaticMaxPositions || d.max_seqs > kStaticMaxSeqs ||
        d.vocab > kStaticMaxVocab)
        return OLIVE_E_LIMIT;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return OLIVE_E_HIP;
    StaticDevice *sd = nullptr;
    if (olive_status e = static_setup(dev, &sd)) return e;
    olive_score_ctx c;   // host-side description of this call only (nothing is allocated)
    c.desc = d;
    c.device = dev;
    c.n_cu = sd->n_cu;
    c.ws = w_student;
    c.wt = w_teacher;
    c.bf16 = d.dtype == OLIVE_BF16;
    c.has_t = true;
    c.mfma_ok = mfma_applies(d, w_student, w_teacher);
    if (!static_carve(&c, sd->base)) return OLIVE_E_LIMIT;
    hipStream_t st = (hipStream_t)hip_stream;
    // the weight-row norms and their maxima bound the rounding of the near-tie decisions
    float *wmax = const_cast<float *>(c.wmax_dev);
    if (launch_row_norms(c.ws, d.vocab, d.d_student, c.bf16, c.wn_s, st) != hipSuccess ||
        launch_row_norms(c.wt, d.vocab, d.d_teacher, c.bf16, c.wn_t, st) != hipSuccess ||
        launch_max_norm(c.wn_s, d.vocab, wmax, st) != hipSuccess ||
        launch_max_norm(c.wn_t, d.vocab, wmax + 1, st) != hipSuccess)
        return OLIVE_E_HIP;
    return run(&c, b, nullptr, kl, nullptr, counts, logp_student, logp_teacher, argmax_student,
               argmax_teacher, ce_per_seq, st);
}

const char *olive_status_string(olive_status s) {
    // A C caller may pass any int: read the argument's bytes rather than the enum value
    // (a value outside the enumerators is undefined as a C++ enum).
    int32_t code;
    static_assert(sizeof(code) == sizeof(s), "olive_status is passed as a 32-bit int");
    std::memcpy(&code, &s, sizeof(code));
    switch (code) {
        case OLIVE_OK: return "OLIVE_OK: success";
        case OLIVE_E_NULL: return "OLIVE_E_NULL: a required pointer is NULL";
        case OLIVE_E_SHAPE: return "OLIVE_E_SHAPE: a size is out of range for this context";
        case OLIVE_E_DTYPE: return "OLIVE_E_DTYPE: unknown dtype or weight layout";
        case OLIVE_E_RANGE: return "OLIVE_E_RANGE: a value is out of range";
        case OLIVE_E_HIP: return "OLIVE_E_HIP: a HIP runtime call failed";
        case OLIVE_E_NOMEM: return "OLIVE_E_NOMEM: device allocation failed";
        case OLIVE_E_UNSUPPORTED: return "OLIVE_E_UNSUPPORTED: not supported by this context";
        case OLIVE_E_LIMIT:
            return "OLIVE_E_LIMIT: beyond the fixed limits of olive_kl_masked_static "
                   "(positions, sequences or vocabulary)";
    }
    return "OLIVE: unknown status";
}

olive_status olive_score_init(olive_score_ctx **out, const olive_score_desc *desc,
                              const void *w_student, const void *w_teacher, void *hip_stream) {
    if (!out || !desc) return OLIVE_E_NULL;
    *out = nullptr;
    const olive_score_desc &d = *desc;
    if (olive_status e = check_desc(d)) return e;
    if (!w_student) return OLIVE_E_NULL;
    if (d.d_teacher > 0 && !w_teacher) return OLIVE_E_NULL;

    olive_score_ctx *c = new (std::nothrow) olive_score_ctx();
    if (!c) return OLIVE_E_NOMEM;
    c->desc = d;
    c->bf16 = d.dtype == OLIVE_BF16;
    c->has_t = d.d_teacher > 0;
    hipStream_t st = (hipStream_t)hip_stream;
    if (hipGetDevice(&c->device) != hipSuccess ||
        hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device) !=
            hipSuccess) {
        release(c);
        return OLIVE_E_HIP;
    }
    c->mfma_ok = mfma_applies(d, w_student, w_teacher);
    c->topk = (d.flags & OLIVE_FLAG_TOPK) != 0;
    if (c->topk && (!c->mfma_ok || !c->has_t || d.vocab < 512 ||
                    d.vocab > (int64_t)MAX_SPLITS * 1024 * MFMA_BV)) {
        release(c);
        return OLIVE_E_UNSUPPORTED;
    }
    c->bw = (d.flags & OLIVE_FLAG_BACKWARD) != 0;
    if (c->bw && !c->mfma_ok) {
        release(c);
        return OLIVE_E_UNSUPPORTED;
    }
    const int esz = c->bf16 ? 2 : 4;
    const int64_t V = d.vocab;
    olive_status s = OLIVE_OK;
    if (d.w_layout == OLIVE_W_DV) {
        s = dev_alloc(&c->ws_own, (size_t)V * d.d_student * esz);
        if (!s && c->has_t) s = dev_alloc(&c->wt_own, (size_t)V * d.d_teacher * esz);
        if (s) { release(c); return s; }
        if (launch_repack(w_student, c->ws_own, d.d_student, V, esz, st) != hipSuccess ||
            (c->has_t && launch_repack(w_teacher, c->wt_own, d.d_teacher, V, esz, st) != hipSuccess)) {
            release(c);
            return OLIVE_E_HIP;
        }
        c->ws = c->ws_own;
        c->wt = c->wt_own;
    } else {
        c->ws = w_student;
        c->wt = c->has_t ? w_teacher : nullptr;
    }
    const int64_t P = d.max_positions;
    c->pstride = (P + 255) / 256 * 256;
    // One near-tie entry per compacted row at most: the list never drops a flagged row.
    c->flag_cap = (int)P;
    c->fx_window = (int)(P < kFixupWindowRows ? P : kFixupWindowRows);
    if (!s) s = dev_alloc(&c->rowmap, (size_t)P * sizeof(uint32_t));
    if (!s) s = dev_alloc(&c->seqbuf, (size_t)seqbuf_entries(d.max_seqs) * sizeof(int32_t));
    if (!s) s = dev_alloc(&c->sched, sizeof(Sched));
    if (!s)
        s = dev_alloc(&c->part, (size_t)(c->topk ? NFIELDS_TOPK : NFIELDS) * MAX_SPLITS *
                                    c->pstride * sizeof(float));
    if (!s && c->topk) {
        s = dev_alloc(&c->tk_buf, topk_work_bytes(P));
        if (!s) c->tkw = topk_carve(c->tk_buf, P, &c->sched->n_tkq[0], &c->sched->n_tk_fb);
    }
    if (!s && c->mfma_ok) {
        s = dev_alloc(&c->fx_buf, filter_queue_bytes(c->flag_cap, FX_CCAP));
        if (!s) {
            c->fxq = filter_queue_carve(c->fx_buf, c->flag_cap, FX_CCAP, &c->sched->n_fxq[0],
                                        &c->sched->n_fx_fb);
            c->fxq.smask = &c->sched->fx_smask[0];   // the greedy filter reads marked splits
        }
    }
    if (!s && c->bw) {
        const int64_t ch = (P + 127) / 128 * 128;
        c->bw_chunk = (int)(ch < kBackwardChunk ? ch : kBackwardChunk);
        c->bw_vp = (V + 63) / 64 * 64;
        const int64_t ds = d.d_student;
        s = dev_alloc(&c->bw_lse, (size_t)P * 2 * sizeof(float));
        if (!s) s = dev_alloc(&c->bw_wt, (size_t)ds * c->bw_vp * 2);
        if (!s) s = dev_alloc(&c->bw_dzt, (size_t)c->bw_chunk * c->bw_vp * 2);
        if (!s) s = dev_alloc(&c->bw_hrt, (size_t)ds * c->bw_chunk * 2);
        if (!s)
            s = dev_alloc(&c->bw_mref,
                          ((size_t)(V + 255) / 256 + 2) * c->bw_chunk * sizeof(float));
        if (!s) s = backward_init(c, st);
    }
    c->wide = c->mfma_ok && !(d.flags & OLIVE_FLAG_NARROW_TILE);
    if (!s && c->wide) {
        c->wp_rows = (V + MFMA_BV - 1) / MFMA_BV * MFMA_BV;
        c->hp_rows = (P + WIDE_BT - 1) / WIDE_BT * WIDE_BT;
        s = dev_alloc(&c->wp_s, (size_t)c->wp_rows * d.d_student * 2);
        if (!s) s = dev_alloc(&c->hp_s, (size_t)c->hp_rows * d.d_student * 2);
        if (!s && c->has_t) s = dev_alloc(&c->wp_t, (size_t)c->wp_rows * d.d_teacher * 2);
        if (!s && c->has_t) s = dev_alloc(&c->hp_t, (size_t)c->hp_rows * d.d_teacher * 2);
        if (!s && (launch_panel_w(c->ws, V, d.d_student, c->wp_rows, c->wp_s, st) != hipSuccess ||
                   (c->has_t &&
                    launch_panel_w(c->wt, V, d.d_teacher, c->wp_rows, c->wp_t, st) != hipSuccess)))
            s = OLIVE_E_HIP;
    }
    if (!s) s = dev_alloc(&c->logp_tmp, (size_t)P * sizeof(float));
    if (!s && c->mfma_ok && c->has_t) s = dev_alloc(&c->lse_buf, (size_t)P * 2 * sizeof(float));
    if (!s) s = dev_alloc(&c->flagged, (size_t)4 * c->flag_cap * sizeof(int32_t));
    if (!s)
        s = dev_alloc(&c->fx_scratch,
                      (size_t)c->fx_window * fixup_chunks(V) * 2 * fixup_result_bytes());
    if (!s) s = dev_alloc(&c->err, sizeof(int32_t));
    if (!s) s = dev_alloc(&c->wn_s, (size_t)V * sizeof(float));
    if (!s && c->has_t) s = dev_alloc(&c->wn_t, (size_t)V * sizeof(float));
    if (s) { release(c); return s; }
    if (launch_row_norms(c->ws, V, d.d_student, c->bf16, c->wn_s, st) != hipSuccess ||
        (c->has_t && launch_row_norms(c->wt, V, d.d_teacher, c->bf16, c->wn_t, st) != hipSuccess)) {
        release(c);
        return OLIVE_E_HIP;
    }
    if (c->mfma_ok) {   // the largest row norms bound the rounding of any logit
        if (hipStreamSynchronize(st) != hipSuccess) {
            release(c);
            return OLIVE_E_HIP;
        }
        std::vector<float> wn((size_t)V);
        for (int m = 0; m < (c->has_t ? 2 : 1); ++m) {
            if (hipMemcpy(wn.data(), m ? c->wn_t : c->wn_s, (size_t)V * sizeof(float),
                          hipMemcpyDeviceToHost) != hipSuccess) {
                release(c);
                return OLIVE_E_HIP;
            }
            float mx = 0.f;
            for (float x : wn) mx = x > mx ? x : mx;
            (m ? c->wmax_t : c->wmax_s) = mx * (1.0f + 0x1p-10f);
        }
    }
    c->timing = (d.flags & OLIVE_FLAG_KERNEL_TIMING) != 0;
    if (c->timing) {
        for (int k = 0; k < 2; ++k)
            for (int i = 0; i < 64; ++i)
                if (hipEventCreate(&c->ev[k][i]) != hipSuccess) { release(c); return OLIVE_E_HIP; }
    }
    if (hipMemsetAsync(c->err, 0, sizeof(int32_t), st) != hipSuccess ||
        hipMemsetAsync(c->sched, 0, sizeof(Sched), st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess) {
        release(c);
        return OLIVE_E_HIP;
    }
    *out = c;
    return OLIVE_OK;
}

olive_status olive_token_logprobs(olive_score_ctx *ctx, const olive_batch *b, float *logp_student,
                                  float *logp_teacher, int32_t *argmax_student,
                                  int32_t *argmax_teacher, void *hip_stream) {
    if (!ctx || !b || !logp_student) return OLIVE_E_NULL;
    return run(ctx, b, nullptr, nullptr, nullptr, nullptr, logp_student, logp_teacher,
               argmax_student, argmax_teacher, nullptr, (hipStream_t)hip_stream);
}

olive_status olive_kl_masked(olive_score_ctx *ctx, const olive_batch *b, float *kl,
                             int64_t *counts, float *logp_student, float *logp_teacher,
                             int32_t *argmax_student, int32_t *argmax_teacher, float *ce_per_seq,
                             void *hip_stream) {
    if (!ctx || !b || !kl) return OLIVE_E_NULL;
    if (!ctx->has_t) return OLIVE_E_UNSUPPORTED;
    return run(ctx, b, nullptr, kl, nullptr, counts, logp_student, logp_teacher, argmax_student,
               argmax_teacher, ce_per_seq, (hipStream_t)hip_stream);
}

static TopkOut topk_of(const olive_score_outputs *out) {
    return TopkOut{out->topk_overlap, out->kl_topk, out->topk_student, out->topk_teacher};
}

// The JSD output of an output set, or NULL when the caller's struct predates the field
// (it then passes the smaller size).
static float *jsd_of(const olive_score_outputs *out) {
    return out->size == (int32_t)sizeof(olive_score_outputs) ? out->jsd : nullptr;
}

static olive_status check_outputs(const olive_score_outputs *out) {
    if (!out) return OLIVE_E_NULL;
    if (out->size != (int32_t)sizeof(olive_score_outputs) &&
        out->size != (int32_t)offsetof(olive_score_outputs, jsd))
        return OLIVE_E_RANGE;
    if (out->flags & ~OLIVE_OUT_REGION_ONLY) return OLIVE_E_RANGE;
    if (!out->kl && !out->kl_reverse && !out->counts && !out->logp_student &&
        !out->logp_teacher && !out->argmax_student && !out->argmax_teacher && !out->ce_per_seq &&
        !out->topk_overlap && !out->kl_topk && !out->topk_student && !out->topk_teacher &&
        !jsd_of(out))
        return OLIVE_E_NULL;
    return OLIVE_OK;
}

olive_status olive_score_batch(olive_score_ctx *ctx, const olive_batch *b,
                               const olive_score_outputs *out, void *hip_stream) {
    if (!ctx || !b) return OLIVE_E_NULL;
    if (olive_status e = check_outputs(out)) return e;
    return run(ctx, b, nullptr, out->kl, out->kl_reverse, out->counts, out->logp_student,
               out->logp_teacher, out->argmax_student, out->argmax_teacher, out->ce_per_seq,
               (hipStream_t)hip_stream, (out->flags & OLIVE_OUT_REGION_ONLY) != 0,
               topk_of(out), jsd_of(out));
}

olive_status olive_score_batch_spans(olive_score_ctx *ctx, const olive_batch *b,
                                     const olive_spans *spans, const olive_score_outputs *out,
                                     void *hip_stream) {
    if (!ctx || !b || !spans) return OLIVE_E_NULL;
    if (olive_status e = check_outputs(out)) return e;
    return run(ctx, b, spans, out->kl, out->kl_reverse, out->counts, out->logp_student,
               out->logp_teacher, out->argmax_student, out->argmax_teacher, out->ce_per_seq,
               (hipStream_t)hip_stream, (out->flags & OLIVE_OUT_REGION_ONLY) != 0,
               topk_of(out), jsd_of(out));
}

olive_status olive_score_backward(olive_score_ctx *ctx, const olive_batch *b,
                                  const olive_spans *spans, const olive_grad_outputs *g,
                                  void *hip_stream) {
    if (!ctx || !b || !g) return OLIVE_E_NULL;
    if (g->size != (int32_t)sizeof(olive_grad_outputs) || (g->flags & ~OLIVE_GRAD_REUSE_FORWARD))
        return OLIVE_E_RANGE;
    if (!std::isfinite(g->w_ce) || !std::isfinite(g->w_kl)) return OLIVE_E_RANGE;
    if (!g->grad_h_student && !g->grad_w_student) return OLIVE_E_NULL;
    if (!ctx->bw) return OLIVE_E_UNSUPPORTED;
    return run_backward(ctx, b, spans, g, (hipStream_t)hip_stream);
}

olive_status olive_score_free(olive_score_ctx *ctx) {
    if (!ctx) return OLIVE_OK;
    hipError_t e = hipDeviceSynchronize();
    release(ctx);
    return e == hipSuccess ? OLIVE_OK : OLIVE_E_HIP;
}

olive_status olive_score_last_error(olive_score_ctx *ctx, int32_t *device_code) {
    if (!ctx || !device_code) return OLIVE_E_NULL;
    if (hipDeviceSynchronize() != hipSuccess) return OLIVE_E_HIP;
    int32_t v = 0;
    if (hipMemcpy(&v, ctx->err, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return OLIVE_E_HIP;
    if (hipMemset(ctx->err, 0, sizeof(int32_t)) != hipSuccess) return OLIVE_E_HIP;
    *device_code = v;
    return OLIVE_OK;
}

olive_status olive_score_last_stats(olive_score_ctx *ctx, int64_t *out) {
    if (!ctx || !out) return OLIVE_E_NULL;
    if (hipDeviceSynchronize() != hipSuccess) return OLIVE_E_HIP;
    Sched s;
    if (hipMemcpy(&s, ctx->sched, sizeof(s), hipMemcpyDeviceToHost) != hipSuccess) return OLIVE_E_HIP;
    out[0] = s.n_splits;
    out[1] = s.n_flagged;
    out[2] = ctx->last_kernel;
    out[3] = ctx->last_grid;
    out[4] = s.n_tkq[0] + s.n_tkq[1];
    out[5] = s.n_tk_fb;
    return OLIVE_OK;
}

olive_status olive_score_kernel_times(olive_score_ctx *ctx, float *out, int32_t n) {
    if (!ctx || !out) return OLIVE_E_NULL;
    if (!ctx->timing) return OLIVE_E_UNSUPPORTED;
    if (n < 1 || n > 64 || n > ctx->n_calls) return OLIVE_E_RANGE;
    if (hipDeviceSynchronize() != hipSuccess) return OLIVE_E_HIP;
    for (int i = 0; i < n; ++i) {
        const int slot = (int)((ctx->n_calls - n + i) % 64);
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, ctx->ev[0][slot], ctx->ev[1][slot]) != hipSuccess)
            return OLIVE_E_HIP;
        out[i] = ms;
    }
    return OLIVE_OK;
}

}  // extern "C"
