// Internal definitions shared by the host ABI and the gfx950 kernels of the
// fused per-position scoring library. Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "olive_score.h"

namespace olive {

// Per-(row, vocabulary split) partial statistics, stored as planes of floats:
// plane (field * max_splits + split) holds one value per compacted row.
//   BEST/SEC: largest and second-largest raw logit (unscaled h.W) seen;
//   IDX:      lowest vocabulary index attaining BEST (int32 bits);
//   Z:        sum_v exp(s * (z_v - BEST)) over the split;
//   A:        sum_v exp(s_T * (zT_v - BEST_T)) * D_v, the teacher-weighted logit
//             difference D_v = zT_v - zS_v (equal scales; multiplied by s at the
//             end) or s_T zT_v - s_S zS_v (different scales);
//   B:        sum_v exp(s_S * (zS_v - BEST_S)) * (-D_v), the student-weighted
//             difference (reverse KL; written only when it is requested).
//   J:        the Jensen-Shannon pass's sum over the split of p_hi g(p_lo / p_hi)
//             (log2 units; see the pass), for scored rows only.
//   ZH:       the 256 x 256 kernel only: sum_v w^_v of the teacher weights it keeps in
//             fp16 (w^_v = 2^15 exp(s_T (zT_v - BEST_T)) rounded), rescaled like Z; its A
//             is sum_v w^_v D_v, so that KL's cross term is A / ZH.
enum Field {
    F_BEST_S = 0, F_SEC_S = 1, F_IDX_S = 2, F_Z_S = 3,
    F_BEST_T = 4, F_SEC_T = 5, F_IDX_T = 6, F_Z_T = 7, F_A = 8, F_B = 9, F_J = 10,
    F_ZH = 11,
    NFIELDS = 12
};
// Top-K planes (contexts built with OLIVE_FLAG_TOPK only), per model m (0 = S, 1 = T)
// from F_TK + m * TK_FIELDS: the split's 8 largest raw logits (descending, lower
// index first among equals), their indices (int32 bits), and a floor that bounds
// every logit of the split not in the list.
constexpr int TK_LIST = 8;
constexpr int TK_FIELDS = 2 * TK_LIST + 1;
constexpr int F_TK = NFIELDS;
constexpr int NFIELDS_TOPK = NFIELDS + 2 * TK_FIELDS;
constexpr int TOPK_K = 16;   // LogProb top-K of the OPD baseline (App. A, Table 3)
constexpr int TK_CAP = 256;  // candidates kept per (row, model) by the vocabulary filter
constexpr int FX_CCAP = 64;  // candidates kept per near-tie pair of the greedy re-decision

// Queue of (compacted row, model) pairs whose decision needs every vocabulary entry
// with an fp32 logit at or above a threshold: the MFMA filter fills in their
// candidates (launch_filter). Carved from one allocation (filter_queue_carve).
struct FilterQueue {
    int32_t *n;          // device [2]: queued pairs per model (Sched fields)
    int32_t *nfb;        // device: pairs sent to the exhaustive scan (a Sched field)
    int32_t *qj;         // [2][cap] compacted row
    float *qthr;         // [2][cap] fp32 threshold on the raw logit h . w
    int32_t *qcnt;       // [2][cap] candidates found (may exceed ccap)
    int32_t *cand;       // [2][cap][ccap] their vocabulary indices
    int32_t *fb;         // [2 cap] (model * cap + slot) of the pairs for the exhaustive scan
    uint32_t *smask;     // device [2] or null: per model, the vocabulary splits (bit s) the
                         // filter reads; null: every split
    int cap, ccap;
};
size_t filter_queue_bytes(int64_t cap, int ccap);
FilterQueue filter_queue_carve(void *base, int64_t cap, int ccap, int32_t *n, int32_t *nfb);

// Device workspace of the top-K statistics (topk_carve): cap = max_positions rows.
struct TopkWork {
    float *lse;        // [cap][2] full-vocabulary log-normalisers (combine)
    float *list_v;     // [cap][2][16] the sets: exact logits (fp32) in rank order
    int32_t *list_i;   //               and their vocabulary indices
    FilterQueue fq;    // pairs whose listed candidates do not settle the set
    int cap;
};
size_t topk_work_bytes(int64_t cap);
TopkWork topk_carve(void *base, int64_t cap, int32_t *n, int32_t *nfb);

// Device-side schedule of one call, written by the preparation kernel.
struct Sched {
    int32_t t_valid;    // compacted rows: valid positions, or only the in-region ones when
                        // the call restricts every output to the region
    int32_t n_ptiles;   // ceil(t_valid / tile_rows) for the kernel in use
    int32_t n_splits;   // vocabulary splits
    int32_t n_units;    // n_ptiles * n_splits
    int64_t n_scored;   // in-region valid positions
    int32_t n_flagged;  // rows queued for the near-tie argmax re-decision
    int32_t cu_bad;     // cu_seqlens malformed: nothing is scored
    int32_t n_tkq[2];   // (row, model) pairs whose top-K field needs the vocabulary filter
    int32_t n_tk_fb;    // pairs of those that need the exhaustive exact scan
    int32_t n_fxq[2];   // near-tie (row, model) pairs of the greedy re-decision (MFMA path)
    int32_t n_fx_fb;    // pairs of those that need the exhaustive exact scan
    uint32_t fx_smask[2];   // per model: vocabulary splits (bit s) the re-decision's filter
                            // must read
};

// Top-K outputs of a call (null pointers: not requested).
struct TopkOut {
    float *overlap;
    float *kl;
    int32_t *idx_s;     // [T][TOPK_K]
    int32_t *idx_t;
    bool any() const { return overlap || kl || idx_s || idx_t; }
};

// Bits of the device error word.
enum {
    ERR_TARGET = 1,
    ERR_CUT = 2,
    ERR_VALID = 4,
    ERR_CU = 8,
    ERR_SPAN = 16,
};

constexpr int MFMA_BV = 256;     // vocabulary rows per tile (MFMA M)
constexpr int MFMA_BT = 128;     // positions per tile (MFMA N)
constexpr int WIDE_BT = 256;     // positions per tile of the 256 x 256 kernel
constexpr int SIMPLE_BT = 16;    // positions per tile of the generic kernel
constexpr int SIMPLE_VC = 256;   // vocabulary chunk of the generic kernel
constexpr int MAX_SPLITS = 32;   // vocabulary splits a call may use

struct ScoreArgs {
    const void *hs, *ht;         // hidden states [T][d] (caller)
    const void *ws, *wt;         // weights [V][d] (repacked or borrowed)
    const uint32_t *rowmap;      // [t_valid]: packed row | in-region << 31
    const Sched *sched;
    float *part;                 // partial planes
    int64_t pstride;             // floats per plane
    int32_t V, ds, dt;
    int32_t n_vtiles;            // vocabulary tiles (MFMA) or chunks (generic)
    float cS, cT;                // s * log2(e)
    float sS, sT;                // logit scales
    float wmax_s, wmax_t;        // largest weight-row L2 norm (top-K rounding bounds)
    const float *wmax_dev;       // device [2]: the same two values formed on the device
                                 // (used instead of wmax_s / wmax_t when set)
    // 256 x 256 kernel: K-blocked panels [d/32][rows][32] of the weights (rows = vpad,
    // zero past V) and of the call's compacted hidden rows (rows = prow)
    const void *wps, *wpt, *hps, *hpt;
    int64_t vpad, prow;
    int32_t wide;                // the partials come from that kernel: 1, KL(T || S)'s cross
                                 // term is A / ZH; 2 (reverse only), KL(S || T)'s is B / ZH
};

// Logit-gradient pass of the backward (scored rows [c0, c0 + chunk) of a call).
struct DzArgs {
    int c0, chunk;               // first compacted scored row, rows per chunk (a multiple
                                 // of the 128-row position tile)
    int64_t vp;                  // V rounded up to 64
    const float *lse;            // [rows][2] forward log-normalisers per compacted row
    const int32_t *targets;      // packed realised tokens
    float w_ce, w_kl;            // loss weights
    uint16_t *dz_t;              // [vp/64][chunk][64] bf16 logit gradient (K-blocked panels)
    // The cross-entropy pass that forms its own normalisers (no forward pass before it):
    float *mref;                 // [vocabulary tiles][chunk] the running max each tile's
                                 // stored weights refer to
    float *gy;                   // [chunk] the realised token's gradient w_ce (p_y - 1)
    int32_t *yrow;               // [chunk] the realised token (-1 when out of range)
};

// Jensen-Shannon pass over the scored rows [0, n_scored) of a forward call (the
// scored rows are compacted first), from that call's log-normalisers.
struct JsdArgs {
    const float *lse;            // [rows][2] log-normalisers per compacted row (combine)
};

// C (+)= alpha * A * B^T on bf16 rows, fp32 C. Each operand is read in K steps of 64
// elements: step kk of row r at base + kk * kstep + r * ld (row-major: kstep = 128,
// ld = the row pitch; K-blocked panels [K/64][rows][64]: ld = 128, kstep = rows * 128).
// N and K are read on the device when their pointers are set: clamp(*p - off, 0, cap).
struct GemmArgs {
    const char *A;
    int64_t lda;                 // bytes between A rows
    int64_t akstep;              // bytes between A's K steps
    const char *B;
    int64_t ldb;
    int64_t bkstep;
    int M, N, K;
    const int32_t *n_dev;
    int n_off, n_cap;
    const int32_t *k_dev;
    int k_off, k_cap;
    float *C;
    int64_t ldc;                 // elements
    const uint32_t *rowmap;      // output row of column n: rowmap[rowmap_off + n] (low 31 bits)
    int rowmap_off;
    float alpha;
    bool trans_out;              // C[n][m] instead of C[m][n]
    bool accumulate;             // C += instead of C =
    int ksplit;                  // 1, or 2: halves of K added into C with atomics
    // A given K-major instead: a_panels > 0 panels of 64 rows m, panel p holding K rows
    // of 128 bytes (64 m values each) at A + (p * a_prows + k) * 128 ([M/64][K][64]); the
    // MFMA operand is formed with LDS transpose reads. lda and akstep are then unused.
    int a_panels;
    int a_prows;
};

// Host-side launchers (each defined beside its kernel).
hipError_t launch_filter(const ScoreArgs &a, const FilterQueue &q, hipStream_t st);
hipError_t launch_repack(const void *w_dv, void *w_vd, int64_t d, int64_t V, int elem_bytes,
                         hipStream_t st);
hipError_t launch_prep(const olive_batch &b, const olive_spans *spans, bool region_only,
                       int64_t V, int32_t *seqbuf, Sched *sched, int32_t *err, int64_t *counts,
                       int tile_rows, int policy, int n_vtiles, int grid, int fixed_splits,
                       int min_splits, hipStream_t st);
hipError_t launch_rowmap(const olive_batch &b, const olive_spans *spans, bool region_only,
                         int64_t V, const int32_t *seqbuf,
                         const Sched *sched, uint32_t *rowmap, int32_t *err, float *logp_s,
                         float *logp_t, int32_t *am_s, int32_t *am_t, float *kl, float *kl_rev,
                         float *jsd, float *logp_tmp, const TopkOut &tk, hipStream_t st);
hipError_t launch_score_simple(const ScoreArgs &a, bool bf16, bool has_t, int64_t max_units,
                               hipStream_t st);
hipError_t launch_score_mfma(const ScoreArgs &a, bool has_t, bool same_scale, bool rev,
                             bool topk, int grid, hipStream_t st);
hipError_t launch_score_wide(const ScoreArgs &a, bool same_scale, bool has_t, bool rev,
                             int grid, hipStream_t st);
hipError_t launch_score_wide_dz(const ScoreArgs &a, const DzArgs &z, int grid, hipStream_t st);
hipError_t launch_score_wide_dz_online(const ScoreArgs &a, const DzArgs &z, int grid,
                                       hipStream_t st);
hipError_t launch_dz_lse(const ScoreArgs &a, const DzArgs &z, int grid, float *lse_out,
                         int32_t *err, hipStream_t st);
hipError_t launch_dz_rescale(const ScoreArgs &a, const DzArgs &z, const float *lse,
                             hipStream_t st);
hipError_t launch_panel_w(const void *w, int64_t V, int d, int64_t vpad, void *out,
                          hipStream_t st);
hipError_t launch_panel_h(const void *h, int d, const uint32_t *rowmap, const Sched *sched,
                          int64_t prow, void *out, hipStream_t st);
hipError_t launch_score_dz(const ScoreArgs &a, const DzArgs &z, bool has_t, int grid,
                           hipStream_t st);
hipError_t launch_score_jsd(const ScoreArgs &a, const JsdArgs &z, int grid, hipStream_t st);
hipError_t launch_jsd_combine(const ScoreArgs &a, float *jsd, int grid, int64_t max_rows,
                              hipStream_t st);
hipError_t launch_gemm(const GemmArgs &g, int grid, hipStream_t st);
hipError_t launch_panel_t(const void *w, int64_t V, int d, int64_t vp, void *out,
                          hipStream_t st);
hipError_t launch_gather_t(const void *h, int d, const uint32_t *rowmap, const Sched *sched,
                           int c0, int chunk, int pitch, uint16_t *out, hipStream_t st);
hipError_t launch_fill(float *p, int64_t n, hipStream_t st);
hipError_t launch_zero_tail(uint16_t *dzt, int64_t vp, int chunk, const Sched *sched, int c0,
                            hipStream_t st);
hipError_t launch_combine(const ScoreArgs &a, bool bf16, bool has_t, bool same_scale,
                          const int32_t *targets, int32_t *err, float *logp_s, float *logp_t,
                          int32_t *am_s, int32_t *am_t, float *kl, float *kl_rev, float *logp_tmp,
                          float *lse_out, int32_t *flagged, int flag_cap, int64_t max_rows,
                          hipStream_t st);
hipError_t launch_topk(const ScoreArgs &a, const TopkWork &w, const TopkOut &out,
                       int64_t max_rows, hipStream_t st);
hipError_t launch_argmax_fix(const ScoreArgs &a, const int32_t *flagged, int flag_cap,
                             const FilterQueue &q, int32_t *am_s, int32_t *am_t,
                             hipStream_t st);
hipError_t launch_fixup_impl(const ScoreArgs &a, bool bf16, const int32_t *flagged, int f_base,
                             int cap, void *scratch, const float *wn_s, const float *wn_t,
                             int32_t *am_s, int32_t *am_t, hipStream_t st);
hipError_t launch_row_norms(const void *w, int64_t V, int d, bool bf16, float *out,
                            hipStream_t st);
hipError_t launch_max_norm(const float *wn, int64_t V, float *out, hipStream_t st);
int fixup_chunks(int64_t V);
size_t fixup_result_bytes();
hipError_t launch_ce(const olive_batch &b, const olive_spans *spans, const int32_t *seqbuf,
                     const Sched *sched, const float *logp_s, float *ce, hipStream_t st);

// Layout of the per-sequence workspace (int32, 5 * (max_seqs + 1) entries).
//   [0, B+1)          exclusive prefix sum of compacted rows per sequence (valid, or
//                     in-region when only the region is compacted)
//   [B+1, 2B+2)       effective valid length per sequence (0 for a bad sequence)
//   [2B+2, 3B+3)      effective cut per sequence
//   [3B+3, 4B+4)      1 when the sequence's cut / valid length was out of range
//   [4B+4, 5B+5)      exclusive prefix sum of in-region valid rows per sequence
inline int64_t seqbuf_entries(int64_t max_seqs) { return 5 * (max_seqs + 1); }

}  // namespace olive
