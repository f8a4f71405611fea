// Top-K statistics of a scored position (K = 16): the top-K overlap ratio of the two
// models (Sec. 4.1) and the top-K approximation of KL(teacher || student) that the
// OPD baseline uses (LogProb top-K = 16, App. A Table 3):
//   TopK_X  = the K largest logits of model X (lower index first among equals),
//   overlap = |TopK_S & TopK_T| / K,
//   kl_topk = sum over v in TopK_T of p_T[v] (log p_T[v] - log p_S[v]),
// with the full-vocabulary normalisers of the scoring pass.
//
// The sets are decided on exact logits, as the greedy token is: fp32 logits only
// narrow the field. Exact logits are bf16 products (exact in fp32) summed in fp64.
// delta = d 2^-23 |h| max_v |w_v| bounds the rounding of any fp32 logit of a row.
// The scoring kernel leaves per (split, row, model) the split's 8 largest fp32 logits,
// each as the lower end of a bucket that holds it (one 2^-7 relative step), and a
// floor above every other fp32 logit of the split. Stages:
//   select  - z16 = the 16th largest listed value. A logit whose exact value can reach
//             the exact top-16 has an fp32 value >= thr = z16 - 2 delta. When no split
//             floor reaches thr, every such logit is listed: their exact values are
//             formed and ranked. Otherwise the (row, model) pair is queued with thr;
//   filter  - for the queued pairs, every fp32 logit of the vocabulary (MFMA, 64
//             queued rows x 128 vocabulary rows per work item; filter.hip); the
//             indices of those >= thr are kept (at most TK_CAP per pair);
//   exact   - exact values of a pair's kept indices, ranked; a pair with more than
//             TK_CAP goes to
//   scan    - every exact logit of the pair's row (one workgroup, fp64 sums);
//   outputs - the overlap, the exact student logits at the teacher's tokens and the
//             top-K KL summed in a fixed order.
#include <hip/hip_runtime.h>

#include "exact.hpp"
#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int TK_CAND = MAX_SPLITS * TK_LIST;   // listed entries of one (row, model)
// Rank n <= TK_CAND candidates (exact values cx, indices ci in LDS; kTkEmpty marks a
// skipped slot) and write the 16 best of row j, model m.
__device__ __forceinline__ void rank_and_write(const double *cx, const int *ci, int n, int lane,
                                               int64_t j, int m, float *list_v,
                                               int32_t *list_i) {
    double kv[4];
    int ki[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int c = lane + 64 * t;
        const bool ok = c < n && cx[c] != kTkEmpty;
        kv[t] = ok ? cx[c] : kTkEmpty;
        ki[t] = ok ? ci[c] : kTkNoIdx;
    }
    for (int r = 0; r < TOPK_K; ++r) {
        double bv = kv[0];
        int bi = ki[0], bt = 0;
#pragma unroll
        for (int t = 1; t < 4; ++t)
            if (tk_before(kv[t], ki[t], bv, bi)) { bv = kv[t]; bi = ki[t]; bt = t; }
        double wv = bv;
        int wi = bi;
        wave_best(wv, wi);
        if (bv == wv && bi == wi) {             // candidate indices are unique
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (t == bt) { kv[t] = kTkEmpty; ki[t] = kTkNoIdx; }
        }
        if (lane == 0) {
            list_v[(j * 2 + m) * TOPK_K + r] = (float)wv;
            list_i[(j * 2 + m) * TOPK_K + r] = wi;
        }
    }
}

// One wavefront per compacted in-region row, for each model in turn.
__global__ void __launch_bounds__(256)
topk_select_kernel(ScoreArgs a, TopkWork w) {
    __shared__ float cv[4][TK_CAND];
    __shared__ int ci[4][TK_CAND];
    __shared__ double cx[4][TK_CAND];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 4 + wid;
    Sched *sched = const_cast<Sched *>(a.sched);
    if (j >= sched->t_valid) return;
    const uint32_t rm = a.rowmap[j];
    if (!(rm >> 31)) return;                     // not scored
    const int64_t g = rm & 0x7fffffffu;
    const int ns = sched->n_splits;
    const int nc = ns * TK_LIST;
    const int64_t ps = a.pstride;
    for (int m = 0; m < 2; ++m) {
        const int d = m ? a.dt : a.ds;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const float hh = wave_sumsq(h, d, lane);
        if (hh == 0.f) {   // h = 0: every exact logit is 0, the set is 0..15
            if (lane < TOPK_K) {
                w.list_v[(j * 2 + m) * TOPK_K + lane] = 0.f;
                w.list_i[(j * 2 + m) * TOPK_K + lane] = lane;
            }
            continue;
        }
        float fl = -__builtin_inff();
        if (lane < ns) {
            for (int e = 0; e < TK_LIST; ++e) {
                cv[wid][lane * TK_LIST + e] =
                    a.part[((F_TK + m * TK_FIELDS + e) * MAX_SPLITS + lane) * ps + j];
                ci[wid][lane * TK_LIST + e] = __float_as_int(
                    a.part[((F_TK + m * TK_FIELDS + TK_LIST + e) * MAX_SPLITS + lane) * ps + j]);
            }
            fl = a.part[((F_TK + m * TK_FIELDS + 2 * TK_LIST) * MAX_SPLITS + lane) * ps + j];
        }
        __builtin_amdgcn_wave_barrier();
        // z16: the 16th largest listed value (lane l < ns walks split l's sorted list)
        int ptr = 0;
        double z16 = kTkEmpty;
        for (int r = 0; r < TOPK_K; ++r) {
            double hv = kTkEmpty;
            int hi = kTkNoIdx;
            if (lane < ns && ptr < TK_LIST) {
                hv = cv[wid][lane * TK_LIST + ptr];
                hi = ci[wid][lane * TK_LIST + ptr];
            }
            double bv = hv;
            int bi = hi;
            wave_best(bv, bi);
            if (lane < ns && ptr < TK_LIST && hv == bv && hi == bi) ++ptr;
            z16 = bv;
        }
        const float delta = (float)d * 0x1p-23f * (sqrtf(hh) * (1.0f + 0x1p-10f)) *
                            (a.wmax_dev ? a.wmax_dev[m] : (m ? a.wmax_t : a.wmax_s));
        const float thr = (float)z16 - 2.f * delta;
        // every logit that can reach the exact top-16 is listed unless a floor reaches
        // thr (a floor or threshold that is not finite queues the pair as well)
        if (__any(lane < ns && !(fl < thr))) {
            if (lane == 0) {
                const FilterQueue &f = w.fq;
                const int q = atomicAdd(&f.n[m], 1);
                if (q < f.cap) {
                    f.qj[m * f.cap + q] = (int32_t)j;
                    f.qthr[m * f.cap + q] = thr;
                    f.qcnt[m * f.cap + q] = 0;
                }
            }
            continue;
        }
        // exact values of the listed entries whose bucket reaches thr (an empty slot,
        // index outside [0, V), never does)
        for (int c = 0; c < nc; ++c) {
            double x = kTkEmpty;
            const int v = ci[wid][c];
            if (bucket_ub(cv[wid][c]) >= thr && (unsigned)v < (unsigned)a.V)
                x = wave_dot_exact(h, W + (int64_t)v * d, d, lane);
            if (lane == 0) cx[wid][c] = x;
        }
        __builtin_amdgcn_wave_barrier();
        rank_and_write(cx[wid], ci[wid], nc, lane, j, m, w.list_v, w.list_i);
        __builtin_amdgcn_wave_barrier();
    }
}

// One wavefront per queued pair: exact values of its kept indices, ranked. A pair
// with more indices than were kept goes to the exhaustive scan.
__global__ void __launch_bounds__(256)
topk_exact_kernel(ScoreArgs a, TopkWork w) {
    __shared__ double cx[4][TK_CAP];
    __shared__ int ci[4][TK_CAP];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const FilterQueue &f = w.fq;
    int nq[2];
    for (int m = 0; m < 2; ++m) {
        const int n = f.n[m];
        nq[m] = n < f.cap ? n : f.cap;
    }
    for (int64_t p = (int64_t)blockIdx.x * 4 + wid; p < nq[0] + nq[1];
         p += (int64_t)gridDim.x * 4) {
        const int m = p < nq[0] ? 0 : 1;
        const int q = (int)(m ? p - nq[0] : p);
        const int n = f.qcnt[m * f.cap + q];
        const int64_t j = f.qj[m * f.cap + q];
        if (n > f.ccap) {
            if (lane == 0) f.fb[atomicAdd(f.nfb, 1)] = m * f.cap + q;
            continue;
        }
        const int d = m ? a.dt : a.ds;
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int32_t *cd = f.cand + ((int64_t)m * f.cap + q) * f.ccap;
        for (int c = 0; c < n; ++c) {
            const int v = cd[c];
            const double x = wave_dot_exact(h, W + (int64_t)v * d, d, lane);
            if (lane == 0) { cx[wid][c] = x; ci[wid][c] = v; }
        }
        __builtin_amdgcn_wave_barrier();
        rank_and_write(cx[wid], ci[wid], n, lane, j, m, w.list_v, w.list_i);
        __builtin_amdgcn_wave_barrier();
    }
}

// One workgroup per pair of the exhaustive scan: the row's 16 best of every exact
// logit of the vocabulary.
__global__ void __launch_bounds__(SCAN_THREADS)
topk_scan_kernel(ScoreArgs a, TopkWork w) {
    extern __shared__ __attribute__((aligned(16))) uint16_t tk_h[];   // [d] bf16
    __shared__ double red_v[SCAN_GROUPS][TOPK_K];
    __shared__ int red_i[SCAN_GROUPS][TOPK_K];
    const FilterQueue &f = w.fq;
    const int nfb = *f.nfb;
    for (int e = blockIdx.x; e < nfb; e += gridDim.x) {
        const int code = f.fb[e];
        const int m = code >= f.cap ? 1 : 0;
        const int q = code - m * f.cap;
        const int64_t j = f.qj[m * f.cap + q];
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        double bv;
        int bi;
        scan_row_top16(h, W, d, a.V, tk_h, red_v, red_i, bv, bi);
        if (threadIdx.x < TOPK_K) {
            w.list_v[(j * 2 + m) * TOPK_K + threadIdx.x] = (float)bv;
            w.list_i[(j * 2 + m) * TOPK_K + threadIdx.x] = bi;
        }
    }
}

// One wavefront per compacted row: the outputs. Rows outside the region get the
// fixed values of unscored positions (overlap 0, kl_topk +0, indices -1).
__global__ void __launch_bounds__(256)
topk_output_kernel(ScoreArgs a, TopkWork w, TopkOut o) {
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= a.sched->t_valid) return;
    const uint32_t rm = a.rowmap[j];
    const int64_t g = rm & 0x7fffffffu;
    if (!(rm >> 31)) {
        if (lane == 0) {
            if (o.overlap) o.overlap[g] = 0.f;
            if (o.kl) o.kl[g] = 0.f;
        }
        if (lane < TOPK_K) {
            if (o.idx_s) o.idx_s[g * TOPK_K + lane] = -1;
            if (o.idx_t) o.idx_t[g * TOPK_K + lane] = -1;
        }
        return;
    }
    // An entry outside [0, V) is an empty slot: with finite logits every list fills
    // from real rows; NaN logits (malformed inputs) leave slots empty.
    int is = lane < TOPK_K ? w.list_i[(j * 2 + 0) * TOPK_K + lane] : -1;
    int it = lane < TOPK_K ? w.list_i[(j * 2 + 1) * TOPK_K + lane] : -1;
    if ((unsigned)is >= (unsigned)a.V) is = -1;
    if ((unsigned)it >= (unsigned)a.V) it = -1;
    const float vt = lane < TOPK_K ? w.list_v[(j * 2 + 1) * TOPK_K + lane] : 0.f;
    if (lane < TOPK_K) {
        if (o.idx_s) o.idx_s[g * TOPK_K + lane] = is;
        if (o.idx_t) o.idx_t[g * TOPK_K + lane] = it;
    }
    if (o.overlap) {
        // lane k < 16 tests whether the teacher's k-th token is among the student's 16
        bool hit = false;
        for (int k = 0; k < TOPK_K; ++k)
            hit |= (lane < TOPK_K) && it >= 0 && (__shfl(is, k) == it);
        const int cnt = __popcll(__ballot(hit));
        if (lane == 0) o.overlap[g] = (float)cnt / (float)TOPK_K;
    }
    if (o.kl) {
        const float lse_s = w.lse[j * 2 + 0], lse_t = w.lse[j * 2 + 1];
        const uint16_t *hs = (const uint16_t *)a.hs + g * a.ds;
        const uint16_t *ws = (const uint16_t *)a.ws;
        float sum = 0.f;
        for (int k = 0; k < TOPK_K; ++k) {       // fixed order: the teacher's ranking
            const int v = __shfl(it, k);
            const float zt = __shfl(vt, k);
            const float zs = v >= 0
                ? (float)wave_dot_exact(hs, ws + (int64_t)v * a.ds, a.ds, lane)
                : __builtin_nanf("");
            const float lpt = a.sT * zt - lse_t;
            const float lps = a.sS * zs - lse_s;
            sum = fmaf(fast_exp2(lpt * kLog2e), lpt - lps, sum);
        }
        if (lane == 0) o.kl[g] = sum;
    }
}

namespace {
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
}

size_t topk_work_bytes(int64_t cap) {
    const size_t c = (size_t)cap;
    return align256(c * 2 * 4) + 2 * align256(c * 2 * TOPK_K * 4) +
           filter_queue_bytes(cap, TK_CAP);
}

TopkWork topk_carve(void *base, int64_t cap, int32_t *n, int32_t *nfb) {
    const size_t c = (size_t)cap;
    char *p = (char *)base;
    TopkWork w;
    w.cap = (int)cap;
    w.lse = (float *)p;        p += align256(c * 2 * 4);
    w.list_v = (float *)p;     p += align256(c * 2 * TOPK_K * 4);
    w.list_i = (int32_t *)p;   p += align256(c * 2 * TOPK_K * 4);
    w.fq = filter_queue_carve(p, cap, TK_CAP, n, nfb);
    return w;
}

hipError_t launch_topk(const ScoreArgs &a, const TopkWork &w, const TopkOut &out,
                       int64_t max_rows, hipStream_t st) {
    if (max_rows <= 0) return hipSuccess;
    const dim3 rows((unsigned)((max_rows + 3) / 4));
    topk_select_kernel<<<rows, 256, 0, st>>>(a, w);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_filter(a, w.fq, st);
    if (e != hipSuccess) return e;
    topk_exact_kernel<<<256, 256, 0, st>>>(a, w);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    topk_scan_kernel<<<256, SCAN_THREADS, (size_t)dmax * 2, st>>>(a, w);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_output_kernel<<<rows, 256, 0, st>>>(a, w, out);
    return hipGetLastError();
}

}  // namespace olive
