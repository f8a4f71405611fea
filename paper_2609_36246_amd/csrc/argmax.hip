// Exact re-decision of the greedy token on the bf16 MFMA path, for the (row, model)
// pairs whose fp32 top-2 logit gap fell inside the fp32 error window (flagged by the
// combine pass with theta, a lower bound of the exact value of the fp32 winner).
//
// The exact maximum is >= theta, and every fp32 logit (in any summation order) lies
// within delta = d 2^-23 |h| max_v |w_v| of its exact value, so every entry that can
// be the exact maximum has an fp32 logit >= thr = theta - delta. The scoring pass left
// per vocabulary split the fp32 maximum, second value (ties counted twice) and argmax
// of the row: a split whose maximum is below thr holds no such entry, one whose second
// value is below thr exactly one, at its argmax. Only splits whose second value reaches
// thr are read again, by the vocabulary filter (MFMA, up to 64 queued rows per read).
// The exact values of all these entries (bf16 products summed in fp64) decide, lower
// index first. A pair with more than FX_CCAP entries takes the exhaustive exact scan.
#include <hip/hip_runtime.h>

#include "exact.hpp"
#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

// One wavefront per flagged row: queue each flagged model with its threshold, its
// candidates from the splits that hold at most one, and mark the other splits for the
// filter. Rows whose hidden state is zero need nothing: every logit is exactly 0 and
// the scoring pass already took index 0.
__device__ __forceinline__ void queue_row(const ScoreArgs &a, const int32_t *__restrict__ flagged,
                                          int f, int ns, int lane, const FilterQueue &q) {
    const int32_t j = flagged[4 * f];
    const int fl = flagged[4 * f + 1];
    const int64_t g = a.rowmap[j] & 0x7fffffffu;
    for (int m = 0; m < 2; ++m) {
        if (!(fl & (1 << m))) continue;
        const int d = m ? a.dt : a.ds;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        const float hh = wave_sumsq(h, d, lane);
        if (hh == 0.f) continue;
        const float theta = __int_as_float(flagged[4 * f + 2 + m]);
        const float delta =
            (float)d * 0x1p-23f * (sqrtf(hh) * (1.0f + 0x1p-10f)) *
            (a.wmax_dev ? a.wmax_dev[m] : (m ? a.wmax_t : a.wmax_s));
        const float thr = theta - delta;
        // lane s < ns: split s's maximum, second value and argmax for this row
        const int fb = m ? F_BEST_T : F_BEST_S;
        float best = kNegInf, sec = kNegInf;
        int idx = 0;
        if (lane < ns) {
            best = a.part[((fb + 0) * MAX_SPLITS + lane) * a.pstride + j];
            sec = a.part[((fb + 1) * MAX_SPLITS + lane) * a.pstride + j];
            idx = __float_as_int(a.part[((fb + 2) * MAX_SPLITS + lane) * a.pstride + j]);
        }
        const bool scan = sec >= thr;
        const bool one = best >= thr && !scan;
        const uint64_t one_mask = __ballot(one);
        const uint64_t scan_mask = __ballot(scan);
        int slot = lane == 0 ? atomicAdd(&q.n[m], 1) : 0;
        slot = __shfl(slot, 0);
        if (slot >= q.cap) continue;
        int32_t *cd = q.cand + ((int64_t)m * q.cap + slot) * q.ccap;
        if (one) cd[__popcll(one_mask & ((1ull << lane) - 1ull))] = idx;
        if (lane == 0) {
            q.qj[m * q.cap + slot] = j;
            q.qthr[m * q.cap + slot] = thr;
            q.qcnt[m * q.cap + slot] = __popcll(one_mask);
            if (scan_mask) atomicOr(&q.smask[m], (uint32_t)scan_mask);
        }
    }
}

__global__ void __launch_bounds__(256)
fx_queue_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int flag_cap,
                FilterQueue q) {
    const int lane = threadIdx.x & 63;
    const int nf_all = a.sched->n_flagged;
    const int nf = nf_all < flag_cap ? nf_all : flag_cap;
    const int ns = a.sched->n_splits;
    for (int f = blockIdx.x * 4 + (threadIdx.x >> 6); f < nf; f += gridDim.x * 4)
        queue_row(a, flagged, f, ns, lane, q);
}

// One wavefront per queued pair: the exact maximum of its candidates (one per lane).
__global__ void __launch_bounds__(256)
fx_exact_kernel(ScoreArgs a, FilterQueue q, int32_t *__restrict__ am_s,
                int32_t *__restrict__ am_t) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    int nq[2];
    for (int m = 0; m < 2; ++m) {
        const int n = q.n[m];
        nq[m] = n < q.cap ? n : q.cap;
    }
    for (int64_t p = (int64_t)blockIdx.x * 4 + wid; p < nq[0] + nq[1];
         p += (int64_t)gridDim.x * 4) {
        const int m = p < nq[0] ? 0 : 1;
        const int s = (int)(m ? p - nq[0] : p);
        const int n = q.qcnt[m * q.cap + s];
        const int64_t j = q.qj[m * q.cap + s];
        if (n > q.ccap) {
            if (lane == 0) q.fb[atomicAdd(q.nfb, 1)] = m * q.cap + s;
            continue;
        }
        if (n == 0) continue;   // cannot happen: the fp32 winner itself reaches theta
        const int d = m ? a.dt : a.ds;
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int32_t *cd = q.cand + ((int64_t)m * q.cap + s) * q.ccap;
        double bv = kTkEmpty;
        int bi = kTkNoIdx;
        for (int c = 0; c < n; ++c) {   // one wavefront dot per candidate
            const int v = cd[c];
            const double x = wave_dot_exact(h, W + (int64_t)v * d, d, lane);
            if (tk_before(x, v, bv, bi)) { bv = x; bi = v; }
        }
        if (lane == 0) (m ? am_t : am_s)[g] = bi;
    }
}

// One workgroup per pair of the exhaustive scan: the best of every exact logit.
__global__ void __launch_bounds__(SCAN_THREADS)
fx_scan_kernel(ScoreArgs a, FilterQueue q, int32_t *__restrict__ am_s,
               int32_t *__restrict__ am_t) {
    extern __shared__ __attribute__((aligned(16))) uint16_t fx_h[];   // [d] bf16
    __shared__ double red_v[SCAN_GROUPS][TOPK_K];
    __shared__ int red_i[SCAN_GROUPS][TOPK_K];
    const int nfb = *q.nfb;
    for (int e = blockIdx.x; e < nfb; e += gridDim.x) {
        const int code = q.fb[e];
        const int m = code >= q.cap ? 1 : 0;
        const int s = code - m * q.cap;
        const int64_t j = q.qj[m * q.cap + s];
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        double bv;
        int bi;
        scan_row_top16(h, W, d, a.V, fx_h, red_v, red_i, bv, bi);
        if (threadIdx.x == 0) (m ? am_t : am_s)[g] = bi;
    }
}

hipError_t launch_argmax_fix(const ScoreArgs &a, const int32_t *flagged, int flag_cap,
                             const FilterQueue &q, int32_t *am_s, int32_t *am_t,
                             hipStream_t st) {
    if (flag_cap <= 0) return hipSuccess;
    // a fixed grid that strides over the flagged rows (their count is on the device)
    const int blocks = (flag_cap + 3) / 4 < 1024 ? (flag_cap + 3) / 4 : 1024;
    fx_queue_kernel<<<blocks, 256, 0, st>>>(a, flagged, flag_cap, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_filter(a, q, st);
    if (e != hipSuccess) return e;
    fx_exact_kernel<<<64, 256, 0, st>>>(a, q, am_s, am_t);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    fx_scan_kernel<<<64, SCAN_THREADS, (size_t)dmax * 2, st>>>(a, q, am_s, am_t);
    return hipGetLastError();
}

}  // namespace olive
