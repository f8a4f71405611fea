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
//             queued rows x 128 vocabulary rows per work item); the indices of those
//             >= thr are kept (at most TK_CAP per pair);
//   exact   - exact values of a pair's kept indices, ranked; a pair with more than
//             TK_CAP goes to
//   scan    - every exact logit of the pair's row (one workgroup, fp64 sums);
//   outputs - the overlap, the exact student logits at the teacher's tokens and the
//             top-K KL summed in a fixed order.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int TK_CAND = MAX_SPLITS * TK_LIST;   // listed entries of one (row, model)
constexpr int TKF_QB = 64;                      // queued rows per filter work item
constexpr int TKF_VR = 128;                     // vocabulary rows per filter work item
constexpr int TKS_THREADS = 256;                // exhaustive scan
constexpr int TKS_GROUPS = TKS_THREADS / 8;
constexpr double kTkEmpty = -0x1p1000;          // empty slot (below every finite logit)
constexpr int kTkNoIdx = 0x7fffffff;

typedef __bf16 tk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float tk_floatx16 __attribute__((ext_vector_type(16)));

// (v, i) ranks before (w, j): larger value first, lower index among equals.
__device__ __forceinline__ bool tk_before(double v, int i, double w, int j) {
    return v > w || (v == w && i < j);
}

// Wave-wide best (value, index) of one candidate per lane.
__device__ __forceinline__ void wave_best(double &v, int &i) {
    for (int off = 32; off > 0; off >>= 1) {
        const double ov = __shfl_xor(v, off);
        const int oi = __shfl_xor(i, off);
        if (tk_before(ov, oi, v, i)) { v = ov; i = oi; }
    }
}

template <int N>
__device__ __forceinline__ void tk_insert(double (&v)[N], int (&ix)[N], double x, int xi) {
#pragma unroll
    for (int j = 0; j < N; ++j) {
        const bool b = tk_before(x, xi, v[j], ix[j]);
        const double nv = b ? x : v[j];
        const int ni = b ? xi : ix[j];
        x = b ? v[j] : x;
        xi = b ? ix[j] : xi;
        v[j] = nv;
        ix[j] = ni;
    }
}

// Sum of the exact products of 8 bf16 pairs, accumulated in fp64.
__device__ __forceinline__ double dot8_f64(const uint4 &p, const uint4 &q, double acc) {
    const uint32_t a[4] = {p.x, p.y, p.z, p.w}, b[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        acc += (double)(bf16_bits_to_f32(a[t] & 0xffffu) * bf16_bits_to_f32(b[t] & 0xffffu));
        acc += (double)(bf16_bits_to_f32(a[t] >> 16) * bf16_bits_to_f32(b[t] >> 16));
    }
    return acc;
}

// Exact logit h . w of one vocabulary row by one wavefront (d a multiple of 8, rows
// 16-byte aligned); every lane returns the sum.
__device__ __forceinline__ double wave_dot_exact(const uint16_t *h, const uint16_t *w, int d,
                                                 int lane) {
    double acc = 0.0;
    for (int k = lane * 8; k < d; k += 512)
        acc = dot8_f64(*(const uint4 *)(h + k), *(const uint4 *)(w + k), acc);
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

// |h|^2 in fp32 by one wavefront.
__device__ __forceinline__ float wave_sumsq(const uint16_t *h, int d, int lane) {
    float acc = 0.f;
    for (int k = lane; k < d; k += 64) {
        const float x = bf16_bits_to_f32(h[k]);
        acc = fmaf(x, x, acc);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

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
                            (m ? a.wmax_t : a.wmax_s);
        const float thr = (float)z16 - 2.f * delta;
        // every logit that can reach the exact top-16 is listed unless a floor reaches
        // thr (a floor or threshold that is not finite queues the pair as well)
        if (__any(lane < ns && !(fl < thr))) {
            if (lane == 0) {
                const int q = atomicAdd(&sched->n_tkq[m], 1);
                if (q < w.cap) {
                    w.qj[m * w.cap + q] = (int32_t)j;
                    w.qthr[m * w.cap + q] = thr;
                    w.qcnt[m * w.cap + q] = 0;
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

// Work item (model, 64 queued rows, 128 vocabulary rows): the fp32 logits by MFMA
// (32x32x16 bf16; vocabulary rows are the A operand, queued rows the B operand, both
// read straight from memory), the indices of those >= the pair's threshold kept. The
// K order inside a 64-wide step is permuted the same way for both operands: lane
// half hf takes k in [32 hf + 8 s, 32 hf + 8 s + 8) at sub-step s, so each lane reads
// 64 contiguous bytes of its row per step.
__global__ void __launch_bounds__(256)
topk_filter_kernel(ScoreArgs a, TopkWork w) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int hf = lane >> 5, c32 = lane & 31;
    const int n_vt = (a.V + TKF_VR - 1) / TKF_VR;
    int nq[2], nqb[2];
    for (int m = 0; m < 2; ++m) {
        const int n = a.sched->n_tkq[m];
        nq[m] = n < w.cap ? n : w.cap;
        nqb[m] = (nq[m] + TKF_QB - 1) / TKF_QB;
    }
    const int64_t items0 = (int64_t)nqb[0] * n_vt;
    const int64_t items = items0 + (int64_t)nqb[1] * n_vt;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int m = it < items0 ? 0 : 1;
        const int64_t rel = m ? it - items0 : it;
        const int qb = (int)(rel % nqb[m]);      // queued batch fastest: a vocabulary
        const int vt = (int)(rel / nqb[m]);      // tile is read by neighbouring items
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const uint16_t *H = (const uint16_t *)(m ? a.ht : a.hs);
        const int r0 = vt * TKF_VR + wid * 32;
        const int vrow = r0 + c32 < a.V ? r0 + c32 : a.V - 1;
        const uint16_t *wr = W + (int64_t)vrow * d + 32 * hf;
        const uint16_t *hr[2];
        for (int cb = 0; cb < 2; ++cb) {
            int q = qb * TKF_QB + cb * 32 + c32;
            q = q < nq[m] ? q : nq[m] - 1;
            const int64_t g = a.rowmap[w.qj[m * w.cap + q]] & 0x7fffffffu;
            hr[cb] = H + g * d + 32 * hf;
        }
        tk_floatx16 acc[2];
        acc[0] = tk_floatx16{0.f};
        acc[1] = tk_floatx16{0.f};
        for (int k0 = 0; k0 < d; k0 += 64) {
            uint4 A[4], B0[4], B1[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                A[s] = *(const uint4 *)(wr + k0 + 8 * s);
                B0[s] = *(const uint4 *)(hr[0] + k0 + 8 * s);
                B1[s] = *(const uint4 *)(hr[1] + k0 + 8 * s);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const tk_bf16x8 av = __builtin_bit_cast(tk_bf16x8, A[s]);
                acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    av, __builtin_bit_cast(tk_bf16x8, B0[s]), acc[0], 0, 0, 0);
                acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    av, __builtin_bit_cast(tk_bf16x8, B1[s]), acc[1], 0, 0, 0);
            }
        }
        // lane holds column c32 (a queued row) and rows 8 (r / 4) + 4 hf + r % 4
        for (int cb = 0; cb < 2; ++cb) {
            const int q = qb * TKF_QB + cb * 32 + c32;
            if (q >= nq[m]) continue;
            const float thr = w.qthr[m * w.cap + q];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = r0 + 8 * (r >> 2) + 4 * hf + (r & 3);
                if (v < a.V && acc[cb][r] >= thr) {
                    const int n = atomicAdd(&w.qcnt[m * w.cap + q], 1);
                    if (n < TK_CAP) w.cand[((int64_t)m * w.cap + q) * TK_CAP + n] = v;
                }
            }
        }
    }
}

// One wavefront per queued pair: exact values of its kept indices, ranked. A pair
// with more indices than were kept goes to the exhaustive scan.
__global__ void __launch_bounds__(256)
topk_exact_kernel(ScoreArgs a, TopkWork w) {
    __shared__ double cx[4][TK_CAP];
    __shared__ int ci[4][TK_CAP];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    Sched *sched = const_cast<Sched *>(a.sched);
    int nq[2];
    for (int m = 0; m < 2; ++m) {
        const int n = sched->n_tkq[m];
        nq[m] = n < w.cap ? n : w.cap;
    }
    for (int64_t p = (int64_t)blockIdx.x * 4 + wid; p < nq[0] + nq[1];
         p += (int64_t)gridDim.x * 4) {
        const int m = p < nq[0] ? 0 : 1;
        const int q = (int)(m ? p - nq[0] : p);
        const int n = w.qcnt[m * w.cap + q];
        const int64_t j = w.qj[m * w.cap + q];
        if (n > TK_CAP) {
            if (lane == 0) {
                const int f = atomicAdd(&sched->n_tk_fb, 1);
                w.fb[f] = m * w.cap + q;
            }
            continue;
        }
        const int d = m ? a.dt : a.ds;
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int32_t *cd = w.cand + ((int64_t)m * w.cap + q) * TK_CAP;
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

// One workgroup per pair of the exhaustive scan: every exact logit of the row (8 lanes
// per vocabulary row, fp64 sums), a top-16 per 8-lane group, merged over the group.
__global__ void __launch_bounds__(TKS_THREADS)
topk_scan_kernel(ScoreArgs a, TopkWork w) {
    extern __shared__ __attribute__((aligned(16))) uint16_t tk_h[];   // [d] bf16
    __shared__ double red_v[TKS_GROUPS][TOPK_K];
    __shared__ int red_i[TKS_GROUPS][TOPK_K];
    const int nfb = a.sched->n_tk_fb;
    const int tid = threadIdx.x, g8 = tid & 7, grp = tid >> 3;
    for (int e = blockIdx.x; e < nfb; e += gridDim.x) {
        const int code = w.fb[e];
        const int m = code >= w.cap ? 1 : 0;
        const int q = code - m * w.cap;
        const int64_t j = w.qj[m * w.cap + q];
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        __syncthreads();
        for (int k = tid * 8; k < d; k += TKS_THREADS * 8)
            *(uint4 *)(tk_h + k) = *(const uint4 *)(h + k);
        __syncthreads();
        double lv[TOPK_K];
        int li[TOPK_K];
#pragma unroll
        for (int t = 0; t < TOPK_K; ++t) { lv[t] = kTkEmpty; li[t] = kTkNoIdx; }
        for (int v0 = 0; v0 < a.V; v0 += TKS_GROUPS) {
            const int v = v0 + grp;
            const bool ok = v < a.V;
            const uint16_t *wr = W + (int64_t)(ok ? v : a.V - 1) * d;
            double z = 0.0;
            for (int k = g8 * 8; k < d; k += 64)
                z = dot8_f64(*(const uint4 *)(tk_h + k), *(const uint4 *)(wr + k), z);
            z += __shfl_xor(z, 1);
            z += __shfl_xor(z, 2);
            z += __shfl_xor(z, 4);
            if (ok && tk_before(z, v, lv[TOPK_K - 1], li[TOPK_K - 1]))
                tk_insert<TOPK_K>(lv, li, z, v);
        }
        if (g8 == 0) {
#pragma unroll
            for (int t = 0; t < TOPK_K; ++t) { red_v[grp][t] = lv[t]; red_i[grp][t] = li[t]; }
        }
        __syncthreads();
        if (tid < 64) {   // merge the 32 group lists: lane l < 32 owns group l's list
            int ptr = 0;
            for (int r = 0; r < TOPK_K; ++r) {
                double hv = kTkEmpty;
                int hi = kTkNoIdx;
                if (tid < TKS_GROUPS && ptr < TOPK_K) { hv = red_v[tid][ptr]; hi = red_i[tid][ptr]; }
                double bv = hv;
                int bi = hi;
                wave_best(bv, bi);
                if (tid < TKS_GROUPS && ptr < TOPK_K && hv == bv && hi == bi) ++ptr;
                if (tid == 0) {
                    w.list_v[(j * 2 + m) * TOPK_K + r] = (float)bv;
                    w.list_i[(j * 2 + m) * TOPK_K + r] = bi;
                }
            }
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
    return align256(c * 2 * 4) + 2 * align256(c * 2 * TOPK_K * 4) + 3 * align256(c * 2 * 4) +
           align256(c * 2 * TK_CAP * 4) + align256(c * 2 * 4);
}

TopkWork topk_carve(void *base, int64_t cap) {
    const size_t c = (size_t)cap;
    char *p = (char *)base;
    TopkWork w;
    w.cap = (int)cap;
    w.lse = (float *)p;        p += align256(c * 2 * 4);
    w.list_v = (float *)p;     p += align256(c * 2 * TOPK_K * 4);
    w.list_i = (int32_t *)p;   p += align256(c * 2 * TOPK_K * 4);
    w.qj = (int32_t *)p;       p += align256(c * 2 * 4);
    w.qthr = (float *)p;       p += align256(c * 2 * 4);
    w.qcnt = (int32_t *)p;     p += align256(c * 2 * 4);
    w.cand = (int32_t *)p;     p += align256(c * 2 * TK_CAP * 4);
    w.fb = (int32_t *)p;
    return w;
}

hipError_t launch_topk(const ScoreArgs &a, const TopkWork &w, const TopkOut &out,
                       int64_t max_rows, hipStream_t st) {
    if (max_rows <= 0) return hipSuccess;
    const dim3 rows((unsigned)((max_rows + 3) / 4));
    topk_select_kernel<<<rows, 256, 0, st>>>(a, w);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_filter_kernel<<<1024, 256, 0, st>>>(a, w);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_exact_kernel<<<256, 256, 0, st>>>(a, w);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    topk_scan_kernel<<<256, TKS_THREADS, (size_t)dmax * 2, st>>>(a, w);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_output_kernel<<<rows, 256, 0, st>>>(a, w, out);
    return hipGetLastError();
}

}  // namespace olive
