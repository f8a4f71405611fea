// Top-K statistics of a scored position (K = 16): the top-K overlap ratio of the two
// models (Sec. 4.1) and the top-K approximation of KL(teacher || student) that the
// OPD baseline uses (LogProb top-K = 16, App. A Table 3):
//   TopK_X  = the K largest logits of model X (lower index first among equals),
//   overlap = |TopK_S & TopK_T| / K,
//   kl_topk = sum over v in TopK_T of p_T[v] (log p_T[v] - log p_S[v]),
// with the full-vocabulary normalisers of the scoring pass.
//
// The scoring kernel leaves per (split, row, model) the split's 8 largest logits and a
// floor above everything else of the split. Here:
//   select  - merges the lists of every split into the row's 16 largest; when some
//             split's floor reaches the 16th value an entry it dropped could belong to
//             the set, and the row is queued for an exact rescan;
//   rescan  - recomputes every logit of a queued row (fp32, per vocabulary chunk) and
//             keeps each chunk's 16 largest; merge picks the row's 16 from the chunks;
//   outputs - forms the overlap, gathers the student logits at the teacher's tokens
//             and sums the top-K KL in a fixed order.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int TKR_CHUNK = 4096;     // vocabulary rows per rescan work item
constexpr int TKR_THREADS = 256;
constexpr int TKR_GROUPS = TKR_THREADS / 8;
constexpr float kTkEmpty = -0x1p99f;   // empty list slot (never a real logit)

struct TkEntry {
    float v;
    int i;
};

// (v, i) ranks before (w, j): larger value first, lower index among equals.
__device__ __forceinline__ bool tk_before(float v, int i, float w, int j) {
    return v > w || (v == w && i < j);
}

// Wave-wide best (value, index) of one candidate per lane.
__device__ __forceinline__ TkEntry wave_best(float v, int i) {
    for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(v, off);
        const int oi = __shfl_xor(i, off);
        if (tk_before(ov, oi, v, i)) { v = ov; i = oi; }
    }
    return TkEntry{v, i};
}

template <int N>
__device__ __forceinline__ void tk_insert(float (&v)[N], int (&ix)[N], float x, int xi) {
#pragma unroll
    for (int j = 0; j < N; ++j) {
        const bool b = tk_before(x, xi, v[j], ix[j]);
        const float nv = b ? x : v[j];
        const int ni = b ? xi : ix[j];
        x = b ? v[j] : x;
        xi = b ? ix[j] : xi;
        v[j] = nv;
        ix[j] = ni;
    }
}

template <int N>
__device__ __forceinline__ void tk_pop(float (&v)[N], int (&ix)[N]) {
#pragma unroll
    for (int j = 0; j + 1 < N; ++j) { v[j] = v[j + 1]; ix[j] = ix[j + 1]; }
    v[N - 1] = kTkEmpty;
    ix[N - 1] = 0x7fffffff;
}

// One wavefront per compacted in-region row: the row's 16 largest logits of each
// model from the split lists (raw, unscaled logits: the order is the same as of the
// scaled ones). Lane l < n_splits walks split l's list, staged in LDS.
__global__ void __launch_bounds__(256)
topk_select_kernel(ScoreArgs a, float *__restrict__ list_v, int32_t *__restrict__ list_i,
                   int32_t *__restrict__ queue, int cap) {
    __shared__ float sv[4][MAX_SPLITS][TK_LIST + 1];
    __shared__ int si[4][MAX_SPLITS][TK_LIST + 1];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 4 + wid;
    Sched *sched = const_cast<Sched *>(a.sched);
    if (j >= sched->t_valid) return;
    if (!(a.rowmap[j] >> 31)) return;            // not scored
    const int ns = sched->n_splits;
    const int64_t ps = a.pstride;
    bool overflow = false;
    for (int m = 0; m < 2; ++m) {
        float fl = kTkEmpty;
        if (lane < ns) {
            for (int e = 0; e < TK_LIST; ++e) {
                sv[wid][lane][e] = a.part[((F_TK + m * TK_FIELDS + e) * MAX_SPLITS + lane) * ps + j];
                si[wid][lane][e] = __float_as_int(
                    a.part[((F_TK + m * TK_FIELDS + TK_LIST + e) * MAX_SPLITS + lane) * ps + j]);
            }
            sv[wid][lane][TK_LIST] = kTkEmpty;   // end of the list
            si[wid][lane][TK_LIST] = 0x7fffffff;
            fl = a.part[((F_TK + m * TK_FIELDS + 2 * TK_LIST) * MAX_SPLITS + lane) * ps + j];
        }
        __builtin_amdgcn_wave_barrier();
        int ptr = 0;
        float mine_v = kTkEmpty;
        int mine_i = 0x7fffffff;
        for (int r = 0; r < TOPK_K; ++r) {
            const float hv = lane < ns ? sv[wid][lane][ptr] : kTkEmpty;
            const int hi = lane < ns ? si[wid][lane][ptr] : 0x7fffffff;
            const TkEntry b = wave_best(hv, hi);
            if (lane < ns && hv == b.v && hi == b.i && ptr < TK_LIST) ++ptr;   // unique indices
            if (lane == r) { mine_v = b.v; mine_i = b.i; }
        }
        const float tau = __shfl(mine_v, TOPK_K - 1);
        overflow |= __any(lane < ns && fl >= tau);
        if (lane < TOPK_K) {
            list_v[(j * 2 + m) * TOPK_K + lane] = mine_v;
            list_i[(j * 2 + m) * TOPK_K + lane] = mine_i;
        }
        __builtin_amdgcn_wave_barrier();
    }
    if (overflow && lane == 0) {
        const int q = atomicAdd(&sched->n_topk_queued, 1);
        if (q < cap) queue[q] = (int32_t)j;
    }
}

// 8 consecutive bf16 of two rows: sum of products into acc (v_dot2, exact products).
typedef __bf16 tk_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float tk_dot8(const uint4 &p, const uint4 &q, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(tk_bf16x2, p.x),
                                          __builtin_bit_cast(tk_bf16x2, q.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(tk_bf16x2, p.y),
                                          __builtin_bit_cast(tk_bf16x2, q.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(tk_bf16x2, p.z),
                                          __builtin_bit_cast(tk_bf16x2, q.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(tk_bf16x2, p.w),
                                          __builtin_bit_cast(tk_bf16x2, q.w), acc, false);
    return acc;
}

// Work item (queued row, model, vocabulary chunk): every logit of the chunk in fp32
// (8 lanes per weight row), the chunk's 16 largest kept per 8-lane group and merged
// over the workgroup. The queued row varies fastest over the items, so workgroups
// running side by side read the same weight chunk.
__global__ void __launch_bounds__(TKR_THREADS)
topk_rescan_kernel(ScoreArgs a, const int32_t *__restrict__ queue, int cap, int n_chunks,
                   TkEntry *__restrict__ out) {
    extern __shared__ __attribute__((aligned(16))) uint16_t tk_h[];   // [d] bf16
    __shared__ float red_v[TKR_GROUPS][TOPK_K];
    __shared__ int red_i[TKR_GROUPS][TOPK_K];
    const int nq_all = a.sched->n_topk_queued;
    const int nq = nq_all < cap ? nq_all : cap;
    const int64_t n_items = (int64_t)nq * 2 * n_chunks;
    const int tid = threadIdx.x, g8 = tid & 7, grp = tid >> 3;
    for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int q = (int)(item % nq);
        const int c = (int)((item / nq) % n_chunks);
        const int m = (int)(item / ((int64_t)nq * n_chunks));
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const int64_t g = a.rowmap[queue[q]] & 0x7fffffffu;
        const uint16_t *h = (const uint16_t *)(m ? a.ht : a.hs) + g * d;
        __syncthreads();
        for (int k = tid; k < d; k += TKR_THREADS) tk_h[k] = h[k];
        __syncthreads();
        float lv[TOPK_K];
        int li[TOPK_K];
#pragma unroll
        for (int e = 0; e < TOPK_K; ++e) { lv[e] = kTkEmpty; li[e] = 0x7fffffff; }
        const int v_end = (c + 1) * TKR_CHUNK < a.V ? (c + 1) * TKR_CHUNK : a.V;
        for (int v0 = c * TKR_CHUNK; v0 < v_end; v0 += TKR_GROUPS) {
            const int v = v0 + grp;
            const bool ok = v < v_end;
            const uint16_t *wr = W + (int64_t)(ok ? v : v_end - 1) * d;
            float z = 0.f;
            for (int k = g8 * 8; k < d; k += 64)
                z = tk_dot8(*(const uint4 *)(tk_h + k), *(const uint4 *)(wr + k), z);
            z += __shfl_xor(z, 1);
            z += __shfl_xor(z, 2);
            z += __shfl_xor(z, 4);
            if (ok && z > lv[TOPK_K - 1]) tk_insert<TOPK_K>(lv, li, z, v);   // v increasing
        }
        if (g8 == 0) {
#pragma unroll
            for (int e = 0; e < TOPK_K; ++e) { red_v[grp][e] = lv[e]; red_i[grp][e] = li[e]; }
        }
        __syncthreads();
        if (tid < 64) {   // merge the 32 group lists: lane l < 32 owns group l's list
            int ptr = 0;
            float cur_v = tid < TKR_GROUPS ? red_v[tid][0] : kTkEmpty;
            int cur_i = tid < TKR_GROUPS ? red_i[tid][0] : 0x7fffffff;
            for (int r = 0; r < TOPK_K; ++r) {
                const TkEntry b = wave_best(cur_v, cur_i);
                if (tid < TKR_GROUPS && cur_v == b.v && cur_i == b.i) {
                    ++ptr;
                    cur_v = ptr < TOPK_K ? red_v[tid][ptr] : kTkEmpty;
                    cur_i = ptr < TOPK_K ? red_i[tid][ptr] : 0x7fffffff;
                }
                if (tid == 0) out[((int64_t)q * 2 + m) * n_chunks * TOPK_K + (int64_t)c * TOPK_K + r] = b;
            }
        }
        __syncthreads();
    }
}

// One wavefront per (queued row, model): the 16 largest over the chunks' lists.
__global__ void __launch_bounds__(256)
topk_rescan_merge_kernel(ScoreArgs a, const int32_t *__restrict__ queue, int cap, int n_chunks,
                         const TkEntry *__restrict__ res, float *__restrict__ list_v,
                         int32_t *__restrict__ list_i) {
    const int lane = threadIdx.x & 63;
    const int nq_all = a.sched->n_topk_queued;
    const int nq = nq_all < cap ? nq_all : cap;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (int64_t)nq * 2) return;
    const int q = (int)(w >> 1), m = (int)(w & 1);
    const TkEntry *r = res + w * n_chunks * TOPK_K;
    // each lane keeps the 16 best of its chunks (lane, lane + 64, ...); every chunk
    // list is sorted, so a chunk is read only while its entries still rank in
    float lv[TOPK_K];
    int li[TOPK_K];
#pragma unroll
    for (int e = 0; e < TOPK_K; ++e) { lv[e] = kTkEmpty; li[e] = 0x7fffffff; }
    for (int c = lane; c < n_chunks; c += 64)
        for (int e = 0; e < TOPK_K; ++e) {
            const TkEntry x = r[(int64_t)c * TOPK_K + e];
            if (!tk_before(x.v, x.i, lv[TOPK_K - 1], li[TOPK_K - 1])) break;
            tk_insert<TOPK_K>(lv, li, x.v, x.i);
        }
    float mine_v = kTkEmpty;
    int mine_i = 0x7fffffff;
    for (int k = 0; k < TOPK_K; ++k) {   // vocabulary indices are unique across chunks
        const TkEntry b = wave_best(lv[0], li[0]);
        if (lv[0] == b.v && li[0] == b.i) tk_pop<TOPK_K>(lv, li);
        if (lane == k) { mine_v = b.v; mine_i = b.i; }
    }
    const int64_t j = queue[q];
    if (lane < TOPK_K) {
        list_v[(j * 2 + m) * TOPK_K + lane] = mine_v;
        list_i[(j * 2 + m) * TOPK_K + lane] = mine_i;
    }
}

// One wavefront per compacted row: the outputs. Rows outside the region get the
// fixed values of unscored positions (overlap 0, kl_topk +0, indices -1).
template <typename E>
__global__ void __launch_bounds__(256)
topk_output_kernel(ScoreArgs a, const float *__restrict__ lse, const float *__restrict__ list_v,
                   const int32_t *__restrict__ list_i, float *__restrict__ overlap,
                   float *__restrict__ kl_topk, int32_t *__restrict__ idx_s,
                   int32_t *__restrict__ idx_t) {
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= a.sched->t_valid) return;
    const uint32_t rm = a.rowmap[j];
    const int64_t g = rm & 0x7fffffffu;
    if (!(rm >> 31)) {
        if (lane == 0) {
            if (overlap) overlap[g] = 0.f;
            if (kl_topk) kl_topk[g] = 0.f;
        }
        if (lane < TOPK_K) {
            if (idx_s) idx_s[g * TOPK_K + lane] = -1;
            if (idx_t) idx_t[g * TOPK_K + lane] = -1;
        }
        return;
    }
    // An entry outside [0, V) is a list's empty slot: with finite logits every list
    // fills from real rows; NaN logits (malformed inputs) leave slots empty.
    int is = lane < TOPK_K ? list_i[(j * 2 + 0) * TOPK_K + lane] : -1;
    int it = lane < TOPK_K ? list_i[(j * 2 + 1) * TOPK_K + lane] : -1;
    if ((unsigned)is >= (unsigned)a.V) is = -1;
    if ((unsigned)it >= (unsigned)a.V) it = -1;
    const float vt = lane < TOPK_K ? list_v[(j * 2 + 1) * TOPK_K + lane] : 0.f;
    if (lane < TOPK_K) {
        if (idx_s) idx_s[g * TOPK_K + lane] = is;
        if (idx_t) idx_t[g * TOPK_K + lane] = it;
    }
    if (overlap) {
        // lane k < 16 tests whether the teacher's k-th token is among the student's 16
        bool hit = false;
        for (int k = 0; k < TOPK_K; ++k) hit |= (lane < TOPK_K) && it >= 0 && (__shfl(is, k) == it);
        const int cnt = __popcll(__ballot(hit));
        if (lane == 0) overlap[g] = (float)cnt / (float)TOPK_K;
    }
    if (kl_topk) {
        const float lse_s = lse[j * 2 + 0], lse_t = lse[j * 2 + 1];
        const E *hs = (const E *)a.hs + g * a.ds;
        const E *ws = (const E *)a.ws;
        float sum = 0.f;
        for (int k = 0; k < TOPK_K; ++k) {       // fixed order: the teacher's ranking
            const int v = __shfl(it, k);
            const float zt = __shfl(vt, k);
            float zs = 0.f;
            if (v >= 0) {
                const E *wr = ws + (int64_t)v * a.ds;
                for (int e = lane; e < a.ds; e += 64)
                    zs = fmaf(load_elem(hs, e), load_elem(wr, e), zs);
                for (int off = 32; off > 0; off >>= 1) zs += __shfl_xor(zs, off);
            } else {
                zs = __builtin_nanf("");
            }
            const float lpt = a.sT * zt - lse_t;
            const float lps = a.sS * zs - lse_s;
            sum = fmaf(fast_exp2(lpt * 1.4426950408889634f), lpt - lps, sum);
        }
        if (lane == 0) kl_topk[g] = sum;
    }
}

size_t topk_rescan_bytes(int64_t V, int cap) {
    const int n_chunks = (int)((V + TKR_CHUNK - 1) / TKR_CHUNK);
    return (size_t)cap * 2 * n_chunks * TOPK_K * sizeof(TkEntry);
}

hipError_t launch_topk(const ScoreArgs &a, bool bf16, const float *lse, float *list_v,
                       int32_t *list_i, int32_t *queue, int cap, void *rescan_buf,
                       float *overlap, float *kl_topk, int32_t *idx_s, int32_t *idx_t,
                       int64_t max_rows, hipStream_t st) {
    if (max_rows <= 0) return hipSuccess;
    if (!bf16) return hipErrorInvalidValue;   // the MFMA path only
    dim3 grid((unsigned)((max_rows + 3) / 4));
    topk_select_kernel<<<grid, 256, 0, st>>>(a, list_v, list_i, queue, cap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int n_chunks = (int)((a.V + TKR_CHUNK - 1) / TKR_CHUNK);
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    topk_rescan_kernel<<<512, TKR_THREADS, (size_t)dmax * 2, st>>>(a, queue, cap, n_chunks,
                                                                   (TkEntry *)rescan_buf);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_rescan_merge_kernel<<<(unsigned)((2 * (int64_t)cap + 3) / 4), 256, 0, st>>>(
        a, queue, cap, n_chunks, (const TkEntry *)rescan_buf, list_v, list_i);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    topk_output_kernel<uint16_t><<<grid, 256, 0, st>>>(a, lse, list_v, list_i, overlap, kl_topk,
                                                       idx_s, idx_t);
    return hipGetLastError();
}

}  // namespace olive
