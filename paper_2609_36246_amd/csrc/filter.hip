// The vocabulary filter of the exact decisions on the bf16 MFMA path: for every
// queued (row, model) pair, the indices of the vocabulary entries whose fp32 logit
// reaches the pair's threshold. The threshold is set so that every entry that can
// win the exact decision is among them; the exact values are formed afterwards. With
// a split mask (the greedy re-decision), only the vocabulary splits it marks are read;
// the candidates of the other splits are already queued.
#include <hip/hip_runtime.h>

#include "olive_internal.hpp"

namespace olive {

constexpr int FL_QB = 64;    // queued rows per work item (two 32-column MFMA blocks)
constexpr int FL_VR = 128;   // vocabulary rows per work item (4 wavefronts x 32)
static_assert(2 * FL_VR == MFMA_BV, "two work-item tiles per tile of the scoring pass");

typedef __bf16 fl_bf16x8 __attribute__((ext_vector_type(8)));
typedef float fl_floatx16 __attribute__((ext_vector_type(16)));

// One 64-wide K step of a lane's operands: its vocabulary row (A) and its two queued
// rows (B0, B1), 4 x 16 bytes each.
__device__ __forceinline__ void fl_load(uint4 (&R)[12], const uint16_t *wr,
                                        const uint16_t *const (&hr)[2], int k0) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        R[s] = *(const uint4 *)(wr + k0 + 8 * s);
        R[4 + s] = *(const uint4 *)(hr[0] + k0 + 8 * s);
        R[8 + s] = *(const uint4 *)(hr[1] + k0 + 8 * s);
    }
}

__device__ __forceinline__ void fl_mma(const uint4 (&R)[12], fl_floatx16 (&acc)[2]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const fl_bf16x8 av = __builtin_bit_cast(fl_bf16x8, R[s]);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            av, __builtin_bit_cast(fl_bf16x8, R[4 + s]), acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            av, __builtin_bit_cast(fl_bf16x8, R[8 + s]), acc[1], 0, 0, 0);
    }
}

// Work item (model, 64 queued rows, 128 vocabulary rows): the fp32 logits by MFMA
// (32x32x16 bf16; vocabulary rows are the A operand, queued rows the B operand, both
// read straight from memory), the indices of those >= the pair's threshold kept. The
// K order inside a 64-wide step is permuted the same way for both operands: lane
// half hf takes k in [32 hf + 8 s, 32 hf + 8 s + 8) at sub-step s, so each lane reads
// 64 contiguous bytes of its row per step.
__global__ void __launch_bounds__(256)
filter_kernel(ScoreArgs a, FilterQueue w) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int hf = lane >> 5, c32 = lane & 31;
    const int n_vt = (a.V + FL_VR - 1) / FL_VR;
    int nq[2], nqb[2];
    for (int m = 0; m < 2; ++m) {
        const int n = w.n[m];
        nq[m] = n < w.cap ? n : w.cap;
        nqb[m] = (nq[m] + FL_QB - 1) / FL_QB;
    }
    // Teacher items first: the wider rows take longer, and the dispatcher hands the
    // cheaper student items to whichever CUs finish early.
    const int64_t items1 = (int64_t)nqb[1] * n_vt;
    const int64_t items = items1 + (int64_t)nqb[0] * n_vt;
    // With a split mask, only the vocabulary tiles of the marked splits of the scoring
    // pass (split s: its 256-row tiles [n_vtiles s / ns, n_vtiles (s + 1) / ns)).
    uint32_t sm[2] = {0xFFFFFFFFu, 0xFFFFFFFFu};
    if (w.smask) {
        sm[0] = w.smask[0];
        sm[1] = w.smask[1];
        if ((sm[0] | sm[1]) == 0u) return;
    }
    const int ns = a.sched->n_splits;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int m = it < items1 ? 1 : 0;
        const int64_t rel = m ? it : it - items1;
        const int qb = (int)(rel % nqb[m]);      // queued batch fastest: a vocabulary
        const int vt = (int)(rel / nqb[m]);      // tile is read by neighbouring items
        if (w.smask) {
            const int64_t t = vt >> 1;           // the scoring pass's 256-row tile
            const int split = (int)(((t + 1) * ns - 1) / a.n_vtiles);
            if (!((sm[m] >> split) & 1u)) continue;
        }
        const int d = m ? a.dt : a.ds;
        const uint16_t *W = (const uint16_t *)(m ? a.wt : a.ws);
        const uint16_t *H = (const uint16_t *)(m ? a.ht : a.hs);
        const int r0 = vt * FL_VR + wid * 32;
        const int vrow = r0 + c32 < a.V ? r0 + c32 : a.V - 1;
        const uint16_t *wr = W + (int64_t)vrow * d + 32 * hf;
        const uint16_t *hr[2];
        for (int cb = 0; cb < 2; ++cb) {
            int q = qb * FL_QB + cb * 32 + c32;
            q = q < nq[m] ? q : nq[m] - 1;
            const int64_t g = a.rowmap[w.qj[m * w.cap + q]] & 0x7fffffffu;
            hr[cb] = H + g * d + 32 * hf;
        }
        fl_floatx16 acc[2];
        acc[0] = fl_floatx16{0.f};
        acc[1] = fl_floatx16{0.f};
        // Two register buffers: the loads of step i+1 are in flight under the MFMAs of
        // step i. Pairs of steps, then an odd last step; after the last pair X reloads
        // the last step (unused when the count is even).
        const int nst = d / 64;
        uint4 X[12], Y[12];
        fl_load(X, wr, hr, 0);
        int i = 0;
        for (; i + 1 < nst; i += 2) {
            fl_load(Y, wr, hr, (i + 1) * 64);
            __builtin_amdgcn_sched_barrier(0);
            fl_mma(X, acc);
            fl_load(X, wr, hr, (i + 2 < nst ? i + 2 : nst - 1) * 64);
            __builtin_amdgcn_sched_barrier(0);
            fl_mma(Y, acc);
        }
        if (i < nst) fl_mma(X, acc);
        // lane holds column c32 (a queued row) and rows 8 (r / 4) + 4 hf + r % 4
        for (int cb = 0; cb < 2; ++cb) {
            const int q = qb * FL_QB + cb * 32 + c32;
            if (q >= nq[m]) continue;
            const float thr = w.qthr[m * w.cap + q];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int v = r0 + 8 * (r >> 2) + 4 * hf + (r & 3);
                if (v < a.V && acc[cb][r] >= thr) {
                    const int n = atomicAdd(&w.qcnt[m * w.cap + q], 1);
                    if (n < w.ccap) w.cand[((int64_t)m * w.cap + q) * w.ccap + n] = v;
                }
            }
        }
    }
}

namespace {
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
}

size_t filter_queue_bytes(int64_t cap, int ccap) {
    const size_t c = (size_t)cap;
    return 3 * align256(c * 2 * 4) + align256(c * 2 * (size_t)ccap * 4) + align256(c * 2 * 4);
}

FilterQueue filter_queue_carve(void *base, int64_t cap, int ccap, int32_t *n, int32_t *nfb) {
    const size_t c = (size_t)cap;
    char *p = (char *)base;
    FilterQueue q;
    q.n = n;
    q.nfb = nfb;
    q.cap = (int)cap;
    q.ccap = ccap;
    q.qj = (int32_t *)p;     p += align256(c * 2 * 4);
    q.qthr = (float *)p;     p += align256(c * 2 * 4);
    q.qcnt = (int32_t *)p;   p += align256(c * 2 * 4);
    q.cand = (int32_t *)p;   p += align256(c * 2 * (size_t)ccap * 4);
    q.fb = (int32_t *)p;
    q.smask = nullptr;
    return q;
}

hipError_t launch_filter(const ScoreArgs &a, const FilterQueue &q, hipStream_t st) {
    // One work item per workgroup for up to 64 queued rows per model (the queue sizes
    // live on the device); larger queues stride.
    const int64_t n_vt = (a.V + FL_VR - 1) / FL_VR;
    const int64_t grid = 2 * n_vt < 65536 ? 2 * n_vt : 65536;
    filter_kernel<<<(unsigned)grid, 256, 0, st>>>(a, q);
    return hipGetLastError();
}

}  // namespace olive
