// The vocabulary filter of the exact decisions on the bf16 MFMA path: for every
// queued (row, model) pair, the indices of the vocabulary entries whose fp32 logit
// reaches the pair's threshold. The threshold is set so that every entry that can
// win the exact decision is among them; the exact values are formed afterwards.
#include <hip/hip_runtime.h>

#include "olive_internal.hpp"

namespace olive {

constexpr int FL_QB = 64;    // queued rows per work item (two 32-column MFMA blocks)
constexpr int FL_VR = 128;   // vocabulary rows per work item (4 wavefronts x 32)

typedef __bf16 fl_bf16x8 __attribute__((ext_vector_type(8)));
typedef float fl_floatx16 __attribute__((ext_vector_type(16)));

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
                const fl_bf16x8 av = __builtin_bit_cast(fl_bf16x8, A[s]);
                acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    av, __builtin_bit_cast(fl_bf16x8, B0[s]), acc[0], 0, 0, 0);
                acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    av, __builtin_bit_cast(fl_bf16x8, B1[s]), acc[1], 0, 0, 0);
            }
        }
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
    return q;
}

hipError_t launch_filter(const ScoreArgs &a, const FilterQueue &q, hipStream_t st) {
    filter_kernel<<<1024, 256, 0, st>>>(a, q);
    return hipGetLastError();
}

}  // namespace olive
