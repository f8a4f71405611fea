// The per-lane fold of the bf16 scoring kernels: running statistics of one position
// column of one model over 32-row blocks of fp32 logits (max, second max, lowest
// argmax, rescaled exp2 sum, and the exp-weighted logit difference to the other model
// that gives the KL sums), and the merge of two such partial records.
#pragma once

#include <hip/hip_runtime.h>

#include "olive_device.hpp"

namespace olive {

// Logit of vocabulary rows outside the tile range: -2^99. A power of two, so that
// kMasked * c is exact and a block whose running max is kMasked folds to exp2(0) = 1
// rather than to the rounding residual of the product; z + kMasked rounds back to
// exactly kMasked for any |z| < 2^74, in both models (their difference is 0).
constexpr float kMasked = -0x1p99f;

// max(a, b) for non-NaN operands as one v_med3_f32 (no NaN canonicalisation).
__device__ __forceinline__ float max2(float a, float b) {
    return __builtin_amdgcn_fmed3f(a, b, __builtin_inff());
}

struct Run {                // running statistics of one position column
    float best, sec, z;
    int idx;
};

// Fold one 32-row block (16 values per lane: rows 8*(r/4) + 4*h + r%4 of the block,
// one column) into a model's running statistics. With DIFF, also the sum of the
// block's exp weights times the logit difference to the other model (z - o with
// equal scales, s_self z - s_other o otherwise) into Aacc: the teacher's forms the
// forward KL, the student's the reverse one. vcode0 is the vocabulary index of the
// lane's first row of the block.
template <bool DIFF, bool SAME>
__device__ __forceinline__ void fold_block(const float (&z)[16], Run &R, float &Aacc,
                                           const float (&o)[16], float c, float s_self,
                                           float s_other, int vcode0) {
    float tm = R.best, ts = R.sec;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        ts = __builtin_amdgcn_fmed3f(z[r], tm, ts);
        tm = max2(tm, z[r]);
    }
    // Branch-free: lowest row of this block equal to the new max (used only when the
    // block raised the max), and the rescale of the running sums (1 when not).
    int code = 0;
#pragma unroll
    for (int r = 15; r >= 0; --r) code = (z[r] == tm) ? 8 * (r >> 2) + (r & 3) : code;
    const bool up = tm > R.best;
    const float resc = fast_exp2((R.best - tm) * c);
    R.z *= resc;
    if (DIFF) Aacc *= resc;
    R.idx = up ? vcode0 + code : R.idx;
    R.best = tm;
    R.sec = ts;
    const float mneg = -tm * c;
    float zsum = 0.f, asum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(fmaf(z[r], c, mneg));
        zsum += e;
        if (DIFF) {
            float dlt;
            {
#pragma clang fp contract(off)
                dlt = SAME ? (z[r] - o[r]) : (s_self * z[r] - s_other * o[r]);
            }
            asum = fmaf(e, dlt, asum);
        }
    }
    R.z += zsum;
    if (DIFF) Aacc += asum;
}

// Merge the partial record y (with its difference sum ya) into x (xa).
__device__ __forceinline__ void merge_run(Run &x, float &xa, const Run &y, float ya, float c) {
    Stat a{x.best, x.sec, x.idx, x.z}, b{y.best, y.sec, y.idx, y.z};
    stat_merge(a, xa, b, ya, c);
    x.best = a.best; x.sec = a.sec; x.idx = a.idx; x.z = a.z;
}

}  // namespace olive
