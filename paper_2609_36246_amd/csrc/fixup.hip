// Exact re-decision of the greedy token for rows whose fp32 top-2 logit gap falls
// inside the fp32 error window.
//
// The scoring kernels take the argmax of fp32 logits. Where the best and second
// best are closer than the window, rounding could have swapped them relative to
// the exact values. For each such (row, model) this pass recomputes every logit of
// the row in fp32 together with a rigorous rounding bound
//   e_v = d * 2^-23 * sum_k |h_k| |w_kv|,
// keeps the entries that could still be the exact maximum
//   z_v + e_v >= theta = (fp32 max of the scoring pass) - (its own bound),
// evaluates those in fp64 and picks the largest, lowest index first. The work is
// split over vocabulary chunks (phase 1) and merged per row in a fixed order
// (phase 2).
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int FX_CHUNK = 2048;
constexpr int FX_THREADS = 256;

struct FxResult {
    double val;
    int32_t idx;
    int32_t pad;
};

template <typename E>
__global__ void __launch_bounds__(FX_THREADS)
fixup_scan_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int cap, int n_chunks,
                  FxResult *__restrict__ out) {
    extern __shared__ float hrow[];
    __shared__ double red_v[FX_THREADS];
    __shared__ int red_i[FX_THREADS];
    const int nf_all = a.sched->n_flagged;
    const int nf = nf_all < cap ? nf_all : cap;
    const int64_t n_items = (int64_t)nf * n_chunks * 2;
    const int tid = threadIdx.x;
    for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int m = (int)(item & 1);
        const int64_t fc = item >> 1;
        const int f = (int)(fc % nf);
        const int c = (int)(fc / nf);
        const int32_t j = flagged[4 * f];
        const int32_t mask = flagged[4 * f + 1];
        const float theta = __int_as_float(flagged[4 * f + 2 + m]);
        double best_v = -__builtin_inf();
        int best_i = 0x7fffffff;
        if (mask & (1 << m)) {
            const int d = m ? a.dt : a.ds;
            const E *h = (const E *)(m ? a.ht : a.hs) + (int64_t)(a.rowmap[j] & 0x7fffffffu) * d;
            const E *w = (const E *)(m ? a.wt : a.ws);
            __syncthreads();
            for (int k = tid; k < d; k += FX_THREADS) hrow[k] = load_elem(h, k);
            __syncthreads();
            const float bound = (float)d * (1.0f / 8388608.0f);
            for (int v = c * FX_CHUNK + tid; v < (c + 1) * FX_CHUNK && v < a.V; v += FX_THREADS) {
                const E *wr = w + (int64_t)v * d;
                float z = 0.f, za = 0.f;
                for (int k = 0; k < d; ++k) {
                    float wv = load_elem(wr, k);
                    z = fmaf(hrow[k], wv, z);
                    za = fmaf(fabsf(hrow[k]), fabsf(wv), za);
                }
                if (z + bound * za >= theta) {
                    double zd = 0.0;
                    for (int k = 0; k < d; ++k) zd = fma((double)hrow[k], (double)load_elem(wr, k), zd);
                    if (zd > best_v || (zd == best_v && v < best_i)) { best_v = zd; best_i = v; }
                }
            }
        }
        red_v[tid] = best_v;
        red_i[tid] = best_i;
        __syncthreads();
        for (int off = FX_THREADS / 2; off > 0; off >>= 1) {
            if (tid < off) {
                double ov = red_v[tid + off];
                int oi = red_i[tid + off];
                if (ov > red_v[tid] || (ov == red_v[tid] && oi < red_i[tid])) {
                    red_v[tid] = ov;
                    red_i[tid] = oi;
                }
            }
            __syncthreads();
        }
        if (tid == 0) {
            out[item].val = red_v[0];
            out[item].idx = red_i[0];
        }
    }
}

__global__ void __launch_bounds__(64)
fixup_merge_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int cap, int n_chunks,
                   const FxResult *__restrict__ res, int32_t *__restrict__ am_s,
                   int32_t *__restrict__ am_t) {
    const int nf_all = a.sched->n_flagged;
    const int nf = nf_all < cap ? nf_all : cap;
    for (int f = blockIdx.x * 64 + threadIdx.x; f < nf; f += gridDim.x * 64) {
        const int32_t j = flagged[4 * f];
        const int32_t mask = flagged[4 * f + 1];
        const int64_t g = a.rowmap[j] & 0x7fffffffu;
        for (int m = 0; m < 2; ++m) {
            if (!(mask & (1 << m))) continue;
            double bv = -__builtin_inf();
            int bi = 0x7fffffff;
            for (int c = 0; c < n_chunks; ++c) {     // chunk order = vocabulary order
                const FxResult r = res[((int64_t)c * nf + f) * 2 + m];
                if (r.val > bv) { bv = r.val; bi = r.idx; }
            }
            if (bi != 0x7fffffff) {
                int32_t *am = m ? am_t : am_s;
                if (am) am[g] = bi;
            }
        }
    }
}

hipError_t launch_fixup_impl(const ScoreArgs &a, bool bf16, const int32_t *flagged, int cap,
                             void *scratch, int32_t *am_s, int32_t *am_t, hipStream_t st) {
    const int n_chunks = (a.V + FX_CHUNK - 1) / FX_CHUNK;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    const size_t lds = (size_t)dmax * sizeof(float);
    FxResult *res = (FxResult *)scratch;
    if (bf16)
        fixup_scan_kernel<uint16_t><<<1024, FX_THREADS, lds, st>>>(a, flagged, cap, n_chunks, res);
    else
        fixup_scan_kernel<float><<<1024, FX_THREADS, lds, st>>>(a, flagged, cap, n_chunks, res);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    fixup_merge_kernel<<<64, 64, 0, st>>>(a, flagged, cap, n_chunks, res, am_s, am_t);
    return hipGetLastError();
}

int fixup_chunks(int64_t V) { return (int)((V + FX_CHUNK - 1) / FX_CHUNK); }
size_t fixup_result_bytes() { return sizeof(FxResult); }

}  // namespace olive
