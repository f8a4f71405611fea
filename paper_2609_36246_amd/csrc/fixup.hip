// Exact re-decision of the greedy token for rows whose fp32 top-2 logit gap falls
// inside the fp32 error window.
//
// The scoring kernels take the argmax of fp32 logits. Where the best and second
// best are closer than the window, rounding could have swapped them relative to
// the exact values. For each such (row, model) this pass recomputes every logit of
// the row in fp32 and bounds its rounding error by
//   e_v = d * 2^-23 * ||h|| * ||w_v||  >=  d * 2^-23 * sum_k |h_k| |w_kv|
// (Cauchy-Schwarz; the weight-row norms are computed once at init). Entries that
// could still be the exact maximum,
//   z_v + e_v >= theta = (fp32 max of the scoring pass) - (its own bound),
// are evaluated in fp64 and the largest wins, lowest index first. The work is split
// over vocabulary chunks (phase 1) and merged per row in a fixed order (phase 2).
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

// 8 consecutive elements of a row as fp32 (one 16-byte load for bf16, two for fp32).
__device__ __forceinline__ void load8(const uint16_t *p, float (&x)[8]) {
    const uint4 q = *(const uint4 *)p;
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8(const float *p, float (&x)[8]) {
    const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// Squared L2 norm of every weight row (init only): one wavefront per row.
template <typename E>
__global__ void __launch_bounds__(256)
row_norm_kernel(const E *__restrict__ w, int64_t V, int d, float *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    for (int64_t v = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); v < V;
         v += (int64_t)gridDim.x * 4) {
        const E *r = w + v * d;
        double acc = 0.0;
        for (int k = lane; k < d; k += 64) {
            const double x = load_elem(r, k);
            acc += x * x;
        }
        for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) out[v] = (float)sqrt(acc) * 1.0001f;   // rounded up
    }
}

template <typename E>
__global__ void __launch_bounds__(FX_THREADS)
fixup_scan_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int cap, int n_chunks,
                  const float *__restrict__ wn_s, const float *__restrict__ wn_t,
                  FxResult *__restrict__ out) {
    extern __shared__ float hrow[];
    __shared__ double red_v[FX_THREADS];
    __shared__ int red_i[FX_THREADS];
    __shared__ float s_hn;
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
        if (mask & (1 << m)) {   // uniform over the workgroup
            const int d = m ? a.dt : a.ds;
            const E *h = (const E *)(m ? a.ht : a.hs) + (int64_t)(a.rowmap[j] & 0x7fffffffu) * d;
            const E *w = (const E *)(m ? a.wt : a.ws);
            const float *wn = m ? wn_t : wn_s;
            __syncthreads();
            for (int k = tid; k < d; k += FX_THREADS) hrow[k] = load_elem(h, k);
            __syncthreads();
            if (tid == 0) {
                double hh = 0.0;
                for (int k = 0; k < d; ++k) hh += (double)hrow[k] * hrow[k];
                s_hn = (float)sqrt(hh) * 1.0001f;
            }
            __syncthreads();
            const float ebound = (float)d * (1.0f / 8388608.0f) * s_hn;
            // 8 lanes per vocabulary row: each pass of a group reads 128 contiguous
            // bytes of its row (coalesced), 8 rows per wavefront at a time.
            const int lane = tid & 63, g8 = lane & 7;
            const int rows_per_pass = FX_THREADS / 8;
            const bool vec = (d & 63) == 0 && (((uintptr_t)w & 15) == 0);
            const int v_end = (c + 1) * FX_CHUNK < a.V ? (c + 1) * FX_CHUNK : a.V;
            for (int v0 = c * FX_CHUNK; v0 < v_end; v0 += rows_per_pass) {
                const int v = v0 + (tid >> 3);
                const bool ok = v < v_end;
                const E *wr = w + (int64_t)(ok ? v : v_end - 1) * d;
                float z = 0.f;
                if (vec) {
                    for (int k = g8 * 8; k < d; k += 64) {
                        float x[8];
                        load8(wr + k, x);
#pragma unroll
                        for (int q = 0; q < 8; ++q) z = fmaf(hrow[k + q], x[q], z);
                    }
                } else {
                    for (int k = g8; k < d; k += 8) z = fmaf(hrow[k], load_elem(wr, k), z);
                }
                z += __shfl_xor(z, 1);
                z += __shfl_xor(z, 2);
                z += __shfl_xor(z, 4);
                if (ok && g8 == 0 && z + ebound * wn[v] >= theta) {
                    double zd = 0.0;
                    for (int k = 0; k < d; ++k)
                        zd = fma((double)hrow[k], (double)load_elem(wr, k), zd);
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
        __syncthreads();
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

hipError_t launch_row_norms(const void *w, int64_t V, int d, bool bf16, float *out,
                            hipStream_t st) {
    const int64_t blocks = (V + 3) / 4 < 4096 ? (V + 3) / 4 : 4096;
    if (bf16)
        row_norm_kernel<uint16_t><<<(unsigned)blocks, 256, 0, st>>>((const uint16_t *)w, V, d, out);
    else
        row_norm_kernel<float><<<(unsigned)blocks, 256, 0, st>>>((const float *)w, V, d, out);
    return hipGetLastError();
}

hipError_t launch_fixup_impl(const ScoreArgs &a, bool bf16, const int32_t *flagged, int cap,
                             void *scratch, const float *wn_s, const float *wn_t, int32_t *am_s,
                             int32_t *am_t, hipStream_t st) {
    const int n_chunks = (a.V + FX_CHUNK - 1) / FX_CHUNK;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    const size_t lds = (size_t)dmax * sizeof(float);
    FxResult *res = (FxResult *)scratch;
    if (bf16)
        fixup_scan_kernel<uint16_t><<<1024, FX_THREADS, lds, st>>>(a, flagged, cap, n_chunks,
                                                                   wn_s, wn_t, res);
    else
        fixup_scan_kernel<float><<<1024, FX_THREADS, lds, st>>>(a, flagged, cap, n_chunks, wn_s,
                                                                wn_t, res);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    fixup_merge_kernel<<<64, 64, 0, st>>>(a, flagged, cap, n_chunks, res, am_s, am_t);
    return hipGetLastError();
}

int fixup_chunks(int64_t V) { return (int)((V + FX_CHUNK - 1) / FX_CHUNK); }
size_t fixup_result_bytes() { return sizeof(FxResult); }

}  // namespace olive
