// Exact re-decision of the greedy token for rows whose fp32 top-2 logit gap falls
// inside the fp32 error window.
//
// The scoring kernels take the argmax of fp32 logits. Where the best and second
// best are closer than the window, rounding could have swapped them relative to
// the exact values. For each such (row, model) this pass recomputes every logit of
// the row in fp32 and bounds its rounding error by
//   e_v = d * 2^-22 * ||h|| * ||w_v||  >=  2 * d * 2^-23 * sum_k |h_k| |w_kv|
// (Cauchy-Schwarz, with a factor 2 over the bound of d fp32 roundings so that the
// packed dot instruction's internal rounding is covered; the weight-row norms are
// computed once at init). Entries that
// could still be the exact maximum,
//   z_v + e_v >= theta = (fp32 max of the scoring pass) - (its own bound),
// are evaluated in fp64 and the largest wins, lowest index first.
//
// Work items are (batch of up to FB flagged rows, vocabulary chunk, model): the
// batch's hidden rows are staged in LDS and every weight row of the chunk is read
// once for all of them, so W streams from HBM once per batch rather than once per
// flagged row. Per-chunk winners are merged per row in a fixed order (phase 2).
// One launch pair covers a window of the flagged list (entries [f_base, f_base +
// cap)); the host runs windows until they cover every row a call can flag, and a
// window past the list's end exits at once.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int FX_CHUNK = 1024;          // vocabulary rows per work item
constexpr int FX_THREADS = 256;
constexpr int FX_GROUPS = FX_THREADS / 8;   // 8 lanes per weight row
constexpr int FX_MAXB = 8;              // flagged rows per pass over W
constexpr int FX_LDS = 65536;           // bytes of staged hidden rows per work item

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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + a.lo * b.lo + a.hi * b.hi for two packed bf16 pairs (v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2bf(uint32_t a, uint32_t b, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), acc, false);
}

// z[i] += sum over 8 elements at k of h_i[k..k+8) * w[k..k+8), for FB staged rows.
template <int FB>
__device__ __forceinline__ void dot8(const uint16_t *hrows, int d, int k, const uint4 &wq,
                                     float (&z)[FB]) {
#pragma unroll
    for (int i = 0; i < FB; ++i) {
        const uint4 hq = *(const uint4 *)(hrows + i * d + k);
        z[i] = dot2bf(hq.x, wq.x, z[i]);
        z[i] = dot2bf(hq.y, wq.y, z[i]);
        z[i] = dot2bf(hq.z, wq.z, z[i]);
        z[i] = dot2bf(hq.w, wq.w, z[i]);
    }
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

template <typename E, int FB>
__global__ void __launch_bounds__(FX_THREADS)
fixup_scan_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int f_base, int cap,
                  int n_chunks, const float *__restrict__ wn_s, const float *__restrict__ wn_t,
                  FxResult *__restrict__ out) {
    extern __shared__ __attribute__((aligned(16))) char fx_smem[];   // [FB][d] of E
    __shared__ float s_eb[FB], s_theta[FB];
    __shared__ double red_v[FX_GROUPS][FB];
    __shared__ int red_i[FX_GROUPS][FB];
    E *hrows = (E *)fx_smem;
    // this window's flagged rows: entries [f_base, f_base + cap) of the list
    const int nf_all = a.sched->n_flagged - f_base;
    const int nf = nf_all < 0 ? 0 : (nf_all < cap ? nf_all : cap);
    flagged += 4 * (int64_t)f_base;
    const int n_batches = (nf + FB - 1) / FB;
    const int64_t n_items = (int64_t)n_batches * n_chunks * 2;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g8 = lane & 7;
    for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int m = (int)(item & 1);
        const int64_t rest = item >> 1;
        const int c = (int)(rest % n_chunks);
        const int f0 = (int)(rest / n_chunks) * FB;
        const int d = m ? a.dt : a.ds;
        const E *H = (const E *)(m ? a.ht : a.hs);
        const E *W = (const E *)(m ? a.wt : a.ws);
        const float *wn = m ? wn_t : wn_s;
        // Stage the batch's hidden rows (zeros for rows absent or not flagged for m)
        // and form each row's error-bound factor d * 2^-23 * ||h|| and its theta.
        __syncthreads();
        for (int i = wave; i < FB; i += FX_THREADS / 64) {
            const int f = f0 + i;
            const bool use = f < nf && (flagged[4 * (f < nf ? f : 0) + 1] & (1 << m));
            const E *h = H + (use ? (int64_t)(a.rowmap[flagged[4 * f]] & 0x7fffffffu) * d : 0);
            double hh = 0.0;
            bool staged = false;
            if constexpr (sizeof(E) == 2) {
                if ((d & 7) == 0 && ((uintptr_t)h & 15) == 0) {
                staged = true;
                for (int k = lane * 8; k < d; k += 512) {     // 16-byte pieces
                    const uint4 q = use ? *(const uint4 *)(h + k) : make_uint4(0, 0, 0, 0);
                    *(uint4 *)(hrows + i * d + k) = q;
                    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double lo = __uint_as_float(w[e] << 16);
                        const double hi = __uint_as_float(w[e] & 0xffff0000u);
                        hh += lo * lo + hi * hi;
                    }
                }
                }
            }
            if (!staged) {
                for (int k = lane; k < d; k += 64) {
                    const E x = use ? h[k] : (E)0;
                    hrows[i * d + k] = x;
                    const double xd = load_elem(&x, 0);
                    hh += xd * xd;
                }
            }
            for (int off = 32; off > 0; off >>= 1) hh += __shfl_xor(hh, off);
            if (lane == 0) {
                s_eb[i] = (float)d * (1.0f / 4194304.0f) * ((float)sqrt(hh) * 1.0001f);
                s_theta[i] = use ? __int_as_float(flagged[4 * f + 2 + m]) : __builtin_inff();
            }
        }
        __syncthreads();
        float eb[FB], th[FB];
        double best_v[FB];
        int best_i[FB];
#pragma unroll
        for (int i = 0; i < FB; ++i) {
            eb[i] = s_eb[i];
            th[i] = s_theta[i];
            best_v[i] = -__builtin_inf();
            best_i[i] = 0x7fffffff;
        }
        // 8 lanes per weight row: each pass of a group reads 128 contiguous bytes of its
        // row (bf16), so a wavefront reads 8 rows at a time, coalesced.
        const bool vec = (d & 63) == 0 && (((uintptr_t)W & 15) == 0);
        const int v_end = (c + 1) * FX_CHUNK < a.V ? (c + 1) * FX_CHUNK : a.V;
        for (int v0 = c * FX_CHUNK; v0 < v_end; v0 += FX_GROUPS) {
            const int v = v0 + (tid >> 3);
            const bool ok = v < v_end;
            const E *wr = W + (int64_t)(ok ? v : v_end - 1) * d;
            float z[FB];
#pragma unroll
            for (int i = 0; i < FB; ++i) z[i] = 0.f;
            if constexpr (sizeof(E) == 2) {
                if (vec) {
                    // 8 independent 16-byte loads in flight per lane (latency, not the
                    // arithmetic, bounds a row scan), then the packed dot products.
                    int k = g8 * 8;
                    for (; k + 7 * 64 < d; k += 8 * 64) {
                        uint4 wq[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) wq[j] = *(const uint4 *)(wr + k + j * 64);
#pragma unroll
                        for (int j = 0; j < 8; ++j) dot8<FB>(hrows, d, k + j * 64, wq[j], z);
                    }
                    for (; k < d; k += 64) dot8<FB>(hrows, d, k, *(const uint4 *)(wr + k), z);
                } else {
                    for (int k = g8; k < d; k += 8) {
                        const float x = load_elem(wr, k);
#pragma unroll
                        for (int i = 0; i < FB; ++i)
                            z[i] = fmaf(load_elem(hrows + i * d, k), x, z[i]);
                    }
                }
            } else if (vec) {
                for (int k = g8 * 8; k < d; k += 64) {
                    float x[8];
                    load8(wr + k, x);
#pragma unroll
                    for (int i = 0; i < FB; ++i) {
                        float hv[8];
                        load8(hrows + i * d + k, hv);
#pragma unroll
                        for (int q = 0; q < 8; ++q) z[i] = fmaf(hv[q], x[q], z[i]);
                    }
                }
            } else {
                for (int k = g8; k < d; k += 8) {
                    const float x = load_elem(wr, k);
#pragma unroll
                    for (int i = 0; i < FB; ++i) z[i] = fmaf(load_elem(hrows + i * d, k), x, z[i]);
                }
            }
            const float wnv = wn[ok ? v : v_end - 1];
#pragma unroll
            for (int i = 0; i < FB; ++i) {
                z[i] += __shfl_xor(z[i], 1);
                z[i] += __shfl_xor(z[i], 2);
                z[i] += __shfl_xor(z[i], 4);
                // Same decision on the 8 lanes of the group; they then form the fp64
                // logit together (fixed split and reduction order).
                if (ok && z[i] + eb[i] * wnv >= th[i]) {
                    double zd = 0.0;
                    for (int k = g8; k < d; k += 8)
                        zd = fma((double)load_elem(hrows + i * d, k), (double)load_elem(wr, k), zd);
                    zd += __shfl_xor(zd, 1, 8);
                    zd += __shfl_xor(zd, 2, 8);
                    zd += __shfl_xor(zd, 4, 8);
                    if (zd > best_v[i] || (zd == best_v[i] && v < best_i[i])) {
                        best_v[i] = zd;
                        best_i[i] = v;
                    }
                }
            }
        }
        if (g8 == 0) {
#pragma unroll
            for (int i = 0; i < FB; ++i) {
                red_v[tid >> 3][i] = best_v[i];
                red_i[tid >> 3][i] = best_i[i];
            }
        }
        __syncthreads();
        if (tid < FB && f0 + tid < nf) {
            double bv = -__builtin_inf();
            int bi = 0x7fffffff;
            for (int g = 0; g < FX_GROUPS; ++g) {
                const double ov = red_v[g][tid];
                const int oi = red_i[g][tid];
                if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
            }
            FxResult r;
            r.val = bv;
            r.idx = bi;
            r.pad = 0;
            out[((int64_t)c * nf + f0 + tid) * 2 + m] = r;
        }
    }
}

__global__ void __launch_bounds__(64)
fixup_merge_kernel(ScoreArgs a, const int32_t *__restrict__ flagged, int f_base, int cap,
                   int n_chunks, const FxResult *__restrict__ res, int32_t *__restrict__ am_s,
                   int32_t *__restrict__ am_t) {
    const int nf_all = a.sched->n_flagged - f_base;
    const int nf = nf_all < 0 ? 0 : (nf_all < cap ? nf_all : cap);
    flagged += 4 * (int64_t)f_base;
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

// out[0] = (1 + 2^-10) max_v wn[v]: the largest weight-row norm with the margin the
// rounding bounds use (one workgroup; max is exact in any order).
__global__ void __launch_bounds__(1024)
max_norm_kernel(const float *__restrict__ wn, int64_t V, float *__restrict__ out) {
    __shared__ float red[1024];
    float m = 0.f;
    for (int64_t v = threadIdx.x; v < V; v += 1024) m = fmaxf(m, wn[v]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int off = 512; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + off]);
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = red[0] * (1.0f + 0x1p-10f);
}

hipError_t launch_max_norm(const float *wn, int64_t V, float *out, hipStream_t st) {
    max_norm_kernel<<<1, 1024, 0, st>>>(wn, V, out);
    return hipGetLastError();
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

template <typename E, int FB>
static void launch_scan(const ScoreArgs &a, const int32_t *flagged, int f_base, int cap,
                        int n_chunks, size_t lds, const float *wn_s, const float *wn_t,
                        FxResult *res, hipStream_t st) {
    fixup_scan_kernel<E, FB><<<1024, FX_THREADS, lds, st>>>(a, flagged, f_base, cap, n_chunks,
                                                             wn_s, wn_t, res);
}

template <typename E>
static void launch_scan_fb(int fb, const ScoreArgs &a, const int32_t *flagged, int f_base,
                           int cap, int n_chunks, size_t lds, const float *wn_s,
                           const float *wn_t, FxResult *res, hipStream_t st) {
#define OLIVE_SCAN(FB_) launch_scan<E, FB_>(a, flagged, f_base, cap, n_chunks, lds, wn_s, wn_t, res, st)
    if (fb >= 8) OLIVE_SCAN(8);
    else if (fb >= 4) OLIVE_SCAN(4);
    else if (fb >= 2) OLIVE_SCAN(2);
    else OLIVE_SCAN(1);
#undef OLIVE_SCAN
}

hipError_t launch_fixup_impl(const ScoreArgs &a, bool bf16, const int32_t *flagged, int f_base,
                             int cap, void *scratch, const float *wn_s, const float *wn_t,
                             int32_t *am_s, int32_t *am_t, hipStream_t st) {
    const int n_chunks = (a.V + FX_CHUNK - 1) / FX_CHUNK;
    const int dmax = a.ds > a.dt ? a.ds : a.dt;
    const int esz = bf16 ? 2 : 4;
    // Rows per batch: as many hidden rows as fit the staging budget, a power of two.
    int fb = FX_LDS / (dmax * esz);
    fb = fb > FX_MAXB ? FX_MAXB : (fb < 1 ? 1 : fb);
    fb = fb >= 8 ? 8 : (fb >= 4 ? 4 : (fb >= 2 ? 2 : 1));
    const size_t lds = (size_t)fb * dmax * esz;
    FxResult *res = (FxResult *)scratch;
    if (bf16)
        launch_scan_fb<uint16_t>(fb, a, flagged, f_base, cap, n_chunks, lds, wn_s, wn_t, res, st);
    else
        launch_scan_fb<float>(fb, a, flagged, f_base, cap, n_chunks, lds, wn_s, wn_t, res, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    fixup_merge_kernel<<<64, 64, 0, st>>>(a, flagged, f_base, cap, n_chunks, res, am_s, am_t);
    return hipGetLastError();
}

int fixup_chunks(int64_t V) { return (int)((V + FX_CHUNK - 1) / FX_CHUNK); }
size_t fixup_result_bytes() { return sizeof(FxResult); }

}  // namespace olive
