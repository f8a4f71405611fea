// Exact-logit helpers of the greedy and top-K decisions on the bf16 MFMA path: a
// logit is formed exactly as bf16 products (exact in fp32) summed in fp64, and
// candidates rank by (value descending, vocabulary index ascending).
#pragma once

#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr double kTkEmpty = -0x1p1000;          // empty slot (below every finite logit)
constexpr int kTkNoIdx = 0x7fffffff;
constexpr int SCAN_THREADS = 256;               // exhaustive scan: 8 lanes per vocabulary row
constexpr int SCAN_GROUPS = SCAN_THREADS / 8;

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

// One workgroup: every exact logit of hidden row h against the vocabulary rows of W
// (8 lanes per row, fp64 sums), a top-16 per 8-lane group merged over the group.
// h_lds holds d bf16 of LDS (16-byte aligned); on return lanes 0..15 of wavefront 0
// hold the row's 16 best in rank order (out_v, out_i). Called by every thread.
__device__ __forceinline__ void scan_row_top16(const uint16_t *h, const uint16_t *W, int d,
                                               int V, uint16_t *h_lds,
                                               double (*red_v)[TOPK_K], int (*red_i)[TOPK_K],
                                               double &out_v, int &out_i) {
    const int tid = threadIdx.x, g8 = tid & 7, grp = tid >> 3;
    __syncthreads();
    for (int k = tid * 8; k < d; k += SCAN_THREADS * 8)
        *(uint4 *)(h_lds + k) = *(const uint4 *)(h + k);
    __syncthreads();
    double lv[TOPK_K];
    int li[TOPK_K];
#pragma unroll
    for (int t = 0; t < TOPK_K; ++t) { lv[t] = kTkEmpty; li[t] = kTkNoIdx; }
    for (int v0 = 0; v0 < V; v0 += SCAN_GROUPS) {
        const int v = v0 + grp;
        const bool ok = v < V;
        const uint16_t *wr = W + (int64_t)(ok ? v : V - 1) * d;
        double z = 0.0;
        for (int k = g8 * 8; k < d; k += 64)
            z = dot8_f64(*(const uint4 *)(h_lds + k), *(const uint4 *)(wr + k), z);
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
    out_v = kTkEmpty;
    out_i = kTkNoIdx;
    if (tid < 64) {   // merge the 32 group lists: lane l < 32 owns group l's list
        int ptr = 0;
        for (int r = 0; r < TOPK_K; ++r) {
            double hv = kTkEmpty;
            int hi = kTkNoIdx;
            if (tid < SCAN_GROUPS && ptr < TOPK_K) { hv = red_v[tid][ptr]; hi = red_i[tid][ptr]; }
            double bv = hv;
            int bi = hi;
            wave_best(bv, bi);
            if (tid < SCAN_GROUPS && ptr < TOPK_K && hv == bv && hi == bi) ++ptr;
            if (tid == r) { out_v = bv; out_i = bi; }
        }
    }
}

}  // namespace olive
