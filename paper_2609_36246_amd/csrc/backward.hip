// Data movement of the backward pass: the scored hidden rows of a chunk gathered
// and transposed into the K-contiguous operand of the dL/dW product, the student's
// weights transposed into K-blocked panels for the dL/dh product, and a zero fill.
#include <hip/hip_runtime.h>

#include "olive_internal.hpp"

namespace olive {

// out[k][t] = h[row(c0 + t)][k] for t < the chunk's scored rows, 0 for the rest of
// the pitch. One 64 (rows) x 64 (k) tile per workgroup, transposed through LDS.
__global__ void __launch_bounds__(256)
gather_t_kernel(const uint16_t *__restrict__ h, int d, const uint32_t *__restrict__ rowmap,
                const Sched *__restrict__ sched, int c0, int chunk, int pitch,
                uint16_t *__restrict__ out) {
    __shared__ uint16_t tile[64][64 + 8];
    const int t_all = sched->t_valid - c0;
    const int t_rows = t_all < 0 ? 0 : (t_all < chunk ? t_all : chunk);
    const int t0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
    const int tid = threadIdx.x;
    {
        const int tl = tid >> 2, kl = (tid & 3) * 16;
        const int t = t0 + tl;
        uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
        if (t < t_rows) {
            const int64_t g = rowmap[c0 + t] & 0x7fffffffu;
            const uint4 *src = (const uint4 *)(h + g * d + k0 + kl);
            a = src[0];
            b = src[1];
        }
        const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            tile[tl][kl + 2 * e] = (uint16_t)(w[e] & 0xffffu);
            tile[tl][kl + 2 * e + 1] = (uint16_t)(w[e] >> 16);
        }
    }
    __syncthreads();
    {
        const int kl = tid >> 2, tl = (tid & 3) * 16;
        uint32_t w[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
            w[e] = (uint32_t)tile[tl + 2 * e][kl] | ((uint32_t)tile[tl + 2 * e + 1][kl] << 16);
        uint4 *dst = (uint4 *)(out + (int64_t)(k0 + kl) * pitch + t0 + tl);
        dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
        dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
}

// Zeros in rows [rows, rows rounded up to 64) of every panel of dz_t ([np][chunk][64]
// bf16), rows = the chunk's scored rows (on the device): the K padding the dL/dW product
// reads in its last K step. One 16-byte piece per lane.
__global__ void __launch_bounds__(256)
zero_tail_kernel(uint16_t *__restrict__ dzt, int np, int chunk, const Sched *__restrict__ sched,
                 int c0) {
    const int t_all = sched->t_valid - c0;
    const int rows = t_all < 0 ? 0 : (t_all < chunk ? t_all : chunk);
    const int pad = ((rows + 63) / 64) * 64 - rows;   // rows to clear per panel
    const int64_t n = (int64_t)np * pad * 8;           // 16-byte pieces
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * 256) {
        const int64_t p = i / (pad * 8);
        const int r = rows + (int)((i / 8) % pad), c = (int)(i % 8);
        *(uint4 *)(dzt + ((p * chunk + r) * 64 + c * 8)) = make_uint4(0, 0, 0, 0);
    }
}

hipError_t launch_zero_tail(uint16_t *dzt, int64_t vp, int chunk, const Sched *sched, int c0,
                            hipStream_t st) {
    const int np = (int)(vp / 64);
    const int64_t most = (int64_t)np * 63 * 8;         // pieces for the widest padding
    const int64_t blocks = (most + 255) / 256 < 2048 ? (most + 255) / 256 : 2048;
    zero_tail_kernel<<<(unsigned)blocks, 256, 0, st>>>(dzt, np, chunk, sched, c0);
    return hipGetLastError();
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float4 *__restrict__ p, int64_t n4) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4;
         i += (int64_t)gridDim.x * 256)
        p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

// out[p][k][j] = W[64 p + j][k] (0 for rows past V): W^T [d][V] cut into panels of 64
// vocabulary columns, [vp/64][d][64], so that one K step of the dL/dh product reads 256
// contiguous 128-byte rows. One 64 (rows) x 64 (k) tile per workgroup through LDS.
__global__ void __launch_bounds__(256)
panel_t_kernel(const uint16_t *__restrict__ w, int64_t V, int d, uint16_t *__restrict__ out) {
    __shared__ uint16_t tile[64][64 + 2];
    const int64_t v0 = (int64_t)blockIdx.x * 64;
    const int k0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const int64_t v = v0 + r;
        tile[r][tx] = v < V ? w[v * d + k0 + tx] : (uint16_t)0;
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4)
        out[((int64_t)blockIdx.x * d + k0 + r) * 64 + tx] = tile[tx][r];
}

hipError_t launch_panel_t(const void *w, int64_t V, int d, int64_t vp, void *out,
                          hipStream_t st) {
    // d and vp are multiples of 64 (the MFMA path's widths, the padded vocabulary)
    if (d % 64 != 0 || vp % 64 != 0 || vp < V) return hipErrorInvalidValue;
    dim3 grid((unsigned)(vp / 64), (unsigned)(d / 64));
    panel_t_kernel<<<grid, 256, 0, st>>>((const uint16_t *)w, V, d, (uint16_t *)out);
    return hipGetLastError();
}

hipError_t launch_gather_t(const void *h, int d, const uint32_t *rowmap, const Sched *sched,
                           int c0, int chunk, int pitch, uint16_t *out, hipStream_t st) {
    // d and pitch are multiples of 64 (the MFMA path's widths, the chunk pitch)
    dim3 grid((unsigned)(pitch / 64), (unsigned)(d / 64));
    gather_t_kernel<<<grid, 256, 0, st>>>((const uint16_t *)h, d, rowmap, sched, c0, chunk,
                                          pitch, out);
    return hipGetLastError();
}

hipError_t launch_fill(float *p, int64_t n, hipStream_t st) {
    // n is a multiple of 4 (whole rows of a width that is a multiple of 64)
    const int64_t n4 = n / 4;
    const int64_t blocks = (n4 + 255) / 256 < 4096 ? (n4 + 255) / 256 : 4096;
    if (blocks <= 0) return hipSuccess;
    fill_zero_kernel<<<(unsigned)blocks, 256, 0, st>>>((float4 *)p, n4);
    return hipGetLastError();
}

}  // namespace olive
