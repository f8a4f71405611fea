// bf16 GEMM for gfx950 with fp32 accumulation and output:
//   C (+)= alpha * A * B^T,   A [M][K], B [N][K] bf16, rows K-contiguous,
// the two GEMMs of the backward pass (dL/dh and dL/dW from the logit gradient).
//
// The operand pipeline is the scoring kernel's: a workgroup (4 wavefronts, 2 x 2)
// owns a 256 x 128 output tile, K advances 64 elements per step, each step's A tile
// (256 rows x 128 B) and B tile (128 rows x 128 B) land in a 3-stage LDS ring through
// global->LDS DMAs issued two steps ahead, and v_mfma_f32_32x32x16_bf16 accumulates
// 128 x 64 per wavefront in AGPRs. Here every lane holds its own row offsets (from the
// tile's first rows) for both operands, so ragged M and N read clamped rows (whose
// results are dropped).
//
// N and K may be read on the device (the scored-row count of a call is known only
// there); the grid is persistent and every workgroup derives the tile count itself.
// With ksplit = 2 each tile's K range is halved over two work units that add into C
// with atomics. C must hold zeros beforehand: then the result is deterministic, since
// 0 + a + b and 0 + b + a round to the same value (the first addition is exact). With
// any other start value c the two orders (c + a) + b and (c + b) + a may differ.
#include <hip/hip_runtime.h>

#include "mfma_pipe.hpp"
#include "olive_internal.hpp"

namespace olive {

namespace {

struct GLane {
    int lane, wid, wv, wt, h, l32;
    int ldsoff[4];
    // K-major A (transposed panels): per lane, the byte offsets of its transpose reads
    // within a stage, for the read of K rows 0..3 or 4..7 of its half (r) and for even or
    // odd 32-row blocks (parity); the block pair and the sub-step add constants
    uint32_t troff[2][2];
    // the tile's first A and B rows (wave-uniform) and, per DMA, the lane's row chunk
    // as a 32-bit offset from them: the K offset is added to the bases in scalar
    // registers, the lane part inside the load
    const char *abase, *bbase;
    int64_t ak, bk;          // bytes from one K step of 64 elements to the next
    uint32_t aoff[W_DMA];    // 8 A DMAs
    uint32_t boff[H_DMA];    // 4 B DMAs
};

struct GFrag {
    bf16x8 A[4], B[2];
};

// DMA q of K step kk (q < 8: A rows 8q .. 8q+7 of the wave's slice; else B DMA q-8)
// into the stage whose wave parts start at la (A) and lb (B).
template <int Q>
__device__ __forceinline__ void g_dma(const GLane &L, uint32_t la, uint32_t lb, int kk) {
    if constexpr (Q < W_DMA)
        dma16_sv<Q * 1024>(L.abase + kk * L.ak, L.aoff[Q], la);
    else
        dma16_sv<(Q - W_DMA) * 1024>(L.bbase + kk * L.bk, L.boff[Q - W_DMA], lb);
}

template <int QB, int QE>
__device__ __forceinline__ void g_dmas(const GLane &L, uint32_t la, uint32_t lb, int kk) {
    if constexpr (QB < QE) {
        g_dma<QB>(L, la, lb, kk);
        g_dmas<QB + 1, QE>(L, la, lb, kk);
    }
}

__device__ __forceinline__ void g_issue(const GLane &L, int st, int kk) {
    const uint32_t base = ring_addr() + (uint32_t)st * STAGE_BYTES;
    const uint32_t la = base + (uint32_t)L.wid * (W_DMA * 1024u);
    const uint32_t lb = base + WT_BYTES + (uint32_t)L.wid * (H_DMA * 1024u);
    g_dmas<0, DMA_PER_STEP>(L, la, lb, kk);
}

// Slot swizzle of the K-major A stage (transpose reads): 16-byte chunk c of row R in slot
// c ^ (4 ((R >> 1) & 1)). A pair of 16-lane groups reads chunks 4 par .. 4 par + 3 of
// rows 4q .. 4q+3; even rows fill banks 0-31 and odd rows banks 32-63, so rows 4q and
// 4q+2 (and 4q+1, 4q+3) must take opposite halves of the 8 slots. With the operand
// stages' swizzle (R >> 1) & 7 they took the same half: 2.3e8 bank-conflict cycles per
// dL/dW product on long_rollout, none with this one (3.55 -> 3.45 ms).
__device__ __forceinline__ int swz_tr(int r) { return ((r >> 1) & 1) << 2; }

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// One ds_read_b64_tr_b16 at byte offset off of the ring. In each group of 16 lanes, lane
// j supplies 4 consecutive 16-bit values M[j][0..3] (8 bytes at its address) and lane i
// receives M[i/4][i%4], M[i/4 + 4][i%4], M[i/4 + 8][i%4], M[i/4 + 12][i%4].
__device__ __forceinline__ i16x4 tr_read(uint32_t off) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4 *)((__attribute__((address_space(3))) char *)(lds_void *)g_ring + off));
}

template <int SUB, bool ATR>
__device__ __forceinline__ void g_read(const GLane &L, int st, GFrag &F) {
    const char *stage = g_ring + st * STAGE_BYTES;
    const char *bb = stage + WT_BYTES + L.wt * 64 * ROWB + L.ldsoff[SUB];
    if constexpr (ATR) {
        // 32-row block vb of the wave = panel 2 wv + vb / 2, columns 32 (vb % 2) ..: two
        // transpose reads give the lane K rows 16 SUB + 8 h + 0..3 and + 4..7 of its row
        const uint32_t sb = (uint32_t)st * STAGE_BYTES;
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) {
            constexpr int kq = SUB * 16 * ROWB;
            const uint32_t bo = sb + (uint32_t)((vb >> 1) * 64 * ROWB + kq);
            const i16x4 lo = tr_read(L.troff[0][vb & 1] + bo);
            const i16x4 hi = tr_read(L.troff[1][vb & 1] + bo);
            const i16x4 both[2] = {lo, hi};
            F.A[vb] = __builtin_bit_cast(bf16x8, both);
        }
    } else {
        const char *ab = stage + L.wv * 128 * ROWB + L.ldsoff[SUB];
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) F.A[vb] = *(const bf16x8 *)(ab + vb * 32 * ROWB);
    }
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) F.B[cb] = *(const bf16x8 *)(bb + cb * 32 * ROWB);
}

__device__ __forceinline__ void g_mma(const GFrag &F, floatx16 (&acc)[4][2]) {
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            __builtin_amdgcn_sched_barrier(0);
            acc[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.A[vb], F.B[cb], acc[vb][cb],
                                                                  0, 0, 0);
        }
    __builtin_amdgcn_sched_barrier(0);
}

// The 8 MFMAs of one sub-step with the DMAs of one third of the next refill
// interleaved (4 of the step's 12).
template <int Q0>
__device__ __forceinline__ void g_mma_issue(const GFrag &F, floatx16 (&acc)[4][2],
                                            const GLane &L, uint32_t la, uint32_t lb, int kk) {
#define OLIVE_GMI(J_)                                                                     \
    __builtin_amdgcn_sched_barrier(0);                                                    \
    acc[(J_) >> 1][(J_) & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                   \
        F.A[(J_) >> 1], F.B[(J_) & 1], acc[(J_) >> 1][(J_) & 1], 0, 0, 0);                \
    __builtin_amdgcn_sched_barrier(0);                                                    \
    if constexpr (((J_) & 1) == 1) g_dma<Q0 + ((J_) >> 1)>(L, la, lb, kk);
    OLIVE_GMI(0)
    OLIVE_GMI(1)
    OLIVE_GMI(2)
    OLIVE_GMI(3)
    OLIVE_GMI(4)
    OLIVE_GMI(5)
    OLIVE_GMI(6)
    OLIVE_GMI(7)
#undef OLIVE_GMI
    __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ void g_arrive() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_imm(DMA_PER_STEP));
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
}

// One step in stage st: barrier, refill the stage of step n-1 with step pk (n+2,
// saturated at the last step), run the four k16 sub-steps; the last one's fragments
// stay pending in P.
template <bool PEND, bool ATR>
__device__ __forceinline__ void g_step(const GLane &L, int st, int pk, floatx16 (&acc)[4][2],
                                       GFrag &P) {
    const int pv = st == 0 ? NST - 1 : st - 1;
    g_arrive();
    const uint32_t base = ring_addr() + (uint32_t)pv * STAGE_BYTES;
    const uint32_t la = base + (uint32_t)L.wid * (W_DMA * 1024u);
    const uint32_t lb = base + WT_BYTES + (uint32_t)L.wid * (H_DMA * 1024u);
    const int off = pk;   // K step of the refill
    GFrag F0, F1, F2;
    g_read<0, ATR>(L, st, F0);
    __builtin_amdgcn_sched_barrier(0);
    if (PEND) {
        g_mma_issue<0>(P, acc, L, la, lb, off);
        g_read<1, ATR>(L, st, F1);
        __builtin_amdgcn_sched_barrier(0);
        g_mma_issue<4>(F0, acc, L, la, lb, off);
        g_read<2, ATR>(L, st, F2);
        __builtin_amdgcn_sched_barrier(0);
        g_mma_issue<8>(F1, acc, L, la, lb, off);
        g_read<3, ATR>(L, st, P);
        __builtin_amdgcn_sched_barrier(0);
        g_mma(F2, acc);
    } else {
        g_read<1, ATR>(L, st, F1);
        __builtin_amdgcn_sched_barrier(0);
        g_mma_issue<0>(F0, acc, L, la, lb, off);
        g_read<2, ATR>(L, st, F2);
        __builtin_amdgcn_sched_barrier(0);
        g_mma_issue<4>(F1, acc, L, la, lb, off);
        g_read<3, ATR>(L, st, P);
        __builtin_amdgcn_sched_barrier(0);
        g_mma_issue<8>(F2, acc, L, la, lb, off);
    }
}

// Tile (mi, ni) of the q-th tile in blocks of GM x GN tiles (bands of GM row tiles, each
// cut into blocks of GN column tiles; the last band and block may be narrower), n
// fastest inside a block. The 32 units one XCD runs together then share 4 A strips and
// 8 B strips: 4 x 32 + 8 x 16 KB fetched per step, the fewest for a 256 x 128 tile.
constexpr int GM = 4, GN = 8;
__device__ __forceinline__ void tile_of(int64_t q, int tm, int tn, int &mi, int &ni) {
    const int64_t per_band = (int64_t)GM * tn;
    const int band = (int)(q / per_band);
    const int hm = tm - GM * band < GM ? tm - GM * band : GM;   // rows of this band
    const int r = (int)(q - band * per_band);
    const int blk = r / (hm * GN);
    const int w = tn - GN * blk < GN ? tn - GN * blk : GN;      // columns of this block
    const int rr = r - blk * hm * GN;
    mi = band * GM + rr / w;
    ni = blk * GN + rr % w;
}

__device__ __forceinline__ int dev_count(const int32_t *p, int off, int cap, int host) {
    if (!p) return host;
    int n = *p - off;
    n = n < 0 ? 0 : n;
    return n < cap ? n : cap;
}

}  // namespace

template <bool ATR>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
gemm_mfma_kernel(GemmArgs g) {
    const int M = g.M;
    const int N = dev_count(g.n_dev, g.n_off, g.n_cap, g.N);
    const int krows = dev_count(g.k_dev, g.k_off, g.k_cap, g.K);
    const int ksteps = (krows + BK - 1) / BK;
    if (ksteps == 0 && g.accumulate) return;     // nothing to add
    const int tm = (M + BV - 1) / BV, tn = (N + BT - 1) / BT;
    const int64_t n_tiles = (int64_t)tm * tn;
    const int ksplit = g.ksplit == 2 ? 2 : 1;
    const int kper = (ksteps + ksplit - 1) / ksplit;
    GLane L;
    L.lane = threadIdx.x & 63;
    L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    L.wv = L.wid & 1;
    L.wt = L.wid >> 1;
    L.h = L.lane >> 5;
    L.l32 = L.lane & 31;
#pragma unroll
    for (int s = 0; s < 4; ++s) L.ldsoff[s] = L.l32 * ROWB + (((2 * s + L.h) ^ swz(L.l32)) << 4);
    if (ATR) {
        // stage row R = 64 (panel in tile) + K row; lane j of 16-lane group gq supplies
        // K row 8 h + 4 r + j / 4 at columns 32 par + 16 (gq % 2) + 4 (j % 4) .. + 3, so
        // that lane i of the group receives column 16 (gq % 2) + i, K rows +0 .. +3
        const int gq = L.lane >> 4, j = L.lane & 15;
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int par = 0; par < 2; ++par) {
                const int R = 2 * L.wv * 64 + 8 * L.h + 4 * r + (j >> 2);
                const int c = 32 * par + 16 * (gq & 1) + 4 * (j & 3);
                L.troff[r][par] = (uint32_t)(R * ROWB + (((c >> 3) ^ swz_tr(R)) << 4) + (c & 7) * 2);
            }
    }
    const int G = gridDim.x;
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;

    for (int64_t u = my; u < n_tiles * ksplit; u += G) {
        const int64_t q = u % n_tiles;
        const int kb = (int)(u / n_tiles) * kper;
        const int kn = ksteps - kb < kper ? ksteps - kb : kper;   // this unit's steps
        int mi, ni;
        tile_of(q, tm, tn, mi, ni);
        const int m0 = mi * BV, n0 = ni * BT;
        // A DMA i of wave wid fills stage rows R = wid*64 + 8i + lane/8, slot lane&7
        // with chunk (lane&7) ^ swz(R) (swz_tr(R) for K-major A); B DMA i rows
        // R = wid*32 + 8i + lane/8. Rows past M (N) read the last one; offsets stay below
        // 256 row pitches.
        L.bbase = g.B + (int64_t)n0 * g.ldb;
        L.bk = g.bkstep;
        if (ATR) {
            // wave wid loads panel m0 / 64 + wid (the last one for panels past M): its 64
            // K rows of the step, 8 KB contiguous
            const int p0 = m0 / 64;
            const int pw = p0 + L.wid < g.a_panels ? L.wid : g.a_panels - 1 - p0;
            L.abase = g.A + (int64_t)p0 * g.a_prows * ROWB;
            L.ak = 64 * ROWB;
#pragma unroll
            for (int i = 0; i < W_DMA; ++i) {
                const int R = L.wid * 8 * W_DMA + 8 * i + (L.lane >> 3);
                const int ch = (L.lane & 7) ^ swz_tr(R);
                L.aoff[i] = (uint32_t)(((int64_t)pw * g.a_prows + 8 * i + (L.lane >> 3)) * ROWB +
                                       ch * 16);
            }
        } else {
            L.abase = g.A + (int64_t)m0 * g.lda;
            L.ak = g.akstep;
#pragma unroll
            for (int i = 0; i < W_DMA; ++i) {
                const int R = L.wid * 8 * W_DMA + 8 * i + (L.lane >> 3);
                const int ch = (L.lane & 7) ^ swz(R);
                const int r = m0 + R < M ? R : M - 1 - m0;
                L.aoff[i] = (uint32_t)((int64_t)r * g.lda + ch * 16);
            }
        }
#pragma unroll
        for (int i = 0; i < H_DMA; ++i) {
            const int R = (L.wid * H_DMA + i) * 8 + (L.lane >> 3);
            const int ch = (L.lane & 7) ^ swz(R);
            const int r = n0 + R < N ? R : N - 1 - n0;
            L.boff[i] = (uint32_t)((int64_t)r * g.ldb + ch * 16);
        }
        floatx16 acc[4][2];
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) acc[vb][cb] = floatx16{0.f};

        if (kn > 0) {
            // prologue: steps 0 and 1 (saturated) into stages 0 and 1
            g_issue(L, 0, kb);
            g_issue(L, 1, kb + (kn > 1 ? 1 : 0));
            int st = 0;
            GFrag P;
            g_step<false, ATR>(L, st, kb + (2 < kn ? 2 : kn - 1), acc, P);
            st = 1;
            for (int n = 1; n < kn; ++n) {
                const int pk = kb + (n + 2 < kn ? n + 2 : kn - 1);
                g_step<true, ATR>(L, st, pk, acc, P);
                st = st + 1 == NST ? 0 : st + 1;
            }
            g_mma(P, acc);
            // every DMA landed (trailing refills included) and every wave is done with
            // the ring before the next tile's prologue refills it
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __builtin_amdgcn_s_barrier();
            compiler_fence();
        }

        // lane holds column n = n0 + wt*64 + cb*32 + l32 and rows
        // m = m0 + wv*128 + vb*32 + 8*(r/4) + 4*h + r%4
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int n = n0 + L.wt * 64 + cb * 32 + L.l32;
            if (n >= N) continue;
            int64_t orow = n;
            if (g.rowmap) orow = g.rowmap[g.rowmap_off + n] & 0x7fffffffu;
#pragma unroll
            for (int vb = 0; vb < 4; ++vb)
#pragma unroll
                for (int rq = 0; rq < 4; ++rq) {
                    const int mb = m0 + L.wv * 128 + vb * 32 + 8 * rq + 4 * L.h;
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = g.alpha * agpr_read(acc[vb][cb][4 * rq + e]);
                    if (ksplit > 1) {
                        for (int e = 0; e < 4; ++e) {
                            if (mb + e >= M) continue;
                            float *c = g.trans_out ? g.C + orow * g.ldc + mb + e
                                                   : g.C + (int64_t)(mb + e) * g.ldc + orow;
                            atomicAdd(c, v[e]);
                        }
                    } else if (g.trans_out) {
                        float *c = g.C + orow * g.ldc + mb;
                        if (mb + 3 < M && ((g.ldc & 3) == 0)) {
                            float4 o = make_float4(v[0], v[1], v[2], v[3]);
                            if (g.accumulate) {
                                const float4 p = *(const float4 *)c;
                                o.x += p.x; o.y += p.y; o.z += p.z; o.w += p.w;
                            }
                            *(float4 *)c = o;
                        } else {
                            for (int e = 0; e < 4; ++e)
                                if (mb + e < M) c[e] = g.accumulate ? c[e] + v[e] : v[e];
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if (mb + e >= M) continue;
                            float *c = g.C + (int64_t)(mb + e) * g.ldc + orow;
                            *c = g.accumulate ? *c + v[e] : v[e];
                        }
                    }
                }
        }
    }
}

hipError_t launch_gemm(const GemmArgs &g, int grid, hipStream_t st) {
    if (grid <= 0 || g.M <= 0) return hipSuccess;
    // lane offsets within a tile are 32-bit: 256 rows of either operand (4 panels of A)
    if (g.ldb <= 0 || g.ldb >= ((int64_t)1 << 24) || g.bkstep <= 0) return hipErrorInvalidValue;
    if (g.a_panels > 0) {
        if (g.a_prows <= 0 || (int64_t)g.a_prows * ROWB * 4 >= ((int64_t)1 << 32) ||
            (int64_t)g.a_panels * 64 < g.M)
            return hipErrorInvalidValue;
        gemm_mfma_kernel<true><<<grid, 256, 0, st>>>(g);
    } else {
        if (g.lda <= 0 || g.lda >= ((int64_t)1 << 24) || g.akstep <= 0)
            return hipErrorInvalidValue;
        gemm_mfma_kernel<false><<<grid, 256, 0, st>>>(g);
    }
    return hipGetLastError();
}

}  // namespace olive
