// Fused bf16 scoring kernel for gfx950 with a 256 x 256 tile (MFMA 16x16x32, LDS ring
// fed by direct global->LDS loads from K-blocked panels).
//
// A workgroup (4 wavefronts) owns 256 vocabulary rows x 256 compacted positions and
// sweeps the vocabulary tiles of one split for one position tile; wavefront w owns all
// 256 rows of positions 64w .. 64w+63 (16 x 4 blocks of v_mfma_f32_16x16x32_bf16, 256
// AGPRs). Per vocabulary tile it accumulates the teacher logits (K = d_T) and then the
// student logits (K = d_S; the other order for the reverse KL alone) of the same block
// in the same AGPRs: one model's fp32 accumulators at a time, where holding both models
// (the other kernel) limits the tile to 256 x 128. The 16x16x32 shape moves half the
// accumulator bytes per MFMA operation of the 32x32x16 one; under this load the chip is
// power-limited, and a pure-MFMA loop of 16x16x32 on random bf16 operands held a 14 %
// higher clock than one of 32x32x16 at the same pipe occupancy.
//
// KL(teacher || student) needs, per vocabulary entry, the teacher's softmax weight
// next to the student's logit. The teacher fold keeps those weights, relative to the
// running teacher max and scaled by 2^15, as fp16 (v_cvt_pk_f16_f32, round to nearest
// even), 128 VGPRs per lane; the student fold consumes them with v_fma_mix_f32. The
// cross term is normalised by the sum of the same fp16 weights,
//   sum_v w^_v (z_T,v - z_S,v) / sum_v w^_v,
// so a common offset of the two logit vectors cancels exactly and the rounding of the
// weights (relative error <= 2^-11, fp16 normals down to 2^-29 of the max) moves the
// expectation by at most 2^-11 / (1 - 2^-11) times the mean absolute deviation of the
// logit difference under p_T, which is at most 2 (KL + TV) nats; the weights below the
// fp16 normal range add at most V * 2^-40 times the largest deviation. The
// log-normalisers use the fp32 weights.
//
// KL(student || teacher) is the same sum with the roles exchanged: the student's block
// comes first in every tile, its fold keeps the student's fp16 weights, and the
// teacher's fold consumes them (the REV instantiation). One call holds one set of
// weights, so a call that asks for both directions takes the other kernel.
//
// Pipeline: K advances 32 elements per step. W and the hidden rows are read from
// K-blocked panels ([d/32][rows][32] bf16, 64 bytes per row per panel), so one step of
// a tile is a contiguous 16 KB for W (256 rows) and for H (256 positions): whole
// 128-byte lines. The two 16 KB tiles land in one of 3 LDS stages (32 KB each) through
// global_load_lds_dwordx4, issued two steps ahead. A step's 64 MFMAs run in two
// halves of 8 row blocks; the second half runs under the next step's operand reads.
// Stage rows are 64 bytes; the 16-byte chunk c of row r sits in slot c ^ ((r >> 1) & 3).
// A ds_read_b128 of a 16x16x32 operand reads 16 rows x 4 chunks; of the XOR swizzles on
// 16-byte slots measured on gfx950 only this one left it free of bank conflicts (the
// 32x32x16 operand's 32 rows x 2 chunks are conflict-free with c ^ ((r >> 2) & 3)
// instead). The panels are written with the swizzle already applied (rows are tile
// rows modulo 256), so each DMA copies 1 KB linearly, whole lines per 8 lanes.
//
// The grid is persistent (one workgroup per CU); work units (position tile, split) are
// ordered so that the 32 workgroups of one XCD share 8 position tiles x 4 splits. They
// share those panel steps through the XCD's L2 only while they stay within some 15 K
// steps of one another; a phase lock (phase_lock.hpp) keeps them there.
#include <hip/hip_runtime.h>

#include "fold.hpp"
#include "mfma_pipe.hpp"
#include "olive_device.hpp"
#include "olive_internal.hpp"
#include "phase_lock.hpp"
#include "wide_pipe.hpp"

namespace olive {

namespace {

constexpr int XSPLIT_GROUP = 4;          // splits that consecutive units cycle through

// Running statistics (best, sec, z, idx) per model, column block and lane, kept in LDS
// between the folds: in registers they would not fit beside the fp16 weights and the
// operand fragments. [model][field][cb][thread], 32 KB.
__shared__ float x_stat[2 * 4 * 4 * 256];

__device__ __forceinline__ Run stat_get(int m, int cb) {
    const float *p = x_stat + (m * 16 + cb) * 256 + threadIdx.x;
    return Run{p[0], p[4 * 256], p[8 * 256], __float_as_int(p[12 * 256])};
}
__device__ __forceinline__ void stat_put(int m, int cb, const Run &R) {
    float *p = x_stat + (m * 16 + cb) * 256 + threadIdx.x;
    p[0] = R.best;
    p[4 * 256] = R.sec;
    p[8 * 256] = R.z;
    p[12 * 256] = __int_as_float(R.idx);
}

typedef _Float16 halfx2 __attribute__((ext_vector_type(2)));

// x, y to a packed fp16 pair (x low), rounded to nearest even (one v_cvt_pk_f16_f32).
// The conversion is left to the compiler, which knows its wait states after the
// exponentials that produce x and y (an inline-assembly conversion read one of them
// before it was written); the empty statement then makes the pair one 32-bit value,
// so that it stays packed in one register.
__device__ __forceinline__ uint32_t pack_f16x2(float x, float y) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    uint32_t r = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){x, y}, halfx2));
    asm volatile("" : "+v"(r));
    return r;
}

// +inf in a register the compiler cannot see through: med3(a, b, inf) then stays one
// v_med3_f32 (max of non-NaN a, b). With a literal inf it becomes v_max_f32 with both
// operands quieted first, since the accumulators come from inline assembly and are not
// known canonical.
__device__ __forceinline__ float opaque_inf() {
    float r;
    asm volatile("v_mov_b32 %0, 0x7f800000" : "=v"(r));
    return r;
}
__device__ __forceinline__ float opaque_one() {
    float r;
    asm volatile("v_mov_b32 %0, 1.0" : "=v"(r));
    return r;
}
__device__ __forceinline__ float f16_lo(uint32_t u) {
    return (float)__builtin_bit_cast(halfx2, u)[0];
}
__device__ __forceinline__ float f16_hi(uint32_t u) {
    return (float)__builtin_bit_cast(halfx2, u)[1];
}

// Running max / second max / lowest argmax of one column over 16 logits (R.z is left
// alone): 4 output blocks of the column, element e at row vcode0 + 16 (e / 4) + e % 4.
// Returns the rescale factor exp2(c (old max - new max)) of the sums.
__device__ __forceinline__ float block_max(const float (&z)[16], Run &R, int vcode0,
                                           float c, float inf) {
    float tm = R.best, ts = R.sec;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        ts = __builtin_amdgcn_fmed3f(z[r], tm, ts);
        tm = __builtin_amdgcn_fmed3f(tm, z[r], inf);
    }
    int code = 0;
#pragma unroll
    for (int r = 15; r >= 0; --r) code = (z[r] == tm) ? 16 * (r >> 2) + (r & 3) : code;
    const bool up = tm > R.best;
    const float resc = fast_exp2((R.best - tm) * c);
    R.idx = up ? vcode0 + code : R.idx;
    R.best = tm;
    R.sec = ts;
    return resc;
}

// The first model of a tile (the one whose weights the KL takes), second pass over a
// column's logits of the tile, once the column's running max over the tile is final
// (the first pass is block_max): mneg = 15 - c max. Adds the weights
// 2^15 exp2(c (z - max)) in fp32 to zsum, keeps them as fp16 in eh, adds the fp16
// values to hsum and their products with the logits to asum. All weights of a tile
// refer to the same max, so those kept for the second model's fold need no rescale.
__device__ __forceinline__ void first_weights(const float (&z)[16], float c, float mneg,
                                                float one, float &zsum, float &hsum,
                                                float &asum, uint32_t (&eh)[8]) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const float e0 = fast_exp2(fmaf(z[2 * q], c, mneg));
        const float e1 = fast_exp2(fmaf(z[2 * q + 1], c, mneg));
        zsum += e0;
        zsum += e1;
        uint32_t p = pack_f16x2(e0, e1);
        // one v_fma_mix_f32 each (1.0 from a register the compiler does not see through;
        // with a literal 1 it would convert and add in two instructions)
        hsum = fmaf(f16_lo(p), one, hsum);
        hsum = fmaf(f16_hi(p), one, hsum);
        asum = fmaf(f16_lo(p), z[2 * q], asum);
        asum = fmaf(f16_hi(p), z[2 * q + 1], asum);
        // a new value for the second fold: it must re-read the packed pair rather than
        // share these conversions (their fp32 results would stay live across its sweep)
        asm volatile("" : "+v"(p));
        eh[q] = p;
    }
}

// The second model of a tile, 16 logits of a column: running statistics, and the sum
// of the first model's fp16 weights times these logits into as.
__device__ __forceinline__ void fold_second(const float (&z)[16], Run &R, float &as,
                                             const uint32_t (&eh)[8], float c, int vcode0,
                                             float inf) {
    R.z *= block_max(z, R, vcode0, c, inf);
    const float mneg = -R.best * c;
    float zsum = R.z, asum = as;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        zsum += fast_exp2(fmaf(z[2 * q], c, mneg));
        zsum += fast_exp2(fmaf(z[2 * q + 1], c, mneg));
        asum = fmaf(f16_lo(eh[q]), z[2 * q], asum);
        asum = fmaf(f16_hi(eh[q]), z[2 * q + 1], asum);
    }
    R.z = zsum;
    as = asum;
}

// Student of a student-only call, 16 logits of a column: running statistics only.
__device__ __forceinline__ void fold_student_only(const float (&z)[16], Run &R, float c,
                                                  int vcode0, float inf) {
    R.z *= block_max(z, R, vcode0, c, inf);
    const float mneg = -R.best * c;
    float zsum = R.z;
#pragma unroll
    for (int q = 0; q < 16; ++q) zsum += fast_exp2(fmaf(z[q], c, mneg));
    R.z = zsum;
}

// Merge the first model's record y (with its difference sum ya and weight sum yz) into x.
__device__ __forceinline__ void merge_weighted(Run &x, float &xa, float &xz, const Run &y,
                                              float ya, float yz, float c) {
    if (y.best == kNegInf) return;
    if (x.best == kNegInf) {
        x = y;
        xa = ya;
        xz = yz;
        return;
    }
    const bool yw = (y.best > x.best) || (y.best == x.best && y.idx < x.idx);
    const Run w = yw ? y : x, l = yw ? x : y;
    const float wa = yw ? ya : xa, la = yw ? xa : ya;
    const float wz = yw ? yz : xz, lz = yw ? xz : yz;
    const float r = fast_exp2((l.best - w.best) * c);
    x.best = w.best;
    x.idx = w.idx;
    x.sec = fmaxf(w.sec, l.best);
    x.z = w.z + l.z * r;
    xa = wa + la * r;
    xz = wz + lz * r;
}

// HAS_T: every tile holds a block of each model, and the first one's fold keeps its fp16
// weights for the cross term of the second's; without it the call is student-only (SAME
// and REV are then unused). REV: the student's block comes first (KL(student ||
// teacher)); otherwise the teacher's (KL(teacher || student)).
template <bool SAME, bool HAS_T, bool REV>
struct Wide {
    static constexpr int M1 = (HAS_T && !REV) ? 1 : 0;   // first block's model (1 = teacher)
    static constexpr int M2 = HAS_T ? 1 - M1 : 0;        // last block's model
    struct Cursor {
        const char *w, *h;       // W and H tile of the step to prefetch
        int64_t wstep, hstep;    // bytes from one panel to the next (0 past the unit's end)
        int m, kk, cnt, vt;      // model block (1 = teacher), step in the block, its length
        int vt1, nS, nT, p;
    };
    using Args = ScoreArgs;
    using Pipe = WidePipe<Wide>;

    template <int M>
    static __device__ __forceinline__ void enter(Cursor &C, const ScoreArgs &a, int vt) {
        C.m = M;
        C.kk = 0;
        C.cnt = M ? C.nT : C.nS;
        C.vt = vt;
        C.w = (const char *)(M ? a.wpt : a.wps) + (int64_t)vt * XV * XROW;
        C.h = (const char *)(M ? a.hpt : a.hps) + (int64_t)C.p * XT * XROW;
        C.wstep = a.vpad * XROW;
        C.hstep = a.prow * XROW;
    }

    // The first model's block of a tile, then the second's, then the next tile's first;
    // past the unit's last block the prefetches repeat its last step.
    static __device__ __forceinline__ void turn(Cursor &C, const ScoreArgs &a) {
        if (C.kk == C.cnt) {
            if (HAS_T && C.m == M1) {
                enter<M2>(C, a, C.vt);
            } else if (C.vt + 1 < C.vt1) {
                enter<M1>(C, a, C.vt + 1);
            } else {
                C.w -= C.wstep;
                C.h -= C.hstep;
                C.wstep = 0;
                C.hstep = 0;
                C.cnt = 0x7fffffff;
            }
        }
    }

    static __device__ __forceinline__ void advance(Cursor &C) {
        C.w += C.wstep;
        C.h += C.hstep;
        C.kk += 1;
    }

    // Add kMasked to the rows at or past V of the padded last tile (one MFMA per block:
    // A holds kMasked in k = 0 of those rows, B ones), so they drop out of every
    // statistic while the accumulators stay MFMA-only.
    static __device__ __forceinline__ void mask_tail(const XLane &L, floatx4 (&acc)[16][4],
                                                     int row0, int V) {
        bf16x8 ones;
#pragma unroll
        for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
#pragma unroll
        for (int vb = 0; vb < 16; ++vb) {
            const int v = row0 + vb * 16 + L.l16;   // A-operand row of this lane
            bf16x8 bias;
#pragma unroll
            for (int e = 0; e < 8; ++e) bias[e] = (__bf16)0.0f;
            if (L.g == 0 && v >= V) bias[0] = (__bf16)kMasked;
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                acc[vb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bias, ones, acc[vb][cb], 0,
                                                                      0, 0);
        }
    }

    // The 16 logits of column cb in row blocks 4q .. 4q+3.
    static __device__ __forceinline__ void col16(const floatx4 (&acc)[16][4], int q, int cb,
                                                 float (&z)[16]) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) z[4 * j + r] = agpr_read(acc[4 * q + j][cb][r]);
    }

    // One model block of COUNT_ K steps into acc: the first step has no pending half, the
    // block's last half runs after the loop.
#define OLIVE_XSTEPS(COUNT_)                                                              \
            {                                                                             \
                XFragA PA;                                                                \
                XFragB PB;                                                                \
                Pipe::template step<0>(a, L, C, st, acc, PA, PB);                         \
                st = st + 1 == XNST ? 0 : st + 1;                                         \
                if ((COUNT_) > 1) {                                                       \
                    Pipe::template step<1>(a, L, C, st, acc, PA, PB);                     \
                    st = st + 1 == XNST ? 0 : st + 1;                                     \
                    for (int k = 2; k < (COUNT_); ++k) {                                  \
                        Pipe::template step<2>(a, L, C, st, acc, PA, PB);                 \
                        st = st + 1 == XNST ? 0 : st + 1;                                 \
                    }                                                                     \
                    Pipe::template mma_half<1, false, 0, 0>(PA, PB, acc, C, L, 0u, x_ring,   \
                                                           PA, PB);               \
                } else {                                                                  \
                    Pipe::template mma_half<1, true, 0, 0>(PA, PB, acc, C, L, 0u, x_ring,    \
                                                          PA, PB);                \
                }                                                                         \
                __builtin_amdgcn_sched_barrier(0);                                        \
            }

    static __device__ __forceinline__ void run(ScoreArgs a) {
        const int t_valid = a.sched->t_valid;
        const int n_p = a.sched->n_ptiles;
        const int ns = a.sched->n_splits;
        const int n_units = a.sched->n_units;
        const XLane L = make_lane();
        const int nS = a.ds / XK, nT = a.dt / XK;
        const int G = gridDim.x;
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        const bool lock = phase_lock_on(G, nS + nT);

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, XSPLIT_GROUP, p, s);
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);

            // per column: the first model's fp16 weight sum, its weighted logit sum, and
            // the same weights times the second model's logits
            float ZH[4], A1[4], A2[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                stat_put(0, cb, Run{kNegInf, kNegInf, 0.f, 0x7fffffff});
                stat_put(1, cb, Run{kNegInf, kNegInf, 0.f, 0x7fffffff});
                ZH[cb] = 0.f;
                A1[cb] = 0.f;
                A2[cb] = 0.f;
            }
            uint32_t eh[4][4][8];   // [row-block quarter][cb][pair]
            floatx4 acc[16][4];

            Cursor C;
            C.vt1 = vt1;
            C.nS = nS;
            C.nT = nT;
            C.p = p;
            enter<M1>(C, a, vt0);
#pragma unroll
            for (int i = 0; i < XNST - 1; ++i) Pipe::issue(a, L, C, i);
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): no scalar load pending
            int st = 0;
            // the first two tiles of a unit only measure the period (it straddles the
            // unit change)
            PhaseClock PH{0u, 0u};
            const float c1 = M1 ? a.cT : a.cS, c2 = M2 ? a.cT : a.cS;
            for (int vt = vt0; vt < vt1; ++vt) {
                const int row0 = vt * XV;
                const int vbase = row0 + 4 * L.g;
                if (lock && L.wid == 0) phase_lock<XDMA_STEP * (XNST - 2)>(PH, G);
                if constexpr (HAS_T) {
                OLIVE_XSTEPS(M1 ? nT : nS)
                if (row0 + XV > a.V) mask_tail(L, acc, row0, a.V);
                {
                    const float inf = opaque_inf(), one = opaque_one();
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        Run R = stat_get(M1, cb);
                        const float m0 = R.best;
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
                            col16(acc, qq, cb, z);
                            (void)block_max(z, R, vbase + qq * 64, c1, inf);
                        }
                        // one rescale per column and tile, to the tile's max
                        const float resc = fast_exp2((m0 - R.best) * c1);
                        float zsum = R.z * resc, hsum = ZH[cb] * resc, asum = A1[cb] * resc;
                        A2[cb] *= resc;
                        const float mneg = fmaf(-R.best, c1, 15.0f);
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
                            col16(acc, qq, cb, z);
                            first_weights(z, c1, mneg, one, zsum, hsum, asum, eh[qq][cb]);
                        }
                        R.z = zsum;
                        ZH[cb] = hsum;
                        A1[cb] = asum;
                        // Pin the weighted sums here: otherwise the compiler sinks them
                        // past the second sweep, keeping the first model's logits alive
                        // (and spilled) across it.
                        asm volatile("" : "+v"(ZH[cb]), "+v"(A1[cb]), "+v"(A2[cb]));
                        stat_put(M1, cb, R);
                    }
                }
                }
                OLIVE_XSTEPS(M2 ? nT : nS)
                if (row0 + XV > a.V) mask_tail(L, acc, row0, a.V);
                {
                    const float inf = opaque_inf();
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        Run R = stat_get(M2, cb);
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
                            col16(acc, qq, cb, z);
                            if constexpr (HAS_T)
                                fold_second(z, R, A2[cb], eh[qq][cb], c2, vbase + qq * 64, inf);
                            else
                                fold_student_only(z, R, a.cS, vbase + qq * 64, inf);
                        }
                        stat_put(M2, cb, R);
                    }
                }
            }

            // The difference sums (first model minus second; unscaled with equal scales,
            // the combine multiplies by s), then the 4 lanes of each column (row groups
            // g = 0..3) merge.
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): trailing prefetches landed
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const float s1 = M1 ? a.sT : a.sS, s2 = M1 ? a.sS : a.sT;
                float aa = SAME ? A1[cb] - A2[cb] : s1 * A1[cb] - s2 * A2[cb];
                float zh = ZH[cb];
                Run R1 = stat_get(M1, cb), R2 = stat_get(M2, cb);
#pragma unroll
                for (int off = 16; off <= 32; off <<= 1) {
                    Run o{__shfl_xor(R2.best, off), __shfl_xor(R2.sec, off),
                          __shfl_xor(R2.z, off), __shfl_xor(R2.idx, off)};
                    float dummy = 0.f;
                    merge_run(R2, dummy, o, 0.f, c2);
                    if constexpr (HAS_T) {
                        Run t{__shfl_xor(R1.best, off), __shfl_xor(R1.sec, off),
                              __shfl_xor(R1.z, off), __shfl_xor(R1.idx, off)};
                        const float ta = __shfl_xor(aa, off), tz = __shfl_xor(zh, off);
                        merge_weighted(R1, aa, zh, t, ta, tz, c1);
                    }
                }
                // the student's record is the last block's unless that is the teacher's
                const Run &RS = M2 == 0 ? R2 : R1, &RT = M2 == 0 ? R1 : R2;
                const int j = p * XT + L.wid * 64 + cb * 16 + L.l16;
                if (L.g == 0 && j < t_valid) {
                    float *P = a.part;
                    const int64_t ps = a.pstride;
                    // the first model's exp-sum carries the weights' 2^15 (exact)
                    const float zs1 = HAS_T ? 0x1p-15f : 1.f;
                    P[(F_BEST_S * MAX_SPLITS + s) * ps + j] = RS.best;
                    P[(F_SEC_S * MAX_SPLITS + s) * ps + j] = RS.sec;
                    P[(F_IDX_S * MAX_SPLITS + s) * ps + j] = __int_as_float(RS.idx);
                    P[(F_Z_S * MAX_SPLITS + s) * ps + j] = M1 ? RS.z : RS.z * zs1;
                    if (!HAS_T) continue;
                    P[(F_BEST_T * MAX_SPLITS + s) * ps + j] = RT.best;
                    P[(F_SEC_T * MAX_SPLITS + s) * ps + j] = RT.sec;
                    P[(F_IDX_T * MAX_SPLITS + s) * ps + j] = __int_as_float(RT.idx);
                    P[(F_Z_T * MAX_SPLITS + s) * ps + j] = M1 ? RT.z * zs1 : RT.z;
                    P[((REV ? F_B : F_A) * MAX_SPLITS + s) * ps + j] = aa;
                    P[(F_ZH * MAX_SPLITS + s) * ps + j] = zh;
                }
            }
            // every wave is past its last read of the ring before the next unit's
            // prologue refills it
            compiler_fence();
            __syncthreads();
        }
    }

    // Logit-gradient pass of the backward's cross-entropy (student only) over the scored
    // rows [c0, c0 + chunk) of the call, from the forward pass's normalisers: per tile,
    // g = w_ce (p_S - onehot(y)), p_S = exp(s_S z_S - lse_S), stored as bf16 (round to
    // nearest even) into dz_t, K-blocked panels [v/64][row][64] of the chunk's rows.
    // a.hps points at the panel row of compacted row c0; the position tiles are 256 rows
    // and c0 a multiple of 256.
    static __device__ __forceinline__ void run_dz(ScoreArgs a, DzArgs z) {
        const int t_all = a.sched->t_valid - z.c0;
        const int t_rows = t_all < 0 ? 0 : (t_all < z.chunk ? t_all : z.chunk);
        const int n_p = (t_rows + XT - 1) / XT;
        const int G = gridDim.x;
        const int ns = pass_splits(n_p, a.n_vtiles, G);
        const int64_t n_units = (int64_t)n_p * ns;
        const XLane L = make_lane();
        const int nS = a.ds / XK, nT = 0;
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        const bool lock = phase_lock_on(G, nS);
        const float wce = z.w_ce;

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, XSPLIT_GROUP, p, s);
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);
            // the lane's 4 columns: chunk row, normaliser (log2 domain), target
            int tcol[4], ycol[4];
            float l2s[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                tcol[cb] = p * XT + L.wid * 64 + cb * 16 + L.l16;
                const bool ok = tcol[cb] < t_rows;
                const int j = z.c0 + (ok ? tcol[cb] : 0);
                l2s[cb] = ok ? z.lse[2 * (int64_t)j] * kLog2e : 0.f;
                ycol[cb] = ok ? z.targets[a.rowmap[j] & 0x7fffffffu] : -1;
                tcol[cb] = ok ? tcol[cb] : -1;
            }
            floatx4 acc[16][4];
            Cursor C;
            C.vt1 = vt1;
            C.nS = nS;
            C.nT = nT;
            C.p = p;
            enter<0>(C, a, vt0);
#pragma unroll
            for (int i = 0; i < XNST - 1; ++i) Pipe::issue(a, L, C, i);
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): no scalar load pending
            int st = 0;
            PhaseClock PH{0u, 0u};
            for (int vt = vt0; vt < vt1; ++vt) {
                const int row0 = vt * XV;
                if (lock && L.wid == 0) phase_lock<XDMA_STEP * (XNST - 2)>(PH, G);
                OLIVE_XSTEPS(nS)
                // Rows at or past V are not stored (dz_t's rows V .. vp-1 stay zero).
                // Lane (l16, g) holds rows 16 vb + 4 g .. +3 of column cb: 8 bytes of one
                // panel row.
#pragma unroll
                for (int vb = 0; vb < 16; ++vb) {
                    __builtin_amdgcn_sched_barrier(0);
                    const int v0 = row0 + vb * 16 + 4 * L.g;
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        float gr[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float zs = agpr_read(acc[vb][cb][e]);
                            gr[e] = wce * fast_exp2(fmaf(zs, a.cS, -l2s[cb]));
                            gr[e] -= (v0 + e == ycol[cb]) ? wce : 0.f;
                        }
                        const int t = tcol[cb];
                        if (t < 0 || v0 >= a.V) continue;
                        uint16_t *dst = z.dz_t + (((int64_t)(v0 >> 6) * z.chunk + t) * 64 +
                                                  (v0 & 63));
                        if (v0 + 4 <= a.V) {
                            *(uint2 *)dst = make_uint2(pack_bf16x2(gr[0], gr[1]),
                                                       pack_bf16x2(gr[2], gr[3]));
                        } else {
                            const uint32_t w0 = pack_bf16x2(gr[0], gr[1]);
                            const uint32_t w1 = pack_bf16x2(gr[2], gr[3]);
                            const uint16_t h4[4] = {(uint16_t)w0, (uint16_t)(w0 >> 16),
                                                    (uint16_t)w1, (uint16_t)(w1 >> 16)};
                            for (int e = 0; e < 4 && v0 + e < a.V; ++e) dst[e] = h4[e];
                        }
                    }
                }
            }
            // every DMA landed and every wave is done with the ring before the next
            // unit's prologue refills it
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __syncthreads();
        }
    }
    // Logit-gradient pass of a cross-entropy-only backward that forms its own
    // normalisers, over the scored rows [c0, c0 + chunk) (no forward pass before it).
    // Per vocabulary tile and column it updates the running max m over the tiles swept
    // so far (this one included) and stores w = 2^15 exp2(c (z - m)) in [0, 2^15] as
    // fp16 (round to nearest even) into dz_t, where the gradient goes; m goes to
    // mref[tile][row], and the split's (m, sum of w 2^-15) to the partial records. The
    // final normaliser (dz_lse_kernel) and the rescale of each tile's weights by
    // 2^-15 w_ce exp(s m - lse) into the bf16 gradient (dz_rescale_kernel) follow.
    static __device__ __forceinline__ void run_dz_online(ScoreArgs a, DzArgs z) {
        const int t_all = a.sched->t_valid - z.c0;
        const int t_rows = t_all < 0 ? 0 : (t_all < z.chunk ? t_all : z.chunk);
        const int n_p = (t_rows + XT - 1) / XT;
        const int G = gridDim.x;
        const int ns = pass_splits(n_p, a.n_vtiles, G);
        const int64_t n_units = (int64_t)n_p * ns;
        const XLane L = make_lane();
        const int nS = a.ds / XK, nT = 0;
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        const bool lock = phase_lock_on(G, nS);

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, XSPLIT_GROUP, p, s);
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);
            // the lane's 4 columns: chunk row (-1 past the rows), running max, weight sum
            int tcol[4];
            // running max and weight sum per column, in LDS between tiles (each thread its
            // own entries): in registers beside the pipeline's they spilled 63 VGPRs
            float *mr = x_stat + threadIdx.x, *zs = x_stat + 1024 + threadIdx.x;
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const int t = p * XT + L.wid * 64 + cb * 16 + L.l16;
                tcol[cb] = t < t_rows ? t : -1;
                mr[cb * 256] = -0x1p127f;   // below every logit, masked rows included
                zs[cb * 256] = 0.f;
            }
            floatx4 acc[16][4];
            Cursor C;
            C.vt1 = vt1;
            C.nS = nS;
            C.nT = nT;
            C.p = p;
            enter<0>(C, a, vt0);
#pragma unroll
            for (int i = 0; i < XNST - 1; ++i) Pipe::issue(a, L, C, i);
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): no scalar load pending
            int st = 0;
            PhaseClock PH{0u, 0u};
            for (int vt = vt0; vt < vt1; ++vt) {
                const int row0 = vt * XV;
                if (lock && L.wid == 0) phase_lock<XDMA_STEP * (XNST - 2)>(PH, G);
                OLIVE_XSTEPS(nS)
                if (row0 + XV > a.V) mask_tail(L, acc, row0, a.V);
                // the column's max over the tile: the lane's 64 rows, then its 4 row groups
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    float tm = agpr_read(acc[0][cb][0]);
#pragma unroll
                    for (int vb = 0; vb < 16; ++vb) {
                        // (the accumulator reads of later blocks are not hoisted)
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (vb || e) tm = fmaxf(tm, agpr_read(acc[vb][cb][e]));
                    }
                    tm = fmaxf(tm, __shfl_xor(tm, 16));
                    tm = fmaxf(tm, __shfl_xor(tm, 32));
                    const float mn = fmaxf(mr[cb * 256], tm);
                    zs[cb * 256] *= fast_exp2((mr[cb * 256] - mn) * a.cS);
                    mr[cb * 256] = mn;
                    if (L.g == 0 && tcol[cb] >= 0) z.mref[(int64_t)vt * z.chunk + tcol[cb]] = mn;
                }
                // the weights: into the sums, and as fp16 into dz_t (rows at or past V are
                // not stored; lane (l16, g) holds rows 16 vb + 4 g .. +3 of column cb)
#pragma unroll
                for (int vb = 0; vb < 16; ++vb) {
                    __builtin_amdgcn_sched_barrier(0);
                    const int v0 = row0 + vb * 16 + 4 * L.g;
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        const float mneg = fmaf(-mr[cb * 256], a.cS, 15.0f);
                        float w[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            w[e] = fast_exp2(fmaf(agpr_read(acc[vb][cb][e]), a.cS, mneg));
                            zs[cb * 256] += w[e];
                        }
                        const int t = tcol[cb];
                        if (t < 0 || v0 >= a.V) continue;
                        uint16_t *dst = z.dz_t + (((int64_t)(v0 >> 6) * z.chunk + t) * 64 +
                                                  (v0 & 63));
                        const uint32_t w01 = pack_f16x2(w[0], w[1]);
                        const uint32_t w23 = pack_f16x2(w[2], w[3]);
                        if (v0 + 4 <= a.V) {
                            *(uint2 *)dst = make_uint2(w01, w23);
                        } else {
                            const uint16_t h4[4] = {(uint16_t)w01, (uint16_t)(w01 >> 16),
                                                    (uint16_t)w23, (uint16_t)(w23 >> 16)};
                            for (int e = 0; e < 4 && v0 + e < a.V; ++e) dst[e] = h4[e];
                        }
                    }
                }
            }
            // the split's records: the 4 row groups of a column share its max, so their
            // weight sums add
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                float zz = zs[cb * 256];
                zz += __shfl_xor(zz, 16);
                zz += __shfl_xor(zz, 32);
                if (L.g == 0 && tcol[cb] >= 0) {
                    const int64_t j = (int64_t)z.c0 + tcol[cb];
                    a.part[(F_BEST_S * MAX_SPLITS + s) * a.pstride + j] = mr[cb * 256];
                    a.part[(F_Z_S * MAX_SPLITS + s) * a.pstride + j] = zz * 0x1p-15f;
                }
            }
            // every DMA landed and every wave is done with the ring before the next
            // unit's prologue refills it
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __syncthreads();
        }
    }
#undef OLIVE_XSTEPS
};

template <bool SAME, bool HAS_T, bool REV>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_wide_kernel(ScoreArgs a) {
    Wide<SAME, HAS_T, REV>::run(a);
}

__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_wide_dz_kernel(ScoreArgs a, DzArgs z) {
    Wide<false, false, false>::run_dz(a, z);
}

__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_wide_dz_online_kernel(ScoreArgs a, DzArgs z) {
    Wide<false, false, false>::run_dz_online(a, z);
}

// Slot of 16-byte chunk q (0..3) of panel row r: the LDS swizzle of the stages, applied
// when the panels are written (tiles start at multiples of 256 rows).
__device__ __forceinline__ int panel_slot(int64_t r, int q) { return q ^ (int)((r >> 1) & 3); }

// [V][d] bf16 weights -> K-blocked panels [d/32][vpad][32] (rows V .. vpad-1 zero), each
// row's chunks in their swizzled slots. Block (64-row group, panel); thread: row t/4,
// 16-byte chunk t&3.
__global__ void __launch_bounds__(256)
panel_w_kernel(const uint16_t *__restrict__ w, int64_t V, int d, int64_t vpad,
               uint16_t *__restrict__ out) {
    const int64_t v = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
    const int pnl = blockIdx.y, q = threadIdx.x & 3;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (v < V) val = *(const uint4 *)(w + v * d + pnl * XK + q * 8);
    *(uint4 *)(out + ((int64_t)pnl * vpad + v) * XK + panel_slot(v, q) * 8) = val;
}

// The compacted hidden rows of a call -> K-blocked panels [d/32][prow][32], chunks in
// their swizzled slots: row j < t_valid is hidden row rowmap[j]; rows t_valid .. up to
// the next multiple of 256 are zero (the last position tile's columns past the rows).
__global__ void __launch_bounds__(256)
panel_h_kernel(const uint16_t *__restrict__ h, int d, const uint32_t *__restrict__ rowmap,
               const Sched *__restrict__ sched, int64_t prow, uint16_t *__restrict__ out) {
    const int t_valid = sched->t_valid;
    const int64_t tpad = ((int64_t)t_valid + XT - 1) / XT * XT;
    const int64_t j = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
    if (j >= tpad || j >= prow) return;
    const int pnl = blockIdx.y, q = threadIdx.x & 3;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (j < t_valid) {
        const int64_t g = rowmap[j] & 0x7fffffffu;
        val = *(const uint4 *)(h + g * d + pnl * XK + q * 8);
    }
    *(uint4 *)(out + ((int64_t)pnl * prow + j) * XK + panel_slot(j, q) * 8) = val;
}

}  // namespace

hipError_t launch_score_wide(const ScoreArgs &a, bool same_scale, bool has_t, bool rev,
                             int grid, hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    if (a.ds <= 0 || a.ds % XK != 0 || a.vpad % XV != 0 || a.prow % XT != 0 || !a.wps ||
        !a.hps)
        return hipErrorInvalidValue;
    if (has_t && (a.dt <= 0 || a.dt % XK != 0 || !a.wpt || !a.hpt)) return hipErrorInvalidValue;
    if (rev && !has_t) return hipErrorInvalidValue;
    if (!has_t)
        score_wide_kernel<false, false, false><<<grid, 256, 0, st>>>(a);
    else if (rev && same_scale)
        score_wide_kernel<true, true, true><<<grid, 256, 0, st>>>(a);
    else if (rev)
        score_wide_kernel<false, true, true><<<grid, 256, 0, st>>>(a);
    else if (same_scale)
        score_wide_kernel<true, true, false><<<grid, 256, 0, st>>>(a);
    else
        score_wide_kernel<false, true, false><<<grid, 256, 0, st>>>(a);
    return hipGetLastError();
}

hipError_t launch_score_wide_dz(const ScoreArgs &a, const DzArgs &z, int grid, hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    if (a.ds <= 0 || a.ds % XK != 0 || a.vpad % XV != 0 || !a.wps || !a.hps || !z.dz_t ||
        z.c0 % XT != 0 || z.chunk <= 0)
        return hipErrorInvalidValue;
    score_wide_dz_kernel<<<grid, 256, 0, st>>>(a, z);
    return hipGetLastError();
}

hipError_t launch_score_wide_dz_online(const ScoreArgs &a, const DzArgs &z, int grid,
                                       hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    if (a.ds <= 0 || a.ds % XK != 0 || a.vpad % XV != 0 || !a.wps || !a.hps || !z.dz_t ||
        !z.mref || !a.part || z.c0 % XT != 0 || z.chunk <= 0)
        return hipErrorInvalidValue;
    score_wide_dz_online_kernel<<<grid, 256, 0, st>>>(a, z);
    return hipGetLastError();
}

hipError_t launch_panel_w(const void *w, int64_t V, int d, int64_t vpad, void *out,
                          hipStream_t st) {
    if (d % XK != 0 || vpad % 64 != 0 || vpad < V) return hipErrorInvalidValue;
    dim3 grid((unsigned)(vpad / 64), (unsigned)(d / XK));
    panel_w_kernel<<<grid, 256, 0, st>>>((const uint16_t *)w, V, d, vpad, (uint16_t *)out);
    return hipGetLastError();
}

hipError_t launch_panel_h(const void *h, int d, const uint32_t *rowmap, const Sched *sched,
                          int64_t prow, void *out, hipStream_t st) {
    if (d % XK != 0 || prow % XT != 0) return hipErrorInvalidValue;
    dim3 grid((unsigned)(prow / 64), (unsigned)(d / XK));
    panel_h_kernel<<<grid, 256, 0, st>>>((const uint16_t *)h, d, rowmap, sched, prow,
                                         (uint16_t *)out);
    return hipGetLastError();
}

}  // namespace olive
