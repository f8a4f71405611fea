// Fused bf16 scoring kernel for gfx950 with a 256 x 256 tile (MFMA 32x32x16, LDS ring
// fed by direct global->LDS loads from K-blocked panels).
//
// A workgroup (4 wavefronts, 2 x 2) owns 256 vocabulary rows x 256 compacted positions
// and sweeps the vocabulary tiles of one split for one position tile. Per vocabulary
// tile it accumulates the teacher logits (K = d_T) and then the student logits
// (K = d_S) of the same 256 x 256 block in the same 256 AGPRs per lane: one model's
// fp32 accumulators at a time, where holding both models (the other kernel) limits
// the tile to 256 x 128. Bytes moved from L2 into LDS per MFMA operation, and LDS reads
// per MFMA, are then two thirds of that kernel's.
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
// Pipeline: K advances 32 elements per step. W and the hidden rows are read from
// K-blocked panels ([d/32][rows][32] bf16, 64 bytes per row per panel), so one step of
// a tile is a contiguous 16 KB for W (256 rows) and for H (256 positions): whole
// 128-byte lines at half the K step of the row-major layout. The two 16 KB tiles land
// in one of 4 LDS stages (32 KB each) through global_load_lds_dwordx4, issued three
// steps ahead. Stage rows are 64 bytes; the 16-byte chunk c of row r sits in slot
// c ^ ((r >> 2) & 3), which keeps the ds_read_b128 operand fetches (16 rows x one chunk
// per 256 bytes of banks) free of bank conflicts. The swizzle is applied on the global
// side of the DMA (each lane fetches the chunk that belongs at its LDS slot).
//
// The grid is persistent (one workgroup per CU); work units (position tile, split) are
// ordered so that the 32 workgroups of one XCD share 8 position tiles x 4 splits.
#include <hip/hip_runtime.h>

#include "fold.hpp"
#include "mfma_pipe.hpp"
#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

namespace {

constexpr int XV = 256;                  // vocabulary rows per tile
constexpr int XT = WIDE_BT;              // positions per tile: 256
constexpr int XK = 32;                   // K elements per step: one panel row
constexpr int XROW = XK * 2;             // 64 bytes
constexpr int XW_BYTES = XV * XROW;      // 16 KB
constexpr int XH_BYTES = XT * XROW;      // 16 KB
constexpr int XNST = 4;                  // ring stages
constexpr int XSTAGE = XW_BYTES + XH_BYTES;   // 32 KB; 4 stages = 128 KB
constexpr int XDMA = 4;                  // 1 KB DMAs per wave per operand per step
constexpr int XDMA_STEP = 2 * XDMA;      // 8
constexpr int XSPLIT_GROUP = 4;          // splits that consecutive units cycle through

__shared__ __attribute__((aligned(1024))) char x_ring[XNST * XSTAGE];
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

__device__ __forceinline__ uint32_t xring_addr() {
    return (uint32_t)(uintptr_t)(lds_void *)x_ring;
}

// One global -> LDS DMA of 16 bytes per lane: lane i's bytes land at the wave-uniform
// LDS address la + OFFL + 16 i; the source is the wave-uniform base plus the lane's
// 32-bit offset. The instruction's own offset field stays 0 (it would move the LDS
// address as well).
template <int OFFL>
__device__ __forceinline__ void xdma(const char *base, uint32_t voff, uint32_t la) {
    la = __builtin_amdgcn_readfirstlane(la);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(la), "v"(voff), "s"(base), "i"(OFFL)
                 : "memory", "m0", "scc");
#pragma clang diagnostic pop
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

struct XLane {
    int lane, wid, wv, wt, h, l32;
    uint32_t voff[XDMA]; // per DMA i of an operand: the lane's byte offset within a
                         // 16 KB tile step (wave part and i * 1 KB included)
    uint32_t lds_a[2];   // operand read offsets of sub-step j within a stage (W part)
    uint32_t lds_b[2];   // (H part)
};

struct XFrag {
    bf16x8 A[4], B[4];
};

// Running max / second max / lowest argmax of one column over one 32-row block (R.z is
// left alone). Returns the rescale factor exp2(c (old max - new max)) of the sums.
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
    for (int r = 15; r >= 0; --r) code = (z[r] == tm) ? 8 * (r >> 2) + (r & 3) : code;
    const bool up = tm > R.best;
    const float resc = fast_exp2((R.best - tm) * c);
    R.idx = up ? vcode0 + code : R.idx;
    R.best = tm;
    R.sec = ts;
    return resc;
}

// Teacher, second pass over a column's blocks of the tile, once the column's running
// max over the tile is final (the first pass is block_max): mneg = 15 - c max. Adds
// the weights 2^15 exp2(c (z - max)) in fp32 to zsum, keeps them as fp16 in eh, adds
// the fp16 values to hsum and their products with the logits to asum. All weights of a
// tile refer to the same max, so those kept for the student fold need no rescale.
__device__ __forceinline__ void teacher_weights(const float (&z)[16], float c, float mneg,
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
        // a new value for the student fold: it must re-read the packed pair rather than
        // share these conversions (their fp32 results would stay live across its sweep)
        asm volatile("" : "+v"(p));
        eh[q] = p;
    }
}

// Student block: running statistics, and the sum of the teacher's fp16 weights times
// the student logits into as.
__device__ __forceinline__ void fold_student(const float (&z)[16], Run &R, float &as,
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

// Merge the teacher record y (with its difference sum ya and weight sum yz) into x.
__device__ __forceinline__ void merge_teacher(Run &x, float &xa, float &xz, const Run &y,
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

template <bool SAME>
struct Wide {
    struct Cursor {
        const char *w, *h;       // W and H tile of the step to prefetch
        int64_t wstep, hstep;    // bytes from one panel to the next (0 past the unit's end)
        int m, kk, cnt, vt;      // model block (1 = teacher), step in the block, its length
        int vt1, nS, nT, p;
    };

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

    // Teacher block of a tile, then its student block, then the next tile's teacher
    // block; past the unit's last block the prefetches repeat its last step.
    static __device__ __forceinline__ void turn(Cursor &C, const ScoreArgs &a) {
        if (C.kk == C.cnt) {
            if (C.m == 1) {
                enter<0>(C, a, C.vt);
            } else if (C.vt + 1 < C.vt1) {
                enter<1>(C, a, C.vt + 1);
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

    // DMA Q of a step (Q < 4: W, else H) into the stage whose wave part starts at lw.
    template <int Q>
    static __device__ __forceinline__ void dma_q(const Cursor &C, const XLane &L, uint32_t lw) {
        if constexpr (Q < XDMA)
            xdma<Q * 1024>(C.w, L.voff[Q], lw);
        else
            xdma<XW_BYTES + (Q - XDMA) * 1024>(C.h, L.voff[Q - XDMA], lw);
    }

    template <int QB, int QE>
    static __device__ __forceinline__ void dmas(const Cursor &C, const XLane &L, uint32_t lw) {
        if constexpr (QB < QE) {
            dma_q<QB>(C, L, lw);
            dmas<QB + 1, QE>(C, L, lw);
        }
    }

    static __device__ __forceinline__ uint32_t stage_w(const XLane &L, int st) {
        return xring_addr() + (uint32_t)st * XSTAGE + (uint32_t)L.wid * (XDMA * 1024u);
    }

    static __device__ __forceinline__ void issue(const ScoreArgs &a, const XLane &L, Cursor &C,
                                                 int st) {
        turn(C, a);
        dmas<0, XDMA_STEP>(C, L, stage_w(L, st));
        advance(C);
    }

    template <int J>
    static __device__ __forceinline__ void read_frag(const XLane &L, int st, XFrag &F) {
        const char *stage = x_ring + st * XSTAGE;
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
            F.A[vb] = *(const bf16x8 *)(stage + L.lds_a[J] + vb * 32 * XROW);
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
            F.B[cb] = *(const bf16x8 *)(stage + L.lds_b[J] + cb * 32 * XROW);
    }

    static __device__ __forceinline__ void mma(const XFrag &F, floatx16 (&acc)[4][4]) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                acc[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.A[vb], F.B[cb],
                                                                      acc[vb][cb], 0, 0, 0);
    }

    // The 16 MFMAs of one sub-step (ZERO: the block's first, onto zero accumulators)
    // with DMAs Q0 .. Q0+NQ-1 of the refill spread between them.
    template <bool ZERO, int Q0, int NQ>
    static __device__ __forceinline__ void mma_issue(const XFrag &F, floatx16 (&acc)[4][4],
                                                     const Cursor &C, const XLane &L,
                                                     uint32_t lw) {
#define OLIVE_XMI(J_, VB_, CB_)                                                             \
        __builtin_amdgcn_sched_barrier(0);                                                \
        acc[VB_][CB_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                            \
            F.A[VB_], F.B[CB_], ZERO ? floatx16{0.f} : acc[VB_][CB_], 0, 0, 0);             \
        __builtin_amdgcn_sched_barrier(0);                                                \
        dmas<Q0 + ((J_) * NQ + 15) / 16, Q0 + ((J_) * NQ + NQ + 15) / 16>(C, L, lw);
        OLIVE_XMI(0, 0, 0)
        OLIVE_XMI(1, 0, 1)
        OLIVE_XMI(2, 0, 2)
        OLIVE_XMI(3, 0, 3)
        OLIVE_XMI(4, 1, 0)
        OLIVE_XMI(5, 1, 1)
        OLIVE_XMI(6, 1, 2)
        OLIVE_XMI(7, 1, 3)
        OLIVE_XMI(8, 2, 0)
        OLIVE_XMI(9, 2, 1)
        OLIVE_XMI(10, 2, 2)
        OLIVE_XMI(11, 2, 3)
        OLIVE_XMI(12, 3, 0)
        OLIVE_XMI(13, 3, 1)
        OLIVE_XMI(14, 3, 2)
        OLIVE_XMI(15, 3, 3)
#undef OLIVE_XMI
        __builtin_amdgcn_sched_barrier(0);
    }

    // Stage barrier of step n: this wave's DMAs of step n have landed (those of steps
    // n+1 and n+2 may be in flight) and its LDS reads of step n-1 have returned; after
    // the barrier every wave's data of step n is in LDS and no wave reads the stage of
    // step n-1, which step n+3 then refills.
    static __device__ __forceinline__ void arrive() {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_imm(XDMA_STEP * (XNST - 2)));
        compiler_fence();
        __builtin_amdgcn_s_barrier();
        compiler_fence();
    }

    // One step in stage st: meet the barrier, read sub-step 0's fragments, run the
    // previous step's sub-step 1 (P) under those reads, read sub-step 1 into P, run
    // sub-step 0. FIRST: the block's first step (no pending sub-step; sub-step 0 starts
    // the accumulators at zero).
    template <bool FIRST>
    static __device__ __forceinline__ void step(const ScoreArgs &a, const XLane &L, Cursor &C,
                                                int st, floatx16 (&acc)[4][4], XFrag &P) {
        const int pv = st == 0 ? XNST - 1 : st - 1;
        turn(C, a);
        arrive();
        const uint32_t lw = stage_w(L, pv);
        XFrag F0;
        read_frag<0>(L, st, F0);
        __builtin_amdgcn_sched_barrier(0);
        if (FIRST) {
            read_frag<1>(L, st, P);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<true, 0, 8>(F0, acc, C, L, lw);
        } else {
            mma_issue<false, 0, 4>(P, acc, C, L, lw);
            read_frag<1>(L, st, P);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<false, 4, 4>(F0, acc, C, L, lw);
        }
        advance(C);
    }

    // Add kMasked to the rows at or past V of the padded last tile (one MFMA per block:
    // A holds kMasked in k = 0 of those rows, B ones), so they drop out of every
    // statistic while the accumulators stay MFMA-only.
    static __device__ __forceinline__ void mask_tail(const XLane &L, floatx16 (&acc)[4][4],
                                                     int row0, int V) {
        bf16x8 ones, bias[4];
#pragma unroll
        for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) {
            const int v = row0 + L.wv * 128 + vb * 32 + L.l32;
#pragma unroll
            for (int e = 0; e < 8; ++e) bias[vb][e] = (__bf16)0.0f;
            if (L.h == 0 && v >= V) bias[vb][0] = (__bf16)kMasked;
        }
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                acc[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bias[vb], ones,
                                                                      acc[vb][cb], 0, 0, 0);
    }

    static __device__ __forceinline__ void run(ScoreArgs a) {
        const int t_valid = a.sched->t_valid;
        const int n_p = a.sched->n_ptiles;
        const int ns = a.sched->n_splits;
        const int n_units = a.sched->n_units;
        XLane L;
        L.lane = threadIdx.x & 63;
        L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        L.wv = L.wid & 1;
        L.wt = L.wid >> 1;
        L.h = L.lane >> 5;
        L.l32 = L.lane & 31;
        // DMA lane: 16 rows x 64 bytes per DMA, row lane/4, LDS slot lane&3 holding the
        // row's chunk (lane&3) ^ ((row >> 2) & 3) = (lane&3) ^ ((lane >> 4) & 3).
#pragma unroll
        for (int i = 0; i < XDMA; ++i)
            L.voff[i] = (uint32_t)(L.wid * XDMA * 1024 + i * 1024 + (L.lane >> 2) * XROW +
                                   (((L.lane & 3) ^ ((L.lane >> 4) & 3)) << 4));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const uint32_t lane_part =
                (uint32_t)(L.l32 * XROW + (((2 * j + L.h) ^ ((L.l32 >> 2) & 3)) << 4));
            L.lds_a[j] = (uint32_t)(L.wv * 128 * XROW) + lane_part;
            L.lds_b[j] = (uint32_t)(XW_BYTES + L.wt * 128 * XROW) + lane_part;
        }
        const int nS = a.ds / XK, nT = a.dt / XK;
        const int G = gridDim.x;
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        constexpr int SG = XSPLIT_GROUP;
        const int nsb = ns / SG, rem = ns % SG;
        const int64_t full_units = (int64_t)nsb * SG * n_p;

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            if (q < full_units) {
                const int64_t w = q % (SG * (int64_t)n_p);
                p = (int)(w / SG);
                s = (int)(q / (SG * (int64_t)n_p)) * SG + (int)(w % SG);
            } else {
                const int64_t w = q - full_units;
                p = (int)(w / rem);
                s = nsb * SG + (int)(w % rem);
            }
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);

            float ZH[4], AT[4], AS[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                stat_put(0, cb, Run{kNegInf, kNegInf, 0.f, 0x7fffffff});
                stat_put(1, cb, Run{kNegInf, kNegInf, 0.f, 0x7fffffff});
                ZH[cb] = 0.f;
                AT[cb] = 0.f;
                AS[cb] = 0.f;
            }
            uint32_t eh[4][4][8];
            floatx16 acc[4][4];

            Cursor C;
            C.vt1 = vt1;
            C.nS = nS;
            C.nT = nT;
            C.p = p;
            enter<1>(C, a, vt0);
#pragma unroll
            for (int i = 0; i < XNST - 1; ++i) issue(a, L, C, i);
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): no scalar load pending
            int st = 0;
#define OLIVE_XSTEPS(COUNT_)                                                              \
            {                                                                             \
                XFrag P;                                                                  \
                step<true>(a, L, C, st, acc, P);                                          \
                st = st + 1 == XNST ? 0 : st + 1;                                         \
                for (int k = 1; k < (COUNT_); ++k) {                                      \
                    step<false>(a, L, C, st, acc, P);                                     \
                    st = st + 1 == XNST ? 0 : st + 1;                                     \
                }                                                                         \
                mma(P, acc);                                                              \
                __builtin_amdgcn_sched_barrier(0);                                        \
            }
            for (int vt = vt0; vt < vt1; ++vt) {
                const int row0 = vt * XV;
                const int vbase = row0 + L.wv * 128 + 4 * L.h;
                OLIVE_XSTEPS(nT)
                if (row0 + XV > a.V) mask_tail(L, acc, row0, a.V);
                {
                    const float inf = opaque_inf(), one = opaque_one();
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        Run R = stat_get(1, cb);
                        const float m0 = R.best;
#pragma unroll
                        for (int vb = 0; vb < 4; ++vb) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
#pragma unroll
                            for (int r = 0; r < 16; ++r) z[r] = agpr_read(acc[vb][cb][r]);
                            (void)block_max(z, R, vbase + vb * 32, a.cT, inf);
                        }
                        // one rescale per column and tile, to the tile's max
                        const float resc = fast_exp2((m0 - R.best) * a.cT);
                        float zsum = R.z * resc, hsum = ZH[cb] * resc, asum = AT[cb] * resc;
                        AS[cb] *= resc;
                        const float mneg = fmaf(-R.best, a.cT, 15.0f);
#pragma unroll
                        for (int vb = 0; vb < 4; ++vb) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
#pragma unroll
                            for (int r = 0; r < 16; ++r) z[r] = agpr_read(acc[vb][cb][r]);
                            teacher_weights(z, a.cT, mneg, one, zsum, hsum, asum, eh[vb][cb]);
                        }
                        R.z = zsum;
                        ZH[cb] = hsum;
                        AT[cb] = asum;
                        // Pin the weighted sums here: otherwise the compiler sinks them
                        // past the student sweep, keeping the teacher logits alive (and
                        // spilled) across it.
                        asm volatile("" : "+v"(ZH[cb]), "+v"(AT[cb]), "+v"(AS[cb]));
                        stat_put(1, cb, R);
                    }
                }
                OLIVE_XSTEPS(nS)
                if (row0 + XV > a.V) mask_tail(L, acc, row0, a.V);
                {
                    const float inf = opaque_inf();
#pragma unroll
                    for (int cb = 0; cb < 4; ++cb) {
                        Run R = stat_get(0, cb);
#pragma unroll
                        for (int vb = 0; vb < 4; ++vb) {
                            __builtin_amdgcn_sched_barrier(0);
                            float z[16];
#pragma unroll
                            for (int r = 0; r < 16; ++r) z[r] = agpr_read(acc[vb][cb][r]);
                            fold_student(z, R, AS[cb], eh[vb][cb], a.cS, vbase + vb * 32, inf);
                        }
                        stat_put(0, cb, R);
                    }
                }
            }
#undef OLIVE_XSTEPS

            // The difference sums (unscaled with equal scales; the combine multiplies by
            // s), then lanes l and l+32 (same columns, interleaved rows).
            float AA[4];
            Run RS[4], RT[4];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                RS[cb] = stat_get(0, cb);
                RT[cb] = stat_get(1, cb);
                AA[cb] = SAME ? AT[cb] - AS[cb] : a.sT * AT[cb] - a.sS * AS[cb];
                Run o{__shfl_xor(RS[cb].best, 32), __shfl_xor(RS[cb].sec, 32),
                      __shfl_xor(RS[cb].z, 32), __shfl_xor(RS[cb].idx, 32)};
                float dummy = 0.f;
                merge_run(RS[cb], dummy, o, 0.f, a.cS);
                Run t{__shfl_xor(RT[cb].best, 32), __shfl_xor(RT[cb].sec, 32),
                      __shfl_xor(RT[cb].z, 32), __shfl_xor(RT[cb].idx, 32)};
                const float ta = __shfl_xor(AA[cb], 32), tz = __shfl_xor(ZH[cb], 32);
                merge_teacher(RT[cb], AA[cb], ZH[cb], t, ta, tz, a.cT);
            }
            // The two vocabulary halves (wv = 1 into wv = 0) through LDS, once the
            // trailing prefetches into the ring have landed.
            float *xs = (float *)x_ring;   // [wt][cb][l32][10]
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __builtin_amdgcn_s_barrier();
            compiler_fence();
            if (L.wv == 1 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    float *o = xs + ((L.wt * 4 + cb) * 32 + L.l32) * 10;
                    o[0] = RS[cb].best; o[1] = RS[cb].sec; o[2] = __int_as_float(RS[cb].idx);
                    o[3] = RS[cb].z;
                    o[4] = RT[cb].best; o[5] = RT[cb].sec; o[6] = __int_as_float(RT[cb].idx);
                    o[7] = RT[cb].z; o[8] = AA[cb]; o[9] = ZH[cb];
                }
            }
            compiler_fence();
            __syncthreads();
            if (L.wv == 0 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    const float *o = xs + ((L.wt * 4 + cb) * 32 + L.l32) * 10;
                    float dummy = 0.f;
                    merge_run(RS[cb], dummy, Run{o[0], o[1], o[3], __float_as_int(o[2])}, 0.f,
                              a.cS);
                    merge_teacher(RT[cb], AA[cb], ZH[cb],
                                  Run{o[4], o[5], o[7], __float_as_int(o[6])}, o[8], o[9], a.cT);
                    const int j = p * XT + L.wt * 128 + cb * 32 + L.l32;
                    if (j < t_valid) {
                        float *P = a.part;
                        const int64_t ps = a.pstride;
                        P[(F_BEST_S * MAX_SPLITS + s) * ps + j] = RS[cb].best;
                        P[(F_SEC_S * MAX_SPLITS + s) * ps + j] = RS[cb].sec;
                        P[(F_IDX_S * MAX_SPLITS + s) * ps + j] = __int_as_float(RS[cb].idx);
                        P[(F_Z_S * MAX_SPLITS + s) * ps + j] = RS[cb].z;
                        P[(F_BEST_T * MAX_SPLITS + s) * ps + j] = RT[cb].best;
                        P[(F_SEC_T * MAX_SPLITS + s) * ps + j] = RT[cb].sec;
                        P[(F_IDX_T * MAX_SPLITS + s) * ps + j] = __int_as_float(RT[cb].idx);
                        // the teacher's exp-sum carries the weights' 2^15 (exact)
                        P[(F_Z_T * MAX_SPLITS + s) * ps + j] = RT[cb].z * 0x1p-15f;
                        P[(F_A * MAX_SPLITS + s) * ps + j] = AA[cb];
                        P[(F_ZH * MAX_SPLITS + s) * ps + j] = ZH[cb];
                    }
                }
            }
            compiler_fence();
            __syncthreads();
        }
    }
};

template <bool SAME>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_wide_kernel(ScoreArgs a) {
    Wide<SAME>::run(a);
}

// [V][d] bf16 weights -> K-blocked panels [d/32][vpad][32] (rows V .. vpad-1 zero).
// Block (64-row group, panel); thread: row t/4, 16-byte chunk t&3.
__global__ void __launch_bounds__(256)
panel_w_kernel(const uint16_t *__restrict__ w, int64_t V, int d, int64_t vpad,
               uint16_t *__restrict__ out) {
    const int64_t v = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
    const int pnl = blockIdx.y, q = threadIdx.x & 3;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (v < V) val = *(const uint4 *)(w + v * d + pnl * XK + q * 8);
    *(uint4 *)(out + ((int64_t)pnl * vpad + v) * XK + q * 8) = val;
}

// The compacted hidden rows of a call -> K-blocked panels [d/32][prow][32]: row j <
// t_valid is hidden row rowmap[j]; rows t_valid .. up to the next multiple of 256 are
// zero (the last position tile's columns past the rows).
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
    *(uint4 *)(out + ((int64_t)pnl * prow + j) * XK + q * 8) = val;
}

}  // namespace

hipError_t launch_score_wide(const ScoreArgs &a, bool same_scale, int grid, hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    if (a.ds % XK != 0 || a.dt % XK != 0 || a.dt <= 0 || a.vpad % XV != 0 || a.prow % XT != 0)
        return hipErrorInvalidValue;
    if (same_scale)
        score_wide_kernel<true><<<grid, 256, 0, st>>>(a);
    else
        score_wide_kernel<false><<<grid, 256, 0, st>>>(a);
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
