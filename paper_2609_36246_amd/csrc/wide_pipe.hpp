// The operand pipeline of the 256 x 256 MFMA kernels for gfx950 (the scoring kernel and
// its logit-gradient pass, the backward's dL/dh product): 4 wavefronts own a 256 x 256
// fp32 tile, wavefront w all 256 A rows of B rows 64w .. 64w+63, as 16 x 4 blocks of
// v_mfma_f32_16x16x32_bf16 in 256 AGPRs. K advances 32 elements per step. A step's A tile
// (256 rows x 64 bytes) and B tile (256 rows x 64 bytes) land in one of 3 LDS stages
// through global_load_lds_dwordx4, issued two steps ahead; the 16-byte chunk c of stage
// row r sits in slot c ^ ((r >> 1) & 3), the one XOR swizzle on 16-byte slots measured
// on gfx950 to keep the 16-row x 4-chunk operand reads free of bank conflicts. The DMA
// lanes' source offsets (XLane::voff) place the swizzle: from panels written
// pre-swizzled they are linear.
//
// A step's 64 MFMAs run in two halves of 8 A row blocks; the previous step's second half
// runs while this step's first operands are read, one read after each MFMA.
//
// The kernel supplies a policy P with its cursor type P::Cursor (fields w and h: the A
// and B tile of the step to prefetch), P::Args, and P::turn(C, a) (called before a
// step's prefetch is issued) and P::advance(C) (after).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma_pipe.hpp"
#include "olive_internal.hpp"

namespace olive {
namespace {

constexpr int XV = 256;                  // A rows (vocabulary rows) per tile
constexpr int XT = WIDE_BT;              // B rows (positions) per tile: 256
constexpr int XK = 32;                   // K elements per step: one panel row
constexpr int XROW = XK * 2;             // 64 bytes
constexpr int XW_BYTES = XV * XROW;      // 16 KB
constexpr int XH_BYTES = XT * XROW;      // 16 KB
constexpr int XNST = 3;                  // ring stages
constexpr int XSTAGE = XW_BYTES + XH_BYTES;   // 32 KB; 3 stages = 96 KB
constexpr int XDMA = 4;                  // 1 KB DMAs per wave per operand per step
constexpr int XDMA_STEP = 2 * XDMA;      // 8

__shared__ __attribute__((aligned(1024))) char x_ring[XNST * XSTAGE];

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

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct XLane {
    int lane, wid, l16, g;   // g = lane / 16: the lane's 4-row group of an output block
                             // and its 8-element K chunk of an operand fragment
    uint32_t voff[XDMA];     // per DMA i of an operand: the lane's byte offset within a
                             // 16 KB tile step (wave part and i * 1 KB included)
    uint32_t lds_a;          // operand read offset within a stage: W row l16 of block 0
    uint32_t lds_b;          // H row (position) 64 wid + l16 of block 0
};

// Operand fragments: one half of a step's A blocks (8 of the 16 row blocks), and the
// step's 4 B blocks (the wavefront's 64 positions).
struct XFragA {
    bf16x8 A[8];
};
struct XFragB {
    bf16x8 B[4];
};

__device__ __forceinline__ XLane make_lane() {
    XLane L;
    L.lane = threadIdx.x & 63;
    L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    L.l16 = L.lane & 15;
    L.g = L.lane >> 4;
    // DMA lane: 16 bytes at 16 lane of a 1 KB piece of the step's tile. The panels
    // hold every row's 16-byte chunks already in their swizzled slots (panel_w,
    // panel_h), so the copy is linear and lands swizzled.
#pragma unroll
    for (int i = 0; i < XDMA; ++i)
        L.voff[i] = (uint32_t)(L.wid * XDMA * 1024 + i * 1024 + L.lane * 16);
    // operand fragment of a 16-row block: row l16, K chunk g, in slot g ^ ((l16 >> 1) & 3)
    const uint32_t lane_part = (uint32_t)(L.l16 * XROW + ((L.g ^ ((L.l16 >> 1) & 3)) << 4));
    L.lds_a = lane_part;
    L.lds_b = (uint32_t)(XW_BYTES + L.wid * 4 * 1024) + lane_part;
    return L;
}


template <class P>
struct WidePipe {
    using Cursor = typename P::Cursor;
    using Args = typename P::Args;

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

    static __device__ __forceinline__ void issue(const Args &a, const XLane &L, Cursor &C,
                                                 int st) {
        P::turn(C, a);
        dmas<0, XDMA_STEP>(C, L, stage_w(L, st));
        P::advance(C);
    }

    // Half H of a step's A blocks (row blocks 8H .. 8H+7), and the step's B blocks.
    template <int H>
    static __device__ __forceinline__ void read_a(const XLane &L, int st, XFragA &F) {
        const char *stage = x_ring + st * XSTAGE;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            F.A[i] = *(const bf16x8 *)(stage + L.lds_a + (8 * H + i) * 1024);
    }
    static __device__ __forceinline__ void read_b(const XLane &L, int st, XFragB &F) {
        const char *stage = x_ring + st * XSTAGE;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
            F.B[cb] = *(const bf16x8 *)(stage + L.lds_b + cb * 1024);
    }

    // Operand reads interleaved with a half's MFMAs (one read after each of its first
    // MFMAs, so that the matrix pipe is fed from the step's first cycle on): RD 1 reads
    // this step's first-half A blocks and its B blocks (12), RD 2 its second-half A
    // blocks (8), RD 0 none.
    template <int RD, int J>
    static __device__ __forceinline__ void read_at(const XLane &L, const char *stage, XFragA &RA,
                                                   XFragB &RB) {
        if constexpr (RD == 1 && J < 8)
            RA.A[J] = *(const bf16x8 *)(stage + L.lds_a + J * 1024);
        else if constexpr (RD == 1 && J >= 8 && J < 12)
            RB.B[J - 8] = *(const bf16x8 *)(stage + L.lds_b + (J - 8) * 1024);
        else if constexpr (RD == 2 && J < 8)
            RA.A[J] = *(const bf16x8 *)(stage + L.lds_a + (8 + J) * 1024);
    }

    // MFMA J (0..31) of half H of a step, then its share of the refill's DMAs Q0 ..
    // Q0+NQ-1 (spread evenly over the 32) and of the interleaved reads, then MFMA J+1.
    // ZERO: onto zero accumulators (the block's first K step).
    template <int H, bool ZERO, int Q0, int NQ, int RD, int J>
    static __device__ __forceinline__ void mma_from(const XFragA &FA, const XFragB &FB,
                                                    floatx4 (&acc)[16][4], const Cursor &C,
                                                    const XLane &L, uint32_t lw,
                                                    const char *stage, XFragA &RA, XFragB &RB) {
        if constexpr (J < 32) {
            constexpr int i = J >> 2, cb = J & 3;
            __builtin_amdgcn_sched_barrier(0);
            acc[8 * H + i][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                FA.A[i], FB.B[cb], ZERO ? floatx4{0.f} : acc[8 * H + i][cb], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            read_at<RD, J>(L, stage, RA, RB);
            __builtin_amdgcn_sched_barrier(0);
            dmas<Q0 + (J * NQ + 31) / 32, Q0 + (J * NQ + NQ + 31) / 32>(C, L, lw);
            mma_from<H, ZERO, Q0, NQ, RD, J + 1>(FA, FB, acc, C, L, lw, stage, RA, RB);
        }
    }
    template <int H, bool ZERO, int Q0, int NQ, int RD = 0>
    static __device__ __forceinline__ void mma_half(const XFragA &FA, const XFragB &FB,
                                                    floatx4 (&acc)[16][4], const Cursor &C,
                                                    const XLane &L, uint32_t lw,
                                                    const char *stage, XFragA &RA, XFragB &RB) {
        mma_from<H, ZERO, Q0, NQ, RD, 0>(FA, FB, acc, C, L, lw, stage, RA, RB);
        __builtin_amdgcn_sched_barrier(0);
    }

    // Stage barrier of step n: this wave's DMAs of step n have landed (those of step
    // n+1 may be in flight) and its LDS reads of step n-1 have returned; after the
    // barrier every wave's data of step n is in LDS and no wave reads the stage of step
    // n-1, which step n+2 then refills.
    static __device__ __forceinline__ void arrive() {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_imm(XDMA_STEP * (XNST - 2)));
        compiler_fence();
        __builtin_amdgcn_s_barrier();
        compiler_fence();
    }

    // One step in stage st: meet the barrier, read the first half's A blocks and the B
    // blocks, run the previous step's second half (PA x PB) under those reads, read this
    // step's second-half A blocks into PA, run the first half. KIND 0: the block's first
    // step (no pending half; the first half starts its accumulators at zero); KIND 1:
    // its second step (the pending half starts its accumulators at zero); KIND 2: later.
    template <int KIND>
    static __device__ __forceinline__ void step(const Args &a, const XLane &L, Cursor &C,
                                                int st, floatx4 (&acc)[16][4], XFragA &PA,
                                                XFragB &PB) {
        const int pv = st == 0 ? XNST - 1 : st - 1;
        P::turn(C, a);
        arrive();
        const uint32_t lw = stage_w(L, pv);
        const char *stage = x_ring + st * XSTAGE;
        XFragA F0;
        XFragB FB;
        if (KIND == 0) {
            read_a<0>(L, st, F0);
            read_b(L, st, FB);
            read_a<1>(L, st, PA);
            __builtin_amdgcn_sched_barrier(0);
            mma_half<0, true, 0, 8>(F0, FB, acc, C, L, lw, stage, F0, FB);
        } else {
            // the previous step's second half, with this step's first reads in between
            mma_half<1, KIND == 1, 0, 4, 1>(PA, PB, acc, C, L, lw, stage, F0, FB);
            // this step's first half, with its second-half reads (into PA) in between
            mma_half<0, false, 4, 4, 2>(F0, FB, acc, C, L, lw, stage, PA, FB);
        }
        PB = FB;
        P::advance(C);
    }
};

}  // namespace
}  // namespace olive
