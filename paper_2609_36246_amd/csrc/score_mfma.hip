// Fused bf16 scoring kernel for gfx950 (MFMA 32x32x16, LDS ring fed by direct
// global->LDS loads).
//
// A workgroup (4 wavefronts) owns a tile of 256 vocabulary rows x 128 compacted
// positions and sweeps the vocabulary tiles of one split for one position tile.
// For every vocabulary tile it accumulates the student logits (K = d_S) and then
// the teacher logits (K = d_T) of the same 256 x 128 block in fp32 registers --
// the [T, V] logits never reach HBM -- and folds both blocks into per-lane running
// statistics: max, second max, lowest argmax and rescaled exp-sum per model, plus
// the teacher-weighted difference sum that yields KL(teacher || student).
//
// Operand roles are swapped (weights are the MFMA A/row operand, hidden states the
// B/column operand) so that every lane owns whole position columns and holds 64
// vocabulary entries of each: the softmax statistics reduce inside registers and
// only lanes l / l+32 and the two vocabulary-half wavefronts need merging at the
// end of a split.
//
// Pipeline: K advances 64 elements (one 128-byte line per row) per step; each step's
// W tile (256 x 128 B) and H tile (128 x 128 B) land in one of 3 LDS stages through
// global_load_lds_dwordx4, issued two steps ahead. Whole-line requests matter: the
// path from L2 to a CU is bound by the number of requests, and 64-byte row pieces
// would halve the bytes per request. Stage rows are XOR-swizzled at 16-byte
// granularity so the ds_read_b128 operand fetches are bank-conflict free. Hidden
// widths must be multiples of 64 (one step).
//
// The grid is persistent (one workgroup per CU). Work units (position tile,
// split) are ordered so that the 32 workgroups of one XCD share 8 position tiles x
// 4 splits at any time and the 8 XCDs share the same 4 splits: W tiles are reused
// across position tiles through L2 and the infinity cache, H tiles across splits.
#include <hip/hip_runtime.h>

#include "fold.hpp"
#include "mfma_pipe.hpp"
#include "phase_lock.hpp"
#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

// Vocabulary splits that consecutive work units cycle through: the 32 workgroups of an
// XCD then share 32 / OLIVE_SPLIT_GROUP position tiles x OLIVE_SPLIT_GROUP splits.
#ifndef OLIVE_SPLIT_GROUP
#define OLIVE_SPLIT_GROUP 4
#endif

struct Lane {
    int lane, wid, wv, wt, h, l32;
    int ldsoff[4];          // operand fetch offsets for the four k16 sub-steps
    uint32_t wvoff[2][2];   // per model, per W DMA parity: lane part of row * rowbytes + chunk * 16
    const char *hp[2][H_DMA];   // per model, per H DMA: pointer to the row chunk
};

// The largest logits a lane keeps of one position column (4), as packed keys in
// descending order (0 = empty): the high 16 bits are the logit's order-preserving
// code rounded toward -inf (the logit lies in [lb(code), lb(code + 1))), the low 16
// bits 0xFFFF minus the lane's ordinal of the row (vocabulary tile of the split x 64 +
// 32-row block x 16 + row of the block), so that among equal codes the lower
// vocabulary index ranks first. Every logit the lane dropped is below lb(c + 1) for c
// the larger code of the 4th key and of the floor key. The lists only narrow the
// field: the top-K sets are decided on exact logits later.
struct Top4 {
    uint32_t k[4];
    uint32_t f;      // floor key: the largest key a block dropped outright (0 = none)
};

// Middle of three unsigned values (one v_med3_u32).
__device__ __forceinline__ uint32_t umed3(uint32_t a, uint32_t b, uint32_t c) {
    const uint32_t lo = a < b ? a : b, hi = a < b ? b : a;
    const uint32_t m = hi < c ? hi : c;
    return lo > m ? lo : m;
}

template <bool HAS_T, bool SAME, bool REV, bool TOPK>
struct Kernel {
    // Issue cursor: the next step to prefetch. Wave-uniform: its model block (vocabulary
    // tile vt, model m, step kk of the block's cnt), the W tile pointer at the step's K
    // offset and the K offset into the hidden rows; per lane: the W row offsets of the 8
    // W DMAs and the hidden-row pointers of the 4 H DMAs, both for model m. A step only
    // adds `inc` (one 128-byte line) to the two offsets; the lane parts change with the
    // model block, twice per vocabulary tile. Past the unit's last step `inc` is 0 and
    // the trailing prefetches repeat the last issued step.
    struct Cursor {
        const char *w;
        int64_t hoff, inc;
        int vt, m, kk, cnt;
        int vt1, nS, nT;
        uint32_t wq[W_DMA];
        const char *hq[H_DMA];
    };

    // Point the cursor at step 0 of block (vt, M).
    template <int M>
    static __device__ __forceinline__ void enter(Cursor &C, const ScoreArgs &a, const Lane &L,
                                                 int vt) {
        const int rb = M ? 2 * a.dt : 2 * a.ds;   // bytes per weight row
        const int row0 = vt * BV < a.V - BV ? vt * BV : a.V - BV;
        C.vt = vt;
        C.m = M;
        C.kk = 0;
        C.cnt = M ? C.nT : C.nS;
        C.inc = ROWB;
        C.w = (const char *)(M ? a.wt : a.ws) + (int64_t)row0 * rb;
        C.hoff = 0;
#pragma unroll
        for (int q = 0; q < W_DMA; ++q) C.wq[q] = L.wvoff[M][q & 1] + (uint32_t)(q * 8 * rb);
#pragma unroll
        for (int i = 0; i < H_DMA; ++i) C.hq[i] = L.hp[M][i];
    }

    // Once the current model block is fully issued, move to the next one: the teacher
    // block of the same tile after a student block, else the next tile's student
    // block; past the unit's last tile, stay on the last issued step (still in L2).
    static __device__ __forceinline__ void turn(Cursor &C, const ScoreArgs &a, const Lane &L) {
        if (C.kk == C.cnt) {
            if (HAS_T && C.m == 0) {
                enter<1>(C, a, L, C.vt);
            } else if (C.vt + 1 < C.vt1) {
                enter<0>(C, a, L, C.vt + 1);
            } else {
                C.w -= ROWB;
                C.hoff -= ROWB;
                C.inc = 0;
                C.cnt = 0x7fffffff;
            }
        }
    }

    static __device__ __forceinline__ void advance(Cursor &C) {
        C.w += C.inc;
        C.hoff += C.inc;
        C.kk += 1;
    }

    // DMA Q of a step (Q < 8: W rows 8Q .. 8Q+7 of the wave's slice; else H DMA Q-8)
    // into the stage whose wave parts start at lw (W) and lh (H).
    template <int Q>
    static __device__ __forceinline__ void dma_q(const Cursor &C, uint32_t lw, uint32_t lh) {
        if constexpr (Q < W_DMA)
            dma16_sv<Q * 1024>(C.w, C.wq[Q], lw);
        else
            dma16_at<(Q - W_DMA) * 1024>(C.hq[Q - W_DMA] + C.hoff, lh);
    }

    // LDS targets of this wave's DMAs into ring stage st.
    static __device__ __forceinline__ uint32_t stage_w(const Lane &L, int st) {
        return ring_addr() + (uint32_t)st * STAGE_BYTES + (uint32_t)L.wid * (W_DMA * 1024u);
    }
    static __device__ __forceinline__ uint32_t stage_h(const Lane &L, int st) {
        return ring_addr() + (uint32_t)st * STAGE_BYTES + WT_BYTES +
               (uint32_t)L.wid * (H_DMA * 1024u);
    }

    // All 12 DMAs of the cursor's step into stage st (the pipeline prologue).
    static __device__ __forceinline__ void issue(const ScoreArgs &a, const Lane &L, Cursor &C,
                                                 int st) {
        turn(C, a, L);
        const uint32_t lw = stage_w(L, st), lh = stage_h(L, st);
        dmas<0, DMA_PER_STEP>(C, lw, lh);
        advance(C);
    }

    // Operand fragments of one k16 sub-step: 4 W row blocks, 2 H column blocks.
    struct Frag {
        bf16x8 A[4], B[2];
    };

    template <int SUB>
    static __device__ __forceinline__ void read_frag(const Lane &L, int st, Frag &F) {
        const char *stage = g_ring + st * STAGE_BYTES;
        const char *wb = stage + L.wv * 128 * ROWB + L.ldsoff[SUB];
        const char *hb = stage + WT_BYTES + L.wt * 64 * ROWB + L.ldsoff[SUB];
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) F.A[vb] = *(const bf16x8 *)(wb + vb * 32 * ROWB);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) F.B[cb] = *(const bf16x8 *)(hb + cb * 32 * ROWB);
    }

    static __device__ __forceinline__ void mma(const Frag &F, floatx16 (&acc)[4][2]) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
                acc[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.A[vb], F.B[cb],
                                                                      acc[vb][cb], 0, 0, 0);
    }

    template <int QB, int QE>
    static __device__ __forceinline__ void dmas(const Cursor &C, uint32_t lw, uint32_t lh) {
        if constexpr (QB < QE) {
            dma_q<QB>(C, lw, lh);
            dmas<QB + 1, QE>(C, lw, lh);
        }
    }

    // The 8 MFMAs of one sub-step with DMAs Q0 .. Q0+NQ-1 of the step's refill spread
    // between them. Each 1 KB DMA holds the CU's address path for about 16 cycles, so
    // the refill is spread over the whole step: issued in a burst, the DMAs back up
    // and stall the wave in front of its next MFMA.
    template <int Q0, int NQ>
    static __device__ __forceinline__ void mma_issue(const Frag &F, floatx16 (&acc)[4][2],
                                                     const Cursor &C, uint32_t lw, uint32_t lh) {
#define OLIVE_MI(J_, VB_, CB_)                                                             \
        __builtin_amdgcn_sched_barrier(0);                                               \
        acc[VB_][CB_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.A[VB_], F.B[CB_],        \
                                                                acc[VB_][CB_], 0, 0, 0); \
        __builtin_amdgcn_sched_barrier(0);                                               \
        dmas<Q0 + ((J_) * NQ + 7) / 8, Q0 + ((J_) * NQ + NQ + 7) / 8>(C, lw, lh);
        OLIVE_MI(0, 0, 0)
        OLIVE_MI(1, 0, 1)
        OLIVE_MI(2, 1, 0)
        OLIVE_MI(3, 1, 1)
        OLIVE_MI(4, 2, 0)
        OLIVE_MI(5, 2, 1)
        OLIVE_MI(6, 3, 0)
        OLIVE_MI(7, 3, 1)
#undef OLIVE_MI
        __builtin_amdgcn_sched_barrier(0);
    }

    // Stage barrier at the start of step n: wait until this wave's DMAs of step n have
    // landed (those of step n+1 may stay in flight) and its LDS reads of step n-1 have
    // returned, then barrier. After it every wave's data of step n is in LDS and no
    // wave reads the stage of step n-1 any more, so step n+2 may be issued into it.
    static __device__ __forceinline__ void arrive() {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_imm(DMA_PER_STEP));
        compiler_fence();
        __builtin_amdgcn_s_barrier();
        compiler_fence();
    }

    // One pipeline step n in stage `st`: meet the stage barrier, prefetch the cursor's
    // step (n+2) into the stage of step n-1, then run the step's four k16 sub-steps,
    // each one's LDS reads issued under the previous one's MFMAs. With PEND, the last
    // sub-step of step n-1 (fragments in P) runs under the first reads. On return P
    // holds this step's last sub-step, still to be run. Every step issues its 12 DMAs
    // (past the end of a unit, those of its last step again), so no DMA sits under a
    // branch.
    template <bool PEND>
    static __device__ __forceinline__ void step(const ScoreArgs &a, const Lane &L, Cursor &C,
                                                int st, floatx16 (&acc)[4][2], Frag &P) {
        const int pv = st == 0 ? NST - 1 : st - 1;
        turn(C, a, L);
        arrive();
        const uint32_t lw = stage_w(L, pv), lh = stage_h(L, pv);
        Frag F0, F1, F2;
        read_frag<0>(L, st, F0);
        __builtin_amdgcn_sched_barrier(0);
        if (PEND) {
            mma_issue<0, 3>(P, acc, C, lw, lh);
            read_frag<1>(L, st, F1);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<3, 3>(F0, acc, C, lw, lh);
            read_frag<2>(L, st, F2);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<6, 3>(F1, acc, C, lw, lh);
            read_frag<3>(L, st, P);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<9, 3>(F2, acc, C, lw, lh);
        } else {
            read_frag<1>(L, st, F1);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<0, 4>(F0, acc, C, lw, lh);
            read_frag<2>(L, st, F2);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<4, 4>(F1, acc, C, lw, lh);
            read_frag<3>(L, st, P);
            __builtin_amdgcn_sched_barrier(0);
            mma_issue<8, 4>(F2, acc, C, lw, lh);
        }
        advance(C);
    }

    // The K sweep of one work unit: for every vocabulary tile vt0 .. vt1-1 the student
    // block (nS steps into accS), then the teacher block (nT steps into accT), then
    // tile_end(vt, row0) on the finished accumulators. Prefetch runs two steps ahead
    // through the cursor, across block and tile ends. LOCK: phase-lock the XCD's
    // workgroups at tile starts (the scoring pass; the backward's passes, whose tile ends
    // hold more live state, leave it off).
    template <bool LOCK, class TileEnd>
    static __device__ __forceinline__ void sweep(const ScoreArgs &a, const Lane &L, int vt0,
                                                 int vt1, int nS, int nT,
                                                 floatx16 (&accS)[4][2], floatx16 (&accT)[4][2],
                                                 TileEnd &&tile_end) {
        Cursor C;
        C.vt1 = vt1;
        C.nS = nS;
        C.nT = nT;
        enter<0>(C, a, L, vt0);
        // Prologue: steps 0 .. NST-2 into stages 0 .. NST-2; the first step's barrier
        // waits for step 0.
#pragma unroll
        for (int i = 0; i < NST - 1; ++i) issue(a, L, C, i);
        // Drain scalar loads before the loops: an SMEM load still pending at a loop
        // header would force lgkmcnt(0) (full LDS waits) inside every step.
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
        int st = 0;   // ring stage of the current step
        // A model block of COUNT_ steps: the first step has no pending sub-step, the
        // block's last sub-step runs after the loop.
#define OLIVE_STEPS(ACC_, COUNT_)                                                        \
        {                                                                                \
            Frag P;                                                                      \
            step<false>(a, L, C, st, ACC_, P);                                           \
            st = st + 1 == NST ? 0 : st + 1;                                             \
            for (int k = 1; k < (COUNT_); ++k) {                                         \
                step<true>(a, L, C, st, ACC_, P);                                        \
                st = st + 1 == NST ? 0 : st + 1;                                         \
            }                                                                            \
            mma(P, ACC_);                                                                \
            __builtin_amdgcn_sched_barrier(0);                                           \
        }
        // Phase lock of the XCD's workgroups (phase_lock.hpp); the first two tiles of a
        // unit only measure the period.
        const int G = gridDim.x;
        const bool lock = LOCK && phase_lock_on(G, 2 * (nS + nT));
        PhaseClock PH{0u, 0u};
        for (int vt = vt0; vt < vt1; ++vt) {
            if (lock && L.wid == 0) phase_lock<DMA_PER_STEP * (NST - 2)>(PH, G);
            // The last tile, when V is not a multiple of 256, is shifted back to end at
            // V; its rows below vt*BV were covered by the previous tile.
            const int row0 = (vt * BV < a.V - BV) ? vt * BV : a.V - BV;
            zero_acc(accS, accT);
            OLIVE_STEPS(accS, nS)
            if (HAS_T) OLIVE_STEPS(accT, nT)
            tile_end(vt, row0);
        }
#undef OLIVE_STEPS
    }

    // Add kMasked to the rows of a shifted last tile whose vocabulary index is below
    // vlo, with one MFMA per block (A: kMasked in k = 0 of masked rows, B: ones), so the
    // accumulators are only ever touched by MFMAs.
    static __device__ __forceinline__ void mask_mma(const Lane &L, floatx16 (&accS)[4][2],
                                                    floatx16 (&accT)[4][2], int row0, int vlo) {
        bf16x8 ones, bias[4];
#pragma unroll
        for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) {
            const int v = row0 + L.wv * 128 + vb * 32 + L.l32;   // A-operand row of this lane
#pragma unroll
            for (int e = 0; e < 8; ++e) bias[vb][e] = (__bf16)0.0f;
            if (L.h == 0 && v < vlo) bias[vb][0] = (__bf16)kMasked;
        }
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                accS[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bias[vb], ones,
                                                                       accS[vb][cb], 0, 0, 0);
                if (HAS_T)
                    accT[vb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bias[vb], ones,
                                                                           accT[vb][cb], 0, 0, 0);
            }
    }

    // Fold the lane's 2 columns x 64 rows of both models, block by block.
    // LISTS: also offer the blocks to the lanes' top-K lists.
    template <bool LISTS>
    static __device__ __forceinline__ void fold(const floatx16 (&accS)[4][2],
                                                const floatx16 (&accT)[4][2], Run (&RS)[2],
                                                Run (&RT)[2], float (&A)[2], float (&Bq)[2],
                                                Top4 (&KS)[2], Top4 (&KT)[2], const ScoreArgs &a,
                                                int vbase, int lvt) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int vb = 0; vb < 4; ++vb) {
                // Keep the scheduler from hoisting accumulator reads of later blocks.
                __builtin_amdgcn_sched_barrier(0);
                float zs[16], zt[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    zs[r] = agpr_read(accS[vb][cb][r]);
                    if (HAS_T) zt[r] = agpr_read(accT[vb][cb][r]);
                }
                fold_block<HAS_T && REV, SAME>(zs, RS[cb], Bq[cb], zt, a.cS, a.sS, a.sT,
                                                 vbase + vb * 32);
                if (HAS_T)
                    fold_block<true, SAME>(zt, RT[cb], A[cb], zs, a.cT, a.sT, a.sS, vbase + vb * 32);
                if (LISTS) {
                    const uint32_t tie0 = 0xFFFFu - (uint32_t)(lvt * 64 + vb * 16);
                    topk_block(zs, KS[cb], tie0);
                    topk_block(zt, KT[cb], tie0);
                }
            }
    }

    // The same for entries of other lanes: (value descending, index ascending) order by
    // comparison. Returns the value pushed off the end.
    template <int N>
    static __device__ __forceinline__ float topk_insert_lex(float (&v)[N], int (&ix)[N], float x,
                                                           int xi) {
#pragma unroll
        for (int j = 0; j < N; ++j) {
            const bool gt = x > v[j] || (x == v[j] && xi < ix[j]);
            const float nv = gt ? x : v[j];
            const int ni = gt ? xi : ix[j];
            x = gt ? v[j] : x;
            xi = gt ? ix[j] : xi;
            v[j] = nv;
            ix[j] = ni;
        }
        return x;
    }

    // Offer one 32-row block (16 values per lane) to a lane's list: the block's three
    // largest keys by a running v_med3_u32 network, the two largest inserted, the
    // third raising the floor key. Every key the lane drops is then at most the list's
    // 4th or some block's third, so the floor bounds it. tie0 = 0xFFFF minus the
    // ordinal of the block's first row.
    static __device__ __forceinline__ void topk_block(const float (&z)[16], Top4 &K,
                                                      uint32_t tie0) {
        uint32_t b1 = 0u, b2 = 0u, b3 = 0u;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t x = (f2ord(z[r]) & 0xFFFF0000u) | (tie0 - (uint32_t)r);
            b3 = umed3(x, b2, b3);
            b2 = umed3(x, b1, b2);
            b1 = b1 > x ? b1 : x;
        }
        K.f = K.f > b3 ? K.f : b3;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            uint32_t x = t ? b2 : b1;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t hi = x > K.k[j] ? x : K.k[j];
                x = x > K.k[j] ? K.k[j] : x;
                K.k[j] = hi;
            }
        }
    }

    static __device__ __forceinline__ void zero_acc(floatx16 (&accS)[4][2],
                                                    floatx16 (&accT)[4][2]) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                accS[vb][cb] = floatx16{0.f};
                if (HAS_T) accT[vb][cb] = floatx16{0.f};
            }
    }

    static __device__ __forceinline__ void run(ScoreArgs a) {
        const int t_valid = a.sched->t_valid;
        const int64_t n_scored = TOPK ? a.sched->n_scored : 0;
        const int n_p = a.sched->n_ptiles;
        const int ns = a.sched->n_splits;
        const int n_units = a.sched->n_units;
        Lane L;
        L.lane = threadIdx.x & 63;
        L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
        L.wv = L.wid & 1;
        L.wt = L.wid >> 1;
        L.h = L.lane >> 5;
        L.l32 = L.lane & 31;
#pragma unroll
        for (int s = 0; s < 4; ++s) L.ldsoff[s] = L.l32 * ROWB + (((2 * s + L.h) ^ swz(L.l32)) << 4);
        const int nS = a.ds / BK, nT = HAS_T ? a.dt / BK : 0;
        // W DMA i of wave wid fills stage rows R = wid*64 + 8i + lane/8, slot lane&7 with
        // chunk (lane&7) ^ swz(R); swz(R) depends on i only through its parity.
#pragma unroll
        for (int par = 0; par < 2; ++par) {
            const int R0 = L.wid * 8 * W_DMA + (L.lane >> 3);
            const int ch = (L.lane & 7) ^ swz(R0 + 8 * par);
            L.wvoff[0][par] = (uint32_t)(R0 * a.ds * 2 + ch * 16);
            L.wvoff[1][par] = HAS_T ? (uint32_t)(R0 * a.dt * 2 + ch * 16) : 0u;
        }
        const int G = gridDim.x;
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, OLIVE_SPLIT_GROUP, p, s);
            // H DMA i of wave wid fills stage rows R = wid*32 + 8i + lane/8.
#pragma unroll
            for (int i = 0; i < H_DMA; ++i) {
                const int R = (L.wid * H_DMA + i) * 8 + (L.lane >> 3);
                const int ch = (L.lane & 7) ^ swz(R);
                int j = p * BT + R;
                j = j < t_valid ? j : t_valid - 1;
                const int64_t g = a.rowmap[j] & 0x7fffffffu;
                L.hp[0][i] = (const char *)a.hs + g * a.ds * 2 + ch * 16;
                L.hp[1][i] = HAS_T ? (const char *)a.ht + g * a.dt * 2 + ch * 16 : nullptr;
            }
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);

            Run RS[2], RT[2];
            float AA[2] = {0.f, 0.f}, BB[2] = {0.f, 0.f};
            Top4 KS[2], KT[2];
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int e = 0; e < 4; ++e) { KS[cb].k[e] = 0u; KT[cb].k[e] = 0u; }
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) { KS[cb].f = 0u; KT[cb].f = 0u; }
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                RS[cb] = Run{kNegInf, kNegInf, 0.f, 0x7fffffff};
                RT[cb] = Run{kNegInf, kNegInf, 0.f, 0x7fffffff};
            }
            floatx16 accS[4][2], accT[4][2];
#pragma unroll
            for (int vb = 0; vb < 4; ++vb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    accS[vb][cb] = floatx16{0.f};
                    accT[vb][cb] = floatx16{0.f};
                }

            // After each tile: the last tile, when V is not a multiple of 256, is shifted
            // back to end at V, and one more MFMA adds kMasked to its rows below vt*BV
            // (the logit is absorbed), so they drop out of every statistic and the fold
            // needs no masking.
            // Top-K lists only where they are used: the scored rows are compacted first,
            // so only position tiles starting below n_scored hold any.
            const bool lists = TOPK && (int64_t)p * BT < n_scored;
            if (lists) {
                sweep<true>(a, L, vt0, vt1, nS, nT, accS, accT, [&](int vt, int row0) {
                    if (row0 != vt * BV) mask_mma(L, accS, accT, row0, vt * BV);
                    fold<true>(accS, accT, RS, RT, AA, BB, KS, KT, a,
                               row0 + L.wv * 128 + 4 * L.h, vt - vt0);
                });
            } else {
                sweep<true>(a, L, vt0, vt1, nS, nT, accS, accT, [&](int vt, int row0) {
                    if (row0 != vt * BV) mask_mma(L, accS, accT, row0, vt * BV);
                    fold<false>(accS, accT, RS, RT, AA, BB, KS, KT, a,
                                row0 + L.wv * 128 + 4 * L.h, vt - vt0);
                });
            }

            // Merge lanes l and l+32 (same columns, interleaved vocabulary rows).
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                Run o{__shfl_xor(RS[cb].best, 32), __shfl_xor(RS[cb].sec, 32),
                      __shfl_xor(RS[cb].z, 32), __shfl_xor(RS[cb].idx, 32)};
                const float ob = REV ? __shfl_xor(BB[cb], 32) : 0.f;
                merge_run(RS[cb], BB[cb], o, ob, a.cS);
                if (HAS_T) {
                    Run q2{__shfl_xor(RT[cb].best, 32), __shfl_xor(RT[cb].sec, 32),
                           __shfl_xor(RT[cb].z, 32), __shfl_xor(RT[cb].idx, 32)};
                    float qa = __shfl_xor(AA[cb], 32);
                    merge_run(RT[cb], AA[cb], q2, qa, a.cT);
                }
            }
            // Top-K: each lane decodes its keys to (lower end of the value's bucket,
            // vocabulary index); lanes l and l+32 combine their top-4 lists into a top-8
            // (nothing is dropped); the floor bounds everything either lane dropped.
            float Q8v[2][2][8], Qfl[2][2];
            int Q8i[2][2][8];
            if (lists) {
#pragma unroll
                for (int m = 0; m < 2; ++m)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) {
                        const Top4 &K = m ? KT[cb] : KS[cb];
                        float kv[4];
                        int ki[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t key = K.k[e];
                            const uint32_t ord = 0xFFFFu - (key & 0xFFFFu);
                            const int vt = vt0 + (int)(ord >> 6);
                            const int r = (int)(ord & 15u);
                            const int row0 = (vt * BV < a.V - BV) ? vt * BV : a.V - BV;
                            kv[e] = key ? key_lb(key) : kMasked;
                            ki[e] = key ? row0 + L.wv * 128 + 4 * L.h + (int)((ord >> 4) & 3u) * 32 +
                                              8 * (r >> 2) + (r & 3)
                                        : 0x7fffffff;
                            Q8v[m][cb][e] = kv[e]; Q8i[m][cb][e] = ki[e];
                            Q8v[m][cb][4 + e] = kMasked; Q8i[m][cb][4 + e] = 0x7fffffff;
                        }
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            topk_insert_lex<8>(Q8v[m][cb], Q8i[m][cb], __shfl_xor(kv[e], 32),
                                               __shfl_xor(ki[e], 32));
                        const uint32_t fk = K.k[3] > K.f ? K.k[3] : K.f;
                        const float f = fk ? key_ub(fk) : kMasked;
                        Qfl[m][cb] = max2(f, __shfl_xor(f, 32));
                    }
            }
            // Merge the two vocabulary halves (wv = 1 into wv = 0) through LDS, once
            // the trailing prefetches into the stages have landed.
            float *xs = (float *)g_ring;   // [wt][cb][l32][10]
            float *xk = xs + 2 * 2 * 32 * 10;   // top-K: [wt][cb][l32][model][17]
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __builtin_amdgcn_s_barrier();
            compiler_fence();
            if (L.wv == 1 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    float *o = xs + ((L.wt * 2 + cb) * 32 + L.l32) * 10;
                    o[0] = RS[cb].best; o[1] = RS[cb].sec; o[2] = __int_as_float(RS[cb].idx);
                    o[3] = RS[cb].z;
                    o[4] = RT[cb].best; o[5] = RT[cb].sec; o[6] = __int_as_float(RT[cb].idx);
                    o[7] = RT[cb].z; o[8] = AA[cb]; o[9] = BB[cb];
                    if (lists) {
#pragma unroll
                        for (int m = 0; m < 2; ++m) {
                            float *q = xk + (((L.wt * 2 + cb) * 32 + L.l32) * 2 + m) * 17;
#pragma unroll
                            for (int e = 0; e < 8; ++e) {
                                q[e] = Q8v[m][cb][e];
                                q[8 + e] = __int_as_float(Q8i[m][cb][e]);
                            }
                            q[16] = Qfl[m][cb];
                        }
                    }
                }
            }
            compiler_fence();
            __syncthreads();
            if (L.wv == 0 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const float *o = xs + ((L.wt * 2 + cb) * 32 + L.l32) * 10;
                    Run ys{o[0], o[1], o[3], __float_as_int(o[2])};
                    merge_run(RS[cb], BB[cb], ys, REV ? o[9] : 0.f, a.cS);
                    if (HAS_T) {
                        Run yt{o[4], o[5], o[7], __float_as_int(o[6])};
                        merge_run(RT[cb], AA[cb], yt, o[8], a.cT);
                    }
                    const int j = p * BT + L.wt * 64 + cb * 32 + L.l32;
                    if (j < t_valid) {
                        float *P = a.part;
                        const int64_t ps = a.pstride;
                        P[(F_BEST_S * MAX_SPLITS + s) * ps + j] = RS[cb].best;
                        P[(F_SEC_S * MAX_SPLITS + s) * ps + j] = RS[cb].sec;
                        P[(F_IDX_S * MAX_SPLITS + s) * ps + j] = __int_as_float(RS[cb].idx);
                        P[(F_Z_S * MAX_SPLITS + s) * ps + j] = RS[cb].z;
                        if (HAS_T) {
                            P[(F_BEST_T * MAX_SPLITS + s) * ps + j] = RT[cb].best;
                            P[(F_SEC_T * MAX_SPLITS + s) * ps + j] = RT[cb].sec;
                            P[(F_IDX_T * MAX_SPLITS + s) * ps + j] = __int_as_float(RT[cb].idx);
                            P[(F_Z_T * MAX_SPLITS + s) * ps + j] = RT[cb].z;
                            P[(F_A * MAX_SPLITS + s) * ps + j] = AA[cb];
                            if (REV) P[(F_B * MAX_SPLITS + s) * ps + j] = BB[cb];
                            if (lists) {
                                // the other half's top-8 into this one's: the 8 dropped
                                // raise the floor
#pragma unroll
                                for (int m = 0; m < 2; ++m) {
                                    const float *q =
                                        xk + (((L.wt * 2 + cb) * 32 + L.l32) * 2 + m) * 17;
                                    float fl = max2(Qfl[m][cb], q[16]);
#pragma unroll
                                    for (int e = 0; e < 8; ++e) {
                                        // a dropped entry's value lies below its bucket's end
                                        const float x = topk_insert_lex<8>(
                                            Q8v[m][cb], Q8i[m][cb], q[e], __float_as_int(q[8 + e]));
                                        fl = max2(fl, x == kMasked ? x : key_ub(f2ord(x)));
                                    }
#pragma unroll
                                    for (int e = 0; e < 8; ++e) {
                                        P[((F_TK + m * TK_FIELDS + e) * MAX_SPLITS + s) * ps + j] =
                                            Q8v[m][cb][e];
                                        P[((F_TK + m * TK_FIELDS + 8 + e) * MAX_SPLITS + s) * ps +
                                          j] = __int_as_float(Q8i[m][cb][e]);
                                    }
                                    P[((F_TK + m * TK_FIELDS + 16) * MAX_SPLITS + s) * ps + j] = fl;
                                }
                            }
                        }
                    }
                }
            }
            compiler_fence();
            __syncthreads();
        }
    }

    // Element (t, v) of the K-blocked dz_t panels [vp/64][chunk][64].
    static __device__ __forceinline__ int64_t dzt_at(const DzArgs &z, int t, int v) {
        return ((int64_t)(v >> 6) * z.chunk + t) * 64 + (v & 63);
    }

    // Logit-gradient pass of the backward: the same units and steps over the scored
    // rows [c0, c0 + chunk) of the call (compacted, region only), with the fold
    // replaced by g = (w_ce + w_kl) p_S - w_ce onehot(y) - w_kl p_T, p_X = exp(s_X z_X -
    // lse_X) with the forward pass's normalisers, stored as bf16 (round to nearest
    // even) into dz_t (K-blocked panels [v/64][row][64]), the operand of both products
    // (the dW product reads it transposed; launch_zero_tail clears its K padding).
    static __device__ __forceinline__ void run_dz(ScoreArgs a, DzArgs z) {
        const int t_all = a.sched->t_valid - z.c0;
        const int t_rows = t_all < 0 ? 0 : (t_all < z.chunk ? t_all : z.chunk);
        const int n_p = (t_rows + BT - 1) / BT;
        const int G = gridDim.x;
        const int ns = pass_splits(n_p, a.n_vtiles, G);
        const int64_t n_units = (int64_t)n_p * ns;
        Lane L;
        L.lane = threadIdx.x & 63;
        L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        L.wv = L.wid & 1;
        L.wt = L.wid >> 1;
        L.h = L.lane >> 5;
        L.l32 = L.lane & 31;
#pragma unroll
        for (int s = 0; s < 4; ++s) L.ldsoff[s] = L.l32 * ROWB + (((2 * s + L.h) ^ swz(L.l32)) << 4);
        const int nS = a.ds / BK, nT = HAS_T ? a.dt / BK : 0;
#pragma unroll
        for (int par = 0; par < 2; ++par) {
            const int R0 = L.wid * 8 * W_DMA + (L.lane >> 3);
            const int ch = (L.lane & 7) ^ swz(R0 + 8 * par);
            L.wvoff[0][par] = (uint32_t)(R0 * a.ds * 2 + ch * 16);
            L.wvoff[1][par] = HAS_T ? (uint32_t)(R0 * a.dt * 2 + ch * 16) : 0u;
        }
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;
        const float wsum = z.w_ce + z.w_kl;

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, OLIVE_SPLIT_GROUP, p, s);
#pragma unroll
            for (int i = 0; i < H_DMA; ++i) {
                const int R = (L.wid * H_DMA + i) * 8 + (L.lane >> 3);
                const int ch = (L.lane & 7) ^ swz(R);
                int t = p * BT + R;
                t = t < t_rows ? t : t_rows - 1;
                const int64_t g = a.rowmap[z.c0 + t] & 0x7fffffffu;
                L.hp[0][i] = (const char *)a.hs + g * a.ds * 2 + ch * 16;
                L.hp[1][i] = HAS_T ? (const char *)a.ht + g * a.dt * 2 + ch * 16 : nullptr;
            }
            // the lane's two columns: scored row, normalisers (log2 domain), target
            int tcol[2];
            bool ok[2];
            float l2s[2], l2t[2];
            int ycol[2];
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                tcol[cb] = p * BT + L.wt * 64 + cb * 32 + L.l32;
                ok[cb] = tcol[cb] < t_rows;
                const int j = z.c0 + (ok[cb] ? tcol[cb] : 0);
                const int64_t g = a.rowmap[j] & 0x7fffffffu;
                l2s[cb] = ok[cb] ? z.lse[2 * (int64_t)j] * kLog2e : 0.f;
                l2t[cb] = ok[cb] && HAS_T ? z.lse[2 * (int64_t)j + 1] * kLog2e : 0.f;
                ycol[cb] = ok[cb] ? z.targets[g] : -1;
            }
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);
            floatx16 accS[4][2], accT[4][2];
            // g of rows v0 .. v0+3 (v0 = the lane's row of 32-row block vb, quad rq) at
            // column cb, as two packed bf16 pairs (zero for columns past the scored rows)
            auto grad4 = [&](int vb, int cb, int rq, int v0) {
                float gr[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float zs = agpr_read(accS[vb][cb][4 * rq + e]);
                    gr[e] = wsum * fast_exp2(fmaf(zs, a.cS, -l2s[cb]));
                    if (HAS_T) {
                        const float zt = agpr_read(accT[vb][cb][4 * rq + e]);
                        gr[e] = fmaf(-z.w_kl, fast_exp2(fmaf(zt, a.cT, -l2t[cb])), gr[e]);
                    }
                    gr[e] -= (v0 + e == ycol[cb]) ? z.w_ce : 0.f;
                }
                uint2 w;
                w.x = ok[cb] ? pack_bf16x2(gr[0], gr[1]) : 0u;
                w.y = ok[cb] ? pack_bf16x2(gr[2], gr[3]) : 0u;
                return w;
            };
            sweep<false>(a, L, vt0, vt1, nS, nT, accS, accT, [&](int vt, int row0) {
                const int vlo = vt * BV;
                const int vw0 = row0 + L.wv * 128;   // the wave's first row
                if (row0 == vlo) {
                    // Whole 16-byte pieces: lanes l and l+32 hold rows 8q .. 8q+3 and
                    // 8q+4 .. 8q+7 of one column for quads q = 2k, 2k+1; one swap of
                    // their upper and lower halves gives each 8 consecutive rows.
#pragma unroll
                    for (int vb = 0; vb < 4; ++vb) {
#pragma unroll
                        for (int cb = 0; cb < 2; ++cb) {
                            __builtin_amdgcn_sched_barrier(0);
                            uint2 w[4];
#pragma unroll
                            for (int rq = 0; rq < 4; ++rq)
                                w[rq] = grad4(vb, cb, rq, vw0 + vb * 32 + 8 * rq + 4 * L.h);
#pragma unroll
                            for (int k = 0; k < 2; ++k) {
                                const auto X = __builtin_amdgcn_permlane32_swap(
                                    w[2 * k].x, w[2 * k + 1].x, false, false);
                                const auto Y = __builtin_amdgcn_permlane32_swap(
                                    w[2 * k].y, w[2 * k + 1].y, false, false);
                                const int v = vw0 + vb * 32 + 16 * k + 8 * L.h;
                                if (ok[cb])
                                    *(uint4 *)(z.dz_t + dzt_at(z, tcol[cb], v)) =
                                        make_uint4(X[0], Y[0], X[1], Y[1]);
                            }
                        }
                    }
                    return;
                }
                // A shifted last tile (V not a multiple of 256) starts at V - 256, which
                // may be any row: its rows below vlo were stored by the previous tile, and
                // its 4-row groups may straddle vlo and sit off 8-byte alignment in dz_t,
                // so it stores row by row.
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int vb = 0; vb < 4; ++vb) {
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int rq = 0; rq < 4; ++rq) {
                            const int v0 = vw0 + vb * 32 + 8 * rq + 4 * L.h;
                            const uint2 w = grad4(vb, cb, rq, v0);
                            const uint16_t q[4] = {(uint16_t)w.x, (uint16_t)(w.x >> 16),
                                                   (uint16_t)w.y, (uint16_t)(w.y >> 16)};
                            const int t = tcol[cb];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                if (v0 + e < vlo) continue;
                                if (ok[cb]) z.dz_t[dzt_at(z, t, v0 + e)] = q[e];
                            }
                        }
                    }
            });
            // every DMA landed and every wave is done with the ring before the next
            // unit's prologue refills it
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __builtin_amdgcn_s_barrier();
            compiler_fence();
        }
    }

    // Jensen-Shannon pass over the scored rows [0, n_scored) (compacted first by every
    // forward call), from the forward pass's log-normalisers. With log2 probabilities
    // l_S = z_S s_S log2(e) - lse_S log2(e) and l_T likewise, the divergence of a row is
    //   JSD = 1/2 sum_v [p_S log p_S + p_T log p_T - (p_S + p_T) log((p_S + p_T) / 2)]
    //       = ln(2)/2 sum_v p_hi g(r),   p_hi = 2^max(l_S, l_T),  r = 2^-|l_S - l_T|,
    //   g(r) = (1 + r)(1 - log2(1 + r)) + r log2(r)   (0 at r = 1, 1 at r = 0),
    // a sum of non-negative terms with no rescaling (the normalisers are known). The
    // same units and K sweep as the scoring kernel recompute both models' logits; per
    // lane and column the terms add in vocabulary order, lanes l / l+32 and the two
    // vocabulary halves merge in a fixed order, and each (split, row) partial goes to
    // plane F_J for the combine.
    static __device__ __forceinline__ void run_jsd(ScoreArgs a, JsdArgs z) {
        const int64_t n_sc = a.sched->n_scored;
        const int t_valid = a.sched->t_valid;
        const int rows = (int)(n_sc < t_valid ? n_sc : t_valid);
        const int n_p = (rows + BT - 1) / BT;
        const int G = gridDim.x;
        const int ns = pass_splits(n_p, a.n_vtiles, G);
        const int64_t n_units = (int64_t)n_p * ns;
        Lane L;
        L.lane = threadIdx.x & 63;
        L.wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        L.wv = L.wid & 1;
        L.wt = L.wid >> 1;
        L.h = L.lane >> 5;
        L.l32 = L.lane & 31;
#pragma unroll
        for (int s = 0; s < 4; ++s) L.ldsoff[s] = L.l32 * ROWB + (((2 * s + L.h) ^ swz(L.l32)) << 4);
        const int nS = a.ds / BK, nT = a.dt / BK;
#pragma unroll
        for (int par = 0; par < 2; ++par) {
            const int R0 = L.wid * 8 * W_DMA + (L.lane >> 3);
            const int ch = (L.lane & 7) ^ swz(R0 + 8 * par);
            L.wvoff[0][par] = (uint32_t)(R0 * a.ds * 2 + ch * 16);
            L.wvoff[1][par] = (uint32_t)(R0 * a.dt * 2 + ch * 16);
        }
        const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
        const int my = (G & 7) == 0 ? xcd * (G >> 3) + slot : (int)blockIdx.x;

        for (int64_t q = my; q < n_units; q += G) {
            int p, s;
            unit_tile_split(q, n_p, ns, OLIVE_SPLIT_GROUP, p, s);
#pragma unroll
            for (int i = 0; i < H_DMA; ++i) {
                const int R = (L.wid * H_DMA + i) * 8 + (L.lane >> 3);
                const int ch = (L.lane & 7) ^ swz(R);
                int t = p * BT + R;
                t = t < rows ? t : rows - 1;
                const int64_t g = a.rowmap[t] & 0x7fffffffu;
                L.hp[0][i] = (const char *)a.hs + g * a.ds * 2 + ch * 16;
                L.hp[1][i] = (const char *)a.ht + g * a.dt * 2 + ch * 16;
            }
            // the lane's two columns: scored row and its normalisers in log2 units
            int tcol[2];
            bool ok[2];
            float l2s[2], l2t[2], acc[2] = {0.f, 0.f};
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                tcol[cb] = p * BT + L.wt * 64 + cb * 32 + L.l32;
                ok[cb] = tcol[cb] < rows;
                const int64_t j = ok[cb] ? tcol[cb] : 0;
                l2s[cb] = ok[cb] ? z.lse[2 * j] * kLog2e : 0.f;
                l2t[cb] = ok[cb] ? z.lse[2 * j + 1] * kLog2e : 0.f;
            }
            const int vt0 = (int)((int64_t)a.n_vtiles * s / ns);
            const int vt1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);
            floatx16 accS[4][2], accT[4][2];
            sweep<false>(a, L, vt0, vt1, nS, nT, accS, accT, [&](int vt, int row0) {
                // rows of a shifted last tile below vt * BV get -2^99 in both models:
                // p_hi = 0 there, and r stays finite
                if (row0 != vt * BV) mask_mma(L, accS, accT, row0, vt * BV);
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int vb = 0; vb < 4; ++vb) {
                        __builtin_amdgcn_sched_barrier(0);
                        float part = 0.f;
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const float ls = fmaf(agpr_read(accS[vb][cb][r]), a.cS, -l2s[cb]);
                            const float lt = fmaf(agpr_read(accT[vb][cb][r]), a.cT, -l2t[cb]);
                            const float ad = fabsf(ls - lt);
                            const float ph = fast_exp2(max2(ls, lt));
                            const float rr = fast_exp2(-ad);
                            const float one_r = 1.0f + rr;
                            const float gv = fmaf(one_r, 1.0f - fast_log2(one_r), -rr * ad);
                            part = fmaf(ph, gv, part);
                        }
                        acc[cb] += part;
                    }
            });
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) acc[cb] += __shfl_xor(acc[cb], 32);
            // the two vocabulary halves (wv = 1 into wv = 0) through LDS, once the
            // trailing prefetches into the stages have landed
            float *xs = (float *)g_ring;   // [wt][cb][l32]
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            compiler_fence();
            __builtin_amdgcn_s_barrier();
            compiler_fence();
            if (L.wv == 1 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) xs[(L.wt * 2 + cb) * 32 + L.l32] = acc[cb];
            }
            compiler_fence();
            __syncthreads();
            if (L.wv == 0 && L.h == 0) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
                    if (ok[cb])
                        a.part[(F_J * MAX_SPLITS + s) * a.pstride + tcol[cb]] =
                            acc[cb] + xs[(L.wt * 2 + cb) * 32 + L.l32];
            }
            compiler_fence();
            __syncthreads();
        }
    }
};

template <bool HAS_T, bool SAME, bool REV, bool TOPK>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_mfma_kernel(ScoreArgs a) {
    Kernel<HAS_T, SAME, REV, TOPK>::run(a);
}

template <bool HAS_T>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_dz_kernel(ScoreArgs a, DzArgs z) {
    Kernel<HAS_T, true, false, false>::run_dz(a, z);
}

__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
score_jsd_kernel(ScoreArgs a, JsdArgs z) {
    Kernel<true, true, false, false>::run_jsd(a, z);
}

hipError_t launch_score_jsd(const ScoreArgs &a, const JsdArgs &z, int grid, hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    score_jsd_kernel<<<grid, 256, 0, st>>>(a, z);
    return hipGetLastError();
}

hipError_t launch_score_dz(const ScoreArgs &a, const DzArgs &z, bool has_t, int grid,
                           hipStream_t st) {
    if (grid <= 0) return hipSuccess;
    if (has_t)
        score_dz_kernel<true><<<grid, 256, 0, st>>>(a, z);
    else
        score_dz_kernel<false><<<grid, 256, 0, st>>>(a, z);
    return hipGetLastError();
}

hipError_t launch_score_mfma(const ScoreArgs &a, bool has_t, bool same_scale, bool rev,
                             bool topk, int grid, hipStream_t st) {
    if (grid <= 0) return hipSuccess;
#define OLIVE_SCORE(S_, R_, K_) score_mfma_kernel<true, S_, R_, K_><<<grid, 256, 0, st>>>(a)
    if (has_t) {
        if (same_scale) {
            if (topk) { if (rev) OLIVE_SCORE(true, true, true); else OLIVE_SCORE(true, false, true); }
            else { if (rev) OLIVE_SCORE(true, true, false); else OLIVE_SCORE(true, false, false); }
        } else {
            if (topk) { if (rev) OLIVE_SCORE(false, true, true); else OLIVE_SCORE(false, false, true); }
            else { if (rev) OLIVE_SCORE(false, true, false); else OLIVE_SCORE(false, false, false); }
        }
    } else {
        score_mfma_kernel<false, true, false, false><<<grid, 256, 0, st>>>(a);
    }
#undef OLIVE_SCORE
    return hipGetLastError();
}

}  // namespace olive
