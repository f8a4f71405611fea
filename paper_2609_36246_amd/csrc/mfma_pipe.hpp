// Pieces of the bf16 MFMA operand pipeline shared by the scoring kernel and the
// GEMM kernels: operand types, the 3-stage LDS ring of (256 x 128-byte, 128 x
// 128-byte) tiles fed by global->LDS DMAs, its swizzle and wait-count encodings.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "olive_internal.hpp"

namespace olive {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BV = MFMA_BV;              // 256
constexpr int BT = MFMA_BT;              // 128
constexpr int BK = 64;                   // K elements per pipeline step
constexpr int ROWB = BK * 2;             // bytes per row per step: one 128-byte line
constexpr int WT_BYTES = BV * ROWB;      // 32 KB
constexpr int HT_BYTES = BT * ROWB;      // 16 KB
// Ring of NST LDS stages; stage i holds the W tile [256 rows x 128 B] followed by
// the H tile [128 rows x 128 B] of one K step.
constexpr int NST = 3;
constexpr int STAGE_BYTES = WT_BYTES + HT_BYTES;     // 48 KB; 3 stages = 144 KB
constexpr int W_DMA = WT_BYTES / 1024 / 4;           // 16-byte-per-lane DMAs per wave: 8
constexpr int H_DMA = HT_BYTES / 1024 / 4;           // 4
constexpr int DMA_PER_STEP = W_DMA + H_DMA;          // 12
__shared__ __attribute__((aligned(1024))) char g_ring[NST * STAGE_BYTES];

__device__ __forceinline__ uint32_t ring_addr() {
    return (uint32_t)(uintptr_t)(lds_void *)g_ring;
}

// s_waitcnt immediates (gfx9 encoding: vmcnt bits [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]): "vmcnt <= n" alone, and together with "lgkmcnt = 0".
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (0xF << 8) | (7 << 4); }
constexpr int vmcnt_lgkm0_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// 16-byte slot swizzle of a 128-byte stage row: slot = chunk ^ ((row >> 1) & 7).
// Measured on gfx950 to keep the ds_read_b128 operand fetches (32 rows x 2 chunks
// per instruction, any of the 4 sub-steps) free of bank conflicts.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Read one accumulator element where it lives (an AGPR). Issuing the read at the
// point of use keeps the register allocator from copying whole accumulator tuples
// into VGPRs ahead of the epilogue.
__device__ __forceinline__ float agpr_read(float x) {
    float y;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(y) : "a"(x));
    return y;
}

__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// One global -> LDS DMA of 16 bytes per lane: lane i's bytes land at the wave-uniform
// LDS address `l` + 16 i. Issued as inline assembly so that the compiler's wait-count
// analysis does not see an LDS write in flight (it would then wait for every LDS read
// with lgkmcnt(0)); completion is ordered by the explicit vmcnt waits and barriers of
// the pipeline. m0 is written here only: the kernel has no other m0 user.
__device__ __forceinline__ void dma16(const char *g, uint32_t la) {
    // The address is wave-uniform by construction; readfirstlane makes that explicit
    // when register pressure has moved it to a VGPR.
    la = __builtin_amdgcn_readfirstlane(la);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    // s_nop: one wait state between the m0 write and the DMA that reads it.
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(la), "v"(g)
                 : "memory", "m0");
#pragma clang diagnostic pop
}

// The same DMA with the LDS address `la` + OFF formed in m0 by one scalar add, from a
// 64-bit lane address (dma16_at) or from a wave-uniform base in SGPRs plus a 32-bit
// lane offset (dma16_sv: the address add happens in the load, not in a VALU op).
template <int OFF>
__device__ __forceinline__ void dma16_at(const char *g, uint32_t la) {
    la = __builtin_amdgcn_readfirstlane(la);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_add_u32 m0, %0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(la), "v"(g), "i"(OFF)
                 : "memory", "m0", "scc");
#pragma clang diagnostic pop
}

template <int OFF>
__device__ __forceinline__ void dma16_sv(const char *base, uint32_t voff, uint32_t la) {
    la = __builtin_amdgcn_readfirstlane(la);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(la), "v"(voff), "s"(base), "i"(OFF)
                 : "memory", "m0", "scc");
#pragma clang diagnostic pop
}

}  // namespace olive
