// Phase lock of the persistent workgroups of one XCD, for the scoring kernels whose
// work units are ordered so that the workgroups of an XCD share weight and hidden-row
// panel steps through that XCD's L2.
//
// The sharing holds only while the workgroups run within some 15 K steps of one
// another. Left alone they drift 20 to 40 steps apart, the bytes fetched from the
// fabric double and, under the power limit, the clock drops. Every workgroup sweeps the
// same K steps in every vocabulary tile, so what matters is the phase: the tile start
// time modulo the tile period D.
//
// At each tile start, wavefront 0 publishes its start time (s_memrealtime ticks, a
// vector store into g_phase) and compares it with the start times its XCD peers had
// published one tile earlier, which a DMA issued at its previous tile start copied into
// x_phase (so the read costs no latency). If the peer furthest behind trails by more
// than D/32 (some 6 steps of 32 K elements on long_rollout), it sleeps the excess, at
// most D/64 per tile. The wait is bounded by the clock alone, never by another
// workgroup's progress, so no workgroup can block another. The entries steer timing
// only: stale or foreign values (another launch on the device) cost at most one bounded
// wait per tile, never a result.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfma_pipe.hpp"

namespace olive {
namespace {

constexpr int PH_MAX_GRID = 2048;
__device__ uint32_t g_phase[PH_MAX_GRID];   // per workgroup: its last tile start
__shared__ uint32_t x_phase[64];            // wavefront 0's copy of its XCD peers' entries

struct PhaseClock {
    uint32_t prev, d;   // this workgroup's last tile start; its tile period (0: unknown)
};

// Where the lock applies: a grid the unit order maps onto the 8 XCDs, with room in
// g_phase, and tiles long enough (steps of 32 K elements) for the clock to resolve.
__device__ __forceinline__ bool phase_lock_on(int G, int k32_steps_per_tile) {
    return (G & 7) == 0 && G <= PH_MAX_GRID && k32_steps_per_tile >= 32;
}

// The peer a lane follows: lanes 0..31 take the XCD's slots (blockIdx.x & 7 is the
// XCD under round-robin dispatch); -1 for this workgroup itself and for lanes past the
// grid or past 32.
__device__ __forceinline__ int phase_peer(int G) {
    const int lane = (int)(threadIdx.x & 63), b = (int)blockIdx.x;
    const int j = lane * 8 + (b & 7);
    return (lane < 32 && j < G && j != b) ? j : -1;
}

// Wavefront 0 at a tile start. WAIT_LEVEL is the kernel's own ring wait (its DMAs in
// flight after a stage barrier): the copy issued at the previous tile start has then
// landed, since the wave has issued at least one K step's DMAs after it.
template <int WAIT_LEVEL>
__device__ __forceinline__ void phase_lock(PhaseClock &P, int G) {
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0_imm(WAIT_LEVEL));
    compiler_fence();
    const int j = phase_peer(G);
    const uint32_t peer_t = x_phase[threadIdx.x & 63];
    const uint32_t now = (uint32_t)__builtin_amdgcn_s_memrealtime();
    const int D = (int)P.d;
    int lag = 0;
    if (D > 0 && j >= 0) {
        // the peer's entry predates the copy, about one tile ago: dt ~ -2D .. -D
        int dt = (int)(peer_t - now);
        if (dt > -3 * D && dt <= 0) {
            dt += D;
            if (dt < 0) dt += D;
            if (dt < 0) dt += D;
            if (dt < D / 2) lag = dt;   // the peer reaches this phase dt ticks later
        }
    }
    // the largest lag over the 32 peer lanes, in scalar registers
    int lmax = 0;
#pragma unroll
    for (int i = 0; i < 32; ++i) lmax = max(lmax, __builtin_amdgcn_readlane(lag, i));
    const int w = min(lmax - (D >> 5), D >> 6);
    if (w > 0) {
        for (int it = 0; it < 4096 && (int)((uint32_t)__builtin_amdgcn_s_memrealtime() - now) < w;
             ++it)
            __builtin_amdgcn_s_sleep(1);
    }
    const uint32_t t1 = (uint32_t)__builtin_amdgcn_s_memrealtime();
    if (threadIdx.x == 0)
        __hip_atomic_store(&g_phase[blockIdx.x], t1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    P.d = P.prev ? t1 - P.prev : 0u;
    P.prev = t1;
    // copy the peers' entries (lanes without a peer copy this workgroup's own) for the
    // next tile start: 4 bytes per lane into x_phase
    const uint32_t voff = (uint32_t)(j >= 0 ? j : (int)blockIdx.x) * 4u;
    const uint32_t la = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void *)x_phase);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2 sc1"
                 :
                 : "s"(la), "v"(voff), "s"((const void *)g_phase)
                 : "memory", "m0");
#pragma clang diagnostic pop
}

}  // namespace
}  // namespace olive
