// Generic scoring kernel: any hidden width, fp32 or bf16 inputs, fp32 FMA.
//
// Used for fp32 batches and for shapes the MFMA kernel does not take (a hidden
// width that is not a multiple of 128, or V < 256). One workgroup scores 16
// compacted rows against one vocabulary split: for each 256-wide vocabulary chunk
// it forms the logits of both models in registers (one vocabulary entry per
// thread), stages them through LDS, and folds them into per-lane running
// statistics (max, second max, lowest argmax, rescaled exp-sums and the teacher-
// and student-weighted logit differences of the two KL directions), merged across
// lanes at the end of the split.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

constexpr int SK = 64;  // hidden-width chunk staged in LDS

template <typename E, bool HAS_T>
__global__ void __launch_bounds__(256)
score_simple_kernel(ScoreArgs a, int same_scale) {
    __shared__ float hsh[SIMPLE_BT][SK];
    __shared__ float zsh[2][SIMPLE_BT][SIMPLE_VC + 1];
    __shared__ int64_t rowg[SIMPLE_BT];
    const int t_valid = a.sched->t_valid;
    const int ns = a.sched->n_splits;
    const int n_units = a.sched->n_units;
    const int u = blockIdx.x;
    if (u >= n_units) return;
    const int p = u / ns, s = u % ns;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int c0 = (int)((int64_t)a.n_vtiles * s / ns);
    const int c1 = (int)((int64_t)a.n_vtiles * (s + 1) / ns);
    if (tid < SIMPLE_BT) {
        int j = p * SIMPLE_BT + tid;
        rowg[tid] = j < t_valid ? (int64_t)(a.rowmap[j] & 0x7fffffffu) : -1;
    }
    const E *hs = (const E *)a.hs;
    const E *ht = (const E *)a.ht;
    const E *ws = (const E *)a.ws;
    const E *wt = (const E *)a.wt;
    Stat st_s[4], st_t[4];
    float acc_a[4], acc_b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st_s[i] = stat_identity();
        st_t[i] = stat_identity();
        acc_a[i] = 0.f;
        acc_b[i] = 0.f;
    }

    for (int c = c0; c < c1; ++c) {
        const int64_t v = (int64_t)c * SIMPLE_VC + tid;
        const bool vok = v < a.V;
#pragma unroll 1
        for (int model = 0; model < (HAS_T ? 2 : 1); ++model) {
            const E *h = model ? ht : hs;
            const E *w = model ? wt : ws;
            const int d = model ? a.dt : a.ds;
            float acc[SIMPLE_BT];
#pragma unroll
            for (int r = 0; r < SIMPLE_BT; ++r) acc[r] = 0.f;
            for (int k0 = 0; k0 < d; k0 += SK) {
                __syncthreads();
                for (int e = tid; e < SIMPLE_BT * SK; e += 256) {
                    int r = e / SK, kk = e % SK;
                    int64_t g = rowg[r];
                    hsh[r][kk] = (g >= 0 && k0 + kk < d) ? load_elem(h, g * d + k0 + kk) : 0.f;
                }
                __syncthreads();
                if (vok) {
                    const int kn = d - k0 < SK ? d - k0 : SK;
                    for (int kk = 0; kk < kn; ++kk) {
                        float wv = load_elem(w, v * d + k0 + kk);
#pragma unroll
                        for (int r = 0; r < SIMPLE_BT; ++r) acc[r] = fmaf(hsh[r][kk], wv, acc[r]);
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < SIMPLE_BT; ++r) zsh[model][r][tid] = acc[r];
        }
        __syncthreads();
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int r = wid * 4 + rr;
            for (int q = 0; q < SIMPLE_VC / 64; ++q) {
                const int vv = lane + 64 * q;
                const int64_t vg = (int64_t)c * SIMPLE_VC + vv;
                if (vg >= a.V) break;
                const float zs = zsh[0][r][vv];
                const float zt = HAS_T ? zsh[1][r][vv] : 0.f;
                float dlt = 0.f;
                if (HAS_T) {
#pragma clang fp contract(off)
                    dlt = same_scale ? (zt - zs) : (a.sT * zt - a.sS * zs);
                }
                Stat &S = st_s[rr];
                if (zs > S.best) {
                    float rs = fast_exp2((S.best - zs) * a.cS);
                    S.z = S.z * rs + 1.f; S.sec = S.best; S.best = zs; S.idx = (int32_t)vg;
                    if (HAS_T) acc_b[rr] = acc_b[rr] * rs - dlt;
                } else {
                    const float e = fast_exp2((zs - S.best) * a.cS);
                    S.z += e; S.sec = fmaxf(S.sec, zs);
                    if (HAS_T) acc_b[rr] = fmaf(-e, dlt, acc_b[rr]);
                }
                if (HAS_T) {
                    Stat &Q = st_t[rr];
                    if (zt > Q.best) {
                        float rt = fast_exp2((Q.best - zt) * a.cT);
                        Q.z = Q.z * rt + 1.f; acc_a[rr] = acc_a[rr] * rt + dlt;
                        Q.sec = Q.best; Q.best = zt; Q.idx = (int32_t)vg;
                    } else {
                        float e = fast_exp2((zt - Q.best) * a.cT);
                        Q.z += e; acc_a[rr] = fmaf(e, dlt, acc_a[rr]); Q.sec = fmaxf(Q.sec, zt);
                    }
                }
            }
        }
    }
    // Lane merge (fixed xor tree: deterministic) and write-out.
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
        for (int off = 32; off > 0; off >>= 1) {
            Stat o;
            o.best = __shfl_xor(st_s[rr].best, off);
            o.sec = __shfl_xor(st_s[rr].sec, off);
            o.idx = __shfl_xor(st_s[rr].idx, off);
            o.z = __shfl_xor(st_s[rr].z, off);
            const float ob = __shfl_xor(acc_b[rr], off);
            stat_merge(st_s[rr], acc_b[rr], o, ob, a.cS);
            if (HAS_T) {
                Stat q;
                q.best = __shfl_xor(st_t[rr].best, off);
                q.sec = __shfl_xor(st_t[rr].sec, off);
                q.idx = __shfl_xor(st_t[rr].idx, off);
                q.z = __shfl_xor(st_t[rr].z, off);
                float qa = __shfl_xor(acc_a[rr], off);
                stat_merge(st_t[rr], acc_a[rr], q, qa, a.cT);
            }
        }
        const int j = p * SIMPLE_BT + wid * 4 + rr;
        if (lane == 0 && j < t_valid) {
            float *P = a.part;
            const int64_t ps = a.pstride;
            P[(F_BEST_S * MAX_SPLITS + s) * ps + j] = st_s[rr].best;
            P[(F_SEC_S * MAX_SPLITS + s) * ps + j] = st_s[rr].sec;
            P[(F_IDX_S * MAX_SPLITS + s) * ps + j] = __int_as_float(st_s[rr].idx);
            P[(F_Z_S * MAX_SPLITS + s) * ps + j] = st_s[rr].z;
            if (HAS_T) {
                P[(F_BEST_T * MAX_SPLITS + s) * ps + j] = st_t[rr].best;
                P[(F_SEC_T * MAX_SPLITS + s) * ps + j] = st_t[rr].sec;
                P[(F_IDX_T * MAX_SPLITS + s) * ps + j] = __int_as_float(st_t[rr].idx);
                P[(F_Z_T * MAX_SPLITS + s) * ps + j] = st_t[rr].z;
                P[(F_A * MAX_SPLITS + s) * ps + j] = acc_a[rr];
                P[(F_B * MAX_SPLITS + s) * ps + j] = acc_b[rr];
            }
        }
    }
}

hipError_t launch_score_simple(const ScoreArgs &a, bool bf16, bool has_t, int64_t max_units,
                               hipStream_t st) {
    if (max_units <= 0) return hipSuccess;
    dim3 grid((unsigned)max_units);
    int same = (a.sS == a.sT) ? 1 : 0;
    if (bf16) {
        if (has_t) score_simple_kernel<uint16_t, true><<<grid, 256, 0, st>>>(a, same);
        else score_simple_kernel<uint16_t, false><<<grid, 256, 0, st>>>(a, same);
    } else {
        if (has_t) score_simple_kernel<float, true><<<grid, 256, 0, st>>>(a, same);
        else score_simple_kernel<float, false><<<grid, 256, 0, st>>>(a, same);
    }
    return hipGetLastError();
}

}  // namespace olive
