// Split combine, realised-token gather and finalisation (one wavefront per row).
//
// For each valid compacted row: merges the per-split partial statistics in a fixed
// order, gathers the realised token's logit of each model as a coalesced dot
// product of the hidden row with the token's weight row, and writes
//   logp_X = s_X z_X[y] - lse_X,   lse_X = s_X best_X + ln Z_X,
//   kl     = A / Z_T - lse_T + lse_S   (KL(teacher || student), in-region only),
//   kl_rev = B / Z_S - lse_S + lse_T   (KL(student || teacher), in-region only),
//   argmax_X = lowest index attaining the max,
// queueing rows whose top-2 gap is inside the fp32 error window for the exact
// re-decision of their greedy token.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

// Relative top-2 gap (in scaled logits) at or below which the greedy token is
// re-decided exactly: 2^-14 max(1, |s M|). The fp32 logits of the MFMA pass differ
// from the exact ones by rounding of the fp32 accumulation only (bf16 products are
// exact in fp32); at the widths and magnitudes of the workloads (|z| up to ~20,
// d up to 5120) that difference stays below ~1e-5, so rows whose top two are more
// than the window apart are decided correctly by the fp32 values.
constexpr float kTieWindow = 1.0f / 16384.0f;

template <typename E>
__device__ __forceinline__ float wave_dot(const E *h, const E *w, int d, int lane);

template <>
__device__ __forceinline__ float wave_dot<uint16_t>(const uint16_t *h, const uint16_t *w, int d,
                                                    int lane) {
    float acc = 0.f;
    if ((d & 7) == 0 && ((uintptr_t)h & 15) == 0 && ((uintptr_t)w & 15) == 0) {
        const uint4 *h4 = (const uint4 *)h;
        const uint4 *w4 = (const uint4 *)w;
        for (int i = lane; i < (d >> 3); i += 64) {
            uint4 x = h4[i], y = w4[i];
            uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc = fmaf(__uint_as_float(xs[q] << 16), __uint_as_float(ys[q] << 16), acc);
                acc = fmaf(__uint_as_float(xs[q] & 0xffff0000u),
                           __uint_as_float(ys[q] & 0xffff0000u), acc);
            }
        }
    } else {
        for (int k = lane; k < d; k += 64)
            acc = fmaf(bf16_bits_to_f32(h[k]), bf16_bits_to_f32(w[k]), acc);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

template <>
__device__ __forceinline__ float wave_dot<float>(const float *h, const float *w, int d, int lane) {
    float acc = 0.f;
    for (int k = lane; k < d; k += 64) acc = fmaf(h[k], w[k], acc);
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

// sum_k |h_k| |w_k| over one row pair (the rounding-bound weight of a dot product).
template <typename E>
__device__ __forceinline__ float wave_absdot(const E *h, const E *w, int d, int lane) {
    float acc = 0.f;
    for (int k = lane; k < d; k += 64)
        acc = fmaf(fabsf(load_elem(h, k)), fabsf(load_elem(w, k)), acc);
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    return acc;
}

__device__ __forceinline__ Stat load_stat(const float *P, int64_t ps, int fb, int s, int64_t j) {
    Stat r;
    r.best = P[((fb + 0) * MAX_SPLITS + s) * ps + j];
    r.sec = P[((fb + 1) * MAX_SPLITS + s) * ps + j];
    r.idx = __float_as_int(P[((fb + 2) * MAX_SPLITS + s) * ps + j]);
    r.z = P[((fb + 3) * MAX_SPLITS + s) * ps + j];
    return r;
}

__device__ __forceinline__ void wave_merge(Stat &st, float &acc, float c) {
    for (int off = 32; off > 0; off >>= 1) {
        Stat o;
        o.best = __shfl_xor(st.best, off);
        o.sec = __shfl_xor(st.sec, off);
        o.idx = __shfl_xor(st.idx, off);
        o.z = __shfl_xor(st.z, off);
        float oa = __shfl_xor(acc, off);
        stat_merge(st, acc, o, oa, c);
    }
}

// The same with a second accumulator rescaled like z (the 256 x 256 kernel's sum of
// the fp16 weights it kept, of the model whose max z follows).
__device__ __forceinline__ void wave_merge2(Stat &st, float &acc, float &acc2, float c) {
    for (int off = 32; off > 0; off >>= 1) {
        Stat o;
        o.best = __shfl_xor(st.best, off);
        o.sec = __shfl_xor(st.sec, off);
        o.idx = __shfl_xor(st.idx, off);
        o.z = __shfl_xor(st.z, off);
        const float oa = __shfl_xor(acc, off), ob = __shfl_xor(acc2, off);
        // both accumulators follow z's rescale: merge (z, acc) and (z, acc2) alike
        Stat s2 = st;
        float a2 = acc2;
        stat_merge(st, acc, o, oa, c);
        stat_merge(s2, a2, o, ob, c);
        acc2 = a2;
    }
}

__device__ __forceinline__ bool near_tie(const Stat &st, float s) {
    float gap = s * (st.best - st.sec);
    float mag = fabsf(s * st.best);
    return gap <= kTieWindow * (mag > 1.f ? mag : 1.f);
}

template <typename E, bool HAS_T>
__global__ void __launch_bounds__(256)
combine_kernel(ScoreArgs a, int same_scale, const int32_t *__restrict__ targets,
               int32_t *__restrict__ err, float *__restrict__ logp_s, float *__restrict__ logp_t,
               int32_t *__restrict__ am_s, int32_t *__restrict__ am_t, float *__restrict__ kl,
               float *__restrict__ kl_rev, float *__restrict__ logp_tmp,
               float *__restrict__ lse_out, int32_t *__restrict__ flagged, int flag_cap) {
    const int lane = threadIdx.x & 63;
    const int64_t j = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    Sched *sched = const_cast<Sched *>(a.sched);
    if (j >= sched->t_valid) return;
    const uint32_t rm = a.rowmap[j];
    const int64_t g = rm & 0x7fffffffu;
    const bool inr = (rm >> 31) != 0;
    const int32_t y = targets[g];
    if (y < 0 || y >= a.V) {
        if (lane == 0) {
            atomicOr(err, ERR_TARGET);
            const float qnan = __builtin_nanf("");
            if (logp_s) logp_s[g] = qnan;
            if (logp_tmp) logp_tmp[g] = qnan;
            if (HAS_T && logp_t) logp_t[g] = qnan;
            if (am_s) am_s[g] = -1;
            if (HAS_T && am_t) am_t[g] = -1;
            if (HAS_T && kl) kl[g] = inr ? qnan : 0.f;
            if (HAS_T && kl_rev) kl_rev[g] = inr ? qnan : 0.f;
            if (lse_out) { lse_out[j * 2] = qnan; lse_out[j * 2 + 1] = qnan; }
        }
        return;
    }
    const E *hs = (const E *)a.hs;
    const E *ws = (const E *)a.ws;
    const float zy_s = wave_dot<E>(hs + g * a.ds, ws + (int64_t)y * a.ds, a.ds, lane);
    float zy_t = 0.f;
    if (HAS_T) {
        const E *ht = (const E *)a.ht;
        const E *wt = (const E *)a.wt;
        zy_t = wave_dot<E>(ht + g * a.dt, wt + (int64_t)y * a.dt, a.dt, lane);
    }
    const int ns = sched->n_splits;
    Stat ss = stat_identity(), st = stat_identity();
    float acc_a = 0.f, acc_b = 0.f, acc_zh = 0.f;
    if (lane < ns) {
        ss = load_stat(a.part, a.pstride, F_BEST_S, lane, j);
        if (HAS_T) {
            st = load_stat(a.part, a.pstride, F_BEST_T, lane, j);
            if (kl) acc_a = a.part[(F_A * MAX_SPLITS + lane) * a.pstride + j];
            if (kl_rev) acc_b = a.part[(F_B * MAX_SPLITS + lane) * a.pstride + j];
            if (a.wide) acc_zh = a.part[(F_ZH * MAX_SPLITS + lane) * a.pstride + j];
        }
    }
    // the 256 x 256 kernel's fp16 weight sums follow the model whose weights it kept
    const bool zh_s = HAS_T && a.wide == 2, zh_t = HAS_T && a.wide == 1;
    if (zh_s) wave_merge2(ss, acc_b, acc_zh, a.cS);
    else wave_merge(ss, acc_b, a.cS);
    if (HAS_T) {
        if (zh_t) wave_merge2(st, acc_a, acc_zh, a.cT);
        else wave_merge(st, acc_a, a.cT);
    }
    // Every lane now holds the merged statistics.
    int fl = (am_s && near_tie(ss, a.sS)) ? 1 : 0;
    if (HAS_T) fl |= (am_t && near_tie(st, a.sT)) ? 2 : 0;
    float theta_s = 0.f, theta_t = 0.f;
    if (fl) {
        // Lower bound of the exact max: fp32 max minus its rounding bound.
        if (fl & 1) {
            float za = wave_absdot<E>(hs + g * a.ds, ws + (int64_t)ss.idx * a.ds, a.ds, lane);
            theta_s = ss.best - (float)a.ds * (1.0f / 8388608.0f) * za;
        }
        if (HAS_T && (fl & 2)) {
            const E *ht = (const E *)a.ht;
            const E *wt = (const E *)a.wt;
            float za = wave_absdot<E>(ht + g * a.dt, wt + (int64_t)st.idx * a.dt, a.dt, lane);
            theta_t = st.best - (float)a.dt * (1.0f / 8388608.0f) * za;
        }
    }
    if (lane != 0) return;
    const float lse_s = a.sS * ss.best + fast_log2(ss.z) * kLn2;
    if (lse_out) lse_out[j * 2] = lse_s;
    const float lp_s = a.sS * zy_s - lse_s;
    if (logp_s) logp_s[g] = lp_s;
    if (logp_tmp) logp_tmp[g] = lp_s;
    if (am_s) am_s[g] = ss.idx;
    if (HAS_T) {
        const float lse_t = a.sT * st.best + fast_log2(st.z) * kLn2;
        if (lse_out) lse_out[j * 2 + 1] = lse_t;
        if (logp_t) logp_t[g] = a.sT * zy_t - lse_t;
        if (am_t) am_t[g] = st.idx;
        if (kl) {
            // the teacher-weighted mean of the logit difference: A / Z_T, or with the
            // 256 x 256 kernel's fp16 weights A / (their sum)
            float an = same_scale ? a.sT * acc_a : acc_a;
            float v = an / (zh_t ? acc_zh : st.z) - lse_t + lse_s;
            kl[g] = inr ? v : 0.f;
        }
        if (kl_rev) {
            // KL(student || teacher) = sum p_S (s_S zS - s_T zT) - lse_S + lse_T, or with
            // the 256 x 256 kernel's fp16 student weights B / (their sum)
            float bn = same_scale ? a.sS * acc_b : acc_b;
            float v = bn / (zh_s ? acc_zh : ss.z) - lse_s + lse_t;
            kl_rev[g] = inr ? v : 0.f;
        }
    }
    if (fl && flagged) {
        int q = atomicAdd(&sched->n_flagged, 1);
        if (q < flag_cap) {
            flagged[4 * q] = (int32_t)j;
            flagged[4 * q + 1] = fl;
            flagged[4 * q + 2] = __float_as_int(theta_s);
            flagged[4 * q + 3] = __float_as_int(theta_t);
        }
    }
}

// Jensen-Shannon outputs (one thread per compacted row): the scored rows [0, n_scored)
// sum their split partials in split order and scale by ln(2)/2; other valid rows get
// +0.0. A scored row whose normalisers are NaN (bad target) stays NaN.
__global__ void __launch_bounds__(256)
jsd_combine_kernel(ScoreArgs a, int grid, float *__restrict__ jsd) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const Sched *sched = a.sched;
    const int t_valid = sched->t_valid;
    if (j >= t_valid) return;
    const int64_t n_sc = sched->n_scored;
    const int rows = (int)(n_sc < t_valid ? n_sc : t_valid);
    const int64_t g = a.rowmap[j] & 0x7fffffffu;
    if (j >= rows) {
        jsd[g] = 0.f;
        return;
    }
    const int ns = pass_splits((rows + MFMA_BT - 1) / MFMA_BT, a.n_vtiles, grid);
    float sum = 0.f;
    for (int s = 0; s < ns; ++s) sum += a.part[(F_J * MAX_SPLITS + s) * a.pstride + j];
    jsd[g] = 0.5f * kLn2 * sum;
}

// Normalisers of the cross-entropy pass that forms its own (one wavefront per scored row
// of the chunk): the split records (max m_s, weight sum z_s relative to m_s) merged in a
// fixed order, lse = s_S M + ln sum_s z_s exp2(c_S (m_s - M)) into lse_out[j][0]; the
// realised token y, and its gradient w_ce (p_y - 1) from the exact-order dot product
// z_y (the rescale writes it in place of the stored weight). A target out of range sets
// the error word and makes the row's normaliser NaN, as the forward combine does.
__global__ void __launch_bounds__(256)
dz_lse_kernel(ScoreArgs a, DzArgs z, int grid, float *__restrict__ lse_out,
              int32_t *__restrict__ err) {
    const int lane = threadIdx.x & 63;
    const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int t_all = a.sched->t_valid - z.c0;
    const int t_rows = t_all < 0 ? 0 : (t_all < z.chunk ? t_all : z.chunk);
    if (t >= t_rows) return;
    const int64_t j = (int64_t)z.c0 + t;
    const int ns = pass_splits((t_rows + WIDE_BT - 1) / WIDE_BT, a.n_vtiles, grid);
    float m = kNegInf, zz = 0.f;
    if (lane < ns) {
        m = a.part[(F_BEST_S * MAX_SPLITS + lane) * a.pstride + j];
        zz = a.part[(F_Z_S * MAX_SPLITS + lane) * a.pstride + j];
    }
    float M = m;
    for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
    zz = lane < ns ? zz * fast_exp2((m - M) * a.cS) : 0.f;
    for (int off = 32; off > 0; off >>= 1) zz += __shfl_xor(zz, off);
    const int64_t g = a.rowmap[j] & 0x7fffffffu;
    const int32_t y = z.targets[g];
    const bool ok = y >= 0 && y < a.V;
    float zy = 0.f;
    if (ok)
        zy = wave_dot<uint16_t>((const uint16_t *)a.hs + g * a.ds,
                                (const uint16_t *)a.ws + (int64_t)y * a.ds, a.ds, lane);
    if (lane != 0) return;
    const float lse = ok ? a.sS * M + fast_log2(zz) * kLn2 : __builtin_nanf("");
    if (!ok) atomicOr(err, ERR_TARGET);
    lse_out[2 * j] = lse;
    z.yrow[t] = ok ? y : -1;
    z.gy[t] = z.w_ce * (fast_exp2((a.sS * zy - lse) * kLog2e) - 1.f);
}

// The gradient of that pass in place: each stored weight w (fp16, 2^15 exp2(c (z - m))
// with m the running max of its tile) becomes 2^-15 w_ce w exp(s m - lse) = w_ce p in
// bf16 (round to nearest even), the realised token's entry w_ce (p_y - 1). Rows at or
// past V and columns past the chunk's rows are left as they are. One 16-byte piece
// (8 entries of one panel row) per thread and step.
__global__ void __launch_bounds__(256)
dz_rescale_kernel(ScoreArgs a, DzArgs z, const float *__restrict__ lse) {
    const int t_all = a.sched->t_valid - z.c0;
    const int t_rows = t_all < 0 ? 0 : (t_all < z.chunk ? t_all : z.chunk);
    const int np = (int)(z.vp / 64);
    const int64_t n = (int64_t)np * t_rows * 8;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * 256) {
        const int64_t P = i / ((int64_t)t_rows * 8);
        const int t = (int)((i / 8) % t_rows), c = (int)(i % 8);
        const int v0 = (int)(P * 64) + 8 * c;
        if (v0 >= a.V) continue;
        const float l2 = lse[2 * ((int64_t)z.c0 + t)] * kLog2e;
        const float mc = z.mref[(int64_t)(v0 >> 8) * z.chunk + t] * a.cS;
        const float f = z.w_ce * 0x1p-15f * fast_exp2(mc - l2);
        uint16_t *q = z.dz_t + ((P * z.chunk + t) * 64 + 8 * c);
        const uint4 in = *(const uint4 *)q;
        const uint32_t wv[4] = {in.x, in.y, in.z, in.w};
        float gv[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const _Float16 lo = __builtin_bit_cast(_Float16, (uint16_t)(wv[e] & 0xffffu));
            const _Float16 hi = __builtin_bit_cast(_Float16, (uint16_t)(wv[e] >> 16));
            gv[2 * e] = (float)lo * f;
            gv[2 * e + 1] = (float)hi * f;
        }
        const int y = z.yrow[t];
        if (y >= v0 && y < v0 + 8) gv[y - v0] = z.gy[t];
        // entries at or past V keep their zeros
        const int nv = a.V - v0 < 8 ? a.V - v0 : 8;
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (e >= nv) gv[e] = 0.f;
        *(uint4 *)q = make_uint4(pack_bf16x2(gv[0], gv[1]), pack_bf16x2(gv[2], gv[3]),
                                 pack_bf16x2(gv[4], gv[5]), pack_bf16x2(gv[6], gv[7]));
    }
}

hipError_t launch_dz_lse(const ScoreArgs &a, const DzArgs &z, int grid, float *lse_out,
                         int32_t *err, hipStream_t st) {
    if (z.chunk <= 0 || !lse_out || !z.gy || !z.yrow || !a.part) return hipErrorInvalidValue;
    dz_lse_kernel<<<(unsigned)((z.chunk + 3) / 4), 256, 0, st>>>(a, z, grid, lse_out, err);
    return hipGetLastError();
}

hipError_t launch_dz_rescale(const ScoreArgs &a, const DzArgs &z, const float *lse,
                             hipStream_t st) {
    if (z.chunk <= 0 || z.vp % 64 != 0 || !z.dz_t || !z.mref || !lse) return hipErrorInvalidValue;
    const int64_t most = z.vp / 64 * (int64_t)z.chunk * 8;   // pieces of a full chunk
    const int64_t blocks = (most + 255) / 256 < 8192 ? (most + 255) / 256 : 8192;
    dz_rescale_kernel<<<(unsigned)blocks, 256, 0, st>>>(a, z, lse);
    return hipGetLastError();
}

hipError_t launch_jsd_combine(const ScoreArgs &a, float *jsd, int grid, int64_t max_rows,
                              hipStream_t st) {
    if (max_rows <= 0) return hipSuccess;
    jsd_combine_kernel<<<(unsigned)((max_rows + 255) / 256), 256, 0, st>>>(a, grid, jsd);
    return hipGetLastError();
}

hipError_t launch_combine(const ScoreArgs &a, bool bf16, bool has_t, bool same_scale,
                          const int32_t *targets, int32_t *err, float *logp_s, float *logp_t,
                          int32_t *am_s, int32_t *am_t, float *kl, float *kl_rev, float *logp_tmp,
                          float *lse_out, int32_t *flagged, int flag_cap, int64_t max_rows,
                          hipStream_t st) {
    if (max_rows <= 0) return hipSuccess;
    dim3 grid((unsigned)((max_rows + 3) / 4));
    int same = same_scale ? 1 : 0;
#define OLIVE_COMBINE(E_, T_)                                                                \
    combine_kernel<E_, T_><<<grid, 256, 0, st>>>(a, same, targets, err, logp_s, logp_t, am_s, \
                                                 am_t, kl, kl_rev, logp_tmp, lse_out, flagged,   \
                                                 flag_cap)
    if (bf16) {
        if (has_t) OLIVE_COMBINE(uint16_t, true);
        else OLIVE_COMBINE(uint16_t, false);
    } else {
        if (has_t) OLIVE_COMBINE(float, true);
        else OLIVE_COMBINE(float, false);
    }
#undef OLIVE_COMBINE
    return hipGetLastError();
}

}  // namespace olive
