// Preparation, row compaction, per-sequence loss and weight repack kernels.
//
// Masks follow Sec. 3.1 (Eq. 1 and the sentence after it): each packed sequence
// is a student prefix (local t < cut) followed by a teacher continuation (t >= cut);
// positions at or past the sequence's valid length (an end-of-sequence) are not
// scored at all. The teacher region is what Eq. 1 sums over. In the multi-turn form
// (Sec. 3.2) the scored region is instead a list of spans per sequence (the
// teacher's actions), the student's turns and the observations staying as context.
#include <hip/hip_runtime.h>

#include "olive_device.hpp"
#include "olive_internal.hpp"

namespace olive {

// Scored spans of a batch in the span region (null otherwise).
struct SpanArgs {
    const int32_t *off;     // [B+1]: spans of sequence b are [off[b], off[b+1])
    const int32_t *pairs;   // [S][2]: local [start, end)
    int32_t n;              // S
};

__device__ __forceinline__ bool in_region(int region, int t, int cut) {
    return region == OLIVE_REGION_TEACHER ? (t >= cut)
           : region == OLIVE_REGION_STUDENT ? (t < cut)
                                             : true;
}

// t inside one of spans [i0, i1) (validated: increasing, disjoint): the last span
// starting at or before t must end after it. Returns that span's index or -1.
__device__ __forceinline__ int span_of(const int32_t *pairs, int i0, int i1, int t) {
    int lo = i0, hi = i1;   // first span with start > t
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (pairs[2 * mid] <= t) lo = mid + 1; else hi = mid;
    }
    return (lo > i0 && t < pairs[2 * (lo - 1) + 1]) ? lo - 1 : -1;
}

// Rank of in-region position t among the sequence's in-region positions (its
// compacted index when only the region is scored).
__device__ __forceinline__ int region_rank(int region, const SpanArgs &sp, int b, int span,
                                           int t, int cut, int vl) {
    if (region == OLIVE_REGION_TEACHER) return t - cut;
    if (region != OLIVE_REGION_SPANS) return t;
    int r = 0;
    for (int i = sp.off[b]; i < span; ++i) {
        const int a = sp.pairs[2 * i], e = sp.pairs[2 * i + 1] < vl ? sp.pairs[2 * i + 1] : vl;
        r += e > a ? e - a : 0;
    }
    return r + (t - sp.pairs[2 * span]);
}

__device__ __forceinline__ int region_count(int region, int vl, int cut) {
    if (region == OLIVE_REGION_TEACHER) return vl > cut ? vl - cut : 0;
    if (region == OLIVE_REGION_STUDENT) return cut < vl ? cut : vl;
    return vl;
}

// Rank of valid position t outside the region among the sequence's valid positions
// outside it. In the span region t lies in no span, so every span that starts before
// t also ends at or before it.
__device__ __forceinline__ int outside_rank(int region, const SpanArgs &sp, int b, int t, int cut,
                                            int vl) {
    if (region == OLIVE_REGION_TEACHER) return t;         // t < cut
    if (region == OLIVE_REGION_STUDENT) return t - cut;   // cut <= t < vl
    int r = 0;
    for (int i = sp.off[b]; i < sp.off[b + 1]; ++i) {
        const int a = sp.pairs[2 * i];
        if (a >= t) break;
        const int e = sp.pairs[2 * i + 1] < vl ? sp.pairs[2 * i + 1] : vl;
        r += e > a ? e - a : 0;
    }
    return t - r;
}

constexpr int PREP_THREADS = 1024;

// One workgroup: validates the batch structure, derives per-sequence effective
// lengths, the compacted-row offsets (exclusive scan of valid lengths), the counts,
// and the vocabulary split of this call.
__global__ void __launch_bounds__(PREP_THREADS)
prep_kernel(const int32_t *__restrict__ cu, const int32_t *__restrict__ cut,
            const int32_t *__restrict__ vlen, int32_t B, int64_t T, int32_t region,
            SpanArgs sp, int32_t region_only, int32_t *__restrict__ seqbuf,
            Sched *__restrict__ sched, int32_t *__restrict__ err, int64_t *__restrict__ counts,
            int32_t tile_rows, int32_t policy, int32_t n_vtiles, int32_t grid,
            int32_t fixed_splits, int32_t min_splits) {
    __shared__ int s_bad, s_badoff;
    __shared__ int s_scan[PREP_THREADS];
    __shared__ int s_scan_sc[PREP_THREADS];
    __shared__ long long s_red[PREP_THREADS];
    __shared__ long long s_val[PREP_THREADS];
    const int tid = threadIdx.x;
    const bool span_mode = region == OLIVE_REGION_SPANS;
    if (tid == 0) { s_bad = 0; s_badoff = 0; }
    __syncthreads();
    if (span_mode) {   // span offsets: 0 = off[0] <= off[1] <= ... <= off[B] = S
        for (int b = tid; b <= B; b += PREP_THREADS) {
            const int o = sp.off[b];
            bool bad = (b == 0 && o != 0) || (b == B && o != sp.n) || (b > 0 && o < sp.off[b - 1]);
            if (bad) atomicOr(&s_badoff, 1);
        }
    }
    for (int b = tid; b <= B; b += PREP_THREADS) {
        int c = cu[b];
        bool bad = (b == 0 && c != 0) || (b == B && (int64_t)c != T) || (b > 0 && c < cu[b - 1]);
        if (bad) atomicOr(&s_bad, 1);
    }
    __syncthreads();
    int32_t *cvalid = seqbuf;
    int32_t *vl_eff = seqbuf + (B + 1);
    int32_t *cut_eff = seqbuf + 2 * (B + 1);
    int32_t *badseq = seqbuf + 3 * (B + 1);
    int32_t *cscored = seqbuf + 4 * (B + 1);
    if (s_bad) {
        for (int b = tid; b <= B; b += PREP_THREADS) {
            cvalid[b] = 0;
            cscored[b] = 0;
            if (b < B) { vl_eff[b] = 0; cut_eff[b] = 0; badseq[b] = 1; }
        }
        if (tid == 0) {
            atomicOr(err, ERR_CU);
            sched->t_valid = 0; sched->n_ptiles = 0; sched->n_splits = 1; sched->n_units = 0;
            sched->n_scored = 0; sched->n_flagged = 0; sched->cu_bad = 1;
            sched->n_tkq[0] = 0; sched->n_tkq[1] = 0; sched->n_tk_fb = 0;
            sched->n_fxq[0] = 0; sched->n_fxq[1] = 0; sched->n_fx_fb = 0;
            sched->fx_smask[0] = 0u; sched->fx_smask[1] = 0u;
            if (counts) { counts[0] = 0; counts[1] = 0; }
        }
        return;
    }
    int carry = 0, carry_sc = 0;
    long long scored = 0, valid = 0;
    for (int base = 0; base < B; base += PREP_THREADS) {
        int b = base + tid;
        int v = 0;            // compacted rows of this sequence
        long long sc = 0;     // its scored positions
        long long vv = 0;     // its valid positions
        if (b < B) {
            int len = cu[b + 1] - cu[b];
            int c = span_mode ? 0 : cut[b];
            int vl = vlen ? vlen[b] : len;
            int e = 0;
            if (c < 0 || c > len) e |= ERR_CUT;
            if (vl < 0 || vl > len) e |= ERR_VALID;
            long long span_sc = 0;
            if (span_mode) {
                if (s_badoff) {
                    e |= ERR_SPAN;
                } else {
                    int prev = 0;
                    for (int i = sp.off[b]; i < sp.off[b + 1]; ++i) {
                        const int a = sp.pairs[2 * i], z = sp.pairs[2 * i + 1];
                        if (a < prev || a > z || z > len) { e |= ERR_SPAN; break; }
                        prev = z;
                        const int zz = z < vl ? z : vl;
                        span_sc += zz > a ? zz - a : 0;
                    }
                }
            }
            if (e) {
                atomicOr(err, e);
                vl_eff[b] = 0; cut_eff[b] = 0; badseq[b] = 1;
            } else {
                vl_eff[b] = vl; cut_eff[b] = c; badseq[b] = 0;
                sc = span_mode ? span_sc : region_count(region, vl, c);
                vv = vl;
                v = region_only ? (int)sc : vl;
            }
        }
        s_scan[tid] = v;
        s_scan_sc[tid] = (int)sc;
        s_red[tid] = sc;
        s_val[tid] = vv;
        __syncthreads();
        for (int off = 1; off < PREP_THREADS; off <<= 1) {   // inclusive scans
            int add = tid >= off ? s_scan[tid - off] : 0;
            int add_sc = tid >= off ? s_scan_sc[tid - off] : 0;
            __syncthreads();
            s_scan[tid] += add;
            s_scan_sc[tid] += add_sc;
            __syncthreads();
        }
        for (int off = PREP_THREADS / 2; off > 0; off >>= 1) {  // fixed-order sums
            if (tid < off) {
                s_red[tid] += s_red[tid + off];
                s_val[tid] += s_val[tid + off];
            }
            __syncthreads();
        }
        if (b < B) {
            cvalid[b] = carry + s_scan[tid] - v;
            cscored[b] = carry_sc + s_scan_sc[tid] - (int)sc;
        }
        carry += s_scan[PREP_THREADS - 1];
        carry_sc += s_scan_sc[PREP_THREADS - 1];
        scored += s_red[0];
        valid += s_val[0];
        __syncthreads();
    }
    if (tid == 0) {
        cvalid[B] = carry;
        cscored[B] = carry_sc;
        int t_valid = carry;   // compacted rows: valid, or in-region when region-only
        int n_p = (t_valid + tile_rows - 1) / tile_rows;
        int ns = 1;
        if (policy == 0) {
            // Minimise (rounds of the persistent grid) x (vocabulary tiles per split).
            long long best = -1;
            int smax = n_vtiles < MAX_SPLITS ? n_vtiles : MAX_SPLITS;
            const int smin = min_splits < smax ? min_splits : smax;
            for (int s = smin; s <= smax; ++s) {
                long long units = (long long)n_p * s;
                long long rounds = (units + grid - 1) / grid;
                long long per = (n_vtiles + s - 1) / s;
                long long cost = rounds * per;
                if (best < 0 || cost < best) { best = cost; ns = s; }
            }
        } else {
            ns = fixed_splits < n_vtiles ? fixed_splits : n_vtiles;
            if (ns < 1) ns = 1;
        }
        sched->t_valid = t_valid;
        sched->n_ptiles = n_p;
        sched->n_splits = ns;
        sched->n_units = n_p * ns;
        sched->n_scored = scored;
        sched->n_flagged = 0;
        sched->n_tkq[0] = 0; sched->n_tkq[1] = 0; sched->n_tk_fb = 0;
        sched->n_fxq[0] = 0; sched->n_fxq[1] = 0; sched->n_fx_fb = 0;
        sched->fx_smask[0] = 0u; sched->fx_smask[1] = 0u;
        sched->cu_bad = 0;
        if (counts) { counts[0] = scored; counts[1] = valid; }
    }
}

// Maps every packed row to its compacted index and writes the fixed outputs of rows
// that are not scored (logp 0, argmax -1, kl +0) and of rows of malformed sequences
// (NaN, argmax -1). With region_only only in-region rows are compacted; otherwise the
// valid rows are, the in-region ones first ([0, n_scored), by sequence and position)
// and then the others, so that work needed only for scored rows covers the leading
// position tiles.
__global__ void __launch_bounds__(256)
rowmap_kernel(const int32_t *__restrict__ cu, int32_t B, int64_t T, int32_t region,
              SpanArgs sp, int32_t region_only, const int32_t *__restrict__ seqbuf,
              const Sched *__restrict__ sched,
              uint32_t *__restrict__ rowmap, float *__restrict__ logp_s,
              float *__restrict__ logp_t, int32_t *__restrict__ am_s, int32_t *__restrict__ am_t,
              float *__restrict__ kl, float *__restrict__ kl_rev, float *__restrict__ jsd,
              float *__restrict__ logp_tmp, TopkOut tk) {
    const int32_t *cvalid = seqbuf;
    const int32_t *vl_eff = seqbuf + (B + 1);
    const int32_t *cut_eff = seqbuf + 2 * (B + 1);
    const int32_t *badseq = seqbuf + 3 * (B + 1);
    const int32_t *cscored = seqbuf + 4 * (B + 1);
    const bool cu_bad = sched->cu_bad != 0;
    const int32_t n_scored = (int32_t)sched->n_scored;
    const float qnan = __builtin_nanf("");
    for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < T;
         g += (int64_t)gridDim.x * blockDim.x) {
        bool bad = cu_bad;
        int b = 0, t = 0;
        if (!bad) {
            int lo = 0, hi = B + 1;              // first index with cu[i] > g
            while (lo < hi) {
                int mid = (lo + hi) >> 1;
                if ((int64_t)cu[mid] <= g) lo = mid + 1; else hi = mid;
            }
            b = lo - 1;
            t = (int)(g - cu[b]);
            bad = badseq[b] != 0;
        }
        if (bad) {
            if (logp_s) logp_s[g] = qnan;
            if (logp_t) logp_t[g] = qnan;
            if (am_s) am_s[g] = -1;
            if (am_t) am_t[g] = -1;
            if (kl) kl[g] = qnan;
            if (kl_rev) kl_rev[g] = qnan;
            if (jsd) jsd[g] = qnan;
            if (logp_tmp) logp_tmp[g] = qnan;
            if (tk.overlap) tk.overlap[g] = qnan;
            if (tk.kl) tk.kl[g] = qnan;
            for (int e = 0; e < TOPK_K; ++e) {
                if (tk.idx_s) tk.idx_s[g * TOPK_K + e] = -1;
                if (tk.idx_t) tk.idx_t[g * TOPK_K + e] = -1;
            }
            continue;
        }
        const int vl = vl_eff[b];
        int span = -1;
        bool r = false;
        if (t < vl) {
            if (region == OLIVE_REGION_SPANS) {
                span = span_of(sp.pairs, sp.off[b], sp.off[b + 1], t);
                r = span >= 0;
            } else {
                r = in_region(region, t, cut_eff[b]);
            }
        }
        if (t < vl && !region_only) {
            const int idx =
                r ? cscored[b] + region_rank(region, sp, b, span, t, cut_eff[b], vl)
                  : n_scored + (cvalid[b] - cscored[b]) +
                        outside_rank(region, sp, b, t, cut_eff[b], vl);
            rowmap[idx] = (uint32_t)g | ((r ? 1u : 0u) << 31);
        } else if (t < vl && r) {
            rowmap[cvalid[b] + region_rank(region, sp, b, span, t, cut_eff[b], vl)] =
                (uint32_t)g | (1u << 31);
        } else {
            if (logp_s) logp_s[g] = 0.f;
            if (logp_t) logp_t[g] = 0.f;
            if (am_s) am_s[g] = -1;
            if (am_t) am_t[g] = -1;
            if (kl) kl[g] = 0.f;
            if (kl_rev) kl_rev[g] = 0.f;
            if (jsd) jsd[g] = 0.f;
            if (logp_tmp) logp_tmp[g] = 0.f;
            if (tk.overlap) tk.overlap[g] = 0.f;
            if (tk.kl) tk.kl[g] = 0.f;
            for (int e = 0; e < TOPK_K; ++e) {
                if (tk.idx_s) tk.idx_s[g * TOPK_K + e] = -1;
                if (tk.idx_t) tk.idx_t[g * TOPK_K + e] = -1;
            }
        }
    }
}

// Eq. 1 per sequence: ce_b = - sum over the in-region valid positions of logp_S,
// accumulated in fp64 in a fixed order (deterministic).
__global__ void __launch_bounds__(256)
ce_kernel(const int32_t *__restrict__ cu, int32_t B, int32_t region, SpanArgs sp,
          const int32_t *__restrict__ seqbuf, const Sched *__restrict__ sched,
          const float *__restrict__ logp_s, float *__restrict__ ce) {
    __shared__ double red[256];
    const int b = blockIdx.x;
    if (b >= B) return;
    const int32_t *vl_eff = seqbuf + (B + 1);
    const int32_t *cut_eff = seqbuf + 2 * (B + 1);
    const int32_t *badseq = seqbuf + 3 * (B + 1);
    if (sched->cu_bad || badseq[b]) {
        if (threadIdx.x == 0) ce[b] = __builtin_nanf("");
        return;
    }
    int vl = vl_eff[b], c = cut_eff[b];
    const int64_t base = cu[b];
    double acc = 0.0;
    if (region == OLIVE_REGION_SPANS) {
        for (int i = sp.off[b]; i < sp.off[b + 1]; ++i) {
            const int lo = sp.pairs[2 * i];
            const int hi = sp.pairs[2 * i + 1] < vl ? sp.pairs[2 * i + 1] : vl;
            for (int t = lo + threadIdx.x; t < hi; t += 256) acc -= (double)logp_s[base + t];
        }
    } else {
        int lo = 0, hi = vl;
        if (region == OLIVE_REGION_TEACHER) lo = c < vl ? c : vl;
        else if (region == OLIVE_REGION_STUDENT) hi = c < vl ? c : vl;
        for (int t = lo + threadIdx.x; t < hi; t += 256) acc -= (double)logp_s[base + t];
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) ce[b] = (float)red[0];
}

// W [d][V] -> W [V][d] through 64 x 64 LDS tiles (init only).
template <typename E>
__global__ void __launch_bounds__(256)
repack_kernel(const E *__restrict__ src, E *__restrict__ dst, int64_t d, int64_t V) {
    __shared__ E tile[64][65];
    const int64_t v0 = (int64_t)blockIdx.x * 64, k0 = (int64_t)blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        int64_t k = k0 + r, v = v0 + tx;
        if (k < d && v < V) tile[r][tx] = src[k * V + v];
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        int64_t v = v0 + r, k = k0 + tx;
        if (k < d && v < V) dst[v * d + k] = tile[tx][r];
    }
}

hipError_t launch_repack(const void *w_dv, void *w_vd, int64_t d, int64_t V, int elem_bytes,
                         hipStream_t st) {
    dim3 grid((unsigned)((V + 63) / 64), (unsigned)((d + 63) / 64));
    if (elem_bytes == 2)
        repack_kernel<uint16_t><<<grid, 256, 0, st>>>((const uint16_t *)w_dv, (uint16_t *)w_vd,
                                                        d, V);
    else
        repack_kernel<float><<<grid, 256, 0, st>>>((const float *)w_dv, (float *)w_vd, d, V);
    return hipGetLastError();
}

static SpanArgs span_args(const olive_spans *s) {
    SpanArgs a;
    a.off = s ? s->span_offsets : nullptr;
    a.pairs = s ? s->spans : nullptr;
    a.n = s ? s->num_spans : 0;
    return a;
}

hipError_t launch_prep(const olive_batch &b, const olive_spans *spans, bool region_only,
                       int64_t V, int32_t *seqbuf, Sched *sched, int32_t *err, int64_t *counts,
                       int tile_rows, int policy, int n_vtiles, int grid, int fixed_splits,
                       int min_splits, hipStream_t st) {
    (void)V;
    prep_kernel<<<1, PREP_THREADS, 0, st>>>(b.cu_seqlens, b.cut, b.valid_len, b.num_seqs,
                                            b.total_positions, b.region, span_args(spans),
                                            region_only ? 1 : 0, seqbuf, sched, err, counts,
                                            tile_rows, policy, n_vtiles, grid, fixed_splits,
                                            min_splits);
    return hipGetLastError();
}

hipError_t launch_rowmap(const olive_batch &b, const olive_spans *spans, bool region_only,
                         int64_t V, const int32_t *seqbuf,
                         const Sched *sched, uint32_t *rowmap, int32_t *err, float *logp_s,
                         float *logp_t, int32_t *am_s, int32_t *am_t, float *kl, float *kl_rev,
                         float *jsd, float *logp_tmp, const TopkOut &tk, hipStream_t st) {
    (void)V; (void)err;
    int64_t T = b.total_positions;
    int64_t blocks = (T + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    rowmap_kernel<<<(unsigned)blocks, 256, 0, st>>>(b.cu_seqlens, b.num_seqs, T, b.region,
                                                    span_args(spans), region_only ? 1 : 0, seqbuf,
                                                    sched, rowmap,
                                                    logp_s, logp_t, am_s,
                                                    am_t, kl, kl_rev, jsd, logp_tmp, tk);
    return hipGetLastError();
}

hipError_t launch_ce(const olive_batch &b, const olive_spans *spans, const int32_t *seqbuf,
                     const Sched *sched, const float *logp_s, float *ce, hipStream_t st) {
    ce_kernel<<<(unsigned)b.num_seqs, 256, 0, st>>>(b.cu_seqlens, b.num_seqs, b.region,
                                                    span_args(spans), seqbuf, sched, logp_s, ce);
    return hipGetLastError();
}

}  // namespace olive
