// Device helpers shared by the scoring kernels: bf16 loads, hardware exp2/log2,
// and the running statistics of one (row, model) over a stream of logits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "olive_internal.hpp"

namespace olive {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Two fp32 values to packed bf16 bits (x in the low half), rounded to nearest even by
// one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float x, float y) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = __builtin_convertvector((f32x2){x, y}, bf16x2);
    return __builtin_bit_cast(uint32_t, v);
}

// 2^x and log2(x) on the transcendental unit (v_exp_f32 / v_log_f32).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Order-preserving image of a float (a larger float maps to a larger unsigned).
__device__ __forceinline__ uint32_t f2ord(float z) {
    const uint32_t b = __float_as_uint(z);
    return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}
__device__ __forceinline__ float ord2f(uint32_t u) {
    return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}
// Top-K list keys: the high 16 bits of f2ord(z) (the logit rounded toward -inf to a
// bucket [lb(code), lb(code + 1))) above a 16-bit tie part. Lower and (exclusive)
// upper end of the bucket of a key's code.
__device__ __forceinline__ float key_lb(uint32_t key) { return ord2f(key & 0xFFFF0000u); }
__device__ __forceinline__ float key_ub(uint32_t key) {
    const uint32_t c = key >> 16;
    return c >= 0xFFFFu ? __builtin_inff() : ord2f((c + 1) << 16);
}

// Exclusive upper end of the bucket of a value that is a bucket's lower end.
__device__ __forceinline__ float bucket_ub(float lb) { return key_ub(f2ord(lb)); }

template <typename T>
__device__ __forceinline__ float load_elem(const T *p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float *p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t *p, int64_t i) {
    return bf16_bits_to_f32(p[i]);
}

// Vocabulary splits of a pass over n_p position tiles on a persistent grid of G
// workgroups: the count minimising (rounds of the grid) x (vocabulary tiles per
// split), the smallest among equals. The passes over the scored rows (logit gradient,
// Jensen-Shannon) and the combine of the latter use it alike.
// Work unit q -> (position tile p, vocabulary split s) of n_p tiles x ns splits: units
// cycle through groups of SG splits, so that the 32 workgroups of an XCD, which take
// consecutive units, share 32 / SG position tiles x SG splits. Two or more splits left
// over (ns % SG) join the last group, which is then SG + rem splits wide; a single one
// stays a group of its own, at the end. (Measured: on a pass of 987 position tiles and
// 7 splits, 3 leftover splits as a group of their own ran 2.2 % slower than joined; on
// one of 90 tiles and 17 splits, the leftover split joined ran 0.5 % slower than alone.)
__device__ __forceinline__ void unit_tile_split(int64_t q, int n_p, int ns, int SG, int &p,
                                                int &s) {
    const int nsb = ns / SG, rem = ns % SG;
    // the groups of SG splits before the last group
    const int nhead = (rem >= 2 && nsb > 0) ? nsb - 1 : nsb;
    const int64_t head_units = (int64_t)nhead * SG * n_p;
    if (q < head_units) {
        const int64_t w = q % (SG * (int64_t)n_p);
        p = (int)(w / SG);
        s = (int)(q / (SG * (int64_t)n_p)) * SG + (int)(w % SG);
    } else {
        // the last group: ns - nhead SG splits (SG + rem, or rem)
        const int wl = ns - nhead * SG;
        const int64_t w = q - head_units;
        p = (int)(w / wl);
        s = nhead * SG + (int)(w % wl);
    }
}

__device__ __forceinline__ int pass_splits(int n_p, int n_vtiles, int G) {
    const int smax = n_vtiles < MAX_SPLITS ? n_vtiles : MAX_SPLITS;
    int ns = 1;
    int64_t best = -1;
    for (int sc = 1; sc <= smax; ++sc) {
        const int64_t cost = (((int64_t)n_p * sc + G - 1) / G) * ((n_vtiles + sc - 1) / sc);
        if (best < 0 || cost < best) { best = cost; ns = sc; }
    }
    return ns;
}

// Running max / second max / lowest argmax / rescaled exp-sum of one model, and
// the teacher-weighted difference accumulator A (teacher only).
struct Stat {
    float best;  // raw logit
    float sec;
    int32_t idx;
    float z;     // sum exp(s * (v - best))
};

__device__ __forceinline__ Stat stat_identity() {
    Stat s;
    s.best = kNegInf;
    s.sec = kNegInf;
    s.idx = 0x7fffffff;
    s.z = 0.f;
    return s;
}

// Merge two partial statistics of the same row and model. The winner is the larger
// best, ties going to the lower index; exp-sums are rescaled to the winner's best.
// `a_acc`, `b_acc` carry the teacher's A accumulator (rescaled like z) when used.
__device__ __forceinline__ void stat_merge(Stat &a, float &a_acc, const Stat &b, float b_acc,
                                           float c) {
    if (b.best == kNegInf) return;              // b saw nothing
    if (a.best == kNegInf) { a = b; a_acc = b_acc; return; }
    bool b_wins = (b.best > a.best) || (b.best == a.best && b.idx < a.idx);
    const Stat &w = b_wins ? b : a;
    const Stat &l = b_wins ? a : b;
    float w_acc = b_wins ? b_acc : a_acc;
    float l_acc = b_wins ? a_acc : b_acc;
    float r = fast_exp2((l.best - w.best) * c);
    Stat o;
    o.best = w.best;
    o.idx = w.idx;
    o.sec = fmaxf(w.sec, l.best);
    o.z = w.z + l.z * r;
    a = o;
    a_acc = w_acc + l_acc * r;
}

}  // namespace olive
