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

// 2^x and log2(x) on the transcendental unit (v_exp_f32 / v_log_f32).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

template <typename T>
__device__ __forceinline__ float load_elem(const T *p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float *p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t *p, int64_t i) {
    return bf16_bits_to_f32(p[i]);
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
