// Running (max, lowest index of the max, scaled sum of exponentials) of a
// row's logits, and its merge -- shared by the streaming vocab pass and the
// LM-head epilogue, which both produce 16-byte partials
// {m, s, idx bits, mL} per (row, vocabulary partition).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace fb {

constexpr float kLog2e = 1.4426950408889634f;

// Running (max, index, scaled sum).  `s` is relative to mL = round(m*log2e).
struct Top {
    float m;
    float mL;
    float s;
    int idx;
};

__device__ inline Top top_empty() { return Top{-INFINITY, -INFINITY, 0.f, 0x7fffffff}; }

// The reference mL must be the rounded product everywhere it is used: with
// contraction, `x - m*log2e` would become an fma on the exact product and
// every merge would scale the sum by the product's rounding error.
__device__ inline float scaled_ref(float m) {
#pragma clang fp contract(off)
    return m * kLog2e;
}

// Order-independent merge of two partial results (commutative bit for bit).
__device__ inline Top top_merge(const Top& a, const Top& b) {
#pragma clang fp contract(off)
    if (a.m == -INFINITY) return b;
    if (b.m == -INFINITY) return a;
    Top r;
    r.m = fmaxf(a.m, b.m);
    r.mL = scaled_ref(r.m);
    r.s = a.s * __builtin_amdgcn_exp2f(a.mL - r.mL) + b.s * __builtin_amdgcn_exp2f(b.mL - r.mL);
    r.idx = a.m > b.m ? a.idx : (b.m > a.m ? b.idx : min(a.idx, b.idx));
    return r;
}

__device__ inline float4 top_pack(const Top& t) {
    return make_float4(t.m, t.s, __int_as_float(t.idx), t.mL);
}

__device__ inline Top top_unpack(const float4& p) {
    return Top{p.x, p.w, p.y, __float_as_int(p.z)};
}

}  // namespace fb
