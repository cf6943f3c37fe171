// mfmae/tcec.hpp -- single-precision emulation on fp16 matrix instructions
// with error correction (Sec. 4.4, eqs. corr-1..corr-5).
//
// An FP32 value x is split in registers into
//     hi = toFP16(x),   lo = toFP16((x - toFP32(hi)) * 2^11)
// (round to nearest even).  For |x| <= 65504 the subtraction and the scaling
// are exact, so the split has exactly two roundings and is bit-reproducible.
// The product of two split operands is then
//     C = hiA.hiB + (loA.hiB + hiA.loB) / 2^11
// where the term loA.loB is dropped (it is at most 2^-22 |a||b|).  The first
// product goes to one FP32 accumulator and both correction products to a
// second one, so the small correction terms are not rounded away against the
// large main sum; the two are combined once, at the end, with one fused
// multiply-add (the 2^-11 scaling is exact).
//
// The fragments are built straight from FP32 values held in registers; no
// fp16 copy of the operands is ever written to memory by these functions.
#pragma once

#include "frag.hpp"

namespace mfmae {
namespace tcec {

constexpr float kLoScale = 2048.0f;            // 2^11
constexpr float kLoScaleInv = 1.0f / 2048.0f;  // 2^-11, exact

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Split one value.  The residual is formed as fma(hi, -2^11, x * 2^11): the
// product x * 2^11 is exact and so is the fused result 2^11 (x - hi), which
// is rounded once, to binary16 -- the same two roundings as the definition.
// (gfx950 evaluates the fma with hi read straight from its binary16 register,
// v_fma_mix, so the residual costs two instructions.)
//
// x must be an FP32 value the compiler cannot re-derive from a wider
// intermediate: a value loaded from memory, say.  For the result of FP32
// arithmetic just before the split use split_rounded.
__device__ inline void split(float x, _Float16& hi, _Float16& lo) {
    hi = static_cast<_Float16>(x);
    lo = static_cast<_Float16>(__builtin_fmaf(static_cast<float>(hi), -kLoScale, x * kLoScale));
}

// The split is defined on the FP32 value.  The empty asm keeps x in a VGPR
// as that value, so the compiler cannot fold the rounding that produced x
// into the conversion: fptrunc(fma(a, b, c)) is otherwise selected as one
// v_fma_mix with a single rounding of the exact a b + c, which differs from
// toFP16(fl32(a b + c)) when fl32(a b + c) is a binary16 tie (the fold is
// made whatever the contraction setting).
__device__ inline float as_fp32(float x) {
    __asm__("" : "+v"(x));
    return x;
}

// split of a value computed by FP32 arithmetic (a rule-built entry).
__device__ inline void split_rounded(float x, _Float16& hi, _Float16& lo) {
    split(as_fp32(x), hi, lo);
}

// Split two values: hi is converted as a pair (one v_cvt_pk_f16_f32) and the
// two residuals read their hi halves from that packed register.  Same
// condition on x0, x1 as for split.
__device__ inline void split_pair(float x0, float x1, half2_t& hi, half2_t& lo) {
    hi = __builtin_convertvector(f32x2_t{x0, x1}, half2_t);
    lo[0] = static_cast<_Float16>(
        __builtin_fmaf(static_cast<float>(hi[0]), -kLoScale, x0 * kLoScale));
    lo[1] = static_cast<_Float16>(
        __builtin_fmaf(static_cast<float>(hi[1]), -kLoScale, x1 * kLoScale));
}

// Split two values into packed (low half = first value) hi and lo words.
__device__ inline void split2(float x0, float x1, uint32_t& hi2, uint32_t& lo2) {
    half2_t h, l;
    split_pair(x0, x1, h, l);
    hi2 = __builtin_bit_cast(uint32_t, h);
    lo2 = __builtin_bit_cast(uint32_t, l);
}

// Split eight consecutive values into one hi and one lo operand vector.
__device__ inline void split8(const float (&x)[8], half8_t& hi, half8_t& lo) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
        half2_t h, l;
        split_pair(x[e], x[e + 1], h, l);
        hi[e] = h[0];
        hi[e + 1] = h[1];
        lo[e] = l[0];
        lo[e + 1] = l[1];
    }
}

// ---------------------------------------------------------------------------
// Fragment-level interface: the same shape of use as the plain fragments
// (fill / build from a rule / mma / read back), with FP32 semantics.
// ---------------------------------------------------------------------------

template <class S, Use U>
struct frag_emu {
    half8_t hi, lo;
};

template <class S>
struct acc_vec;
template <>
struct acc_vec<Shape16> {
    using type = f32x4_t;
};
template <>
struct acc_vec<Shape32> {
    using type = f32x16_t;
};

template <class S>
struct acc_emu {
    using vec = typename acc_vec<S>::type;
    static constexpr int num_elements = layout<S, Use::Acc>::num_elements;
    vec main;  // sum of hi.hi
    vec corr;  // sum of lo.hi + hi.lo, in units of 2^-11
};

template <class S>
__device__ inline void fill_zero(acc_emu<S>& d) {
#pragma unroll
    for (int e = 0; e < acc_emu<S>::num_elements; ++e) {
        d.main[e] = 0.0f;
        d.corr[e] = 0.0f;
    }
}

// Build an operand fragment from a rule: value(i, j) returns the FP32 entry
// at matrix position (i, j); it is split in registers (foreach_ij over the
// operand map, Sec. 4.2, applied to the FP32 emulation of Sec. 4.4).
template <class S, Use U, class Fn>
__device__ inline void build(frag_emu<S, U>& f, Fn&& value) {
    using L = layout<S, U>;
    const int l = lane_id();
#pragma unroll
    for (int e = 0; e < L::num_elements; ++e) {
        _Float16 h, lo;
        split_rounded(value(L::row(l, e), L::col(l, e)), h, lo);
        f.hi[e] = h;
        f.lo[e] = lo;
    }
}

// d += a . b with error correction (3 MFMAs) or without (1 MFMA).
template <bool EC, class S>
__device__ inline void mma(acc_emu<S>& d, const frag_emu<S, Use::A>& a,
                           const frag_emu<S, Use::B>& b) {
    d.main = mfmae::mma(S{}, a.hi, b.hi, d.main);
    if constexpr (EC) {
        d.corr = mfmae::mma(S{}, a.lo, b.hi, d.corr);
        d.corr = mfmae::mma(S{}, a.hi, b.lo, d.corr);
    }
}

// The FP32 result of element e of this lane: main + corr * 2^-11, one
// rounding.
template <class S>
__device__ inline float result(const acc_emu<S>& d, int e) {
    return __builtin_fmaf(d.corr[e], kLoScaleInv, d.main[e]);
}

}  // namespace tcec
}  // namespace mfmae
