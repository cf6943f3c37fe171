// mfmae/wmma_tcec.hpp -- FP32 matrix-multiply-accumulate fragments with the
// interface of a fragment API (fragment / fill_fragment / load_matrix_sync /
// mma_sync / store_matrix_sync, Sec. 2.3.1), computed by the single-precision
// emulation of Sec. 4.4 on the gfx950 fp16 MFMA instructions.
//
// Code written for fp16 fragments switches to emulated FP32 by changing the
// element type to float and the namespace to mfmae::wmma::tcec; the
// interface of the paper's error-correcting extension follows the same idea
// (Sec. 4.4).  What differs from a plain fp16 fragment:
//
//   * A and B fragments hold two fp16 vectors, hi = toFP16(x) and
//     lo = toFP16((x - hi) 2^11), formed in registers when the fragment is
//     loaded (or set element by element); no fp16 copy of the input is ever
//     written to memory (Fig. 6, bottom).
//   * Accumulator fragments hold two FP32 vectors: the sum of hi.hi products
//     and the sum of the correction products lo.hi + hi.lo in units of
//     2^-11; the FP32 value of an element is acc + cor 2^-11, formed once,
//     when it is read or stored.
//   * A policy template parameter chooses, per fragment, whether the
//     correction products are computed (EC on: 3 MFMAs per mma_sync; off: 1,
//     the hi.hi product only), after the policy-based design of Sec. 4.4.
//
// Shapes (M, N, K): (32, 32, 16) on v_mfma_f32_32x32x16_f16 and (16, 16, 32)
// on v_mfma_f32_16x16x32_f16.  The element maps are those of mfmae/frag.hpp
// (every element held by exactly one lane).  All functions must be called
// by all 64 lanes of a wavefront with the same arguments (except where an
// argument is documented as per lane).
//
// Memory contract of load_matrix_sync / store_matrix_sync: p points to
// element (0, 0); row_major stores element (i, j) at p[i ld + j], col_major
// at p[j ld + i].  p must be 16-byte aligned and ld a multiple of 4 (as a
// fragment API requires for 32-bit elements): along the contiguous direction
// each lane then moves 8 (A, B) or 4 (accumulator) elements with 16-byte
// accesses.  The *_bounded variants take any p and ld, touch only elements
// with i < rows and j < cols, and read the others as zero.  The stores take an
// optional last argument `nontemporal` (default false): true marks the writes
// as streaming, for output that is not read again soon; the values written
// are the same either way.
#pragma once

#include "frag.hpp"
#include "tcec.hpp"

namespace mfmae {
namespace wmma {

struct matrix_a {};
struct matrix_b {};
struct accumulator {};
struct row_major {};
struct col_major {};
enum layout_t { mem_row_major = 0, mem_col_major = 1 };

namespace tcec {

// Policy: error correction on (3 MFMAs per product) or off (1 MFMA).
template <bool EC = true>
struct policy {
    static constexpr bool ec = EC;
};
using default_policy = policy<true>;

namespace detail {

template <int M, int N, int K>
struct shape_of;
template <>
struct shape_of<32, 32, 16> {
    using type = Shape32;
};
template <>
struct shape_of<16, 16, 32> {
    using type = Shape16;
};

template <class U>
struct use_of;
template <>
struct use_of<matrix_a> {
    static constexpr Use value = Use::A;
};
template <>
struct use_of<matrix_b> {
    static constexpr Use value = Use::B;
};
template <>
struct use_of<accumulator> {
    static constexpr Use value = Use::Acc;
};

typedef float f32x4 __attribute__((ext_vector_type(4)));

// one store, streaming (nontemporal) or ordinary
template <class T>
__device__ inline void put(T* q, T v, bool nontemporal) {
    if (nontemporal)
        __builtin_nontemporal_store(v, q);
    else
        *q = v;
}

}  // namespace detail

// fragment<Use, M, N, K, float, Layout, Policy>; Layout is row_major or
// col_major for matrix_a / matrix_b and void for the accumulator.
template <class UseT, int M, int N, int K, class T, class Layout = void,
          class Policy = default_policy>
struct fragment;

template <class UseT, int M, int N, int K, class Layout, class Policy>
struct fragment<UseT, M, N, K, float, Layout, Policy> {
    using shape = typename detail::shape_of<M, N, K>::type;
    using map_t = layout<shape, detail::use_of<UseT>::value>;
    using layout_type = Layout;
    using policy_type = Policy;
    static constexpr int num_elements = map_t::num_elements;  // 8
    half8_t hi, lo;
};

template <int M, int N, int K, class Policy>
struct fragment<accumulator, M, N, K, float, void, Policy> {
    using shape = typename detail::shape_of<M, N, K>::type;
    using map_t = layout<shape, Use::Acc>;
    using policy_type = Policy;
    using vec = typename mfmae::tcec::acc_vec<shape>::type;
    static constexpr int num_elements = map_t::num_elements;  // 16 or 4
    vec acc;  // sum of hi.hi
    vec cor;  // sum of lo.hi + hi.lo, in units of 2^-11
};

// ---- element access -------------------------------------------------------

// Operand element e of this lane := x (split into hi and lo; x may be the
// result of FP32 arithmetic, e.g. an entry built from a rule).
template <class F>
__device__ inline void set_element(F& f, int e, float x) {
    _Float16 h, l;
    mfmae::tcec::split_rounded(x, h, l);
    f.hi[e] = h;
    f.lo[e] = l;
}

// Accumulator element e of this lane := x (exact: the correction part is 0).
template <int M, int N, int K, class P>
__device__ inline void set_element(fragment<accumulator, M, N, K, float, void, P>& f, int e,
                                   float x) {
    f.acc[e] = x;
    f.cor[e] = 0.0f;
}

// FP32 value of accumulator element e: acc + cor 2^-11, rounded once.
template <int M, int N, int K, class P>
__device__ inline float get_element(const fragment<accumulator, M, N, K, float, void, P>& f,
                                    int e) {
    return __builtin_fmaf(f.cor[e], mfmae::tcec::kLoScaleInv, f.acc[e]);
}

// For every element this lane holds, fn(e, i, j) with its matrix position
// (Sec. 4.2): build a fragment from a rule with set_element, no memory.
template <class F, class Fn>
__device__ inline void foreach_ij(Fn&& fn) {
    using L = typename F::map_t;
    const int l = lane_id();
#pragma unroll
    for (int e = 0; e < F::num_elements; ++e) fn(e, L::row(l, e), L::col(l, e));
}

// Matrix position (i, j) -> (lane, element) that holds it (Sec. 4.3).
template <class F>
__host__ __device__ constexpr void map(int& lane, int& elem, int i, int j) {
    using L = typename F::map_t;
    lane = L::lane_of(i, j);
    elem = L::elem_of(i, j);
}

// ---- fill -------------------------------------------------------------------

template <class UseT, int M, int N, int K, class L, class P>
__device__ inline void fill_fragment(fragment<UseT, M, N, K, float, L, P>& f, float v) {
    _Float16 h, l;
    mfmae::tcec::split_rounded(v, h, l);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        f.hi[e] = h;
        f.lo[e] = l;
    }
}

template <int M, int N, int K, class P>
__device__ inline void fill_fragment(fragment<accumulator, M, N, K, float, void, P>& f,
                                     float v) {
#pragma unroll
    for (int e = 0; e < f.num_elements; ++e) {
        f.acc[e] = v;
        f.cor[e] = 0.0f;
    }
}

// ---- loads ------------------------------------------------------------------

namespace detail {

// Offset of element (i, j) for a storage layout.
template <class L>
__device__ inline int64_t offset(int i, int j, int64_t ld) {
    if constexpr (__is_same(L, row_major)) return (int64_t)i * ld + j;
    else return (int64_t)j * ld + i;
}

// The 8 elements an operand lane holds are consecutive along k: for A that
// is the column index, for B the row index.  They are contiguous in memory
// when A is row_major or B is col_major.
template <class UseT, class L>
constexpr bool operand_contiguous() {
    return (__is_same(UseT, matrix_a) && __is_same(L, row_major)) ||
           (__is_same(UseT, matrix_b) && __is_same(L, col_major));
}

}  // namespace detail

template <class UseT, int M, int N, int K, class L, class P>
__device__ inline void load_matrix_sync(fragment<UseT, M, N, K, float, L, P>& f, const float* p,
                                        unsigned ld) {
    using F = fragment<UseT, M, N, K, float, L, P>;
    using Map = typename F::map_t;
    const int l = lane_id();
    float x[8];
    if constexpr (detail::operand_contiguous<UseT, L>()) {
        // element 0 of this lane and the 7 after it, two 16-byte loads
        const float* q = p + detail::offset<L>(Map::row(l, 0), Map::col(l, 0), ld);
        const detail::f32x4 v0 = *reinterpret_cast<const detail::f32x4*>(q);
        const detail::f32x4 v1 = *reinterpret_cast<const detail::f32x4*>(q + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[e] = v0[e];
            x[e + 4] = v1[e];
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = p[detail::offset<L>(Map::row(l, e), Map::col(l, e), ld)];
    }
    mfmae::tcec::split8(x, f.hi, f.lo);
}

template <class UseT, int M, int N, int K, class L, class P>
__device__ inline void load_matrix_bounded(fragment<UseT, M, N, K, float, L, P>& f,
                                           const float* p, int64_t ld, int rows, int cols) {
    using F = fragment<UseT, M, N, K, float, L, P>;
    using Map = typename F::map_t;
    const int l = lane_id();
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int i = Map::row(l, e), j = Map::col(l, e);
        x[e] = (i < rows && j < cols) ? p[detail::offset<L>(i, j, ld)] : 0.0f;
    }
    mfmae::tcec::split8(x, f.hi, f.lo);
}

// Accumulator elements come in runs of 4 consecutive rows per lane (e = 4q
// .. 4q + 3), contiguous in memory when stored col_major.
template <int M, int N, int K, class P>
__device__ inline void load_matrix_sync(fragment<accumulator, M, N, K, float, void, P>& f,
                                        const float* p, unsigned ld, layout_t layout) {
    using Map = typename fragment<accumulator, M, N, K, float, void, P>::map_t;
    const int l = lane_id();
    if (layout == mem_col_major) {
#pragma unroll
        for (int q = 0; q < f.num_elements / 4; ++q) {
            const detail::f32x4 v = *reinterpret_cast<const detail::f32x4*>(
                p + detail::offset<col_major>(Map::row(l, 4 * q), Map::col(l, 4 * q), ld));
#pragma unroll
            for (int t = 0; t < 4; ++t) f.acc[4 * q + t] = v[t];
        }
    } else {
#pragma unroll
        for (int e = 0; e < f.num_elements; ++e)
            f.acc[e] = p[detail::offset<row_major>(Map::row(l, e), Map::col(l, e), ld)];
    }
#pragma unroll
    for (int e = 0; e < f.num_elements; ++e) f.cor[e] = 0.0f;
}

template <int M, int N, int K, class P>
__device__ inline void load_matrix_bounded(fragment<accumulator, M, N, K, float, void, P>& f,
                                           const float* p, int64_t ld, layout_t layout, int rows,
                                           int cols) {
    using Map = typename fragment<accumulator, M, N, K, float, void, P>::map_t;
    const int l = lane_id();
#pragma unroll
    for (int e = 0; e < f.num_elements; ++e) {
        const int i = Map::row(l, e), j = Map::col(l, e);
        const int64_t o = layout == mem_col_major ? detail::offset<col_major>(i, j, ld)
                                                  : detail::offset<row_major>(i, j, ld);
        f.acc[e] = (i < rows && j < cols) ? p[o] : 0.0f;
        f.cor[e] = 0.0f;
    }
}

// ---- stores -----------------------------------------------------------------

template <int M, int N, int K, class P>
__device__ inline void store_matrix_sync(float* p,
                                         const fragment<accumulator, M, N, K, float, void, P>& f,
                                         unsigned ld, layout_t layout,
                                         bool nontemporal = false) {
    using Map = typename fragment<accumulator, M, N, K, float, void, P>::map_t;
    const int l = lane_id();
    if (layout == mem_col_major) {
#pragma unroll
        for (int q = 0; q < f.num_elements / 4; ++q) {
            detail::f32x4 v;
#pragma unroll
            for (int t = 0; t < 4; ++t) v[t] = get_element(f, 4 * q + t);
            detail::put(reinterpret_cast<detail::f32x4*>(p + detail::offset<col_major>(
                            Map::row(l, 4 * q), Map::col(l, 4 * q), ld)),
                        v, nontemporal);
        }
    } else {
#pragma unroll
        for (int e = 0; e < f.num_elements; ++e)
            detail::put(&p[detail::offset<row_major>(Map::row(l, e), Map::col(l, e), ld)],
                        get_element(f, e), nontemporal);
    }
}

template <int M, int N, int K, class P>
__device__ inline void store_matrix_bounded(
    float* p, const fragment<accumulator, M, N, K, float, void, P>& f, int64_t ld,
    layout_t layout, int rows, int cols, bool nontemporal = false) {
    using Map = typename fragment<accumulator, M, N, K, float, void, P>::map_t;
    const int l = lane_id();
#pragma unroll
    for (int e = 0; e < f.num_elements; ++e) {
        const int i = Map::row(l, e), j = Map::col(l, e);
        const int64_t o = layout == mem_col_major ? detail::offset<col_major>(i, j, ld)
                                                  : detail::offset<row_major>(i, j, ld);
        if (i < rows && j < cols) detail::put(&p[o], get_element(f, e), nontemporal);
    }
}

// ---- multiply-accumulate ------------------------------------------------------

// d = a . b + c (d may be c).  With error correction
//   d.acc = a.hi b.hi + c.acc,  d.cor = a.lo b.hi + a.hi b.lo + c.cor;
// without, only the first product (d.cor = c.cor).
template <int M, int N, int K, class LA, class LB, class P>
__device__ inline void mma_sync(fragment<accumulator, M, N, K, float, void, P>& d,
                                const fragment<matrix_a, M, N, K, float, LA, P>& a,
                                const fragment<matrix_b, M, N, K, float, LB, P>& b,
                                const fragment<accumulator, M, N, K, float, void, P>& c) {
    using S = typename detail::shape_of<M, N, K>::type;
    const auto cor = c.cor;
    d.acc = mfmae::mma(S{}, a.hi, b.hi, c.acc);
    if constexpr (P::ec) {
        d.cor = mfmae::mma(S{}, a.lo, b.hi, cor);
        d.cor = mfmae::mma(S{}, a.hi, b.lo, d.cor);
    } else {
        d.cor = cor;
    }
}

}  // namespace tcec
}  // namespace wmma
}  // namespace mfmae
