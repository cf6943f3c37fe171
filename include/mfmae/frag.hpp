// mfmae/frag.hpp -- register fragments of the gfx950 fp16 matrix instructions
// and the primitives that build them from a rule instead of from memory.
//
// The paper's extension library exposes the mapping between a matrix element
// (i, j) and the (lane, element) of the register array that holds it, so a
// fragment can be generated from a structural rule without a round trip
// through shared memory: foreach_ij (Sec. 4.2), map (Sec. 4.3) and the
// all-equal fill (Sec. 4.1).  This header gives the same primitives for the
// CDNA4 MFMA operands, where a wavefront is 64 lanes and every matrix element
// is held exactly once (no duplication across lanes).
//
// Shapes (D = A.B + C, A: M x K, B: K x N, C/D: M x N, fp16 inputs, FP32
// accumulate):
//   Shape16 : v_mfma_f32_16x16x32_f16  (M = N = 16, K = 32)
//   Shape32 : v_mfma_f32_32x32x16_f16  (M = N = 32, K = 16)
//
// Operand layouts (l = lane 0..63, v = element index):
//   Shape16  A: l holds A[l % 16][8 (l / 16) + v], v = 0..7
//            B: l holds B[8 (l / 16) + v][l % 16], v = 0..7
//            C: l holds C[4 (l / 16) + v][l % 16], v = 0..3
//   Shape32  A: l holds A[l % 32][8 (l / 32) + v], v = 0..7
//            B: l holds B[8 (l / 32) + v][l % 32], v = 0..7
//            C: l holds C[8 (v / 4) + 4 (l / 32) + v % 4][l % 32], v = 0..15
//
// The row index of A, the column index of B and the whole accumulator map
// are observable through the instruction's result.  The k index of an A/B
// element is observable only jointly: any relabelling of k applied to both
// operands gives the same product.  The k order above is the one this
// library uses everywhere, on both operands.
//
// All functions are constexpr __host__ __device__ so the host-side map
// queries of the C ABI and the kernels use one definition.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace mfmae {

enum class Use : int { A = 0, B = 1, Acc = 2 };

struct Shape16 {
    static constexpr int M = 16, N = 16, K = 32;
    static constexpr int id = 0;
};
struct Shape32 {
    static constexpr int M = 32, N = 32, K = 16;
    static constexpr int id = 1;
};

constexpr int kWave = 64;

// Number of elements each lane holds for (shape, use).
template <class S, Use U>
struct layout;

template <class S>
struct layout<S, Use::A> {
    static constexpr int rows = S::M, cols = S::K;
    static constexpr int num_elements = rows * cols / kWave;  // 8
    static constexpr int groups = kWave / S::M;               // lanes per row
    __host__ __device__ static constexpr int row(int lane, int) { return lane % S::M; }
    __host__ __device__ static constexpr int col(int lane, int e) {
        return num_elements * (lane / S::M) + e;
    }
    __host__ __device__ static constexpr int lane_of(int i, int j) {
        return i + S::M * (j / num_elements);
    }
    __host__ __device__ static constexpr int elem_of(int, int j) { return j % num_elements; }
};

template <class S>
struct layout<S, Use::B> {
    static constexpr int rows = S::K, cols = S::N;
    static constexpr int num_elements = rows * cols / kWave;  // 8
    __host__ __device__ static constexpr int row(int lane, int e) {
        return num_elements * (lane / S::N) + e;
    }
    __host__ __device__ static constexpr int col(int lane, int) { return lane % S::N; }
    __host__ __device__ static constexpr int lane_of(int i, int j) {
        return j + S::N * (i / num_elements);
    }
    __host__ __device__ static constexpr int elem_of(int i, int) { return i % num_elements; }
};

template <>
struct layout<Shape16, Use::Acc> {
    static constexpr int rows = 16, cols = 16;
    static constexpr int num_elements = 4;
    __host__ __device__ static constexpr int row(int lane, int e) { return 4 * (lane / 16) + e; }
    __host__ __device__ static constexpr int col(int lane, int) { return lane % 16; }
    __host__ __device__ static constexpr int lane_of(int i, int j) { return j + 16 * (i / 4); }
    __host__ __device__ static constexpr int elem_of(int i, int) { return i % 4; }
};

template <>
struct layout<Shape32, Use::Acc> {
    static constexpr int rows = 32, cols = 32;
    static constexpr int num_elements = 16;
    __host__ __device__ static constexpr int row(int lane, int e) {
        return 8 * (e / 4) + 4 * (lane / 32) + e % 4;
    }
    __host__ __device__ static constexpr int col(int lane, int) { return lane % 32; }
    __host__ __device__ static constexpr int lane_of(int i, int j) { return j + 32 * ((i / 4) % 2); }
    __host__ __device__ static constexpr int elem_of(int i, int) { return 4 * (i / 8) + i % 4; }
};

// ---------------------------------------------------------------------------
// Fragment storage
// ---------------------------------------------------------------------------

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <class S, Use U, class T>
struct fragment;

template <class S, class T>
struct fragment<S, Use::A, T> {
    static constexpr int num_elements = layout<S, Use::A>::num_elements;
    T x[num_elements];
};
template <class S, class T>
struct fragment<S, Use::B, T> {
    static constexpr int num_elements = layout<S, Use::B>::num_elements;
    T x[num_elements];
};
template <class S>
struct fragment<S, Use::Acc, float> {
    static constexpr int num_elements = layout<S, Use::Acc>::num_elements;
    float x[num_elements];
};

template <class F>
struct frag_traits;
template <class S, Use U, class T>
struct frag_traits<fragment<S, U, T>> {
    using shape = S;
    static constexpr Use use = U;
    using layout_t = layout<S, U>;
};

__device__ inline int lane_id() { return __lane_id(); }

// ---------------------------------------------------------------------------
// Primitives
// ---------------------------------------------------------------------------

// Set every element of a fragment to v (Sec. 4.1).
template <class F, class V>
__device__ inline void fill(F& f, V v) {
#pragma unroll
    for (int e = 0; e < F::num_elements; ++e) f.x[e] = v;
}

// For every element this lane holds, call fn(elem, i, j) with the element
// index and its matrix position (Sec. 4.2).  Each (i, j) is visited by
// exactly one (lane, elem) of the wavefront.  The index arithmetic is a
// function of the lane only; with `fn` inlined it is evaluated once and
// reused by every fragment the callback writes (the amortisation that makes
// rule-built fragments pay off).
template <class F, class Fn>
__device__ inline void foreach_ij(Fn&& fn) {
    using L = typename frag_traits<F>::layout_t;
    const int l = lane_id();
#pragma unroll
    for (int e = 0; e < F::num_elements; ++e) fn(e, L::row(l, e), L::col(l, e));
}

// Position (i, j) -> the lane that holds it and its element index there
// (Sec. 4.3).
template <class F>
__host__ __device__ constexpr void map(int& lane, int& elem, int i, int j) {
    using L = typename frag_traits<F>::layout_t;
    lane = L::lane_of(i, j);
    elem = L::elem_of(i, j);
}

// Raw vector views used by the mma wrappers.
template <class S>
__device__ inline half8_t pack(const fragment<S, Use::A, _Float16>& f) {
    half8_t r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = f.x[e];
    return r;
}
template <class S>
__device__ inline half8_t pack(const fragment<S, Use::B, _Float16>& f) {
    half8_t r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = f.x[e];
    return r;
}

// One fp16 MFMA on raw operand vectors: acc += a . b.
__device__ inline f32x4_t mma(Shape16, half8_t a, half8_t b, f32x4_t acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc, 0, 0, 0);
}
__device__ inline f32x16_t mma(Shape32, half8_t a, half8_t b, f32x16_t acc) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc, 0, 0, 0);
}

}  // namespace mfmae
