// Small device utilities behind the C ABI: the elementwise split (so the
// split can be checked bit for bit against its definition) and a one-MFMA
// probe that takes operands lane by lane (the register-level counterpart of
// the paper's mapping probe, Sec. 2.3.2).
#include "internal.h"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"
#include "sgemm_emu.h"
#include "tiling.hpp"

namespace sgemm_emu {

// Each thread splits one group of 8 consecutive values with the chosen
// device function; a group cut short by the end of x is split one value at
// a time.  An element of a vector is copied to a scalar before its bits are
// taken: this clang reads element 0 when __builtin_bit_cast is applied to
// an indexed vector element directly.
template <int FORM>
__global__ __launch_bounds__(256) void split_kernel(int64_t count, const float* __restrict__ x,
                                                    uint16_t* __restrict__ hi,
                                                    uint16_t* __restrict__ lo) {
    const int64_t groups = (count + 7) / 8;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < groups; g += stride) {
        const int64_t i0 = 8 * g;
        if (FORM != SGEMM_EMU_SPLIT_SCALAR && i0 + 8 <= count) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = x[i0 + e];
            if constexpr (FORM == SGEMM_EMU_SPLIT_EIGHT) {
                mfmae::half8_t h, l;
                mfmae::tcec::split8(v, h, l);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const _Float16 he = h[e], le = l[e];
                    hi[i0 + e] = __builtin_bit_cast(uint16_t, he);
                    lo[i0 + e] = __builtin_bit_cast(uint16_t, le);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    mfmae::tcec::half2_t h, l;
                    mfmae::tcec::split_pair(v[e], v[e + 1], h, l);
                    const _Float16 h0 = h[0], h1 = h[1], l0 = l[0], l1 = l[1];
                    hi[i0 + e] = __builtin_bit_cast(uint16_t, h0);
                    hi[i0 + e + 1] = __builtin_bit_cast(uint16_t, h1);
                    lo[i0 + e] = __builtin_bit_cast(uint16_t, l0);
                    lo[i0 + e + 1] = __builtin_bit_cast(uint16_t, l1);
                }
            }
            continue;
        }
        for (int64_t i = i0; i < count && i < i0 + 8; ++i) {
            _Float16 h, l;
            mfmae::tcec::split(x[i], h, l);
            hi[i] = __builtin_bit_cast(uint16_t, h);
            lo[i] = __builtin_bit_cast(uint16_t, l);
        }
    }
}

hipError_t launch_split(int64_t count, const float* x, uint16_t* hi, uint16_t* lo, int form,
                        hipStream_t stream) {
    if (count == 0) return hipSuccess;
    int64_t blocks = ((count + 7) / 8 + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (form == SGEMM_EMU_SPLIT_EIGHT)
        hipLaunchKernelGGL(split_kernel<SGEMM_EMU_SPLIT_EIGHT>, dim3((unsigned)blocks), dim3(256),
                           0, stream, count, x, hi, lo);
    else if (form == SGEMM_EMU_SPLIT_PAIR)
        hipLaunchKernelGGL(split_kernel<SGEMM_EMU_SPLIT_PAIR>, dim3((unsigned)blocks), dim3(256),
                           0, stream, count, x, hi, lo);
    else
        hipLaunchKernelGGL(split_kernel<SGEMM_EMU_SPLIT_SCALAR>, dim3((unsigned)blocks),
                           dim3(256), 0, stream, count, x, hi, lo);
    return hipGetLastError();
}

// Measurement reference: the read-A, read-B, write-C traffic of a batched
// product without its arithmetic.  One workgroup per item (item =
// blockIdx.x + item0), 16-byte loads, nontemporal 16-byte stores (as the
// full-tile kernel stores C).
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int NT>
__global__ __launch_bounds__(NT) void stream_probe_kernel(int64_t item0, int64_t n4,
                                                          const f32x4_t* __restrict__ A,
                                                          const f32x4_t* __restrict__ B,
                                                          f32x4_t* __restrict__ C) {
    const int64_t base = (item0 + blockIdx.x) * n4;
    for (int64_t i = threadIdx.x; i < n4; i += NT) {
        const f32x4_t v = A[base + i] + B[base + i];
        __builtin_nontemporal_store(v, &C[base + i]);
    }
}

hipError_t launch_stream_probe(int64_t items, int64_t n, const float* A, const float* B, float* C,
                               int threads, hipStream_t stream) {
    const int64_t n4 = n / 4;
    const auto* a = reinterpret_cast<const f32x4_t*>(A);
    const auto* b = reinterpret_cast<const f32x4_t*>(B);
    auto* c = reinterpret_cast<f32x4_t*>(C);
    const int64_t per_launch = (int64_t(1) << 31) / threads - 1;
    for (int64_t i0 = 0; i0 < items; i0 += per_launch) {
        const unsigned g = (unsigned)(items - i0 < per_launch ? items - i0 : per_launch);
        if (threads == 256)
            hipLaunchKernelGGL(stream_probe_kernel<256>, dim3(g), dim3(256), 0, stream, i0, n4, a, b, c);
        else if (threads == 512)
            hipLaunchKernelGGL(stream_probe_kernel<512>, dim3(g), dim3(512), 0, stream, i0, n4, a, b, c);
        else
            hipLaunchKernelGGL(stream_probe_kernel<1024>, dim3(g), dim3(1024), 0, stream, i0, n4, a, b,
                               c);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Measurement reference for the full-tile kernel's 128 x 256 tile: the same
// grid, task numbering, waves (eight of 64 x 64, two per SIMD), MFMA
// instruction (v_mfma_f32_32x32x16_f16), product order per k step (hi.hi for
// the four blocks, then lo.hi, then hi.lo into the correction accumulator) and
// epilogue, with the operand fragments of the tile's first k chunk built once
// (split from A[.][0..31] and B[0..31][.]) and held in registers: the k loop
// runs the products alone, without global loads, split or LDS traffic.  C
// receives k / 32 times the emulated product of the first chunk,
// A[.][0..31] B[0..31][.].
struct MfmaProbeParams {
    const float* A;
    int64_t lda;
    const float* B;
    int64_t ldb;
    float* C;
    int64_t ldc;
    int tiles_m, tiles_n;
    int nk;  // k chunks of 32
};

__global__ __launch_bounds__(512, 2) void mfma_probe_kernel(MfmaProbeParams p) {
    using mfmae::half8_t;
    const int task = xcd_task(blockIdx.x, gridDim.x);
    const int tiles = p.tiles_m * p.tiles_n;  // the grid: one task per tile
    const TileRC rc = block_order_applies(p.tiles_m, p.tiles_n, tiles)
                          ? block_tile(task, p.tiles_m, p.tiles_n)
                          : grouped_tile(task, p.tiles_m, p.tiles_n);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    const int g = l >> 5, j = l & 31;
    const int r0 = rc.tm * 128 + (wave / 4) * 64;  // the wave's 64 x 64 sub-tile
    const int c0 = rc.tn * 256 + (wave % 4) * 64;
    // [k step][block]: lane (j, g) holds k = 16 s + 8 g + 0..7 of row / column j
    half8_t ahi[2][2], alo[2][2], bhi[2][2], blo[2][2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            float x[8];
            const float* ap = p.A + (int64_t)(r0 + 32 * t + j) * p.lda + 16 * s + 8 * g;
#pragma unroll
            for (int v = 0; v < 8; ++v) x[v] = ap[v];
            mfmae::tcec::split8(x, ahi[s][t], alo[s][t]);
            const float* bp = p.B + (int64_t)(16 * s + 8 * g) * p.ldb + c0 + 32 * t + j;
#pragma unroll
            for (int v = 0; v < 8; ++v) x[v] = bp[(int64_t)v * p.ldb];
            mfmae::tcec::split8(x, bhi[s][t], blo[s][t]);
        }
    mfmae::f32x16_t acc[2][2], cor[2][2];
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[tm][tn][e] = 0.0f;
                cor[tm][tn][e] = 0.0f;
            }
    for (int c = 0; c < p.nk; ++c) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
#pragma unroll
            for (int tm = 0; tm < 2; ++tm)
#pragma unroll
                for (int tn = 0; tn < 2; ++tn)
                    acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[s][tm], bhi[s][tn],
                                                                         acc[tm][tn], 0, 0, 0);
#pragma unroll
            for (int tm = 0; tm < 2; ++tm)
#pragma unroll
                for (int tn = 0; tn < 2; ++tn)
                    cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[s][tm], bhi[s][tn],
                                                                         cor[tm][tn], 0, 0, 0);
#pragma unroll
            for (int tm = 0; tm < 2; ++tm)
#pragma unroll
                for (int tn = 0; tn < 2; ++tn)
                    cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[s][tm], blo[s][tn],
                                                                         cor[tm][tn], 0, 0, 0);
        }
    }
    // element e of a 32 x 32 block is row 8 (e / 4) + 4 g + e % 4, column j
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
            float* cp = p.C + (int64_t)(r0 + 32 * tm + 4 * g) * p.ldc + c0 + 32 * tn + j;
#pragma unroll
            for (int e = 0; e < 16; ++e)
                __builtin_nontemporal_store(
                    __builtin_fmaf(cor[tm][tn][e], mfmae::tcec::kLoScaleInv, acc[tm][tn][e]),
                    &cp[(int64_t)(8 * (e >> 2) + (e & 3)) * p.ldc]);
        }
}

hipError_t launch_mfma_probe(int m, int n, int k, const float* A, int64_t lda, const float* B,
                             int64_t ldb, float* C, int64_t ldc, hipStream_t stream) {
    MfmaProbeParams p;
    p.A = A;
    p.lda = lda;
    p.B = B;
    p.ldb = ldb;
    p.C = C;
    p.ldc = ldc;
    p.tiles_m = m / 128;
    p.tiles_n = n / 256;
    p.nk = k / 32;
    hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)(p.tiles_m * p.tiles_n)), dim3(512), 0,
                       stream, p);
    return hipGetLastError();
}

template <class S>
__global__ __launch_bounds__(64) void mma_probe_kernel(const uint16_t* __restrict__ a,
                                                       const uint16_t* __restrict__ b,
                                                       float* __restrict__ d) {
    const int l = threadIdx.x;
    mfmae::half8_t va, vb;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        va[e] = __builtin_bit_cast(_Float16, a[l * 8 + e]);
        vb[e] = __builtin_bit_cast(_Float16, b[l * 8 + e]);
    }
    constexpr int n = mfmae::layout<S, mfmae::Use::Acc>::num_elements;
    typename mfmae::tcec::acc_vec<S>::type acc;
#pragma unroll
    for (int e = 0; e < n; ++e) acc[e] = 0.0f;
    acc = mfmae::mma(S{}, va, vb, acc);
#pragma unroll
    for (int e = 0; e < n; ++e) d[l * n + e] = acc[e];
}

hipError_t launch_mma_probe(int shape, const uint16_t* a, const uint16_t* b, float* d,
                            hipStream_t stream) {
    if (shape == MFMAE_SHAPE_16x16x32)
        hipLaunchKernelGGL(mma_probe_kernel<mfmae::Shape16>, dim3(1), dim3(64), 0, stream, a, b, d);
    else
        hipLaunchKernelGGL(mma_probe_kernel<mfmae::Shape32>, dim3(1), dim3(64), 0, stream, a, b, d);
    return hipGetLastError();
}

}  // namespace sgemm_emu
