// Batched Householder application C = (I - 2 u u^T) B with the reflector
// built directly in the MFMA A-operand registers (Sec. 4.2.1, eq. householder;
// the rule-built fragment of Sec. 4.2), in emulated FP32 (Sec. 4.4).
//
// One wavefront handles one batch item (n = 64) and up to 64 columns of B.
// H is never stored: each lane evaluates, for every A-operand element it
// holds, h_ij = fmaf(-2 u_i, u_j, delta_ij) and splits it into hi/lo in
// registers.  Per
// 16-wide k step one foreach_ij over the A-operand map fills both 32-row
// blocks of the reflector (the index computation is shared by the two
// fragments, and -2 u_i of the lane's rows is computed once), which is what
// keeps rule-built fragments cheaper than a trip through memory.
//
// B is read straight from global memory into the B-operand registers.  When
// rows allow 8-byte accesses the two 32-column blocks interleave their
// columns, so for a fixed k the 32 lanes of a half-wave read one 256-byte row
// segment with one 8-byte load each (and C is written the same way);
// otherwise lane l holds column l % 32 of each block (128-byte segments).
// Neither H nor B goes through LDS; the kernel is bound by HBM traffic (u, B
// read once, C written once).
#include "internal.h"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"

namespace sgemm_emu {

using mfmae::f32x16_t;
using mfmae::half8_t;
using mfmae::Shape32;
using mfmae::Use;

struct HhParams {
    int ncols;
    const float* u;
    int64_t su;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int batch;   // items of this launch
    int64_t item0;  // first item of this launch
};

constexpr int kHhWaves = 4;  // waves (tasks) per workgroup

// PAIR: the two 32-column blocks interleave their columns (column j of
// block cb is c0 + 2 j + cb), so one 8-byte load of a B row and one 8-byte
// store of a C row serve both blocks; needs 8-byte aligned, even-length B
// and C rows.  Otherwise block cb holds columns c0 + 32 cb + j.
template <bool PAIR>
__global__ __launch_bounds__(64 * kHhWaves, 2) void householder64_kernel(HhParams p) {
    // wave index as a wave-uniform (scalar) value, so that the per-item base
    // pointers below live in SGPRs and loads use scalar-base addressing
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    // one wave per (item, group of 64 columns)
    const int64_t task = (int64_t)blockIdx.x * kHhWaves + wave;
    const int ngroups = (p.ncols + 63) / 64;
    const int64_t local = task / ngroups;
    const int c0 = (int)(task - local * ngroups) * 64;
    if (local >= p.batch) return;  // whole wave; the kernel has no barrier
    const int64_t item = local + p.item0;

    const float* __restrict__ u = p.u + item * p.su;
    const float* __restrict__ Bi = p.B + item * p.sb;
    float* __restrict__ Ci = p.C + item * p.sc;

    using FragA = mfmae::fragment<Shape32, Use::A, _Float16>;

    // Row of each of the two 32-row blocks of H this lane holds.
    float urow[2];
    mfmae::foreach_ij<FragA>([&](int e, int i, int) {
        if (e == 0) {
            urow[0] = -2.0f * u[i];
            urow[1] = -2.0f * u[32 + i];
        }
    });

    const int j = l & 31;
    // first column of this lane in block 0, and whether it (and, paired,
    // its neighbour) lies inside B
    const int col0 = PAIR ? c0 + 2 * j : c0 + j;
    const bool ok0 = col0 < p.ncols;
    const bool ok1 = PAIR ? ok0 : col0 + 32 < p.ncols;

    f32x16_t acc[2][2], cor[2][2];
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[tm][cb][e] = 0.0f;
                cor[tm][cb][e] = 0.0f;
            }

#pragma unroll
    for (int s = 0; s < 4; ++s) {
        // B operands of this 16-wide k step for both column blocks: lane l
        // holds rows 16 s + 8 (l / 32) + e; the row start of (s, e) is
        // wave-uniform and the lane part is a 32-bit offset.
        half8_t bh[2], bl[2];
        const int lane_off = 8 * (l >> 5) * (int)p.ldb + col0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float* rowp = Bi + (int64_t)(16 * s + e) * p.ldb;
            float x[2];
            if constexpr (PAIR) {
                typedef float f32x2 __attribute__((ext_vector_type(2)));
                f32x2 v = {0.0f, 0.0f};
                if (ok0) v = *reinterpret_cast<const f32x2*>(rowp + lane_off);
                x[0] = v[0];
                x[1] = v[1];
            } else {
                x[0] = ok0 ? rowp[lane_off] : 0.0f;
                x[1] = ok1 ? rowp[lane_off + 32] : 0.0f;
            }
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                _Float16 vh, vl;
                mfmae::tcec::split(x[cb], vh, vl);
                bh[cb][e] = vh;
                bl[cb][e] = vl;
            }
        }
        // Reflector operands of this k step for both row blocks, built
        // from the rule h_ij = fmaf(-2 u_i, u_j, delta_ij).
        half8_t hh[2], hl[2];
        const float* us = u + 16 * s + 8 * (l >> 5);
        mfmae::foreach_ij<FragA>([&](int e, int i, int jj) {
            const int gj = 16 * s + jj;
            const float uj = us[e];  // u[gj]: jj = 8 (l / 32) + e
#pragma unroll
            for (int tm = 0; tm < 2; ++tm) {
                const float h = __builtin_fmaf(urow[tm], uj, (32 * tm + i) == gj ? 1.0f : 0.0f);
                _Float16 vh, vl;
                mfmae::tcec::split(h, vh, vl);
                hh[tm][e] = vh;
                hl[tm][e] = vl;
            }
        });
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                acc[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hh[tm], bh[cb], acc[tm][cb], 0, 0, 0);
                cor[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hl[tm], bh[cb], cor[tm][cb], 0, 0, 0);
                cor[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hh[tm], bl[cb], cor[tm][cb], 0, 0, 0);
            }
    }

    // C = main + corr * 2^-11; element e of a block is row
    // 8 (e / 4) + 4 (l / 32) + e % 4 of it.
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int row = 32 * tm + mfmae::layout<Shape32, Use::Acc>::row(l, e);
            float v[2];
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
                v[cb] = __builtin_fmaf(cor[tm][cb][e], mfmae::tcec::kLoScaleInv, acc[tm][cb][e]);
            float* dst = Ci + (int64_t)row * p.ldc + col0;
            if constexpr (PAIR) {
                typedef float f32x2 __attribute__((ext_vector_type(2)));
                if (ok0) *reinterpret_cast<f32x2*>(dst) = f32x2{v[0], v[1]};
            } else {
                if (ok0) dst[0] = v[0];
                if (ok1) dst[32] = v[1];
            }
        }
}

hipError_t launch_householder64(const HouseholderArgs& a, hipStream_t stream) {
    HhParams p;
    p.ncols = a.ncols;
    p.u = a.u;
    p.su = a.su;
    p.B = a.B;
    p.ldb = a.ldb;
    p.sb = a.sb;
    p.C = a.C;
    p.ldc = a.ldc;
    p.sc = a.sc;
    const bool pair = ((uintptr_t)a.B % 8 == 0) && ((uintptr_t)a.C % 8 == 0) && a.ldb % 2 == 0 &&
                      a.ldc % 2 == 0 && a.sb % 2 == 0 && a.sc % 2 == 0 && a.ncols % 2 == 0;
    // one launch stays below 2^31 work-items (the dispatch packet counts
    // work-items in 32 bits); larger batches take several launches
    const int64_t ngroups = (a.ncols + 63) / 64;
    const int64_t max_blocks = (int64_t(1) << 31) / (64 * kHhWaves) - 1;
    const int64_t items_per_launch = max_blocks * kHhWaves / ngroups;
    if (items_per_launch == 0) return hipErrorInvalidConfiguration;
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        p.batch = (int)items;
        p.item0 = i0;
        const int64_t blocks = (items * ngroups + kHhWaves - 1) / kHhWaves;
        if (pair)
            hipLaunchKernelGGL(householder64_kernel<true>, dim3((unsigned)blocks),
                               dim3(64 * kHhWaves), 0, stream, p);
        else
            hipLaunchKernelGGL(householder64_kernel<false>, dim3((unsigned)blocks),
                               dim3(64 * kHhWaves), 0, stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace sgemm_emu
