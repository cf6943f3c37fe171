// Batched D = op(A) . op(B) + C in emulated FP32, written entirely with the
// fragment interface of mfmae/wmma_tcec.hpp: the multiply-accumulate form of
// a fragment API (Sec. 2.3.1) with the error-correcting emulation of Sec. 4.4
// behind the same calls (load_matrix_sync, mma_sync, store_matrix_sync).
//
// Each wavefront owns a 2 x 2 block of fragments (64 x 64 outputs with the
// 32 x 32 x 16 instruction, 32 x 32 with 16 x 16 x 32) of one batch item and
// walks k one instruction depth at a time: two A and two B fragments are
// loaded from global memory straight into registers (split there), four
// mma_sync calls update the block.  Edge tiles and the k tail use the
// bounded loads and stores.  No LDS: operands are reused from L2.
//
// The operand layouts are template parameters, as in a fragment API: A
// row_major (stored m x k) or col_major (stored as its k x m transpose), B
// row_major (k x n) or col_major (n x k); C and D share a runtime layout.
#include "internal.h"
#include "mfmae/wmma_tcec.hpp"
#include "sgemm_emu.h"

namespace sgemm_emu {

namespace {

namespace tw = mfmae::wmma;
namespace tt = mfmae::wmma::tcec;

constexpr int kWaves = 4;

template <int M, int N, int K, bool EC, class LA, class LB>
__global__ __launch_bounds__(64 * kWaves, 2) void gemm_acc_kernel(AccArgs p, int64_t task0,
                                                                  int64_t ntasks) {
    using P = tt::policy<EC>;
    using FA = tt::fragment<tw::matrix_a, M, N, K, float, LA, P>;
    using FB = tt::fragment<tw::matrix_b, M, N, K, float, LB, P>;
    using FC = tt::fragment<tw::accumulator, M, N, K, float, void, P>;
    constexpr bool a_row = __is_same(LA, tw::row_major);
    constexpr bool b_row = __is_same(LB, tw::row_major);

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t task = task0 + (int64_t)blockIdx.x * kWaves + wave;
    if (task >= task0 + ntasks) return;  // whole wave; no barrier below
    const int64_t tiles_m = ((int64_t)p.m + 2 * M - 1) / (2 * M);
    const int64_t tiles_n = ((int64_t)p.n + 2 * N - 1) / (2 * N);
    const int64_t per_item = tiles_m * tiles_n;
    const int64_t item = task / per_item;
    const int64_t t = task - item * per_item;
    const int m0 = (int)(t / tiles_n) * 2 * M;
    const int n0 = (int)(t % tiles_n) * 2 * N;

    const float* Ai = p.A + item * p.sa;
    const float* Bi = p.B + item * p.sb;
    float* Di = p.D + item * p.sd;
    const tw::layout_t lcd = p.cd_col ? tw::mem_col_major : tw::mem_row_major;
    // offset of element (i, j) of C or D
    auto cd_off = [&](int i, int j, int64_t ld) {
        return p.cd_col ? (int64_t)j * ld + i : (int64_t)i * ld + j;
    };

    FC d[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int r0 = m0 + a * M, c0 = n0 + b * N;
            if (p.C == nullptr) {
                tt::fill_fragment(d[a][b], 0.0f);
            } else {
                const float* Ci = p.C + item * p.sc + cd_off(r0, c0, p.ldc);
                if (p.vec_c && r0 + M <= p.m && c0 + N <= p.n)
                    tt::load_matrix_sync(d[a][b], Ci, (unsigned)p.ldc, lcd);
                else
                    tt::load_matrix_bounded(d[a][b], Ci, p.ldc, lcd, p.m - r0, p.n - c0);
            }
        }

    for (int k0 = 0; k0 < p.k; k0 += K) {
        const bool full_k = k0 + K <= p.k;
        FA fa[2];
        FB fb[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            const int r0 = m0 + a * M;
            const float* q = Ai + (a_row ? (int64_t)r0 * p.lda + k0 : (int64_t)k0 * p.lda + r0);
            if (p.vec_a && full_k && r0 + M <= p.m)
                tt::load_matrix_sync(fa[a], q, (unsigned)p.lda);
            else
                tt::load_matrix_bounded(fa[a], q, p.lda, p.m - r0, p.k - k0);
        }
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int c0 = n0 + b * N;
            const float* q = Bi + (b_row ? (int64_t)k0 * p.ldb + c0 : (int64_t)c0 * p.ldb + k0);
            if (p.vec_b && full_k && c0 + N <= p.n)
                tt::load_matrix_sync(fb[b], q, (unsigned)p.ldb);
            else
                tt::load_matrix_bounded(fb[b], q, p.ldb, p.k - k0, p.n - c0);
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) tt::mma_sync(d[a][b], fa[a], fb[b], d[a][b]);
    }

    // D is written once and not read again here: streaming stores (measured 5%
    // faster on the batched 128^3 accumulate)
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int r0 = m0 + a * M, c0 = n0 + b * N;
            float* q = Di + cd_off(r0, c0, p.ldd);
            if (p.vec_d && r0 + M <= p.m && c0 + N <= p.n)
                tt::store_matrix_sync(q, d[a][b], (unsigned)p.ldd, lcd, true);
            else
                tt::store_matrix_bounded(q, d[a][b], p.ldd, lcd, p.m - r0, p.n - c0, true);
        }
}

template <int M, int N, int K, bool EC, class LA, class LB>
hipError_t launch_acc_cfg(const AccArgs& a, hipStream_t stream) {
    const int64_t tiles =
        (((int64_t)a.m + 2 * M - 1) / (2 * M)) * (((int64_t)a.n + 2 * N - 1) / (2 * N));
    const int64_t total = tiles * a.batch;
    // one launch stays below 2^31 work-items
    const int64_t max_tasks = ((int64_t(1) << 31) / (64 * kWaves) - 1) * kWaves;
    for (int64_t t0 = 0; t0 < total; t0 += max_tasks) {
        const int64_t nt = total - t0 < max_tasks ? total - t0 : max_tasks;
        const int64_t blocks = (nt + kWaves - 1) / kWaves;
        hipLaunchKernelGGL((gemm_acc_kernel<M, N, K, EC, LA, LB>), dim3((unsigned)blocks),
                           dim3(64 * kWaves), 0, stream, a, t0, nt);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int M, int N, int K, bool EC>
hipError_t launch_acc_layouts(const AccArgs& a, hipStream_t stream) {
    using R = tw::row_major;
    using Cm = tw::col_major;
    if (!a.a_trans && !a.b_trans) return launch_acc_cfg<M, N, K, EC, R, R>(a, stream);
    if (a.a_trans && !a.b_trans) return launch_acc_cfg<M, N, K, EC, Cm, R>(a, stream);
    if (!a.a_trans && a.b_trans) return launch_acc_cfg<M, N, K, EC, R, Cm>(a, stream);
    return launch_acc_cfg<M, N, K, EC, Cm, Cm>(a, stream);
}

}  // namespace

hipError_t launch_gemm_acc(const AccArgs& a, int shape, bool ec, hipStream_t stream) {
    if (shape == 1)
        return ec ? launch_acc_layouts<32, 32, 16, true>(a, stream)
                  : launch_acc_layouts<32, 32, 16, false>(a, stream);
    return ec ? launch_acc_layouts<16, 16, 32, true>(a, stream)
              : launch_acc_layouts<16, 16, 32, false>(a, stream);
}

}  // namespace sgemm_emu
