// Batched inclusive scan y_j = sum_{i <= j} x_i of every row, as the product
// x^T U with the upper-triangular all-ones U (Sec. 4.1, eq. scan-mat, rule
// u-rule), in emulated FP32 (Sec. 4.4).
//
// One wavefront scans 32 rows, 64 columns (a chunk) at a time.  The chunk is
// the 32 x 64 A operand X (split into hi and lo in registers); U's 64 x 64
// block is the B operand, built once per wave with foreach_ij from the rule
// u_ij = [i <= j] and never stored: its 16 x 32 pieces for k step s and
// column block cb are all-zero for cb = 0, s >= 2, so a chunk takes 6 piece
// products.  U's entries are 0 and 1, whose lo parts are 0, so the
// correction reduces to lo(X) U: two MFMAs per piece instead of three.
// Chunks are chained by a carry: the running total of each row (column 63
// of the previous chunk's result, broadcast from the lanes that hold it)
// is added to every output of the row.  The next chunk's X is loaded while
// the current one is multiplied.
#include "internal.h"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"

namespace sgemm_emu {

namespace {

using mfmae::f32x16_t;
using mfmae::half8_t;
using mfmae::Shape32;
using mfmae::Use;

typedef float f32x4 __attribute__((ext_vector_type(4)));
using FragB = mfmae::fragment<Shape32, Use::B, _Float16>;

constexpr int kWaves = 4;

// The 8 values lane l holds of a 32-row, 16-column piece of X at k step s:
// row r0 + l % 32, columns c0 + 16 s + 8 (l / 32) .. + 7.
struct Chunk {
    float x[4][8];
};

__device__ inline void load_chunk(Chunk& ch, const ScanArgs& p, int64_t r0, int c0, bool fast) {
    const int l = threadIdx.x & 63;
    const int64_t row = r0 + (l & 31);
    const int col = c0 + 8 * (l >> 5);
    if (fast) {
        const float* q = p.X + row * p.ldx + col;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const f32x4 v0 = *reinterpret_cast<const f32x4*>(q + 16 * s);
            const f32x4 v1 = *reinterpret_cast<const f32x4*>(q + 16 * s + 4);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                ch.x[s][v] = v0[v];
                ch.x[s][v + 4] = v1[v];
            }
        }
    } else {
        const bool row_ok = row < p.rows;
        const float* q = p.X + (row_ok ? row : 0) * p.ldx;
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const int cc = col + 16 * s + v;
                ch.x[s][v] = (row_ok && cc < p.len) ? q[cc] : 0.0f;
            }
    }
}

__global__ __launch_bounds__(64 * kWaves, 2) void scan_kernel(ScanArgs p) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    const int64_t group = (int64_t)blockIdx.x * kWaves + wave;
    const int64_t r0 = group * 32;
    if (r0 >= p.rows) return;  // whole wave; no barrier below
    const bool rows_full = r0 + 32 <= p.rows;

    // U pieces (k step s, column block cb): element (kk, j) is
    // [16 s + kk <= 32 cb + j]; hi only (lo is 0 for 0 and 1).
    half8_t U[4][2];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
            mfmae::foreach_ij<FragB>([&](int e, int kk, int j) {
                U[s][cb][e] = (16 * s + kk <= 32 * cb + j) ? (_Float16)1.0f : (_Float16)0.0f;
            });

    float carry[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) carry[e] = 0.0f;

    auto fast_at = [&](int c0) { return p.vec && rows_full && c0 + 64 <= p.len; };
    Chunk cur;
    load_chunk(cur, p, r0, 0, fast_at(0));
    for (int c0 = 0; c0 < p.len; c0 += 64) {
        Chunk nxt;
        const int c1 = c0 + 64;
        if (c1 < p.len) load_chunk(nxt, p, r0, c1, fast_at(c1));

        half8_t xh[4], xl[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) mfmae::tcec::split8(cur.x[s], xh[s], xl[s]);
        f32x16_t acc[2], cor[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[cb][e] = 0.0f;
                cor[cb][e] = 0.0f;
            }
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                if (cb == 0 && s >= 2) continue;  // that piece of U is zero
                acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(xh[s], U[s][cb], acc[cb], 0, 0, 0);
                cor[cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(xl[s], U[s][cb], cor[cb], 0, 0, 0);
            }

        // y = carry + (acc + cor 2^-11); element e of block cb is row
        // 8 (e / 4) + 4 (l / 32) + e % 4, column c0 + 32 cb + l % 32
        float y[2][16];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                y[cb][e] = carry[e] +
                           __builtin_fmaf(cor[cb][e], mfmae::tcec::kLoScaleInv, acc[cb][e]);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int col = c0 + 32 * cb + (l & 31);
            if (col < p.len) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int64_t row = r0 + mfmae::layout<Shape32, Use::Acc>::row(l, e);
                    if (rows_full || row < p.rows) p.Y[row * p.ldy + col] = y[cb][e];
                }
            }
        }
        // running totals: column 63 of this chunk, held by lane 31 + 32 (l / 32)
        // for the same rows as this lane's elements
        const int src = 31 + 32 * (l >> 5);
#pragma unroll
        for (int e = 0; e < 16; ++e) carry[e] = __shfl(y[1][e], src, 64);
        if (c1 < p.len) cur = nxt;
    }
}

}  // namespace

hipError_t launch_scan(const ScanArgs& a, hipStream_t stream) {
    const int64_t groups = (a.rows + 31) / 32;
    const int64_t blocks = (groups + kWaves - 1) / kWaves;
    if (blocks >= (int64_t(1) << 31) / (64 * kWaves)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(scan_kernel, dim3((unsigned)blocks), dim3(64 * kWaves), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sgemm_emu
