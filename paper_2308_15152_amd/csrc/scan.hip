// Batched inclusive scan y_j = sum_{i <= j} x_i of every row, as the product
// x^T U with the upper-triangular all-ones U (Sec. 4.1, eq. scan-mat, rule
// u-rule), in emulated FP32 (Sec. 4.4).
//
// A wavefront scans whole rows, 1024 values (a block) at a time.  The block
// is read as a 32 x 32 matrix Z of 32 consecutive segments (Z[n][k] is value
// 32 n + k of the block) and scanned in two levels:
//   * within segments, as the transposed product S^T = U^T Z^T: U^T's
//     32 x 32 block is the A operand, built once per wave with foreach_ij
//     from the rule (element (i, k) of U^T is [k <= i]) and never stored; Z
//     is the B operand (two 16-wide k steps, split into hi and lo in
//     registers).  U's entries are 0 and 1, whose lo parts are 0, so the
//     correction reduces to U^T lo(Z^T): four MFMAs per block;
//   * across segments, an exclusive scan of the 32 segment totals over the
//     lanes (five shuffle steps), plus the running total of the row's
//     earlier blocks, added to every value of the segment.
// Lane (n, g) = (l % 32, l / 32) holds values 32 n + 16 s + 8 g .. + 7 of the
// block as its operand and, as its accumulator, outputs 32 n + 8 q + 4 g ..
// + 3 for q = 0..3: every load and store is 16 bytes, and one wave's
// instructions together cover a contiguous 4 KiB.  Over whole blocks of
// 16-byte aligned rows the loads of the next kBuf blocks are in flight while
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
using FragA = mfmae::fragment<Shape32, Use::A, _Float16>;

constexpr int kWaves = 4;

constexpr int kBuf = 4;         // block buffers per wave
constexpr int kRowsPerWave = 8;  // rows a wave scans, one after another

// The 16 values lane (n, g) holds of a block as B operand: block values
// 32 n + 16 s + 8 g + v, s = 0, 1, v = 0..7.
struct Block {
    float x[2][8];
};

// A block as loaded on the whole-block path: lane l holds values
// 256 i + 4 l .. + 3, i = 0..3, so every load instruction reads 1 KiB of
// whole cache lines.
struct Raw {
    f32x4 v[4];
};

// Whole block inside a 16-byte aligned row: four contiguous 16-byte loads.
__device__ inline void load_fast(Raw& b, const float* row, int c0) {
    const int l = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < 4; ++i) b.v[i] = *reinterpret_cast<const f32x4*>(row + c0 + 256 * i + 4 * l);
}

// The wave's LDS copy of one block: segment n (32 values) at 36 n floats.
// With this pitch the 16-byte accesses of the operand and accumulator
// layouts (lanes n = 0..15 at 36 n + c) fall on distinct banks.
constexpr int kSegPitch = 36;
constexpr int kStageFloats = 32 * kSegPitch;

__device__ inline int staged(int value) { return kSegPitch * (value >> 5) + (value & 31); }

// Regroup a contiguous block into the operand layout through the wave's
// LDS buffer (other lanes' values: ordered by the wave fence).
__device__ inline void to_operand(const Raw& r, float* buf, Block& b) {
    const int l = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<f32x4*>(buf + staged(256 * i + 4 * l)) = r.v[i];
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
    const float* q = buf + kSegPitch * (l & 31) + 8 * (l >> 5);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const f32x4 v0 = *reinterpret_cast<const f32x4*>(q + 16 * s);
        const f32x4 v1 = *reinterpret_cast<const f32x4*>(q + 16 * s + 4);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            b.x[s][v] = v0[v];
            b.x[s][v + 4] = v1[v];
        }
    }
}

// Any block: element loads, zero past the row's end.
__device__ inline void load_bounded(Block& b, const float* row, int c0, int len) {
    const int l = threadIdx.x & 63;
    const int base = c0 + 32 * (l & 31) + 8 * (l >> 5);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            const int cc = base + 16 * s + v;
            b.x[s][v] = cc < len ? row[cc] : 0.0f;
        }
}

// y = carry + scan of the block; carry becomes the row's running total
// after it.  Accumulator element e of lane (n, g) is block value
// 32 n + 8 (e / 4) + 4 g + e % 4.
__device__ inline void scan_block(const Block& b, const half8_t (&Ut)[2], float& carry,
                                  float (&y)[16]) {
    const int l = threadIdx.x & 63;
    const int n = l & 31;
    f32x16_t acc, cor;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        acc[e] = 0.0f;
        cor[e] = 0.0f;
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        half8_t xh, xl;
        mfmae::tcec::split8(b.x[s], xh, xl);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(Ut[s], xh, acc, 0, 0, 0);
        cor = __builtin_amdgcn_mfma_f32_32x32x16_f16(Ut[s], xl, cor, 0, 0, 0);
    }
    // scans within the segments
    float z[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) z[e] = __builtin_fmaf(cor[e], mfmae::tcec::kLoScaleInv, acc[e]);
    // segment totals: the last value of segment n is element 15 of lane
    // 32 + n; inclusive scan of the totals over n (both half-waves hold it)
    float incl = __shfl(z[15], 32 + n, 64);
#pragma unroll
    for (int d = 1; d < 32; d *= 2) {
        const float u = __shfl_up(incl, d, 32);
        if (n >= d) incl += u;
    }
    const float before = __shfl_up(incl, 1, 32);  // total of segments 0..n-1
    const float offset = n == 0 ? carry : carry + before;
#pragma unroll
    for (int e = 0; e < 16; ++e) y[e] = offset + z[e];
    carry = carry + __shfl(incl, 31, 64);
}

// Outputs in the accumulator layout, regrouped through the wave's LDS
// buffer and stored as four contiguous 1 KiB instructions, nontemporal: y
// is not read again (measured 2.7% faster; the rule-built kernels, whose
// output stores interleave with the next item's loads, ran 2-3% slower
// with them).
__device__ inline void store_fast(float* row, int c0, const float (&y)[16], float* buf) {
    const int l = threadIdx.x & 63;
    float* q = buf + kSegPitch * (l & 31) + 4 * (l >> 5);
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");  // operand reads done
#pragma unroll
    for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(q + 8 * g) = f32x4{y[4 * g], y[4 * g + 1], y[4 * g + 2],
                                                     y[4 * g + 3]};
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
#pragma unroll
    for (int i = 0; i < 4; ++i)
        __builtin_nontemporal_store(*reinterpret_cast<const f32x4*>(buf + staged(256 * i + 4 * l)),
                                    reinterpret_cast<f32x4*>(row + c0 + 256 * i + 4 * l));
}

__device__ inline void store_bounded(float* row, int c0, int len, const float (&y)[16]) {
    const int l = threadIdx.x & 63;
    const int base = c0 + 32 * (l & 31) + 4 * (l >> 5);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int col = base + 8 * (e >> 2) + (e & 3);
        if (col < len) row[col] = y[e];
    }
}

__global__ __launch_bounds__(64 * kWaves, 2) void scan_kernel(ScanArgs p) {
    __shared__ __attribute__((aligned(16))) float stage[kWaves][kStageFloats];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t r_first = ((int64_t)blockIdx.x * kWaves + wave) * kRowsPerWave;
    if (r_first >= p.rows) return;  // whole wave; no barrier below
    const int nrows = (int)min((int64_t)kRowsPerWave, p.rows - r_first);

    // U^T's diagonal block for k step s: element (i, kk) is [16 s + kk <= i];
    // hi only (lo is 0 for 0 and 1).
    half8_t Ut[2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
        mfmae::foreach_ij<FragA>([&](int e, int i, int kk) {
            Ut[s][e] = (16 * s + kk <= i) ? (_Float16)1.0f : (_Float16)0.0f;
        });

    float carry = 0.0f;
    float y[16];

    if (p.vec && p.len % 1024 == 0) {
        // Whole blocks of aligned rows, as one sequence f = (row, block) of
        // nf blocks: kBuf block buffers in turn.  A step scans one buffer's
        // block, stores it and reloads the buffer with block f + kBuf.  Loads
        // are unconditional (past the end they re-read the last block) and
        // the first round of steps is peeled, so the loop is entered with the
        // same memory operations pending as on every later iteration and the
        // wait before each block covers that block's loads only.
        const int nb = p.len / 1024;
        const int nf = nrows * nb;
        const int last = nf - 1;
        auto row_in = [&](int f) { return p.X + (r_first + f / nb) * p.ldx; };
        auto row_out = [&](int f) { return p.Y + (r_first + f / nb) * p.ldy; };
        float* sb = stage[wave];
        auto load = [&](Raw& b, int f) {
            const int fc = min(f, last);
            load_fast(b, row_in(fc), 1024 * (fc % nb));
        };
        // the scheduling barrier keeps each step's reload in place, so the
        // blocks really are loaded kBuf steps ahead
        auto step = [&](Raw& r, int f) {
            if (f % nb == 0) carry = 0.0f;
            Block b;
            to_operand(r, sb, b);
            scan_block(b, Ut, carry, y);
            store_fast(row_out(f), 1024 * (f % nb), y, sb);
            load(r, f + kBuf);
            __builtin_amdgcn_sched_barrier(0);
        };
        Raw buf[kBuf];
#pragma unroll
        for (int i = 0; i < kBuf; ++i) load(buf[i], i);
        int f = 0;
        if (nf >= kBuf) {
#pragma unroll
            for (int i = 0; i < kBuf; ++i) step(buf[i], i);
            for (f = kBuf; f + kBuf <= nf; f += kBuf) {
#pragma unroll
                for (int i = 0; i < kBuf; ++i) step(buf[i], f + i);
            }
        }
        // buf[i] holds block f + i for the remaining blocks
#pragma unroll
        for (int i = 0; i < kBuf - 1; ++i) {
            if (f + i < nf) {
                if ((f + i) % nb == 0) carry = 0.0f;
                Block b;
                to_operand(buf[i], sb, b);
                scan_block(b, Ut, carry, y);
                store_fast(row_out(f + i), 1024 * ((f + i) % nb), y, sb);
            }
        }
        return;
    }
    // any length or alignment: element loads and stores, one block at a time
    for (int r = 0; r < nrows; ++r) {
        const float* xin = p.X + (r_first + r) * p.ldx;
        float* yout = p.Y + (r_first + r) * p.ldy;
        carry = 0.0f;
        for (int c0 = 0; c0 < p.len; c0 += 1024) {
            Block b;
            load_bounded(b, xin, c0, p.len);
            scan_block(b, Ut, carry, y);
            store_bounded(yout, c0, p.len, y);
        }
    }
}

}  // namespace

hipError_t launch_scan(const ScanArgs& a, hipStream_t stream) {
    // one launch stays below 2^31 work-items (the dispatch packet counts
    // work-items in 32 bits); more rows take several launches, each on its
    // own range of rows
    const int64_t max_blocks = (int64_t(1) << 31) / (64 * kWaves) - 1;
    const int64_t rows_per_launch = max_blocks * kWaves * kRowsPerWave;
    for (int64_t r0 = 0; r0 < a.rows; r0 += rows_per_launch) {
        ScanArgs c = a;
        c.rows = a.rows - r0 < rows_per_launch ? a.rows - r0 : rows_per_launch;
        c.X = a.X + r0 * a.ldx;
        c.Y = a.Y + r0 * a.ldy;
        const int64_t waves = (c.rows + kRowsPerWave - 1) / kRowsPerWave;
        const int64_t blocks = (waves + kWaves - 1) / kWaves;
        hipLaunchKernelGGL(scan_kernel, dim3((unsigned)blocks), dim3(64 * kWaves), 0, stream, c);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace sgemm_emu
