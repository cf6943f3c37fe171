// Emulated SGEMM for large products (Sec. 4.4): full 256 x 128 tiles of C,
// split once per workgroup at staging, hi/lo planes in LDS.
//
// Per k chunk of 32, every thread loads 24 FP32 operand elements from global
// memory into registers (A: two runs of 8 consecutive k of one row; B: 8
// consecutive k of one column, one 256-byte row segment per wave and load),
// splits them there and writes 16-byte hi and lo pieces to LDS, so each
// element is split once per workgroup and LDS holds 2 + 2 bytes per element,
// the footprint of the FP32 data.  Eight waves of 64 x 64 read their operand
// vectors with one 16-byte LDS read per fragment and run 3 MFMAs per 32 x 32
// block and 16-wide k step (v_mfma_f32_32x32x16_f16), main and correction
// products in separate accumulators.
//
// LDS layout: a plane (A hi, A lo, B hi, B lo) is [row][4 pieces of 8
// halves], 64 bytes per row, no padding; piece q of row r is stored at
// position q ^ ((r ^ (r >> 2)) & 3).  Measured on gfx950 (16-byte LDS
// accesses, timed against a linear pattern), this swizzle makes all three
// access patterns conflict-free: the fragment reads (lanes 0..31 rows
// r..r+31 at one piece, lanes 32..63 the next piece), the A staging writes (4
// lanes per row, one piece each) and the B staging writes (one row per lane,
// one piece); unswizzled 64-byte rows give 4-way conflicts on the reads.
//
// Pipeline: two LDS stages and two register stages.  In iteration c the
// workgroup computes chunk c, writes chunk c + 1 (loaded two iterations
// earlier) to LDS, issues the loads of chunk c + 3 into the registers just
// freed, and meets at one barrier that orders LDS only (global loads stay in
// flight across it).  Every load and store of the loop is unconditional --
// chunk indices past the end are clamped to the last chunk -- so the waits
// before each use are for that stage's loads only.
//
// Only full tiles: m % 256 == 0, n % 128 == 0, k % 32 == 0, 16-byte aligned
// rows; other shapes take the general LDS kernel.
#include "internal.h"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"
#include "sgemm_emu.h"
#include "tiling.hpp"

namespace sgemm_emu {

using mfmae::f32x16_t;
using mfmae::half8_t;

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 256, BN = 128, BK = 32;
constexpr int WM = 64, WN = 64, WAVES_N = BN / WN;
constexpr int NT = 512;  // 8 waves, two per SIMD
constexpr int TM = WM / 32, TN = WN / 32;
constexpr int ROW_BYTES = 2 * BK;  // one row of a binary16 plane
constexpr int A_PLANE = BM * ROW_BYTES;
constexpr int B_PLANE = BN * ROW_BYTES;
constexpr int STAGE_BYTES = 2 * A_PLANE + 2 * B_PLANE;  // 48 KiB
constexpr int LDS_BYTES = 2 * STAGE_BYTES;              // 96 KiB
constexpr int A_UNITS = BM * (BK / 8) / NT;             // 8-element A runs per thread: 2

struct BigParams {
    int k;
    const float* A;
    int64_t lda, sa;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int tiles_m, tiles_n;
    int ntasks;  // (items of this launch) x (tiles per item)
    int item0;
};

// Byte offset of piece q (8 halves) of row r in a plane.
__device__ inline int piece(int r, int q) {
    return r * ROW_BYTES + 16 * (q ^ ((r ^ (r >> 2)) & 3));
}

// Registers of one staged chunk.
struct Stage {
    f32x4 a[A_UNITS][2];
    float b[8];
};

// Per-thread staging coordinates (constant over the k loop).
struct StageMap {
    const float* a[A_UNITS];  // A[m0 + row][8 q]
    const float* b;           // B[8 kg][n0 + n]
    int64_t ldb;
    int a_lds[A_UNITS];       // piece(row, q)
    int b_lds;                // piece(n, kg)
};

__device__ inline void load_stage(Stage& st, const StageMap& sm, int k0) {
#pragma unroll
    for (int u = 0; u < A_UNITS; ++u) {
        st.a[u][0] = *reinterpret_cast<const f32x4*>(sm.a[u] + k0);
        st.a[u][1] = *reinterpret_cast<const f32x4*>(sm.a[u] + k0 + 4);
    }
    const float* bp = sm.b + (int64_t)k0 * sm.ldb;
#pragma unroll
    for (int v = 0; v < 8; ++v) st.b[v] = bp[(int64_t)v * sm.ldb];
}

// Split the staged chunk and write its hi and lo pieces to LDS stage `buf`.
__device__ inline void store_stage(const Stage& st, const StageMap& sm, unsigned char* buf) {
    unsigned char* a_hi = buf;
    unsigned char* a_lo = buf + A_PLANE;
    unsigned char* b_hi = buf + 2 * A_PLANE;
    unsigned char* b_lo = b_hi + B_PLANE;
#pragma unroll
    for (int u = 0; u < A_UNITS; ++u) {
        const float x[8] = {st.a[u][0][0], st.a[u][0][1], st.a[u][0][2], st.a[u][0][3],
                            st.a[u][1][0], st.a[u][1][1], st.a[u][1][2], st.a[u][1][3]};
        half8_t hi, lo;
        mfmae::tcec::split8(x, hi, lo);
        *reinterpret_cast<half8_t*>(a_hi + sm.a_lds[u]) = hi;
        *reinterpret_cast<half8_t*>(a_lo + sm.a_lds[u]) = lo;
    }
    half8_t hi, lo;
    mfmae::tcec::split8(st.b, hi, lo);
    *reinterpret_cast<half8_t*>(b_hi + sm.b_lds) = hi;
    *reinterpret_cast<half8_t*>(b_lo + sm.b_lds) = lo;
}

// Both 16-wide k steps of one chunk from LDS stage `buf`.
__device__ inline void compute_stage(f32x16_t (&acc)[TM][TN], f32x16_t (&cor)[TM][TN],
                                     const unsigned char* buf, int wrow, int wcol, int g, int j) {
    const unsigned char* a_hi = buf;
    const unsigned char* a_lo = buf + A_PLANE;
    const unsigned char* b_hi = buf + 2 * A_PLANE;
    const unsigned char* b_lo = b_hi + B_PLANE;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
        const int q = 2 * s + g;  // k = 16 s + 8 g + (0..7), the same for A and B
        half8_t ahi[TM], alo[TM], bhi[TN], blo[TN];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
            const int o = piece(wrow + 32 * tm + j, q);
            ahi[tm] = *reinterpret_cast<const half8_t*>(a_hi + o);
            alo[tm] = *reinterpret_cast<const half8_t*>(a_lo + o);
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
            const int o = piece(wcol + 32 * tn + j, q);
            bhi[tn] = *reinterpret_cast<const half8_t*>(b_hi + o);
            blo[tn] = *reinterpret_cast<const half8_t*>(b_lo + o);
        }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
                acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], bhi[tn], acc[tm][tn],
                                                                     0, 0, 0);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
                cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[tm], bhi[tn], cor[tm][tn],
                                                                     0, 0, 0);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
                cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], blo[tn], cor[tm][tn],
                                                                     0, 0, 0);
    }
}

// Barrier that orders LDS accesses only: outstanding global loads stay in
// flight across it.
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__global__ __launch_bounds__(NT, 2) void bgemm_big_kernel(BigParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_BYTES];

    const int task = xcd_task(blockIdx.x, gridDim.x);
    if (task >= p.ntasks) return;  // the whole workgroup leaves together
    const int tiles = p.tiles_m * p.tiles_n;
    const int item = task / tiles;
    const int t = task - item * tiles;
    // tiles in groups of 8 tile rows, so that the workgroups running at the
    // same time on one XCD share B columns
    constexpr int GROUP_M = 8;
    const int group_size = GROUP_M * p.tiles_n;
    const int grp = t / group_size;
    const int first_m = grp * GROUP_M;
    const int gm = min(p.tiles_m - first_m, GROUP_M);
    const int r = t - grp * group_size;
    const int m0 = (first_m + r % gm) * BM;
    const int n0 = (r / gm) * BN;

    const int64_t it = (int64_t)item + p.item0;
    const float* __restrict__ Ab = p.A + it * p.sa;
    const float* __restrict__ Bb = p.B + it * p.sb;
    float* __restrict__ Cb = p.C + it * p.sc;

    const int tid = threadIdx.x;
    StageMap sm;
#pragma unroll
    for (int u = 0; u < A_UNITS; ++u) {
        const int unit = u * NT + tid;
        const int row = unit >> 2, q = unit & 3;
        sm.a[u] = Ab + (int64_t)(m0 + row) * p.lda + 8 * q;
        sm.a_lds[u] = piece(row, q);
    }
    {
        const int n = tid & (BN - 1), kg = tid / BN;
        sm.b = Bb + (int64_t)(8 * kg) * p.ldb + n0 + n;
        sm.ldb = p.ldb;
        sm.b_lds = piece(n, kg);
    }

    const int wave = tid >> 6;
    const int l = tid & 63;
    const int g = l >> 5, j = l & 31;
    const int wrow = (wave / WAVES_N) * WM;
    const int wcol = (wave % WAVES_N) * WN;

    f32x16_t acc[TM][TN], cor[TM][TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[tm][tn][e] = 0.0f;
                cor[tm][tn][e] = 0.0f;
            }

    const int nk = p.k / BK;  // >= 1
    const int last = nk - 1;
    unsigned char* buf0 = smem;
    unsigned char* buf1 = smem + STAGE_BYTES;
    Stage r0, r1;
    load_stage(r0, sm, 0);
    load_stage(r1, sm, BK * min(1, last));
    store_stage(r0, sm, buf0);
    load_stage(r0, sm, BK * min(2, last));
    lds_barrier();
    // iteration c: compute chunk c, store chunk c + 1, load chunk c + 3.
    // The MFMAs of chunk c are issued first; they run in the matrix unit
    // while the same wave splits chunk c + 1 on the VALU.
    int c = 0;
    for (; c + 2 <= nk; c += 2) {
        compute_stage(acc, cor, buf0, wrow, wcol, g, j);
        store_stage(r1, sm, buf1);
        load_stage(r1, sm, BK * min(c + 3, last));
        lds_barrier();
        compute_stage(acc, cor, buf1, wrow, wcol, g, j);
        store_stage(r0, sm, buf0);
        load_stage(r0, sm, BK * min(c + 4, last));
        lds_barrier();
    }
    if (c < nk) compute_stage(acc, cor, buf0, wrow, wcol, g, j);

    // Epilogue: C = main + corr * 2^-11.  Element e of a 32 x 32 block is
    // row 8 (e / 4) + 4 g + e % 4, column j.
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
            float* cp = Cb + (int64_t)(m0 + wrow + 32 * tm + 4 * g) * p.ldc + n0 + wcol + 32 * tn + j;
#pragma unroll
            for (int e = 0; e < 16; ++e)
                cp[(int64_t)(8 * (e >> 2) + (e & 3)) * p.ldc] =
                    __builtin_fmaf(cor[tm][tn][e], mfmae::tcec::kLoScaleInv, acc[tm][tn][e]);
        }
}

}  // namespace

bool big_supported(const GemmArgs& a) {
    return a.m % BM == 0 && a.n % BN == 0 && a.k % BK == 0 && a.k > 0 && a.vec_a && a.vec_b;
}

hipError_t launch_gemm_big(const GemmArgs& a, hipStream_t stream) {
    if (!big_supported(a)) return hipErrorInvalidValue;
    BigParams p;
    p.k = a.k;
    p.A = a.A;
    p.lda = a.lda;
    p.sa = a.sa;
    p.B = a.B;
    p.ldb = a.ldb;
    p.sb = a.sb;
    p.C = a.C;
    p.ldc = a.ldc;
    p.sc = a.sc;
    p.tiles_m = a.m / BM;
    p.tiles_n = a.n / BN;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    // one launch stays below 2^31 work-items
    const int64_t max_tasks = (int64_t(1) << 31) / NT - 1;
    if (tiles > max_tasks) return hipErrorInvalidConfiguration;
    const int64_t items_per_launch = max_tasks / tiles;
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        p.ntasks = (int)(items * tiles);
        p.item0 = (int)i0;
        hipLaunchKernelGGL(bgemm_big_kernel, dim3((unsigned)p.ntasks), dim3(NT), 0, stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace sgemm_emu
