// Batched emulated SGEMM with register-direct operand fragments (Sec. 4.2 and
// 4.4): every wave loads its A and B operand elements from global memory
// straight into the VGPRs the MFMA operands are built from, splits them there
// and issues the three products.  Nothing goes through LDS and the kernel has
// no barrier, so each wave streams independently and the hardware keeps the
// loads of every resident wave in flight at once.  This is the flow for
// batches of small products, which are bound by HBM bandwidth: what limits
// them is keeping enough bytes in flight while the splits and MFMAs run, not
// LDS or MFMA throughput.  Two waves per SIMD let one wave's split overlap
// the other's MFMAs and loads.
//
// Work split: a workgroup of WAVES_M x WAVES_N waves covers a BM x BN tile
// of one item; a wave owns a WM x WN sub-tile made of TM x TN blocks of
// 32 x 32 (v_mfma_f32_32x32x16_f16).  Waves that share A rows or B columns
// share them through the L1/L2 caches.
//
// Operand loads per 16-wide k step (g = lane / 32, j = lane % 32):
//   A block tm: lane reads A[row(tm, j)][k0 + 8 g .. k0 + 8 g + 7], two
//     16-byte loads of consecutive k (the operand's own k order);
//   B: the TN blocks of a wave interleave their columns: column j of block tn
//     is global column n0 + TN j + tn.  A lane then needs, for each of its
//     eight k rows, the TN consecutive floats B[k][n0 + TN j .. + TN - 1],
//     one TN-wide vector load, and 32 lanes read TN * 128 contiguous bytes
//     of a row.  The permutation of output columns is undone by the store,
//     which writes the same TN-wide vectors to C.
//
// D k steps are in flight per wave (a register ring of depth D): the loads
// of step s + D are issued as soon as step s has been split, so they overlap
// the MFMAs of the steps in between.
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

template <int N>
struct fvec;
template <>
struct fvec<1> {
    typedef float type;
    __device__ static float get(type v, int) { return v; }
    __device__ static type make(const float* x) { return x[0]; }
};
template <>
struct fvec<2> {
    typedef float type __attribute__((ext_vector_type(2)));
    __device__ static float get(type v, int i) { return v[i]; }
    __device__ static type make(const float* x) { return type{x[0], x[1]}; }
};
template <>
struct fvec<4> {
    typedef float type __attribute__((ext_vector_type(4)));
    __device__ static float get(type v, int i) { return v[i]; }
    __device__ static type make(const float* x) { return type{x[0], x[1], x[2], x[3]}; }
};

template <int TM_, int TN_, int D_, int WAVES_PER_SIMD_, int WAVES_M_, int WAVES_N_, bool EC_>
struct RegCfg {
    static constexpr int TM = TM_, TN = TN_;
    static constexpr int D = D_;  // k steps in flight per wave
    static constexpr int WAVES_PER_SIMD = WAVES_PER_SIMD_;
    static constexpr bool EC = EC_;
    static constexpr int WM = 32 * TM, WN = 32 * TN;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int NT = 64 * WAVES_M * WAVES_N;
    static constexpr int BM = WAVES_M * WM, BN = WAVES_N * WN;
    using bvec = fvec<TN>;
    using bvec_t = typename bvec::type;
};

// Raw FP32 operand elements of one 16-wide k step.
template <class CF>
struct Slot {
    f32x4 a[CF::TM][2];
    typename CF::bvec_t b[8];
};

// Addressing of one wave's sub-tile: wave-uniform base pointers (scalar
// registers) plus one 32-bit byte offset per lane, so every load is a
// scalar-base + vector-offset global load and advancing k is scalar work.
template <class CF>
struct Lanes {
    const float* a;          // A[wm0][0] of this item
    const float* b;          // B[0][wn0] of this item
    int64_t ldb;
    uint32_t a_off[CF::TM];  // bytes to A[row of block tm][8 g]
    uint32_t b_off;          // bytes to B[8 g][this lane's first column]
};

template <class T>
__device__ inline T load_at(const float* base, uint32_t byte_off) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}

template <class CF>
__device__ inline void load_full(Slot<CF>& s, const Lanes<CF>& ln, int k0) {
    const float* ak = ln.a + k0;
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm) {
        s.a[tm][0] = load_at<f32x4>(ak, ln.a_off[tm]);
        s.a[tm][1] = load_at<f32x4>(ak, ln.a_off[tm] + 16);
    }
#pragma unroll
    for (int v = 0; v < 8; ++v)
        s.b[v] = load_at<typename CF::bvec_t>(ln.b + (int64_t)(k0 + v) * ln.ldb, ln.b_off);
}

// The last, partial k step: elements with k >= K read as zero.  kk is this
// lane's first k (k0 + 8 g).
template <class CF>
__device__ inline void load_tail(Slot<CF>& s, const Lanes<CF>& ln, int k0, int kk, int K) {
    const float* ak = ln.a + k0;
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k = kk + 4 * h + e;
                s.a[tm][h][e] = k < K ? load_at<float>(ak, ln.a_off[tm] + 16 * h + 4 * e) : 0.0f;
            }
#pragma unroll
    for (int v = 0; v < 8; ++v) {
        if (kk + v < K) {
            s.b[v] = load_at<typename CF::bvec_t>(ln.b + (int64_t)(k0 + v) * ln.ldb, ln.b_off);
        } else {
            const float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            s.b[v] = CF::bvec::make(z);
        }
    }
}

// Split one k step in registers and issue its MFMAs.
template <class CF>
__device__ inline void compute(f32x16_t (&acc)[CF::TM][CF::TN], f32x16_t (&cor)[CF::TM][CF::TN],
                               const Slot<CF>& s) {
    half8_t ahi[CF::TM], alo[CF::TM], bhi[CF::TN], blo[CF::TN];
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm) {
        const float x[8] = {s.a[tm][0][0], s.a[tm][0][1], s.a[tm][0][2], s.a[tm][0][3],
                            s.a[tm][1][0], s.a[tm][1][1], s.a[tm][1][2], s.a[tm][1][3]};
        mfmae::tcec::split8(x, ahi[tm], alo[tm]);
    }
#pragma unroll
    for (int tn = 0; tn < CF::TN; ++tn) {
        float x[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) x[v] = CF::bvec::get(s.b[v], tn);
        mfmae::tcec::split8(x, bhi[tn], blo[tn]);
    }
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < CF::TN; ++tn)
            acc[tm][tn] =
                __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], bhi[tn], acc[tm][tn], 0, 0, 0);
    if constexpr (CF::EC) {
#pragma unroll
        for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                cor[tm][tn] =
                    __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[tm], bhi[tn], cor[tm][tn], 0, 0, 0);
#pragma unroll
        for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                cor[tm][tn] =
                    __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], blo[tn], cor[tm][tn], 0, 0, 0);
    }
}

struct RegParams {
    int m, n, k;
    const float* A;
    int64_t lda, sa;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int tiles_m, tiles_n;
    int ntasks;  // (items of this launch) x (tiles per item)
    int item0;
    int vec_c;   // TN-wide vector stores to C are legal
};

template <class CF>
__global__ __launch_bounds__(CF::NT, CF::WAVES_PER_SIMD) void bgemm_reg_kernel(RegParams p) {
    // Items of one tile share no operand: plain dispatch order (measured 5-7%
    // faster than the XCD-aware numbering on 4096 x 128^3 with 128 x 128
    // tiles); otherwise an item's tiles stay in one XCD's L2.
    const int task =
        p.tiles_m * p.tiles_n == 1 ? (int)blockIdx.x : xcd_task(blockIdx.x, gridDim.x);
    if (task >= p.ntasks) return;
    const int tiles = p.tiles_m * p.tiles_n;
    const int item = task / tiles;
    const TileRC rc = grouped_tile(task - item * tiles, p.tiles_m, p.tiles_n);
    const int tile_m = rc.tm;
    const int tile_n = rc.tn;

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    const int g = l >> 5, j = l & 31;
    const int wm0 = tile_m * CF::BM + (wave / CF::WAVES_N) * CF::WM;
    const int wn0 = tile_n * CF::BN + (wave % CF::WAVES_N) * CF::WN;
    // A wave whose whole sub-tile lies outside C has nothing to do (the
    // kernel has no barrier, so it may leave on its own).
    if (wm0 >= p.m || wn0 >= p.n) return;

    const int64_t it = (int64_t)item + p.item0;
    const float* __restrict__ Ab = p.A + it * p.sa;
    const float* __restrict__ Bb = p.B + it * p.sb;
    float* __restrict__ Cb = p.C + it * p.sc;

    // Rows beyond m and column groups beyond n read the last valid row /
    // group (their results are never stored); n is a multiple of TN here,
    // and wm0 < m, wn0 <= n - TN, so every offset is non-negative.
    Lanes<CF> ln;
    ln.a = Ab + (int64_t)wm0 * p.lda;
    ln.b = Bb + wn0;
    ln.ldb = p.ldb;
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm) {
        const int row = min(wm0 + 32 * tm + j, p.m - 1);
        ln.a_off[tm] = (uint32_t)(((row - wm0) * p.lda + 8 * g) * 4);
    }
    const int col = wn0 + CF::TN * j;
    ln.b_off = (uint32_t)(((int64_t)(8 * g) * p.ldb + min(col, p.n - CF::TN) - wn0) * 4);

    f32x16_t acc[CF::TM][CF::TN], cor[CF::TM][CF::TN];
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < CF::TN; ++tn)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[tm][tn][e] = 0.0f;
                cor[tm][tn][e] = 0.0f;
            }

    // k steps, D in flight.  The first nfull % D steps run one at a time;
    // the rest, a multiple of D, stream through the register ring: the
    // loads of step s + D are issued as soon as step s is split, and every
    // load is issued on a path with no data-dependent branch between it and
    // the steps it overlaps, so the wait before a step is for that step's
    // own loads only.
    const int nfull = p.k / 16;
    const int lead = nfull % CF::D;
    Slot<CF> ring[CF::D];
    for (int e = 0; e < lead; ++e) {
        load_full<CF>(ring[0], ln, 16 * e);
        compute<CF>(acc, cor, ring[0]);
    }
    const int nring = nfull - lead;
    if (nring > 0) {
#pragma unroll
        for (int d = 0; d < CF::D; ++d) load_full<CF>(ring[d], ln, 16 * (lead + d));
        for (int s = lead; s + CF::D < nfull; s += CF::D) {
#pragma unroll
            for (int d = 0; d < CF::D; ++d) {
                compute<CF>(acc, cor, ring[d]);
                load_full<CF>(ring[d], ln, 16 * (s + CF::D + d));
            }
        }
#pragma unroll
        for (int d = 0; d < CF::D; ++d) compute<CF>(acc, cor, ring[d]);
    }
    Slot<CF>& s0 = ring[0];
    if (p.k % 16 != 0) {
        const int k0 = 16 * nfull;
        load_tail<CF>(s0, ln, k0, k0 + 8 * g, p.k);
        compute<CF>(acc, cor, s0);
    }

    // Epilogue: C = main + corr * 2^-11.  Element e of block (tm, tn) is row
    // 8 (e / 4) + 4 g + e % 4 of the block and global column col + tn.
    if (col >= p.n) return;
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int row = wm0 + 32 * tm + 8 * (e >> 2) + 4 * g + (e & 3);
            if (row >= p.m) continue;
            float v[CF::TN];
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                v[tn] = CF::EC ? __builtin_fmaf(cor[tm][tn][e], mfmae::tcec::kLoScaleInv,
                                                acc[tm][tn][e])
                               : acc[tm][tn][e];
            float* dst = Cb + (int64_t)row * p.ldc + col;
            if (p.vec_c) {
                *reinterpret_cast<typename CF::bvec_t*>(dst) = CF::bvec::make(v);
            } else {
#pragma unroll
                for (int tn = 0; tn < CF::TN; ++tn) dst[tn] = v[tn];
            }
        }
}

template <class CF>
hipError_t launch_reg_cfg(const GemmArgs& a, hipStream_t stream) {
    RegParams p;
    p.m = a.m;
    p.n = a.n;
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
    p.tiles_m = cdiv(a.m, CF::BM);
    p.tiles_n = cdiv(a.n, CF::BN);
    p.vec_c = ((uintptr_t)a.C % (4 * CF::TN) == 0) && a.ldc % CF::TN == 0 && a.sc % CF::TN == 0;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    // one launch stays below 2^31 work-items (the dispatch packet counts
    // work-items in 32 bits); larger batches take several launches
    const int64_t max_tasks = (int64_t(1) << 31) / CF::NT - 1;
    if (tiles > max_tasks) return hipErrorInvalidConfiguration;
    const int64_t items_per_launch = max_tasks / tiles;
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        p.ntasks = (int)(items * tiles);
        p.item0 = (int)i0;
        hipLaunchKernelGGL(bgemm_reg_kernel<CF>, dim3((unsigned)p.ntasks), dim3(CF::NT), 0, stream,
                           p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int TM, int TN, int D, int W, int WAVES_M, int WAVES_N>
hipError_t launch_reg_tn(const GemmArgs& a, bool ec, hipStream_t stream) {
    return ec ? launch_reg_cfg<RegCfg<TM, TN, D, W, WAVES_M, WAVES_N, true>>(a, stream)
              : launch_reg_cfg<RegCfg<TM, TN, D, W, WAVES_M, WAVES_N, false>>(a, stream);
}

// B (and C) vector width of the 128x128 tile: 4 if the B rows allow 16-byte
// loads (waves of 32 x 128, four blocks interleaved), else 2 if they allow
// 8-byte loads (waves of 64 x 64), else 0.
int reg_width_128(const GemmArgs& a) {
    auto ok = [&](int w) {
        return ((uintptr_t)a.B % (4 * w) == 0) && a.ldb % w == 0 && a.sb % w == 0 && a.n % w == 0;
    };
    return ok(4) ? 4 : ok(2) ? 2 : 0;
}

}  // namespace

bool reg_flow_supported(const GemmArgs& a, int tile) {
    if (tile != SGEMM_EMU_TILE_64x64 && tile != SGEMM_EMU_TILE_128x128) return false;
    // per-lane byte offsets are 32-bit: 64 rows of A, 8 rows of B
    if (a.lda >= (int64_t(1) << 23) || a.ldb >= (int64_t(1) << 25)) return false;
    if (!a.vec_a) return false;  // 16-byte A loads along k
    return tile == SGEMM_EMU_TILE_64x64 || reg_width_128(a) > 0;
}

hipError_t launch_gemm_reg(const GemmArgs& a, int tile, bool ec, hipStream_t stream) {
    if (!reg_flow_supported(a, tile)) return hipErrorInvalidValue;
    // Two waves per SIMD in every variant: while one wave splits, the other's
    // MFMAs and loads proceed.  The register ring depth D is what fits in
    // the 256 registers a wave then has next to its accumulators.
    //   64x64 tile:   2 x 2 waves of 32 x 32,  3 k steps in flight
    //   128x128 tile: 4 x 1 waves of 32 x 128 (16-byte B loads), or
    //                 2 x 2 waves of 64 x 64 (8-byte B loads), 2 in flight
    if (tile == SGEMM_EMU_TILE_64x64) return launch_reg_tn<1, 1, 3, 2, 2, 2>(a, ec, stream);
    if (reg_width_128(a) == 4) return launch_reg_tn<1, 4, 2, 2, 4, 1>(a, ec, stream);
    return launch_reg_tn<2, 2, 2, 2, 2, 2>(a, ec, stream);
}

}  // namespace sgemm_emu
