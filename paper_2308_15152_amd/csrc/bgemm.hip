// Batched single-precision-emulating GEMM on gfx950 fp16 MFMA (Sec. 4.4).
//
// One workgroup computes a BM x BN tile of one batch item's C; its waves own
// WM x WN sub-tiles made of 32x32 MFMA blocks (v_mfma_f32_32x32x16_f16).
// The k dimension is walked in chunks of BK: FP32 tiles of A (BM x BK) and
// B (BK x BN) come from global memory in 16-byte coalesced loads into
// registers one chunk ahead, are written to a double-buffered LDS panel, and
// every wave reads its operand fragments from LDS with 16-byte conflict-free
// reads.  Per 16-wide k step and per 32x32 block three MFMAs run:
//     main += hiA.hiB,   corr += loA.hiB,   corr += hiA.loB
// and the epilogue stores C = main + corr * 2^-11 (one fma per element).
//
// Where the split to hi/lo happens is the FLOW policy:
//   FLOW_SPLIT  : split in registers between the global load and the LDS
//                 store; LDS holds hi and lo planes (2 + 2 bytes per element,
//                 the same footprint as FP32).  Each element is split once
//                 per workgroup.
//   FLOW_DIRECT : LDS holds FP32; each wave reads FP32 fragments and splits
//                 them in registers (the paper's direct fragment build,
//                 Fig. 6 bottom).  Each element is split once per wave that
//                 reads it.
//   FLOW_STAGED : LDS holds FP32; each wave converts its rows/columns to
//                 hi/lo, writes them to a private LDS area and reloads them
//                 as fragments (Fig. 6 top: the flow a load-only fragment
//                 API forces).  Measurement only.
//
// LDS rows are padded so that the 16-byte fragment reads of 16 consecutive
// lanes (16 rows, same k offset) fall into distinct banks: a row pitch of
// BK + 8 halves (80 bytes at BK = 32) or BK + 4 floats (144 bytes) moves
// consecutive rows by 20 or 36 dwords, i.e. by 4 * odd banks.
//
// B is stored transposed in LDS ([n][k], k contiguous) so that a lane's
// eight consecutive-k B elements are one 16-byte read, exactly like A.
// The transpose happens in registers during staging: a thread loads four
// consecutive rows of four consecutive columns and writes each column's four
// k values together.
#include <atomic>
#include <type_traits>

#include "internal.h"
#include "tiling.hpp"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"
#include "sgemm_emu.h"

namespace sgemm_emu {

using mfmae::f32x16_t;
using mfmae::half8_t;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum { FLOW_SPLIT = SGEMM_EMU_FLOW_SPLIT, FLOW_DIRECT = SGEMM_EMU_FLOW_DIRECT,
       FLOW_STAGED = SGEMM_EMU_FLOW_STAGED };


// Split four FP32 values into packed hi and lo halves (element e of the
// input goes to half e of the output pairs).
__device__ inline void split4(float x0, float x1, float x2, float x3, u32x2& hi, u32x2& lo) {
    uint32_t h0, l0, h1, l1;
    mfmae::tcec::split2(x0, x1, h0, l0);
    mfmae::tcec::split2(x2, x3, h1, l1);
    hi = u32x2{h0, h1};
    lo = u32x2{l0, l1};
}

template <int BM_, int BN_, int BK_, int WM_, int WN_, int FLOW_, bool EC_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int FLOW = FLOW_;
    static constexpr bool EC = EC_;
    static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
    static constexpr int NWAVES = WAVES_M * WAVES_N;
    static constexpr int NT = NWAVES * 64;
    static constexpr int TM = WM / 32, TN = WN / 32;
    static constexpr int KSTEPS = BK / 16;
    // staging: A in float4 along k, B in 4x4 (k x n) units
    static constexpr int A_F4 = BM * BK / 4;
    static constexpr int A_LOADS = cdiv(A_F4, NT);
    static constexpr int B_UNITS = (BK / 4) * (BN / 4);
    static constexpr int B_LOADS = cdiv(B_UNITS, NT);
    // LDS layout
    static constexpr int PH = BK + 8;  // halves per row, hi/lo planes
    static constexpr int PF = BK + 4;  // floats per row, FP32 panels
    static constexpr int PLANE_A = BM * PH * 2;  // bytes of one hi (or lo) A plane
    static constexpr int PLANE_B = BN * PH * 2;
    static constexpr int STAGE_SPLIT = 2 * PLANE_A + 2 * PLANE_B;
    static constexpr int STAGE_F32 = (BM + BN) * PF * 4;
    static constexpr int STAGE = FLOW == FLOW_SPLIT ? STAGE_SPLIT : STAGE_F32;
    static constexpr int WAVE_SCRATCH = FLOW == FLOW_STAGED ? (WM + WN) * PH * 2 * 2 : 0;
    static constexpr int LDS_BYTES = 2 * STAGE + NWAVES * WAVE_SCRATCH;

    static_assert(BM % WM == 0 && BN % WN == 0, "tile");
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile is made of 32x32 blocks");
    static_assert(BK % 16 == 0, "k chunk is a multiple of the MFMA k");
    static constexpr bool FITS = LDS_BYTES <= 160 * 1024;  // LDS of one CU
    // Waves per SIMD the register allocation must allow: two resident waves
    // per SIMD cap a wave at 256 registers (VGPR + AGPR).
    static constexpr int MIN_WAVES = 2;
};

// ---------------------------------------------------------------------------
// Global -> register staging of one k chunk.
// ---------------------------------------------------------------------------
template <class CF>
struct Stage {
    f32x4 a[CF::A_LOADS];
    f32x4 b[CF::B_LOADS][4];  // four consecutive k rows of four columns
};

template <class CF>
__device__ inline void load_chunk(Stage<CF>& st, const KParams& p, const float* __restrict__ Ab,
                                  const float* __restrict__ Bb, int m0, int n0, int k0) {
    const int t = threadIdx.x;
    const bool fullA = p.vec_a && (m0 + CF::BM <= p.m) && (k0 + CF::BK <= p.k);
    const bool fullB = p.vec_b && (n0 + CF::BN <= p.n) && (k0 + CF::BK <= p.k);
#pragma unroll
    for (int q = 0; q < CF::A_LOADS; ++q) {
        const int f = q * CF::NT + t;
        if (CF::A_F4 % CF::NT != 0 && f >= CF::A_F4) break;
        const int r = f / (CF::BK / 4);
        const int c4 = f % (CF::BK / 4);
        const int gr = m0 + r;
        const int gk = k0 + 4 * c4;
        if (fullA) {
            st.a[q] = *reinterpret_cast<const f32x4*>(Ab + (int64_t)gr * p.lda + gk);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                st.a[q][e] = (gr < p.m && gk + e < p.k) ? Ab[(int64_t)gr * p.lda + gk + e] : 0.0f;
        }
    }
#pragma unroll
    for (int q = 0; q < CF::B_LOADS; ++q) {
        const int u = q * CF::NT + t;
        if (CF::B_UNITS % CF::NT != 0 && u >= CF::B_UNITS) break;
        const int n4 = u % (CF::BN / 4);
        const int kr = u / (CF::BN / 4);
        const int gk = k0 + 4 * kr;
        const int gn = n0 + 4 * n4;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            if (fullB) {
                st.b[q][rr] = *reinterpret_cast<const f32x4*>(Bb + (int64_t)(gk + rr) * p.ldb + gn);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    st.b[q][rr][e] = (gk + rr < p.k && gn + e < p.n)
                                         ? Bb[(int64_t)(gk + rr) * p.ldb + gn + e]
                                         : 0.0f;
            }
        }
    }
}

// Register -> LDS store of one staged chunk into stage buffer `buf`.
template <class CF>
__device__ inline void store_chunk(const Stage<CF>& st, unsigned char* buf) {
    const int t = threadIdx.x;
    if constexpr (CF::FLOW == FLOW_SPLIT) {
        _Float16* a_hi = reinterpret_cast<_Float16*>(buf);
        _Float16* a_lo = a_hi + CF::BM * CF::PH;
        _Float16* b_hi = a_lo + CF::BM * CF::PH;
        _Float16* b_lo = b_hi + CF::BN * CF::PH;
#pragma unroll
        for (int q = 0; q < CF::A_LOADS; ++q) {
            const int f = q * CF::NT + t;
            if (CF::A_F4 % CF::NT != 0 && f >= CF::A_F4) break;
            const int r = f / (CF::BK / 4);
            const int c4 = f % (CF::BK / 4);
            u32x2 hi, lo;
            split4(st.a[q][0], st.a[q][1], st.a[q][2], st.a[q][3], hi, lo);
            const int off = r * CF::PH + 4 * c4;
            *reinterpret_cast<u32x2*>(a_hi + off) = hi;
            *reinterpret_cast<u32x2*>(a_lo + off) = lo;
        }
#pragma unroll
        for (int q = 0; q < CF::B_LOADS; ++q) {
            const int u = q * CF::NT + t;
            if (CF::B_UNITS % CF::NT != 0 && u >= CF::B_UNITS) break;
            const int n4 = u % (CF::BN / 4);
            const int kr = u / (CF::BN / 4);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                u32x2 hi, lo;
                split4(st.b[q][0][c], st.b[q][1][c], st.b[q][2][c], st.b[q][3][c], hi, lo);
                const int off = (4 * n4 + c) * CF::PH + 4 * kr;
                *reinterpret_cast<u32x2*>(b_hi + off) = hi;
                *reinterpret_cast<u32x2*>(b_lo + off) = lo;
            }
        }
    } else {
        float* as = reinterpret_cast<float*>(buf);
        float* bs = as + CF::BM * CF::PF;
#pragma unroll
        for (int q = 0; q < CF::A_LOADS; ++q) {
            const int f = q * CF::NT + t;
            if (CF::A_F4 % CF::NT != 0 && f >= CF::A_F4) break;
            const int r = f / (CF::BK / 4);
            const int c4 = f % (CF::BK / 4);
            *reinterpret_cast<f32x4*>(as + r * CF::PF + 4 * c4) = st.a[q];
        }
#pragma unroll
        for (int q = 0; q < CF::B_LOADS; ++q) {
            const int u = q * CF::NT + t;
            if (CF::B_UNITS % CF::NT != 0 && u >= CF::B_UNITS) break;
            const int n4 = u % (CF::BN / 4);
            const int kr = u / (CF::BN / 4);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                f32x4 v = {st.b[q][0][c], st.b[q][1][c], st.b[q][2][c], st.b[q][3][c]};
                *reinterpret_cast<f32x4*>(bs + (4 * n4 + c) * CF::PF + 4 * kr) = v;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Fragment reads for one 16-wide k step.
// ---------------------------------------------------------------------------
template <class CF>
struct Frags {
    half8_t ahi[CF::TM], alo[CF::TM], bhi[CF::TN], blo[CF::TN];
};

// Read 8 FP32 values (32 bytes) and split them into operand vectors.
__device__ inline void read_split8(const float* src, half8_t& hi, half8_t& lo) {
    const f32x4 v0 = *reinterpret_cast<const f32x4*>(src);
    const f32x4 v1 = *reinterpret_cast<const f32x4*>(src + 4);
    float x[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
    mfmae::tcec::split8(x, hi, lo);
}

// FLOW_SPLIT / FLOW_STAGED: read ready hi/lo vectors from planes with row
// pitch PH.  Row of lane = base_row + 32 t + l % 32, k offset 16 s + 8 (l / 32).
template <class CF, int T>
__device__ inline void read_planes(const _Float16* hi_plane, const _Float16* lo_plane, int base_row,
                                   int s, half8_t (&hi)[T], half8_t (&lo)[T]) {
    const int l = threadIdx.x & 63;
    const int koff = 16 * s + 8 * (l >> 5);
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const int off = (base_row + 32 * t + (l & 31)) * CF::PH + koff;
        hi[t] = *reinterpret_cast<const half8_t*>(hi_plane + off);
        if constexpr (CF::EC) lo[t] = *reinterpret_cast<const half8_t*>(lo_plane + off);
    }
}

template <class CF, int T>
__device__ inline void read_f32_split(const float* panel, int base_row, int s, half8_t (&hi)[T],
                                      half8_t (&lo)[T]) {
    const int l = threadIdx.x & 63;
    const int koff = 16 * s + 8 * (l >> 5);
#pragma unroll
    for (int t = 0; t < T; ++t) {
        read_split8(panel + (base_row + 32 * t + (l & 31)) * CF::PF + koff, hi[t], lo[t]);
    }
}

// FLOW_STAGED: the wave converts its WM rows of A and WN columns of B of the
// current chunk from the FP32 panels into its private hi/lo planes.
template <class CF>
__device__ inline void stage_wave_planes(const float* as, const float* bs, _Float16* scratch,
                                         int wrow, int wcol) {
    const int l = threadIdx.x & 63;
    _Float16* a_hi = scratch;
    _Float16* a_lo = a_hi + CF::WM * CF::PH;
    _Float16* b_hi = a_lo + CF::WM * CF::PH;
    _Float16* b_lo = b_hi + CF::WN * CF::PH;
    constexpr int F4_ROW = CF::BK / 4;
#pragma unroll
    for (int f = l; f < CF::WM * F4_ROW; f += 64) {
        const int r = f / F4_ROW, c4 = f % F4_ROW;
        const f32x4 v = *reinterpret_cast<const f32x4*>(as + (wrow + r) * CF::PF + 4 * c4);
        u32x2 hi, lo;
        split4(v[0], v[1], v[2], v[3], hi, lo);
        *reinterpret_cast<u32x2*>(a_hi + r * CF::PH + 4 * c4) = hi;
        *reinterpret_cast<u32x2*>(a_lo + r * CF::PH + 4 * c4) = lo;
    }
#pragma unroll
    for (int f = l; f < CF::WN * F4_ROW; f += 64) {
        const int r = f / F4_ROW, c4 = f % F4_ROW;
        const f32x4 v = *reinterpret_cast<const f32x4*>(bs + (wcol + r) * CF::PF + 4 * c4);
        u32x2 hi, lo;
        split4(v[0], v[1], v[2], v[3], hi, lo);
        *reinterpret_cast<u32x2*>(b_hi + r * CF::PH + 4 * c4) = hi;
        *reinterpret_cast<u32x2*>(b_lo + r * CF::PH + 4 * c4) = lo;
    }
}

// ---------------------------------------------------------------------------
// One k chunk of MFMA work from the LDS stage `cur`.
// ---------------------------------------------------------------------------
template <class CF>
__device__ inline void compute_chunk(f32x16_t (&acc)[CF::TM][CF::TN], f32x16_t (&cor)[CF::TM][CF::TN],
                                     unsigned char* smem, const unsigned char* cur, int wave,
                                     int wrow, int wcol) {
    if constexpr (CF::FLOW == FLOW_STAGED) {
        _Float16* scratch =
            reinterpret_cast<_Float16*>(smem + 2 * CF::STAGE + wave * CF::WAVE_SCRATCH);
        const float* as = reinterpret_cast<const float*>(cur);
        stage_wave_planes<CF>(as, as + CF::BM * CF::PF, scratch, wrow, wcol);
        __builtin_amdgcn_wave_barrier();
    }
#pragma unroll
    for (int s = 0; s < CF::KSTEPS; ++s) {
        Frags<CF> fr;
        if constexpr (CF::FLOW == FLOW_SPLIT) {
            const _Float16* a_hi = reinterpret_cast<const _Float16*>(cur);
            const _Float16* a_lo = a_hi + CF::BM * CF::PH;
            const _Float16* b_hi = a_lo + CF::BM * CF::PH;
            const _Float16* b_lo = b_hi + CF::BN * CF::PH;
            read_planes<CF>(a_hi, a_lo, wrow, s, fr.ahi, fr.alo);
            read_planes<CF>(b_hi, b_lo, wcol, s, fr.bhi, fr.blo);
        } else if constexpr (CF::FLOW == FLOW_DIRECT) {
            const float* as = reinterpret_cast<const float*>(cur);
            read_f32_split<CF>(as, wrow, s, fr.ahi, fr.alo);
            read_f32_split<CF>(as + CF::BM * CF::PF, wcol, s, fr.bhi, fr.blo);
        } else {
            const _Float16* a_hi =
                reinterpret_cast<const _Float16*>(smem + 2 * CF::STAGE + wave * CF::WAVE_SCRATCH);
            const _Float16* a_lo = a_hi + CF::WM * CF::PH;
            const _Float16* b_hi = a_lo + CF::WM * CF::PH;
            const _Float16* b_lo = b_hi + CF::WN * CF::PH;
            read_planes<CF>(a_hi, a_lo, 0, s, fr.ahi, fr.alo);
            read_planes<CF>(b_hi, b_lo, 0, s, fr.bhi, fr.blo);
        }
#pragma unroll
        for (int i = 0; i < CF::TM; ++i)
#pragma unroll
            for (int j = 0; j < CF::TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fr.ahi[i], fr.bhi[j], acc[i][j],
                                                                   0, 0, 0);
        if constexpr (CF::EC) {
#pragma unroll
            for (int i = 0; i < CF::TM; ++i)
#pragma unroll
                for (int j = 0; j < CF::TN; ++j)
                    cor[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fr.alo[i], fr.bhi[j],
                                                                       cor[i][j], 0, 0, 0);
#pragma unroll
            for (int i = 0; i < CF::TM; ++i)
#pragma unroll
                for (int j = 0; j < CF::TN; ++j)
                    cor[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fr.ahi[i], fr.blo[j],
                                                                       cor[i][j], 0, 0, 0);
        }
    }
}

template <class CF>
__device__ inline void zero_acc(f32x16_t (&acc)[CF::TM][CF::TN], f32x16_t (&cor)[CF::TM][CF::TN]) {
#pragma unroll
    for (int i = 0; i < CF::TM; ++i)
#pragma unroll
        for (int j = 0; j < CF::TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[i][j][e] = 0.0f;
                cor[i][j][e] = 0.0f;
            }
}

// Epilogue: C = main + corr * 2^-11, accumulator layout of the 32x32 MFMA:
// element e of lane l is row 8 (e / 4) + 4 (l / 32) + e % 4, column l % 32.
template <class CF>
__device__ inline void store_tile(const f32x16_t (&acc)[CF::TM][CF::TN],
                                  const f32x16_t (&cor)[CF::TM][CF::TN], const KParams& p,
                                  const TaskPos& q, int wrow, int wcol) {
    const int l = threadIdx.x & 63;
    const bool full = (q.m0 + CF::BM <= p.m) && (q.n0 + CF::BN <= p.n);
#pragma unroll
    for (int i = 0; i < CF::TM; ++i)
#pragma unroll
        for (int j = 0; j < CF::TN; ++j) {
            const int col = q.n0 + wcol + 32 * j + (l & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = q.m0 + wrow + 32 * i + 8 * (e >> 2) + 4 * (l >> 5) + (e & 3);
                const float v = CF::EC ? __builtin_fmaf(cor[i][j][e], mfmae::tcec::kLoScaleInv,
                                                        acc[i][j][e])
                                       : acc[i][j][e];
                if (full || (row < p.m && col < p.n)) q.C[(int64_t)row * p.ldc + col] = v;
            }
        }
}

// ---------------------------------------------------------------------------
// The kernel.
// ---------------------------------------------------------------------------
template <class CF>
__global__ __launch_bounds__(CF::NT, CF::MIN_WAVES) void bgemm_emu_kernel(KParams p) {
    static_assert(CF::FITS, "LDS budget of one CU");
    __shared__ __attribute__((aligned(16))) unsigned char smem[CF::LDS_BYTES];

    const int G = gridDim.x;
    int task = first_task(p);
    if (task >= p.ntasks) return;  // the whole workgroup leaves together

    const int wave = threadIdx.x >> 6;
    const int wrow = (wave / CF::WAVES_N) * CF::WM;  // within the tile
    const int wcol = (wave % CF::WAVES_N) * CF::WN;

    f32x16_t acc[CF::TM][CF::TN], cor[CF::TM][CF::TN];
    zero_acc<CF>(acc, cor);

    const int nchunks = cdiv(p.k, CF::BK);
    if (nchunks == 0) {  // empty sum: every tile is zero
        for (; task < p.ntasks; task += G) store_tile<CF>(acc, cor, p, task_pos<CF::BM, CF::BN>(p, task), wrow, wcol);
        return;
    }

    TaskPos cur_t = task_pos<CF::BM, CF::BN>(p, task);
    Stage<CF> st;
    load_chunk<CF>(st, p, cur_t.A, cur_t.B, cur_t.m0, cur_t.n0, 0);
    store_chunk<CF>(st, smem);
    __syncthreads();

    int c = 0, buf = 0;
    for (;;) {
        // the chunk after this one: the next k chunk of this task, or the
        // first chunk of this workgroup's next task
        int ntask = task, nc = c + 1;
        if (nc == nchunks) {
            ntask += G;
            nc = 0;
        }
        const bool more = ntask < p.ntasks;
        TaskPos next_t = cur_t;
        if (more) {
            if (ntask != task) next_t = task_pos<CF::BM, CF::BN>(p, ntask);
            load_chunk<CF>(st, p, next_t.A, next_t.B, next_t.m0, next_t.n0, nc * CF::BK);
        }

        compute_chunk<CF>(acc, cor, smem, smem + buf * CF::STAGE, wave, wrow, wcol);

        if (c == nchunks - 1) {
            store_tile<CF>(acc, cor, p, cur_t, wrow, wcol);
            zero_acc<CF>(acc, cor);
        }
        if (more) store_chunk<CF>(st, smem + (buf ^ 1) * CF::STAGE);
        __syncthreads();
        if (!more) break;
        task = ntask;
        cur_t = next_t;
        c = nc;
        buf ^= 1;
    }
}

// ---------------------------------------------------------------------------
// Instances and launch.
// ---------------------------------------------------------------------------
template <int TILE>
struct TileShape;
template <>
struct TileShape<SGEMM_EMU_TILE_64x64> {
    static constexpr int BM = 64, BN = 64, BK = 32, WM = 32, WN = 32;
};
template <>
struct TileShape<SGEMM_EMU_TILE_128x128> {
    static constexpr int BM = 128, BN = 128, BK = 32, WM = 64, WN = 64;
};
template <>
struct TileShape<SGEMM_EMU_TILE_256x128> {
    static constexpr int BM = 256, BN = 128, BK = 32, WM = 64, WN = 64;
};

template <int TILE, int FLOW, bool EC>
using CfgOf = Cfg<TileShape<TILE>::BM, TileShape<TILE>::BN, TileShape<TILE>::BK,
                  TileShape<TILE>::WM, TileShape<TILE>::WN, FLOW, EC>;

template <int TILE, int FLOW>
constexpr bool variant_fits() {
    return CfgOf<TILE, FLOW, true>::FITS;
}

// Workgroups of one instance that fit on the device at once (cached; the
// device of the calling thread is used).
template <class CF>
static int resident_blocks() {
    // one value per device, computed on first use; atomic so that threads
    // calling for the first time at once (all computing the same value) do
    // not race; devices past the table are computed on every call
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    const bool cached = dev < 64;
    if (cached) {
        const int r = cache[dev].load(std::memory_order_relaxed);
        if (r > 0) return r;
    }
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, bgemm_emu_kernel<CF>, CF::NT, 0) !=
        hipSuccess)
        return 0;
    const int r = cus * (per_cu > 0 ? per_cu : 1);
    if (cached) cache[dev].store(r, std::memory_order_relaxed);
    return r;
}

template <class CF>
static hipError_t launch_cfg(const GemmArgs& a, hipStream_t stream) {
    KParams p;
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
    p.vec_a = a.vec_a;
    p.vec_b = a.vec_b;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    // task ids are 32-bit: split a batch whose task count would not fit
    const int64_t max_tasks = (int64_t(1) << 31) - 1;
    if (tiles > max_tasks) return hipErrorInvalidConfiguration;
    const int64_t items_per_launch = max_tasks / tiles;
    int resident = resident_blocks<CF>();
    if (resident <= 0) {
        hipError_t e = hipGetLastError();
        return e != hipSuccess ? e : hipErrorInvalidDeviceFunction;
    }
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        const int64_t ntasks = items * tiles;
        int64_t blocks = ntasks < resident ? ntasks : resident;
        if (blocks >= 8) blocks -= blocks % 8;
        p.ntasks = (int)ntasks;
        p.item0 = (int)i0;
        hipLaunchKernelGGL(bgemm_emu_kernel<CF>, dim3((unsigned)blocks), dim3(CF::NT), 0, stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int TILE, int FLOW>
static hipError_t launch_tf(const GemmArgs& a, bool ec, hipStream_t stream) {
    if constexpr (!variant_fits<TILE, FLOW>()) {
        return hipErrorInvalidConfiguration;
    } else {
        return ec ? launch_cfg<CfgOf<TILE, FLOW, true>>(a, stream)
                  : launch_cfg<CfgOf<TILE, FLOW, false>>(a, stream);
    }
}

template <int TILE>
static hipError_t launch_t(const GemmArgs& a, int flow, bool ec, hipStream_t stream) {
    switch (flow) {
        case FLOW_SPLIT: return launch_tf<TILE, FLOW_SPLIT>(a, ec, stream);
        case FLOW_DIRECT: return launch_tf<TILE, FLOW_DIRECT>(a, ec, stream);
        case FLOW_STAGED: return launch_tf<TILE, FLOW_STAGED>(a, ec, stream);
        default: return hipErrorInvalidValue;
    }
}

bool gemm_variant_exists(int tile, int flow) {
    auto fits = [&](auto tile_tag) {
        constexpr int T = decltype(tile_tag)::value;
        switch (flow) {
            case FLOW_SPLIT: return variant_fits<T, FLOW_SPLIT>();
            case FLOW_DIRECT: return variant_fits<T, FLOW_DIRECT>();
            case FLOW_STAGED: return variant_fits<T, FLOW_STAGED>();
            default: return false;
        }
    };
    switch (tile) {
        case SGEMM_EMU_TILE_64x64: return fits(std::integral_constant<int, SGEMM_EMU_TILE_64x64>{});
        case SGEMM_EMU_TILE_128x128:
            return fits(std::integral_constant<int, SGEMM_EMU_TILE_128x128>{});
        case SGEMM_EMU_TILE_256x128:
            return fits(std::integral_constant<int, SGEMM_EMU_TILE_256x128>{});
        default: return false;
    }
}

hipError_t launch_gemm(const GemmArgs& a, int tile, int flow, bool ec, hipStream_t stream) {
    switch (tile) {
        case SGEMM_EMU_TILE_64x64: return launch_t<SGEMM_EMU_TILE_64x64>(a, flow, ec, stream);
        case SGEMM_EMU_TILE_128x128: return launch_t<SGEMM_EMU_TILE_128x128>(a, flow, ec, stream);
        case SGEMM_EMU_TILE_256x128: return launch_t<SGEMM_EMU_TILE_256x128>(a, flow, ec, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace sgemm_emu
