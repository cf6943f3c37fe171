// Emulated SGEMM on full tiles of C (Sec. 4.4): split once per workgroup at
// staging, hi/lo planes in LDS.
//
// Per k chunk of 32, every thread loads its part of the chunk from global
// memory into registers with 16-byte loads along the rows of A and of B (A:
// 8 consecutive k of one row; B: 4 consecutive n of one k row, one 1 KiB row
// per wave and load), splits the values there and writes hi and lo to LDS,
// so each element is split once per workgroup and LDS holds 2 + 2 bytes per
// element, the footprint of the FP32 data.  Waves of 64 x 64 build their
// operand vectors from LDS and run 3 MFMAs per 32 x 32 block and 16-wide k
// step (v_mfma_f32_32x32x16_f16), main and correction products in separate
// accumulators.
//
// LDS layout, A planes (A hi, A lo): [row][4 pieces of 8 halves], 64 bytes
// per row, no padding; piece q of row r is stored at position
// q ^ ((r ^ (r >> 2)) & 3).  Measured on gfx950 (16-byte LDS accesses, timed
// against a linear pattern), this swizzle makes the fragment reads (lanes
// 0..31 rows r..r+31 at one piece, lanes 32..63 the next piece) and the
// staging writes (4 lanes per row, one piece each) conflict-free.
//
// B planes (B hi, B lo): n-major, [k][BN halves], quad q (4 halves) of row k
// at position q ^ (8 (k & 3)).  The MFMA wants 8 consecutive k of one column
// per lane; gfx950's transposing LDS read (ds_read_b64_tr_b16) delivers them
// from this layout, two 8-byte reads per fragment: in a group of 16 lanes,
// lane 4i + c receives element c of the reads of lanes i, i + 4, i + 8 and
// i + 12 of the group (lane layout checked on the device).  The swizzle puts
// the 4 rows one half-wave reads (64 bytes each) and the 256-byte half-rows
// the staging writes on distinct banks.  Loading B as whole rows instead of
// 8 strided rows per lane cuts its vector-memory instructions by 4, which
// was the binding limit of the k loop (measured: with half of those loads
// the loop runs as fast as with none).
//
// Pipeline: two LDS stages and two register stages.  In iteration c the
// workgroup computes chunk c, writes chunk c + 1 (loaded two iterations
// earlier) to LDS, issues the loads of chunk c + 3 into the registers just
// freed, and meets at one barrier that orders LDS only (global loads stay in
// flight across it).  Every load and store of the loop is unconditional --
// chunk indices past the end are clamped to the last chunk -- so the waits
// before each use are for that stage's loads only.
//
// Flows (where the split happens, the policy of Sec. 4.4 / Fig. 6):
//   SPLIT  (production) as above: split once per workgroup at staging.
//   DIRECT LDS holds the FP32 chunk ([row][8 pieces of 4 floats], 128-byte
//          rows, piece p of row r at p ^ ((r ^ (r >> 3)) & 7), measured
//          conflict-free for these patterns); every wave reads FP32 operand
//          values and splits them itself -- the paper's extension-library
//          flow, fragments built from FP32 shared memory.
//   STAGED LDS holds the FP32 chunk; every wave converts its own rows and
//          columns to hi/lo, writes them to a private LDS area and reloads
//          them as fragments -- the flow a load-only fragment API forces
//          (three LDS passes per element, twice the footprint).
// The three have the same tiles, loads and pipeline, so they differ only in
// LDS traffic and footprint and in where the split's VALU work is done.
//
// Only full tiles (m and n multiples of the tile, k of 32) with 16-byte
// aligned rows; other shapes take the general LDS kernel or the
// register-direct flow.
#include <atomic>

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

// Tile configuration: BM x BN workgroup tile, WAVES_M x WAVES_N waves of
// WM x WN (made of 32 x 32 blocks), W waves per SIMD.
enum { BIG_SPLIT = SGEMM_EMU_FLOW_SPLIT, BIG_DIRECT = SGEMM_EMU_FLOW_DIRECT,
       BIG_STAGED = SGEMM_EMU_FLOW_STAGED };

template <int BM_, int BN_, int WAVES_M_, int WAVES_N_, int W_, int VALU_PER_MFMA_ = 0,
          int FLOW_ = BIG_SPLIT, bool EC_ = true>
struct BigCfg {
    static constexpr int BM = BM_, BN = BN_, BK = 32;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, W = W_;
    static constexpr int FLOW = FLOW_;
    // error correction: false keeps the hi.hi product only (staging converts
    // hi alone; the lo planes are neither written nor read)
    static constexpr bool EC = EC_;
    static_assert(EC || FLOW == BIG_SPLIT, "EC off is built for the split flow");
    static constexpr int MFMAS_PER_BLOCK = EC ? 3 : 1;
    // 0: compiler's own schedule; else the MFMAs of a chunk are interleaved
    // with this many VALU instructions each (the split of the next chunk)
    static constexpr int VALU_PER_MFMA = VALU_PER_MFMA_;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    static constexpr int NT = 64 * WAVES_M * WAVES_N;
    static constexpr int TM = WM / 32, TN = WN / 32;
    static constexpr int ROW_BYTES = 2 * BK;  // one row of a binary16 plane
    static constexpr int A_PLANE = BM * ROW_BYTES;
    static constexpr int B_PLANE = BN * ROW_BYTES;
    // a stage holds the chunk: hi and lo planes (split flow) or the FP32
    // rows (direct, staged): the same bytes
    static constexpr int STAGE_BYTES = 2 * A_PLANE + 2 * B_PLANE;
    // staged flow: each wave's private hi and lo planes of its WM + WN rows
    static constexpr int WAVE_BYTES = FLOW == BIG_STAGED ? 2 * (WM + WN) * ROW_BYTES : 0;
    static constexpr int LDS_BYTES = 2 * STAGE_BYTES + (NT / 64) * WAVE_BYTES;
    // staging units: 8 consecutive k of one A row or one B column
    static constexpr int A_UNITS = BM * (BK / 8) / NT;
    static constexpr int B_UNITS = BN * (BK / 8) / NT;
    static_assert(A_UNITS * NT == BM * (BK / 8) && B_UNITS * NT == BN * (BK / 8), "staging");
    // split flow, B: quads of 4 consecutive n of one k row; one pass of the
    // workgroup covers B_PASS_ROWS rows, each thread loads B_QUADS quads
    static constexpr int B_QUADS = BK * BN / 4 / NT;
    static constexpr int B_PASS_ROWS = NT / (BN / 4);
    static_assert(B_QUADS * NT * 4 == BK * BN && B_PASS_ROWS % 4 == 0, "B quads");
    static_assert(WM % 32 == 0 && WN % 32 == 0, "blocks");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS of one CU");
};

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

// Byte offset of piece q (8 halves) of row r in a plane of 64-byte rows.
__device__ inline int piece(int r, int q) {
    return r * 64 + 16 * (q ^ ((r ^ (r >> 2)) & 3));
}

// Byte offset of piece p (4 floats) of row r in FP32 rows of 128 bytes.
// Pieces 2q and 2q + 1 sit at offsets that differ only in bit 4.
__device__ inline int piece32(int r, int p) {
    return r * 128 + 16 * (p ^ ((r ^ (r >> 3)) & 7));
}

// Byte offset of quad q (4 halves) of row k in an n-major B plane of BN
// halves per row.  The swizzle flips bits 3 and 4 of q, so q stays in the
// row (BN / 4 is a multiple of 32).
template <class CF>
__device__ inline int bquad(int k, int q) {
    return k * (2 * CF::BN) + 8 * (q ^ (8 * (k & 3)));
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));

// Transposing 8-byte LDS read (ds_read_b64_tr_b16).
__device__ inline half4_t read_tr(const unsigned char* p) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    return __builtin_bit_cast(half4_t,
                              __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p)));
}

// Registers of one staged chunk.
template <class CF>
struct Stage {
    f32x4 a[CF::A_UNITS][2];
    f32x4 bq[CF::B_QUADS];    // split flow
    float b[CF::B_UNITS][8];  // FP32 flows
};

// Per-thread staging coordinates.  The task's corner addresses are the same
// for the whole workgroup (scalar registers); each thread adds a 32-bit byte
// offset.  The loads are buffer loads on a descriptor made from the chunk's
// corner (scalar), the thread's offset (vector) and the row's offset
// (scalar), so no load needs 64-bit address arithmetic on the VALU.
template <class CF>
struct StageMap {
    const float* a;               // A[m0][0] of the task
    const float* b;               // B[0][n0] of the task
    int64_t ldb;
    uint32_t a_off[CF::A_UNITS];  // bytes from a to A[m0 + row][8 q]
    uint32_t b_off[CF::B_UNITS];  // FP32 flows: bytes from b to B[8 kg][n0 + n]
    uint32_t bq_off;              // split flow: bytes from b to B[row][n0 + 4 q]
    int a_lds[CF::A_UNITS];       // piece(row, q), or piece32(row, 2q) for FP32 stages
    int b_lds[CF::B_UNITS];       // FP32 flows: piece32(n, 2kg)
    int bq_lds;                   // split flow: bquad(row, q)
};

// Raw buffer descriptor on p: byte offsets up to 2^32 - 1, no stride, 32-bit
// data format (the fourth word as for every gfx9 raw buffer).
__device__ inline __amdgpu_buffer_rsrc_t raw_rsrc(const float* p) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), 0, -1, 0x00020000);
}

template <class CF>
__device__ inline void load_stage(Stage<CF>& st, const StageMap<CF>& sm, int k0) {
    const __amdgpu_buffer_rsrc_t ra = raw_rsrc(sm.a + k0);
#pragma unroll
    for (int u = 0; u < CF::A_UNITS; ++u) {
        st.a[u][0] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, sm.a_off[u], 0, 0));
        st.a[u][1] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, sm.a_off[u] + 16, 0, 0));
    }
    const __amdgpu_buffer_rsrc_t rb = raw_rsrc(sm.b + (int64_t)k0 * sm.ldb);
    const uint32_t row = (uint32_t)sm.ldb * 4u;  // bytes; a chunk spans under 2^31 (offsets_fit)
    if constexpr (CF::FLOW == BIG_SPLIT) {
#pragma unroll
        for (int r = 0; r < CF::B_QUADS; ++r)
            st.bq[r] = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                           rb, sm.bq_off, (int)(row * (uint32_t)(r * CF::B_PASS_ROWS)), 0));
    } else {
#pragma unroll
        for (int v = 0; v < 8; ++v)
#pragma unroll
            for (int u = 0; u < CF::B_UNITS; ++u)
                st.b[u][v] = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(rb, sm.b_off[u],
                                                                (int)(row * (uint32_t)v), 0));
    }
}

// The byte offsets of StageMap and the row offsets of load_stage stay below
// 2^31, so that no buffer offset depends on how the hardware treats the top
// bit of a 32-bit offset.  Larger leading dimensions (128 rows of over 2^22
// floats, 32 rows of over 2^24) take the general kernel, which addresses
// with 64-bit pointers.
template <class CF>
bool offsets_fit(const GemmArgs& a) {
    const int64_t lim = (int64_t)1 << 31;
    return ((int64_t)CF::BM * a.lda + CF::BK) * 4 < lim &&
           ((int64_t)CF::BK * a.ldb + CF::BN) * 4 < lim;
}

// Write the staged chunk to LDS stage `buf`: split into hi and lo pieces
// (split flow) or as FP32 (direct and staged flows).
template <class CF>
__device__ inline void store_stage(const Stage<CF>& st, const StageMap<CF>& sm,
                                   unsigned char* buf) {
    if constexpr (CF::FLOW != BIG_SPLIT) {
        unsigned char* a32 = buf;
        unsigned char* b32 = buf + 2 * CF::A_PLANE;
#pragma unroll
        for (int u = 0; u < CF::A_UNITS; ++u) {
            *reinterpret_cast<f32x4*>(a32 + sm.a_lds[u]) = st.a[u][0];
            *reinterpret_cast<f32x4*>(a32 + (sm.a_lds[u] ^ 16)) = st.a[u][1];
        }
#pragma unroll
        for (int u = 0; u < CF::B_UNITS; ++u) {
            const f32x4 v0 = {st.b[u][0], st.b[u][1], st.b[u][2], st.b[u][3]};
            const f32x4 v1 = {st.b[u][4], st.b[u][5], st.b[u][6], st.b[u][7]};
            *reinterpret_cast<f32x4*>(b32 + sm.b_lds[u]) = v0;
            *reinterpret_cast<f32x4*>(b32 + (sm.b_lds[u] ^ 16)) = v1;
        }
        return;
    }
    unsigned char* a_hi = buf;
    unsigned char* a_lo = buf + CF::A_PLANE;
    unsigned char* b_hi = buf + 2 * CF::A_PLANE;
    unsigned char* b_lo = b_hi + CF::B_PLANE;
    if constexpr (!CF::EC) {
#pragma unroll
        for (int u = 0; u < CF::A_UNITS; ++u) {
            const half4_t h0 = __builtin_convertvector(st.a[u][0], half4_t);
            const half4_t h1 = __builtin_convertvector(st.a[u][1], half4_t);
            *reinterpret_cast<half8_t*>(a_hi + sm.a_lds[u]) =
                half8_t{h0[0], h0[1], h0[2], h0[3], h1[0], h1[1], h1[2], h1[3]};
        }
#pragma unroll
        for (int r = 0; r < CF::B_QUADS; ++r)
            *reinterpret_cast<half4_t*>(b_hi + sm.bq_lds + r * CF::B_PASS_ROWS * 2 * CF::BN) =
                __builtin_convertvector(st.bq[r], half4_t);
        return;
    }
#pragma unroll
    for (int u = 0; u < CF::A_UNITS; ++u) {
        const float x[8] = {st.a[u][0][0], st.a[u][0][1], st.a[u][0][2], st.a[u][0][3],
                            st.a[u][1][0], st.a[u][1][1], st.a[u][1][2], st.a[u][1][3]};
        half8_t hi, lo;
        mfmae::tcec::split8(x, hi, lo);
        *reinterpret_cast<half8_t*>(a_hi + sm.a_lds[u]) = hi;
        *reinterpret_cast<half8_t*>(a_lo + sm.a_lds[u]) = lo;
    }
#pragma unroll
    for (int r = 0; r < CF::B_QUADS; ++r) {
        mfmae::tcec::half2_t h0, l0, h1, l1;
        mfmae::tcec::split_pair(st.bq[r][0], st.bq[r][1], h0, l0);
        mfmae::tcec::split_pair(st.bq[r][2], st.bq[r][3], h1, l1);
        const int o = sm.bq_lds + r * CF::B_PASS_ROWS * 2 * CF::BN;
        *reinterpret_cast<half4_t*>(b_hi + o) = half4_t{h0[0], h0[1], h1[0], h1[1]};
        *reinterpret_cast<half4_t*>(b_lo + o) = half4_t{l0[0], l0[1], l1[0], l1[1]};
    }
}

// Read 8 FP32 values (pieces 2q, 2q + 1 of row r) and split them.
__device__ inline void read_split32(const unsigned char* plane, int r, int q, half8_t& hi,
                                    half8_t& lo) {
    const int o = piece32(r, 2 * q);
    const f32x4 v0 = *reinterpret_cast<const f32x4*>(plane + o);
    const f32x4 v1 = *reinterpret_cast<const f32x4*>(plane + (o ^ 16));
    const float x[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
    mfmae::tcec::split8(x, hi, lo);
}

// Staged flow: the wave converts its WM rows of A and WN columns of B of the
// FP32 stage `buf` to hi/lo pieces in its private planes `priv` (rows
// 0..WM-1 for A, WM..WM+WN-1 for B).
template <class CF>
__device__ inline void stage_private(const unsigned char* buf, unsigned char* priv, int wrow,
                                     int wcol, int l) {
    const unsigned char* a32 = buf;
    const unsigned char* b32 = buf + 2 * CF::A_PLANE;
    unsigned char* p_hi = priv;
    unsigned char* p_lo = priv + (CF::WM + CF::WN) * CF::ROW_BYTES;
#pragma unroll
    for (int i = 0; i < (CF::WM + CF::WN) * 4 / 64; ++i) {
        const int u = i * 64 + l;
        const int r = u >> 2, q = u & 3;
        half8_t hi, lo;
        if (r < CF::WM) read_split32(a32, wrow + r, q, hi, lo);
        else read_split32(b32, wcol + r - CF::WM, q, hi, lo);
        *reinterpret_cast<half8_t*>(p_hi + piece(r, q)) = hi;
        *reinterpret_cast<half8_t*>(p_lo + piece(r, q)) = lo;
    }
    // the fragments read below were written by other lanes of this wave
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
}

// Both 16-wide k steps of one chunk from LDS stage `buf` (and, for the
// staged flow, the wave's private planes `priv`).
template <class CF>
__device__ inline void compute_stage(f32x16_t (&acc)[CF::TM][CF::TN],
                                     f32x16_t (&cor)[CF::TM][CF::TN], const unsigned char* buf,
                                     unsigned char* priv, int wrow, int wcol, int g, int j) {
    const unsigned char* a_hi = buf;
    const unsigned char* a_lo = buf + CF::A_PLANE;
    const unsigned char* b_hi = buf + 2 * CF::A_PLANE;
    const unsigned char* b_lo = b_hi + CF::B_PLANE;
    int arow = wrow, brow = wcol;
    if constexpr (CF::FLOW == BIG_STAGED) {
        stage_private<CF>(buf, priv, wrow, wcol, threadIdx.x & 63);
        a_hi = priv;
        a_lo = priv + (CF::WM + CF::WN) * CF::ROW_BYTES;
        b_hi = a_hi;
        b_lo = a_lo;
        arow = 0;
        brow = CF::WM;
    }
#pragma unroll
    for (int s = 0; s < CF::BK / 16; ++s) {
        const int q = 2 * s + g;  // k = 16 s + 8 g + (0..7), the same for A and B
        half8_t ahi[CF::TM], alo[CF::TM], bhi[CF::TN], blo[CF::TN];
        if constexpr (CF::FLOW == BIG_DIRECT) {
            // one B block at a time, to keep the split's temporaries few
            const unsigned char* a32 = buf;
            const unsigned char* b32 = buf + 2 * CF::A_PLANE;
#pragma unroll
            for (int tm = 0; tm < CF::TM; ++tm)
                read_split32(a32, wrow + 32 * tm + j, q, ahi[tm], alo[tm]);
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn) {
                half8_t bh, bl;
                read_split32(b32, wcol + 32 * tn + j, q, bh, bl);
#pragma unroll
                for (int tm = 0; tm < CF::TM; ++tm) {
                    acc[tm][tn] =
                        __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], bh, acc[tm][tn], 0, 0, 0);
                    cor[tm][tn] =
                        __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[tm], bh, cor[tm][tn], 0, 0, 0);
                    cor[tm][tn] =
                        __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], bl, cor[tm][tn], 0, 0, 0);
                }
            }
            continue;
        } else {
#pragma unroll
            for (int tm = 0; tm < CF::TM; ++tm) {
                const int o = piece(arow + 32 * tm + j, q);
                ahi[tm] = *reinterpret_cast<const half8_t*>(a_hi + o);
                if constexpr (CF::EC) alo[tm] = *reinterpret_cast<const half8_t*>(a_lo + o);
            }
            if constexpr (CF::FLOW == BIG_SPLIT) {
                // lane 16 G + sl reads row 8 (G / 2) + sl / 4 (+ 4 for the
                // second half of the 8 k) at quad 4 (G % 2) + sl % 4 of the
                // block; the transpose hands lane (j, g) rows 16 s + 8 g + 0..7
                // of column j
                const int l = threadIdx.x & 63;
                const int sl = l & 15, G = l >> 4;
                const int kl = 16 * s + 8 * (G >> 1) + (sl >> 2);
                const int ql = 4 * (G & 1) + (sl & 3);
#pragma unroll
                for (int tn = 0; tn < CF::TN; ++tn) {
                    const int o = bquad<CF>(kl, 8 * ((brow >> 5) + tn) + ql);
                    const int o4 = o + 4 * 2 * CF::BN;  // rows + 4: same swizzle
                    const half4_t h0 = read_tr(b_hi + o), h1 = read_tr(b_hi + o4);
                    bhi[tn] = half8_t{h0[0], h0[1], h0[2], h0[3], h1[0], h1[1], h1[2], h1[3]};
                    if constexpr (CF::EC) {
                        const half4_t l0 = read_tr(b_lo + o), l1 = read_tr(b_lo + o4);
                        blo[tn] =
                            half8_t{l0[0], l0[1], l0[2], l0[3], l1[0], l1[1], l1[2], l1[3]};
                    }
                }
            } else {
#pragma unroll
                for (int tn = 0; tn < CF::TN; ++tn) {
                    const int o = piece(brow + 32 * tn + j, q);
                    bhi[tn] = *reinterpret_cast<const half8_t*>(b_hi + o);
                    blo[tn] = *reinterpret_cast<const half8_t*>(b_lo + o);
                }
            }
        }
#pragma unroll
        for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], bhi[tn], acc[tm][tn],
                                                                     0, 0, 0);
        if constexpr (!CF::EC) continue;
#pragma unroll
        for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[tm], bhi[tn], cor[tm][tn],
                                                                     0, 0, 0);
#pragma unroll
        for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < CF::TN; ++tn)
                cor[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[tm], blo[tn], cor[tm][tn],
                                                                     0, 0, 0);
    }
}

// Ask the scheduler to interleave the chunk's MFMAs with the VALU work of
// the split, so one wave issues both while the matrix unit is busy.
template <class CF>
__device__ inline void interleave() {
    if constexpr (CF::VALU_PER_MFMA > 0) {
#pragma unroll
        for (int i = 0; i < CF::MFMAS_PER_BLOCK * (CF::BK / 16) * CF::TM * CF::TN; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, CF::VALU_PER_MFMA, 0);  // VALU
        }
    }
}

// Barrier that orders LDS accesses only: outstanding global loads stay in
// flight across it.
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <class CF>
__global__ __launch_bounds__(CF::NT, CF::W) void bgemm_big_kernel(BigParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[CF::LDS_BYTES];

    const int task = xcd_task(blockIdx.x, gridDim.x);
    if (task >= p.ntasks) return;  // the whole workgroup leaves together
    const int tiles = p.tiles_m * p.tiles_n;
    const int item = task / tiles;
    // one large product on the 128 x 256 tile: tiles in device-wide blocks
    const TileRC rc =
        CF::BM == 128 && CF::BN == 256 && block_order_applies(p.tiles_m, p.tiles_n, p.ntasks)
            ? block_tile(task - item * tiles, p.tiles_m, p.tiles_n)
            : grouped_tile(task - item * tiles, p.tiles_m, p.tiles_n);
    const int m0 = rc.tm * CF::BM;
    const int n0 = rc.tn * CF::BN;

    const int64_t it = (int64_t)item + p.item0;
    const float* __restrict__ Ab = p.A + it * p.sa;
    const float* __restrict__ Bb = p.B + it * p.sb;
    float* __restrict__ Cb = p.C + it * p.sc;

    const int tid = threadIdx.x;
    StageMap<CF> sm;
    sm.a = Ab + (int64_t)m0 * p.lda;
    sm.b = Bb + n0;
    sm.ldb = p.ldb;
#pragma unroll
    for (int u = 0; u < CF::A_UNITS; ++u) {
        const int unit = u * CF::NT + tid;
        const int row = unit >> 2, q = unit & 3;
        sm.a_off[u] = (uint32_t)(row * p.lda + 8 * q) * 4u;
        sm.a_lds[u] = CF::FLOW == BIG_SPLIT ? piece(row, q) : piece32(row, 2 * q);
    }
#pragma unroll
    for (int u = 0; u < CF::B_UNITS; ++u) {
        const int unit = u * CF::NT + tid;
        const int n = unit % CF::BN, kg = unit / CF::BN;
        sm.b_off[u] = (uint32_t)(8 * kg * p.ldb + n) * 4u;
        sm.b_lds[u] = piece32(n, 2 * kg);
    }
    {
        const int q = tid % (CF::BN / 4), row = tid / (CF::BN / 4);
        sm.bq_off = (uint32_t)(row * p.ldb + 4 * q) * 4u;
        sm.bq_lds = bquad<CF>(row, q);
    }

    const int wave = tid >> 6;
    const int l = tid & 63;
    const int g = l >> 5, j = l & 31;
    const int wrow = (wave / CF::WAVES_N) * CF::WM;
    const int wcol = (wave % CF::WAVES_N) * CF::WN;

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

    const int nk = p.k / CF::BK;  // >= 1
    const int last = nk - 1;
    unsigned char* buf0 = smem;
    unsigned char* buf1 = smem + CF::STAGE_BYTES;
    unsigned char* priv = smem + 2 * CF::STAGE_BYTES + wave * CF::WAVE_BYTES;
    Stage<CF> r0, r1;
    load_stage<CF>(r0, sm, 0);
    load_stage<CF>(r1, sm, CF::BK * min(1, last));
    store_stage<CF>(r0, sm, buf0);
    load_stage<CF>(r0, sm, CF::BK * min(2, last));
    lds_barrier();
    // iteration c: compute chunk c, store chunk c + 1, load chunk c + 3.
    // The MFMAs of chunk c are issued first; they run in the matrix unit
    // while the same wave splits chunk c + 1 on the VALU.
    int c = 0;
    for (; c + 2 <= nk; c += 2) {
        compute_stage<CF>(acc, cor, buf0, priv, wrow, wcol, g, j);
        store_stage<CF>(r1, sm, buf1);
        load_stage<CF>(r1, sm, CF::BK * min(c + 3, last));
        interleave<CF>();
        lds_barrier();
        compute_stage<CF>(acc, cor, buf1, priv, wrow, wcol, g, j);
        store_stage<CF>(r0, sm, buf0);
        load_stage<CF>(r0, sm, CF::BK * min(c + 4, last));
        interleave<CF>();
        lds_barrier();
    }
    if (c < nk) compute_stage<CF>(acc, cor, buf0, priv, wrow, wcol, g, j);

    // Epilogue: C = main + corr * 2^-11.  Element e of a 32 x 32 block is
    // row 8 (e / 4) + 4 g + e % 4, column j.  C is written once and not read
    // again here: nontemporal stores (measured 5% faster on the batched
    // 128^3 and 256^3 products, neutral on 8192^3).
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < CF::TN; ++tn) {
            float* cp = Cb + (int64_t)(m0 + wrow + 32 * tm + 4 * g) * p.ldc + n0 + wcol +
                        32 * tn + j;
#pragma unroll
            for (int e = 0; e < 16; ++e)
                __builtin_nontemporal_store(
                    CF::EC ? __builtin_fmaf(cor[tm][tn][e], mfmae::tcec::kLoScaleInv,
                                            acc[tm][tn][e])
                           : acc[tm][tn][e],
                    &cp[(int64_t)(8 * (e >> 2) + (e & 3)) * p.ldc]);
        }
}

// Geometry of one task (one tile of one item).
struct TaskGeo {
    const float* A;  // item bases
    const float* B;
    float* C;
    int m0, n0;
};

template <class CF>
__device__ inline TaskGeo task_geo(const BigParams& p, int task) {
    const int tiles = p.tiles_m * p.tiles_n;
    const int item = task / tiles;
    const TileRC rc = grouped_tile(task - item * tiles, p.tiles_m, p.tiles_n);
    TaskGeo q;
    const int64_t it = (int64_t)item + p.item0;
    q.A = p.A + it * p.sa;
    q.B = p.B + it * p.sb;
    q.C = p.C + it * p.sc;
    q.m0 = rc.tm * CF::BM;
    q.n0 = rc.tn * CF::BN;
    return q;
}

// Global addresses of this thread's staging units for task geometry q.
template <class CF>
__device__ inline void map_task(StageMap<CF>& sm, const BigParams& p, const TaskGeo& q) {
    sm.a = q.A + (int64_t)q.m0 * p.lda;
    sm.b = q.B + q.n0;
}

// Byte offsets and LDS offsets of this thread's staging units (the same for
// every task).
template <class CF>
__device__ inline void map_lds(StageMap<CF>& sm, const BigParams& p) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < CF::A_UNITS; ++u) {
        const int unit = u * CF::NT + tid;
        const int row = unit >> 2, q = unit & 3;
        sm.a_off[u] = (uint32_t)(row * p.lda + 8 * q) * 4u;
        sm.a_lds[u] = CF::FLOW == BIG_SPLIT ? piece(row, q) : piece32(row, 2 * q);
    }
#pragma unroll
    for (int u = 0; u < CF::B_UNITS; ++u) {
        const int unit = u * CF::NT + tid;
        const int n = unit % CF::BN, kg = unit / CF::BN;
        sm.b_off[u] = (uint32_t)(8 * kg * p.ldb + n) * 4u;
        sm.b_lds[u] = piece32(n, 2 * kg);
    }
    {
        const int q = tid % (CF::BN / 4), row = tid / (CF::BN / 4);
        sm.bq_off = (uint32_t)(row * p.ldb + 4 * q) * 4u;
        sm.bq_lds = bquad<CF>(row, q);
    }
}

// C = main + corr * 2^-11 for the wave's sub-tile (nontemporal stores, as
// in bgemm_big_kernel), and zero the accumulators.  Element e of a 32 x 32
// block is row 8 (e / 4) + 4 g + e % 4, column j.
template <class CF>
__device__ inline void store_c(f32x16_t (&acc)[CF::TM][CF::TN], f32x16_t (&cor)[CF::TM][CF::TN],
                               const BigParams& p, const TaskGeo& q, int wrow, int wcol, int g,
                               int j) {
#pragma unroll
    for (int tm = 0; tm < CF::TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < CF::TN; ++tn) {
            float* cp = q.C + (int64_t)(q.m0 + wrow + 32 * tm + 4 * g) * p.ldc + q.n0 + wcol +
                        32 * tn + j;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                __builtin_nontemporal_store(
                    __builtin_fmaf(cor[tm][tn][e], mfmae::tcec::kLoScaleInv, acc[tm][tn][e]),
                    &cp[(int64_t)(8 * (e >> 2) + (e & 3)) * p.ldc]);
                acc[tm][tn][e] = 0.0f;
                cor[tm][tn][e] = 0.0f;
            }
        }
}

// Persistent form: a grid of about as many workgroups as fit on the GPU at
// once; each walks its tasks (task t0 + i G) as one stream of k chunks, so
// the loads of a task's first chunks are issued while the previous task's
// last chunks are computed and its C is stored, and there is no pipeline
// fill per tile.
template <class CF>
__global__ __launch_bounds__(CF::NT, CF::W) void bgemm_big_stream_kernel(BigParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char smem[CF::LDS_BYTES];

    const int G = gridDim.x;
    const int t0 = xcd_task(blockIdx.x, G);
    if (t0 >= p.ntasks) return;  // the whole workgroup leaves together
    const int ntw = (p.ntasks - 1 - t0) / G + 1;  // tasks of this workgroup
    const int nk = p.k / CF::BK;                  // chunks per task, >= 1
    const int total = ntw * nk;                   // chunks in the stream

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int l = tid & 63;
    const int g = l >> 5, j = l & 31;
    const int wrow = (wave / CF::WAVES_N) * CF::WM;
    const int wcol = (wave % CF::WAVES_N) * CF::WN;

    StageMap<CF> sm;
    map_lds<CF>(sm, p);
    sm.ldb = p.ldb;
    map_task<CF>(sm, p, task_geo<CF>(p, t0));
    // load cursor: task index li of this workgroup, chunk lc.  Past the end
    // it stays on the last chunk (re-loading it keeps every load
    // unconditional).
    int li = 0, lc = 0;
    auto load_next = [&](Stage<CF>& st) {
        load_stage<CF>(st, sm, CF::BK * lc);
        if (++lc == nk) {
            if (li + 1 < ntw) {
                ++li;
                lc = 0;
                map_task<CF>(sm, p, task_geo<CF>(p, t0 + li * G));
            } else {
                lc = nk - 1;
            }
        }
    };

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

    unsigned char* buf0 = smem;
    unsigned char* buf1 = smem + CF::STAGE_BYTES;
    unsigned char* priv = smem + 2 * CF::STAGE_BYTES + wave * CF::WAVE_BYTES;
    // compute cursor: task index ci, chunk cc
    int ci = 0, cc = 0;
    auto finish_chunk = [&]() {
        if (++cc == nk) {
            store_c<CF>(acc, cor, p, task_geo<CF>(p, t0 + ci * G), wrow, wcol, g, j);
            ++ci;
            cc = 0;
        }
    };
    Stage<CF> r0, r1;
    load_next(r0);  // chunk 0
    load_next(r1);  // chunk 1
    store_stage<CF>(r0, sm, buf0);
    load_next(r0);  // chunk 2
    lds_barrier();
    // position s: compute chunk s, store chunk s + 1, load chunk s + 3
    for (int s = 0; s < total; s += 2) {
        compute_stage<CF>(acc, cor, buf0, priv, wrow, wcol, g, j);
        finish_chunk();
        store_stage<CF>(r1, sm, buf1);
        load_next(r1);
        interleave<CF>();
        lds_barrier();
        if (s + 1 < total) {
            compute_stage<CF>(acc, cor, buf1, priv, wrow, wcol, g, j);
            finish_chunk();
        }
        store_stage<CF>(r0, sm, buf0);
        load_next(r0);
        interleave<CF>();
        lds_barrier();
    }
}

// Workgroups of one instance that fit on the device at once (cached per
// device).
template <class CF, class K>
int resident_wgs(K kernel) {
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
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, CF::NT, 0) != hipSuccess)
        return 0;
    const int r = cus * (per_cu > 0 ? per_cu : 1);
    if (cached) cache[dev].store(r, std::memory_order_relaxed);
    return r;
}

template <class CF>
hipError_t launch_big_cfg(const GemmArgs& a, hipStream_t stream) {
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
    p.tiles_m = a.m / CF::BM;
    p.tiles_n = a.n / CF::BN;
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    // one launch stays below 2^31 work-items
    const int64_t max_tasks = (int64_t(1) << 31) / CF::NT - 1;
    if (tiles > max_tasks) return hipErrorInvalidConfiguration;
    const int64_t items_per_launch = max_tasks / tiles;
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        p.ntasks = (int)(items * tiles);
        p.item0 = (int)i0;
        hipLaunchKernelGGL(bgemm_big_kernel<CF>, dim3((unsigned)p.ntasks), dim3(CF::NT), 0, stream,
                           p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <class CF>
hipError_t launch_big_stream_cfg(const GemmArgs& a, hipStream_t stream) {
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
    p.tiles_m = a.m / CF::BM;
    p.tiles_n = a.n / CF::BN;
    const int resident = resident_wgs<CF>(bgemm_big_stream_kernel<CF>);
    if (resident <= 0) {
        hipError_t e = hipGetLastError();
        return e != hipSuccess ? e : hipErrorInvalidDeviceFunction;
    }
    const int64_t tiles = (int64_t)p.tiles_m * p.tiles_n;
    const int64_t max_tasks = (int64_t(1) << 31) - 1;  // task ids are 32-bit
    if (tiles > max_tasks) return hipErrorInvalidConfiguration;
    const int64_t items_per_launch = max_tasks / tiles;
    for (int64_t i0 = 0; i0 < a.batch; i0 += items_per_launch) {
        const int64_t items = a.batch - i0 < items_per_launch ? a.batch - i0 : items_per_launch;
        p.ntasks = (int)(items * tiles);
        p.item0 = (int)i0;
        const int grid = p.ntasks < resident ? p.ntasks : resident;
        hipLaunchKernelGGL(bgemm_big_stream_kernel<CF>, dim3((unsigned)grid), dim3(CF::NT), 0,
                           stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// The three full-tile configurations.  128 x 256 (eight 64 x 64 waves, the
// MFMAs of a chunk interleaved with four VALU instructions each) for large
// products; 256 x 128 for batches of 256-row products; 128 x 128 (four
// 64 x 64 waves, two workgroups per CU) for batches of 128-row products.
using Big128x256 = BigCfg<128, 256, 2, 4, 2, 4>;
using Big256x128 = BigCfg<256, 128, 4, 2, 2>;
using Big128x128 = BigCfg<128, 128, 2, 2, 2>;
// the paper's two data flows, for measurement, on the 128 x 128 tile
using Big128x128Direct = BigCfg<128, 128, 2, 2, 2, 0, BIG_DIRECT>;
using Big128x128Staged = BigCfg<128, 128, 2, 2, 2, 0, BIG_STAGED>;
// error correction off (the hi.hi product alone), for measuring what the
// correction costs on the same kernel and tiles
using Big128x256NoEC = BigCfg<128, 256, 2, 4, 2, 4, BIG_SPLIT, false>;
using Big128x128NoEC = BigCfg<128, 128, 2, 2, 2, 0, BIG_SPLIT, false>;

template <class CF>
bool fits(const GemmArgs& a) {
    return a.m % CF::BM == 0 && a.n % CF::BN == 0 && a.k % CF::BK == 0 && a.k > 0 && a.vec_a &&
           a.vec_b && offsets_fit<CF>(a);
}

}  // namespace

bool big_supported(const GemmArgs& a, int tile, int flow, bool ec) {
    if (!ec) {
        if (flow != SGEMM_EMU_FLOW_SPLIT) return false;
        if (tile == SGEMM_EMU_TILE_128x128) return fits<Big128x128NoEC>(a);
        return tile == SGEMM_EMU_TILE_128x256 && fits<Big128x256NoEC>(a);
    }
    if (flow != SGEMM_EMU_FLOW_SPLIT)
        return tile == SGEMM_EMU_TILE_128x128 &&
               (flow == SGEMM_EMU_FLOW_DIRECT || flow == SGEMM_EMU_FLOW_STAGED) &&
               fits<Big128x128>(a);
    switch (tile) {
        case SGEMM_EMU_TILE_128x128: return fits<Big128x128>(a);
        case SGEMM_EMU_TILE_256x128: return fits<Big256x128>(a);
        case SGEMM_EMU_TILE_128x256: return fits<Big128x256>(a);
        default: return false;
    }
}

// 256x128 runs one workgroup per CU: with few k chunks per tile, the
// persistent stream hides the per-tile pipeline fill (measured 1.14x on
// 1024 x 256^3); long k loops amortize it themselves.
bool big_streams(const GemmArgs& a, int tile, int flow) {
    return flow == SGEMM_EMU_FLOW_SPLIT && tile == SGEMM_EMU_TILE_256x128 && a.k <= 2048;
}

hipError_t launch_gemm_big(const GemmArgs& a, int tile, int flow, bool ec, hipStream_t stream) {
    if (!big_supported(a, tile, flow, ec)) return hipErrorInvalidValue;
    if (!ec)
        return tile == SGEMM_EMU_TILE_128x128 ? launch_big_cfg<Big128x128NoEC>(a, stream)
                                               : launch_big_cfg<Big128x256NoEC>(a, stream);
    if (flow == SGEMM_EMU_FLOW_DIRECT) return launch_big_cfg<Big128x128Direct>(a, stream);
    if (flow == SGEMM_EMU_FLOW_STAGED) return launch_big_cfg<Big128x128Staged>(a, stream);
    switch (tile) {
        case SGEMM_EMU_TILE_128x128: return launch_big_cfg<Big128x128>(a, stream);
        case SGEMM_EMU_TILE_256x128:
            return big_streams(a, tile, flow) ? launch_big_stream_cfg<Big256x128>(a, stream)
                                              : launch_big_cfg<Big256x128>(a, stream);
        default: return launch_big_cfg<Big128x256>(a, stream);
    }
}

}  // namespace sgemm_emu
