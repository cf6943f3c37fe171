// Internal declarations shared by the C ABI and the kernel translation units.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace sgemm_emu {

struct GemmArgs {
    int m, n, k;
    const float* A;
    int64_t lda, sa;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int batch;
    bool vec_a, vec_b;  // 16-byte vector loads are legal for A / B
};

// Launch the batched emulated GEMM with the given tile / flow / ec choice.
// Returns hipSuccess or the launch error.  Arguments are already validated.
hipError_t launch_gemm(const GemmArgs& a, int tile, int flow, bool ec, hipStream_t stream);

// True if (tile, flow) is a compiled combination.
bool gemm_variant_exists(int tile, int flow);

// Register-direct flow (no LDS): true if the operands allow its vector loads
// for this tile choice.
bool reg_flow_supported(const GemmArgs& a, int tile);
hipError_t launch_gemm_reg(const GemmArgs& a, int tile, bool ec, hipStream_t stream);

// Pipelined full-tile kernels (split flow: tiles 128x128, 256x128,
// 128x256; direct and staged flows: tile 128x128; error correction off:
// split flow, tiles 128x128 and 128x256): true if the shape and alignment
// allow the tile.
bool big_supported(const GemmArgs& a, int tile, int flow, bool ec);
hipError_t launch_gemm_big(const GemmArgs& a, int tile, int flow, bool ec, hipStream_t stream);
// True if launch_gemm_big runs the persistent stream form of the kernel
// (error correction on).
bool big_streams(const GemmArgs& a, int tile, int flow);

struct HouseholderArgs {
    int mode;  // SGEMM_EMU_HOUSEHOLDER_RULE or _LDS
    int ncols;
    const float* u;
    int64_t su;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int batch;
};

hipError_t launch_householder64(const HouseholderArgs& a, hipStream_t stream);

struct GivensArgs {
    int ncols;
    int i, j;  // rotation plane
    const float* c;
    const float* s;
    int64_t scs;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int batch;
    int mode;  // SGEMM_EMU_GIVENS_MAP, _EMBEDDED or _LDS (resolved, not AUTO)
};

// True if the plane (i, j) of n = 64 has a compile-time kernel instance.
bool givens_embedded(int i, int j);
hipError_t launch_givens64(const GivensArgs& a, hipStream_t stream);

// D = op(A) op(B) + C through the fragment interface (C may be null: zero).
struct AccArgs {
    int m, n, k;
    const float* A;
    int64_t lda, sa;
    const float* B;
    int64_t ldb, sb;
    const float* C;
    int64_t ldc, sc;
    float* D;
    int64_t ldd, sd;
    int batch;
    bool a_trans, b_trans, cd_col;
    bool vec_a, vec_b, vec_c, vec_d;  // 16-byte accesses legal (contiguous direction)
};

// shape: 0 = 16x16x32, 1 = 32x32x16.
hipError_t launch_gemm_acc(const AccArgs& a, int shape, bool ec, hipStream_t stream);

// Inclusive scan of each row of X (rows x len, row stride ldx) into Y.
struct ScanArgs {
    int64_t rows;
    int len;
    const float* X;
    int64_t ldx;
    float* Y;
    int64_t ldy;
    bool vec;  // X and Y 16-byte aligned, ldx and ldy multiples of 4
};

hipError_t launch_scan(const ScanArgs& a, hipStream_t stream);

// form: SGEMM_EMU_SPLIT_SCALAR, _PAIR or _EIGHT.
hipError_t launch_split(int64_t count, const float* x, uint16_t* hi, uint16_t* lo, int form,
                        hipStream_t stream);

// C_t = A_t + B_t over items of n floats, one workgroup of `threads` per item.
hipError_t launch_stream_probe(int64_t items, int64_t n, const float* A, const float* B, float* C,
                               int threads, hipStream_t stream);

// m a multiple of 128, n of 256, k of 32 (k > 0); reads A[.][0..31], B[0..31][.].
hipError_t launch_mfma_probe(int m, int n, int k, const float* A, int64_t lda, const float* B,
                             int64_t ldb, float* C, int64_t ldc, hipStream_t stream);

hipError_t launch_mma_probe(int shape, const uint16_t* a, const uint16_t* b, float* d,
                            hipStream_t stream);

}  // namespace sgemm_emu
