// C ABI of the library (declared in include/sgemm_emu.h): argument
// validation, kernel choice and launch.  Validation runs entirely on the host
// before any HIP call, so every error path is free of side effects.
#include <stdint.h>

#include <initializer_list>

#include "internal.h"
#include "mfmae/frag.hpp"
#include "sgemm_emu.h"
#include "tiling.hpp"

namespace {

thread_local int g_last_hip_error = 0;

int hip_fail(hipError_t e) {
    g_last_hip_error = (int)e;
    return SGEMM_EMU_ERR_HIP;
}

struct Extent {
    uintptr_t lo, hi;  // [lo, hi) in bytes; empty if lo == hi
    bool ok;           // false: the span runs past the end of the address space
};

// Bytes spanned by `items` row-major matrices of rows x cols with leading
// dimension ld and item stride s (elements of `elem` bytes), starting at p.
// All arguments are non-negative; the span is computed in 128 bits, so no
// stride or leading dimension can wrap it.
Extent extent(const void* p, int64_t items, int64_t rows, int64_t cols, int64_t ld, int64_t s,
              int64_t elem = sizeof(float)) {
    Extent e{(uintptr_t)p, (uintptr_t)p, true};
    if (items <= 0 || rows <= 0 || cols <= 0) return e;
    const __int128 last = (__int128)(items - 1) * s + (__int128)(rows - 1) * ld + cols;
    const __int128 bytes = last * elem;
    if (bytes > (__int128)(UINTPTR_MAX - e.lo)) {
        e.ok = false;
        return e;
    }
    e.hi = e.lo + (uintptr_t)bytes;
    return e;
}

bool all_ok(std::initializer_list<Extent> es) {
    for (const Extent& e : es)
        if (!e.ok) return false;
    return true;
}

bool overlap(Extent a, Extent b) {
    if (a.lo == a.hi || b.lo == b.hi) return false;
    return a.lo < b.hi && b.lo < a.hi;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int pick_tile(int m, int n, int batch) {
    if (m <= 64 && n <= 64) return SGEMM_EMU_TILE_64x64;
    const int64_t big = (int64_t)((m + 255) / 256) * ((n + 127) / 128) * batch;
    if (m >= 256 && big >= 1024) return SGEMM_EMU_TILE_256x128;
    return SGEMM_EMU_TILE_128x128;
}

// AUTO tile under a flow the caller named: a tile that flow is built for.
// The register-direct flow has 64x64 and 128x128 tiles (128x128 only when
// B's rows allow its vector loads); the direct and staged flows run on
// 64x64 and 128x128 everywhere (the full-tile kernel has them on 128x128
// only, the staged flow's general kernel stops at 128x128).  The split flow
// takes the shape-based choice.
int pick_tile_for_flow(const sgemm_emu::GemmArgs& a, int flow, int batch) {
    const bool small = a.m <= 64 && a.n <= 64;
    switch (flow) {
        case SGEMM_EMU_FLOW_REG:
            if (small) return SGEMM_EMU_TILE_64x64;
            return sgemm_emu::reg_flow_supported(a, SGEMM_EMU_TILE_128x128)
                       ? SGEMM_EMU_TILE_128x128
                       : SGEMM_EMU_TILE_64x64;
        case SGEMM_EMU_FLOW_DIRECT:
        case SGEMM_EMU_FLOW_STAGED:
            return small ? SGEMM_EMU_TILE_64x64 : SGEMM_EMU_TILE_128x128;
        default: return pick_tile(a.m, a.n, batch);
    }
}

// Validation shared by the two GEMM entry points.
int check_gemm(int m, int n, int k, const float* A, int lda, const float* B, int ldb, float* C,
               int ldc, int batch, sgemm_emu_stride_t st) {
    if (m < 0 || n < 0 || k < 0 || batch < 0) return SGEMM_EMU_ERR_DIM;
    if (lda < (k > 1 ? k : 1) || ldb < (n > 1 ? n : 1) || ldc < (n > 1 ? n : 1))
        return SGEMM_EMU_ERR_LD;
    if (m == 0 || n == 0 || batch == 0) return SGEMM_EMU_OK;
    if (C == nullptr) return SGEMM_EMU_ERR_NULL;
    if (k > 0 && (A == nullptr || B == nullptr)) return SGEMM_EMU_ERR_NULL;
    if (st.a < 0 || st.b < 0 || st.c < 0) return SGEMM_EMU_ERR_STRIDE;
    if (batch > 1 && st.c < (int64_t)(m - 1) * ldc + n) return SGEMM_EMU_ERR_STRIDE;
    const Extent ec = extent(C, batch, m, n, ldc, st.c);
    if (!ec.ok) return SGEMM_EMU_ERR_STRIDE;
    if (k > 0) {
        const Extent ea = extent(A, st.a == 0 ? 1 : batch, m, k, lda, st.a);
        const Extent eb = extent(B, st.b == 0 ? 1 : batch, k, n, ldb, st.b);
        if (!all_ok({ea, eb})) return SGEMM_EMU_ERR_STRIDE;
        if (overlap(ec, ea) || overlap(ec, eb)) return SGEMM_EMU_ERR_ALIAS;
    }
    return SGEMM_EMU_OK;
}

// The kernels a GEMM call can run.  K_NONE: an empty problem (nothing to
// run).  K_TILED: a large product whose shape does not fill whole tiles, run
// as its interior of whole tiles on the full-tile kernel, a k tail (k mod 32
// values) added in place by the accumulate kernel, and the edge strips on
// the register-flow kernel.
enum Kernel { K_NONE, K_REG, K_BIG, K_LDS, K_TILED };

const char* kernel_name(Kernel k) {
    switch (k) {
        case K_REG: return "bgemm_reg_kernel";
        case K_BIG: return "bgemm_big_kernel";
        case K_LDS: return "bgemm_emu_kernel";
        case K_TILED: return "bgemm_big_kernel+bgemm_reg_kernel";
        default: return "";
    }
}

int tile_rows(int tile) { return tile == SGEMM_EMU_TILE_256x128 ? 256 : 128; }
int tile_cols(int tile) { return tile == SGEMM_EMU_TILE_128x256 ? 256 : 128; }

// Interior of whole tiles and whole 32-deep k chunks.
struct Interior {
    int m, n, k;
};

Interior interior(const sgemm_emu::GemmArgs& a, int tile) {
    return {a.m - a.m % tile_rows(tile), a.n - a.n % tile_cols(tile), a.k - a.k % 32};
}

// Validate, then resolve the policy (flow and tile, AUTO replaced by the
// library's choice), fill the kernel arguments and name the kernel.
int resolve_gemm(int m, int n, int k, const float* A, int lda, const float* B, int ldb, float* C,
                 int ldc, int batch, sgemm_emu_stride_t st, int& flow, int ec, int& tile,
                 sgemm_emu::GemmArgs& a, Kernel& kern) {
    kern = K_NONE;
    int rc = check_gemm(m, n, k, A, lda, B, ldb, C, ldc, batch, st);
    if (rc != SGEMM_EMU_OK) return rc;
    if (flow < SGEMM_EMU_FLOW_AUTO || flow > SGEMM_EMU_FLOW_REG) return SGEMM_EMU_ERR_POLICY;
    if (ec != 0 && ec != 1) return SGEMM_EMU_ERR_POLICY;
    if (tile < SGEMM_EMU_TILE_AUTO || tile > SGEMM_EMU_TILE_128x256) return SGEMM_EMU_ERR_POLICY;
    if (m == 0 || n == 0 || batch == 0) return SGEMM_EMU_OK;
    a.m = m;
    a.n = n;
    a.k = k;
    a.A = A;
    a.lda = lda;
    a.sa = st.a;
    a.B = B;
    a.ldb = ldb;
    a.sb = st.b;
    a.C = C;
    a.ldc = ldc;
    a.sc = st.c;
    a.batch = batch;
    a.vec_a = aligned16(A) && lda % 4 == 0 && st.a % 4 == 0;
    a.vec_b = aligned16(B) && ldb % 4 == 0 && st.b % 4 == 0;
    if (flow == SGEMM_EMU_FLOW_AUTO) {
        // Full tiles take the pipelined split-flow kernel (each element
        // split once per workgroup).  Other products take the barrier-free
        // register-direct flow, which keeps the most bytes in flight: 1.8-5x
        // the general LDS kernel's rate on every shape measured (1100 x 1500
        // x 2000: 76 against 397 us; 8000^3: 5.9 against 7.2 ms).  From
        // 2^35 multiply-adds on, a large ragged product whose whole tiles
        // cover nearly all of C runs faster decomposed: those tiles on the
        // full-tile kernel, the rest on the accumulate and register-flow
        // kernels (4000^3: 557 against 613 us; 8000^3: 3.5 against 5.9 ms;
        // 3000^3: 338 against 320 us).  The general kernel is left for
        // unaligned operands.
        int big_tile = SGEMM_EMU_TILE_AUTO;
        const bool wide = k >= 1024 && (int64_t)m * n * batch >= (int64_t)2048 * 2048;
        // 128x256 pays off for long k loops over much output (measured on
        // 8192^3 and on 256 x 1024 x 1024 x k for k >= 1024)
        const int order[3] = {wide ? SGEMM_EMU_TILE_128x256 : SGEMM_EMU_TILE_256x128,
                              SGEMM_EMU_TILE_256x128, SGEMM_EMU_TILE_128x128};
        for (int t : order)
            if (big_tile == SGEMM_EMU_TILE_AUTO && (tile == SGEMM_EMU_TILE_AUTO || tile == t) &&
                sgemm_emu::big_supported(a, t, SGEMM_EMU_FLOW_SPLIT, ec == 1))
                big_tile = t;
        const double work = (double)batch * m * n * k;  // multiply-adds (no overflow)
        const double kDecompose = 34359738368.0;         // 2^35
        // the decomposition: whole tiles covering at least 95% of C, at least
        // one per CU (measured: 0.95-0.98 coverage won or tied, 0.92-0.94 lost
        // to the register-direct flow by 1.2-1.4x)
        int tiled = SGEMM_EMU_TILE_AUTO;
        if (big_tile == SGEMM_EMU_TILE_AUTO && ec == 1 && tile == SGEMM_EMU_TILE_AUTO &&
            a.vec_a && a.vec_b && m > 1024 && n > 1024 && k >= 32 &&
            work >= kDecompose && sgemm_emu::reg_flow_supported(a, SGEMM_EMU_TILE_64x64)) {
            // (the 128 x 128 interior lost on every shape measured)
            for (int t : {order[0], order[1]}) {
                const Interior in = interior(a, t);
                const int64_t ntiles =
                    (int64_t)(in.m / tile_rows(t)) * (in.n / tile_cols(t)) * batch;
                if (tiled == SGEMM_EMU_TILE_AUTO && ntiles >= 256 &&
                    (int64_t)in.m * in.n * 20 >= (int64_t)m * n * 19)
                    tiled = t;
            }
        }
        // register-direct tile: 64x64 for products inside one such tile or
        // B rows that allow no vector loads (that one only below 2^35
        // multiply-adds: measured only there), else 128x128
        int reg_tile = SGEMM_EMU_TILE_AUTO;
        if (m <= 64 && n <= 64) {
            if (sgemm_emu::reg_flow_supported(a, SGEMM_EMU_TILE_64x64))
                reg_tile = SGEMM_EMU_TILE_64x64;
        } else if (sgemm_emu::reg_flow_supported(a, SGEMM_EMU_TILE_128x128)) {
            reg_tile = SGEMM_EMU_TILE_128x128;
        } else if (work < kDecompose && sgemm_emu::reg_flow_supported(a, SGEMM_EMU_TILE_64x64)) {
            reg_tile = SGEMM_EMU_TILE_64x64;
        }
        if (tile != SGEMM_EMU_TILE_AUTO && tile != reg_tile) reg_tile = SGEMM_EMU_TILE_AUTO;
        if (big_tile != SGEMM_EMU_TILE_AUTO) {
            flow = SGEMM_EMU_FLOW_SPLIT;
            tile = big_tile;
        } else if (tiled != SGEMM_EMU_TILE_AUTO) {
            flow = SGEMM_EMU_FLOW_SPLIT;
            tile = tiled;
            kern = K_TILED;
            return SGEMM_EMU_OK;
        } else if (reg_tile != SGEMM_EMU_TILE_AUTO) {
            flow = SGEMM_EMU_FLOW_REG;
            tile = reg_tile;
        } else {
            flow = SGEMM_EMU_FLOW_SPLIT;
        }
    }
    if (tile == SGEMM_EMU_TILE_AUTO) tile = pick_tile_for_flow(a, flow, batch);
    if (flow == SGEMM_EMU_FLOW_REG) {
        if (!sgemm_emu::reg_flow_supported(a, tile)) return SGEMM_EMU_ERR_POLICY;
        kern = K_REG;
    } else if (sgemm_emu::big_supported(a, tile, flow, ec == 1)) {
        kern = K_BIG;  // full tiles: the pipelined kernel
    } else if (tile != SGEMM_EMU_TILE_128x256 && sgemm_emu::gemm_variant_exists(tile, flow)) {
        kern = K_LDS;
    } else {
        return SGEMM_EMU_ERR_POLICY;
    }
    return SGEMM_EMU_OK;
}

// An edge strip (at most one tile deep, long k): the barrier-free register
// flow on 64 x 64 tiles runs 4-6x faster than the LDS-tiled general kernel
// there (measured on 7936 x 64 x 8000 and 64 x 8000 x 8000), since the
// strip has too few tiles to hide the general kernel's per-step barriers.
// The strips share A's row alignment and both leading dimensions with the
// whole product, which was checked for this flow before K_TILED was chosen.
hipError_t run_strip(const sgemm_emu::GemmArgs& s, hipStream_t stream) {
    return sgemm_emu::launch_gemm_reg(s, SGEMM_EMU_TILE_64x64, true, stream);
}

// K_TILED, in stream order: the interior C[0:mi, 0:ni] = A[0:mi, 0:ki]
// B[0:ki, 0:ni] on the full-tile kernel; the k tail C[0:mi, 0:ni] +=
// A[0:mi, ki:k] B[ki:k, 0:ni] in place; the right strip C[0:mi, ni:n] and
// the bottom strip C[mi:m, 0:n] over the whole k on the register-flow
// kernel (64 x 64 tiles).  Every piece is a view of the same operands (same
// ld and item strides).
hipError_t run_tiled(const sgemm_emu::GemmArgs& a, int tile, hipStream_t stream) {
    const Interior in = interior(a, tile);
    sgemm_emu::GemmArgs g = a;
    g.m = in.m;
    g.n = in.n;
    g.k = in.k;
    hipError_t e = sgemm_emu::launch_gemm_big(g, tile, SGEMM_EMU_FLOW_SPLIT, true, stream);
    if (e != hipSuccess) return e;
    if (in.k < a.k) {
        sgemm_emu::AccArgs t{};
        t.m = in.m;
        t.n = in.n;
        t.k = a.k - in.k;
        t.A = a.A + in.k;
        t.lda = a.lda;
        t.sa = a.sa;
        t.B = a.B + (int64_t)in.k * a.ldb;
        t.ldb = a.ldb;
        t.sb = a.sb;
        t.C = a.C;
        t.ldc = a.ldc;
        t.sc = a.sc;
        t.D = a.C;
        t.ldd = a.ldc;
        t.sd = a.sc;
        t.batch = a.batch;
        t.a_trans = t.b_trans = t.cd_col = false;
        t.vec_a = a.vec_a;  // ki is a multiple of 32: rows stay 16-byte aligned
        // row-major B (k x n) and row-major C, D: the fragment loads and
        // stores move single elements along those layouts, so these flags
        // only select the whole-tile path and set no alignment requirement
        t.vec_b = t.vec_c = t.vec_d = true;
        e = sgemm_emu::launch_gemm_acc(t, MFMAE_SHAPE_32x32x16, true, stream);
        if (e != hipSuccess) return e;
    }
    if (in.n < a.n) {
        sgemm_emu::GemmArgs r = a;
        r.m = in.m;
        r.n = a.n - in.n;
        r.B = a.B + in.n;
        r.C = a.C + in.n;
        r.vec_b = a.vec_b && in.n % 4 == 0;
        e = run_strip(r, stream);
        if (e != hipSuccess) return e;
    }
    if (in.m < a.m) {
        sgemm_emu::GemmArgs b = a;
        b.m = a.m - in.m;
        b.A = a.A + (int64_t)in.m * a.lda;
        b.C = a.C + (int64_t)in.m * a.ldc;
        e = run_strip(b, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

int run_gemm(int m, int n, int k, const float* A, int lda, const float* B, int ldb, float* C,
             int ldc, int batch, sgemm_emu_stride_t st, int flow, int ec, int tile,
             hipStream_t stream) {
    sgemm_emu::GemmArgs a;
    Kernel kern;
    int rc = resolve_gemm(m, n, k, A, lda, B, ldb, C, ldc, batch, st, flow, ec, tile, a, kern);
    if (rc != SGEMM_EMU_OK || kern == K_NONE) return rc;
    hipError_t e;
    switch (kern) {
        case K_REG: e = sgemm_emu::launch_gemm_reg(a, tile, ec != 0, stream); break;
        case K_BIG: e = sgemm_emu::launch_gemm_big(a, tile, flow, ec != 0, stream); break;
        case K_TILED: e = run_tiled(a, tile, stream); break;
        default: e = sgemm_emu::launch_gemm(a, tile, flow, ec != 0, stream); break;
    }
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

template <class S>
int map_impl(int use, int i, int j, int* lane, int* elem) {
    using namespace mfmae;
    switch (use) {
        case MFMAE_USE_A:
            if (i < 0 || i >= S::M || j < 0 || j >= S::K) return SGEMM_EMU_ERR_DIM;
            *lane = layout<S, Use::A>::lane_of(i, j);
            *elem = layout<S, Use::A>::elem_of(i, j);
            return SGEMM_EMU_OK;
        case MFMAE_USE_B:
            if (i < 0 || i >= S::K || j < 0 || j >= S::N) return SGEMM_EMU_ERR_DIM;
            *lane = layout<S, Use::B>::lane_of(i, j);
            *elem = layout<S, Use::B>::elem_of(i, j);
            return SGEMM_EMU_OK;
        case MFMAE_USE_ACC:
            if (i < 0 || i >= S::M || j < 0 || j >= S::N) return SGEMM_EMU_ERR_DIM;
            *lane = layout<S, Use::Acc>::lane_of(i, j);
            *elem = layout<S, Use::Acc>::elem_of(i, j);
            return SGEMM_EMU_OK;
        default: return SGEMM_EMU_ERR_UNSUPPORTED;
    }
}

template <class L>
void foreach_fill(int lane, int* i_out, int* j_out) {
    for (int e = 0; e < L::num_elements; ++e) {
        i_out[e] = L::row(lane, e);
        j_out[e] = L::col(lane, e);
    }
}

template <class S>
int foreach_impl(int use, int lane, int* i_out, int* j_out) {
    using namespace mfmae;
    switch (use) {
        case MFMAE_USE_A: foreach_fill<layout<S, Use::A>>(lane, i_out, j_out); return SGEMM_EMU_OK;
        case MFMAE_USE_B: foreach_fill<layout<S, Use::B>>(lane, i_out, j_out); return SGEMM_EMU_OK;
        case MFMAE_USE_ACC:
            foreach_fill<layout<S, Use::Acc>>(lane, i_out, j_out);
            return SGEMM_EMU_OK;
        default: return SGEMM_EMU_ERR_UNSUPPORTED;
    }
}

}  // namespace

extern "C" {

int sgemm_emu_batched(int m, int n, int k, const float* A, int lda, const float* B, int ldb,
                      float* C, int ldc, int batch, sgemm_emu_stride_t stride,
                      hipStream_t stream) {
    return run_gemm(m, n, k, A, lda, B, ldb, C, ldc, batch, stride, SGEMM_EMU_FLOW_AUTO, 1,
                    SGEMM_EMU_TILE_AUTO, stream);
}

int sgemm_emu_batched_ex(int m, int n, int k, const float* A, int lda, const float* B, int ldb,
                         float* C, int ldc, int batch, sgemm_emu_stride_t stride,
                         const sgemm_emu_policy_t* policy, hipStream_t stream) {
    sgemm_emu_policy_t pol{SGEMM_EMU_FLOW_AUTO, 1, SGEMM_EMU_TILE_AUTO};
    if (policy) pol = *policy;
    return run_gemm(m, n, k, A, lda, B, ldb, C, ldc, batch, stride, pol.flow, pol.ec, pol.tile,
                    stream);
}

int sgemm_emu_resolve_policy(int m, int n, int k, const float* A, int lda, const float* B,
                             int ldb, float* C, int ldc, int batch, sgemm_emu_stride_t stride,
                             const sgemm_emu_policy_t* policy, sgemm_emu_policy_t* out,
                             const char** kernel) {
    if (out == nullptr) return SGEMM_EMU_ERR_NULL;
    sgemm_emu_policy_t pol{SGEMM_EMU_FLOW_AUTO, 1, SGEMM_EMU_TILE_AUTO};
    if (policy) pol = *policy;
    sgemm_emu::GemmArgs a;
    Kernel kern;
    int rc = resolve_gemm(m, n, k, A, lda, B, ldb, C, ldc, batch, stride, pol.flow, pol.ec,
                          pol.tile, a, kern);
    if (rc != SGEMM_EMU_OK) return rc;
    *out = pol;
    if (kernel)
        *kernel = kern == K_BIG && sgemm_emu::big_streams(a, pol.tile, pol.flow)
                      ? "bgemm_big_stream_kernel"
                      : kernel_name(kern);
    return SGEMM_EMU_OK;
}

int sgemm_emu_xcd_order(int grid, int* task_of_workgroup) {
    if (grid < 1) return SGEMM_EMU_ERR_DIM;
    if (task_of_workgroup == nullptr) return SGEMM_EMU_ERR_NULL;
    for (int b = 0; b < grid; ++b) task_of_workgroup[b] = sgemm_emu::xcd_task(b, grid);
    return SGEMM_EMU_OK;
}

int sgemm_emu_tile_order(int tiles_m, int tiles_n, int* tile_row, int* tile_col) {
    if (tiles_m < 1 || tiles_n < 1 || (int64_t)tiles_m * tiles_n > INT32_MAX)
        return SGEMM_EMU_ERR_DIM;
    if (tile_row == nullptr || tile_col == nullptr) return SGEMM_EMU_ERR_NULL;
    const int tiles = tiles_m * tiles_n;
    for (int t = 0; t < tiles; ++t) {
        const sgemm_emu::TileRC rc = sgemm_emu::grouped_tile(t, tiles_m, tiles_n);
        tile_row[t] = rc.tm;
        tile_col[t] = rc.tn;
    }
    return SGEMM_EMU_OK;
}

int sgemm_emu_block_order(int tiles_m, int tiles_n, int* tile_row, int* tile_col) {
    if (tiles_m < 1 || tiles_n < 1 || (int64_t)tiles_m * tiles_n > INT32_MAX ||
        !sgemm_emu::block_order_applies(tiles_m, tiles_n, tiles_m * tiles_n))
        return SGEMM_EMU_ERR_DIM;
    if (tile_row == nullptr || tile_col == nullptr) return SGEMM_EMU_ERR_NULL;
    const int tiles = tiles_m * tiles_n;
    for (int t = 0; t < tiles; ++t) {
        const sgemm_emu::TileRC rc = sgemm_emu::block_tile(t, tiles_m, tiles_n);
        tile_row[t] = rc.tm;
        tile_col[t] = rc.tn;
    }
    return SGEMM_EMU_OK;
}

int sgemm_emu_batched_acc(int op_a, int op_b, int layout_cd, int m, int n, int k, const float* A,
                          int lda, const float* B, int ldb, const float* C, int ldc, float* D,
                          int ldd, int batch, sgemm_emu_stride4_t stride, int shape, int ec,
                          hipStream_t stream) {
    if ((op_a != SGEMM_EMU_OP_N && op_a != SGEMM_EMU_OP_T) ||
        (op_b != SGEMM_EMU_OP_N && op_b != SGEMM_EMU_OP_T) ||
        (layout_cd != SGEMM_EMU_ROW_MAJOR && layout_cd != SGEMM_EMU_COL_MAJOR) ||
        (shape != MFMAE_SHAPE_16x16x32 && shape != MFMAE_SHAPE_32x32x16) || (ec != 0 && ec != 1))
        return SGEMM_EMU_ERR_POLICY;
    if (m < 0 || n < 0 || k < 0 || batch < 0) return SGEMM_EMU_ERR_DIM;
    const bool at = op_a == SGEMM_EMU_OP_T, bt = op_b == SGEMM_EMU_OP_T;
    const bool cdc = layout_cd == SGEMM_EMU_COL_MAJOR;
    // stored shapes (rows x cols, row-major with the given ld)
    const int ar = at ? k : m, ac = at ? m : k;
    const int br = bt ? n : k, bc = bt ? k : n;
    const int cr = cdc ? n : m, cc = cdc ? m : n;
    auto ld_ok = [](int ld, int cols) { return ld >= (cols > 1 ? cols : 1); };
    if (!ld_ok(lda, ac) || !ld_ok(ldb, bc) || !ld_ok(ldd, cc) || (C && !ld_ok(ldc, cc)))
        return SGEMM_EMU_ERR_LD;
    if (m == 0 || n == 0 || batch == 0) return SGEMM_EMU_OK;
    // tile and k-step indices are formed in 32 bits with room for one tile
    if (m >= (1 << 30) || n >= (1 << 30) || k >= (1 << 30)) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (D == nullptr || (k > 0 && (A == nullptr || B == nullptr))) return SGEMM_EMU_ERR_NULL;
    if (stride.a < 0 || stride.b < 0 || stride.c < 0 || stride.d < 0) return SGEMM_EMU_ERR_STRIDE;
    if (batch > 1 && stride.d < (int64_t)(cr - 1) * ldd + cc) return SGEMM_EMU_ERR_STRIDE;
    const Extent ed = extent(D, batch, cr, cc, ldd, stride.d);
    const Extent none{0, 0, true};
    const Extent ea = k > 0 ? extent(A, stride.a == 0 ? 1 : batch, ar, ac, lda, stride.a) : none;
    const Extent eb = k > 0 ? extent(B, stride.b == 0 ? 1 : batch, br, bc, ldb, stride.b) : none;
    const Extent ecx = C ? extent(C, stride.c == 0 ? 1 : batch, cr, cc, ldc, stride.c) : none;
    if (!all_ok({ed, ea, eb, ecx})) return SGEMM_EMU_ERR_STRIDE;
    if (overlap(ed, ea) || overlap(ed, eb)) return SGEMM_EMU_ERR_ALIAS;
    if (C) {
        const bool in_place = C == D && ldc == ldd && stride.c == stride.d;
        if (!in_place && overlap(ed, ecx)) return SGEMM_EMU_ERR_ALIAS;
    }
    auto vec_ok = [](const void* p, int64_t ld, int64_t s) {
        return ((uintptr_t)p % 16 == 0) && ld % 4 == 0 && s % 4 == 0;
    };
    sgemm_emu::AccArgs a;
    a.m = m;
    a.n = n;
    a.k = k;
    a.A = A;
    a.lda = lda;
    a.sa = stride.a;
    a.B = B;
    a.ldb = ldb;
    a.sb = stride.b;
    a.C = C;
    a.ldc = ldc;
    a.sc = stride.c;
    a.D = D;
    a.ldd = ldd;
    a.sd = stride.d;
    a.batch = batch;
    a.a_trans = at;
    a.b_trans = bt;
    a.cd_col = cdc;
    // 16-byte accesses happen only along a contiguous direction: A stored
    // m x k, B stored n x k, C and D stored column-major
    a.vec_a = at || vec_ok(A, lda, stride.a);
    a.vec_b = !bt || vec_ok(B, ldb, stride.b);
    a.vec_c = C == nullptr || !cdc || vec_ok(C, ldc, stride.c);
    a.vec_d = !cdc || vec_ok(D, ldd, stride.d);
    hipError_t e = sgemm_emu::launch_gemm_acc(a, shape, ec == 1, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int householder_emu_batched(int n, const float* u, int64_t stride_u, const float* B, int ldb,
                            int64_t stride_b, int ncols, float* C, int ldc, int64_t stride_c,
                            int batch, hipStream_t stream) {
    return householder_emu_batched_ex(n, u, stride_u, B, ldb, stride_b, ncols, C, ldc, stride_c,
                                      batch, SGEMM_EMU_HOUSEHOLDER_RULE, stream);
}

int householder_emu_batched_ex(int n, const float* u, int64_t stride_u, const float* B, int ldb,
                               int64_t stride_b, int ncols, float* C, int ldc, int64_t stride_c,
                               int batch, int mode, hipStream_t stream) {
    if (mode != SGEMM_EMU_HOUSEHOLDER_RULE && mode != SGEMM_EMU_HOUSEHOLDER_LDS)
        return SGEMM_EMU_ERR_POLICY;
    if (n < 0 || ncols < 0 || batch < 0) return SGEMM_EMU_ERR_DIM;
    if (ldb < (ncols > 1 ? ncols : 1) || ldc < (ncols > 1 ? ncols : 1)) return SGEMM_EMU_ERR_LD;
    if (n == 0 || ncols == 0 || batch == 0) return SGEMM_EMU_OK;
    if (n != 64) return SGEMM_EMU_ERR_UNSUPPORTED;
    // the kernel forms 8 * ldb + column as a 32-bit lane offset
    if (ldb >= (1 << 27)) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (u == nullptr || B == nullptr || C == nullptr) return SGEMM_EMU_ERR_NULL;
    if (stride_u < 0 || stride_b < 0 || stride_c < 0) return SGEMM_EMU_ERR_STRIDE;
    if (batch > 1 && stride_c < (int64_t)(n - 1) * ldc + ncols) return SGEMM_EMU_ERR_STRIDE;
    const Extent ec = extent(C, batch, n, ncols, ldc, stride_c);
    const Extent eu = extent(u, stride_u == 0 ? 1 : batch, 1, n, n, stride_u);
    const Extent eb = extent(B, stride_b == 0 ? 1 : batch, n, ncols, ldb, stride_b);
    if (!all_ok({ec, eu, eb})) return SGEMM_EMU_ERR_STRIDE;
    if (overlap(ec, eu) || overlap(ec, eb)) return SGEMM_EMU_ERR_ALIAS;
    sgemm_emu::HouseholderArgs a;
    a.mode = mode;
    a.ncols = ncols;
    a.u = u;
    a.su = stride_u;
    a.B = B;
    a.ldb = ldb;
    a.sb = stride_b;
    a.C = C;
    a.ldc = ldc;
    a.sc = stride_c;
    a.batch = batch;
    hipError_t e = sgemm_emu::launch_householder64(a, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int givens_emu_batched(int n, int i, int j, const float* c, const float* s, int64_t stride_cs,
                       const float* B, int ldb, int64_t stride_b, int ncols, float* C, int ldc,
                       int64_t stride_c, int batch, int mode, hipStream_t stream) {
    if (n < 0 || ncols < 0 || batch < 0) return SGEMM_EMU_ERR_DIM;
    if (mode < SGEMM_EMU_GIVENS_AUTO || mode > SGEMM_EMU_GIVENS_LDS) return SGEMM_EMU_ERR_POLICY;
    if (ldb < (ncols > 1 ? ncols : 1) || ldc < (ncols > 1 ? ncols : 1)) return SGEMM_EMU_ERR_LD;
    if (n == 0 || ncols == 0 || batch == 0) return SGEMM_EMU_OK;
    if (i < 0 || j < 0 || i >= n || j >= n || i == j) return SGEMM_EMU_ERR_DIM;
    if (n != 64) return SGEMM_EMU_ERR_UNSUPPORTED;
    // the kernel forms 8 * ldb + column as a 32-bit lane offset
    if (ldb >= (1 << 27)) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (mode == SGEMM_EMU_GIVENS_AUTO)
        mode = sgemm_emu::givens_embedded(i, j) ? SGEMM_EMU_GIVENS_EMBEDDED : SGEMM_EMU_GIVENS_MAP;
    if (mode == SGEMM_EMU_GIVENS_EMBEDDED && !sgemm_emu::givens_embedded(i, j))
        return SGEMM_EMU_ERR_UNSUPPORTED;
    if (c == nullptr || s == nullptr || B == nullptr || C == nullptr) return SGEMM_EMU_ERR_NULL;
    if (stride_cs < 0 || stride_b < 0 || stride_c < 0) return SGEMM_EMU_ERR_STRIDE;
    if (batch > 1 && stride_c < (int64_t)(n - 1) * ldc + ncols) return SGEMM_EMU_ERR_STRIDE;
    const Extent ec = extent(C, batch, n, ncols, ldc, stride_c);
    const Extent ecs = extent(c, stride_cs == 0 ? 1 : batch, 1, 1, 1, stride_cs);
    const Extent ess = extent(s, stride_cs == 0 ? 1 : batch, 1, 1, 1, stride_cs);
    const Extent eb = extent(B, stride_b == 0 ? 1 : batch, n, ncols, ldb, stride_b);
    if (!all_ok({ec, ecs, ess, eb})) return SGEMM_EMU_ERR_STRIDE;
    if (overlap(ec, ecs) || overlap(ec, ess) || overlap(ec, eb)) return SGEMM_EMU_ERR_ALIAS;
    sgemm_emu::GivensArgs a;
    a.ncols = ncols;
    a.i = i;
    a.j = j;
    a.c = c;
    a.s = s;
    a.scs = stride_cs;
    a.B = B;
    a.ldb = ldb;
    a.sb = stride_b;
    a.C = C;
    a.ldc = ldc;
    a.sc = stride_c;
    a.batch = batch;
    a.mode = mode;
    hipError_t e = sgemm_emu::launch_givens64(a, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int sgemm_emu_scan(int64_t rows, int len, const float* X, int64_t ldx, float* Y, int64_t ldy,
                   hipStream_t stream) {
    if (rows < 0 || len < 0) return SGEMM_EMU_ERR_DIM;
    if (ldx < (len > 1 ? len : 1) || ldy < (len > 1 ? len : 1)) return SGEMM_EMU_ERR_LD;
    if (rows == 0 || len == 0) return SGEMM_EMU_OK;
    if (X == nullptr || Y == nullptr) return SGEMM_EMU_ERR_NULL;
    const Extent ex = extent(X, 1, rows, len, ldx, 0);
    const Extent ey = extent(Y, 1, rows, len, ldy, 0);
    if (!all_ok({ex, ey})) return SGEMM_EMU_ERR_LD;
    const bool in_place = X == Y && ldx == ldy;
    if (!in_place && overlap(ex, ey)) return SGEMM_EMU_ERR_ALIAS;
    sgemm_emu::ScanArgs a;
    a.rows = rows;
    a.len = len;
    a.X = X;
    a.ldx = ldx;
    a.Y = Y;
    a.ldy = ldy;
    // 16-byte loads of X and 16-byte stores of Y
    a.vec = ((uintptr_t)X % 16 == 0) && ldx % 4 == 0 && ((uintptr_t)Y % 16 == 0) && ldy % 4 == 0;
    hipError_t e = sgemm_emu::launch_scan(a, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int sgemm_emu_split(int64_t count, const float* x, uint16_t* hi, uint16_t* lo, int form,
                    hipStream_t stream) {
    if (count < 0) return SGEMM_EMU_ERR_DIM;
    if (form < SGEMM_EMU_SPLIT_SCALAR || form > SGEMM_EMU_SPLIT_EIGHT) return SGEMM_EMU_ERR_POLICY;
    if (count == 0) return SGEMM_EMU_OK;
    if (x == nullptr || hi == nullptr || lo == nullptr) return SGEMM_EMU_ERR_NULL;
    const Extent ex = extent(x, 1, 1, count, count, 0, 4);
    const Extent eh = extent(hi, 1, 1, count, count, 0, 2);
    const Extent el = extent(lo, 1, 1, count, count, 0, 2);
    if (!all_ok({ex, eh, el})) return SGEMM_EMU_ERR_DIM;
    if (overlap(ex, eh) || overlap(ex, el) || overlap(eh, el)) return SGEMM_EMU_ERR_ALIAS;
    hipError_t e = sgemm_emu::launch_split(count, x, hi, lo, form, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int mfmae_num_elements(int shape, int use) {
    if (use < MFMAE_USE_A || use > MFMAE_USE_ACC) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (shape == MFMAE_SHAPE_16x16x32) return use == MFMAE_USE_ACC ? 4 : 8;
    if (shape == MFMAE_SHAPE_32x32x16) return use == MFMAE_USE_ACC ? 16 : 8;
    return SGEMM_EMU_ERR_UNSUPPORTED;
}

int mfmae_map(int shape, int use, int i, int j, int* lane, int* elem) {
    if (lane == nullptr || elem == nullptr) return SGEMM_EMU_ERR_NULL;
    if (shape == MFMAE_SHAPE_16x16x32) return map_impl<mfmae::Shape16>(use, i, j, lane, elem);
    if (shape == MFMAE_SHAPE_32x32x16) return map_impl<mfmae::Shape32>(use, i, j, lane, elem);
    return SGEMM_EMU_ERR_UNSUPPORTED;
}

int mfmae_foreach(int shape, int use, int lane, int* i_out, int* j_out) {
    if (mfmae_num_elements(shape, use) < 0) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (lane < 0 || lane >= 64) return SGEMM_EMU_ERR_DIM;
    if (i_out == nullptr || j_out == nullptr) return SGEMM_EMU_ERR_NULL;
    if (shape == MFMAE_SHAPE_16x16x32) return foreach_impl<mfmae::Shape16>(use, lane, i_out, j_out);
    return foreach_impl<mfmae::Shape32>(use, lane, i_out, j_out);
}

int mfmae_mma_probe(int shape, const uint16_t* a, const uint16_t* b, float* d,
                    hipStream_t stream) {
    if (shape != MFMAE_SHAPE_16x16x32 && shape != MFMAE_SHAPE_32x32x16)
        return SGEMM_EMU_ERR_UNSUPPORTED;
    if (a == nullptr || b == nullptr || d == nullptr) return SGEMM_EMU_ERR_NULL;
    hipError_t e = sgemm_emu::launch_mma_probe(shape, a, b, d, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int sgemm_emu_stream_probe(int64_t items, int64_t item_elems, const float* A, const float* B,
                           float* C, int threads, hipStream_t stream) {
    if (items < 0 || item_elems < 0) return SGEMM_EMU_ERR_DIM;
    if (items == 0) return SGEMM_EMU_OK;
    if (A == nullptr || B == nullptr || C == nullptr) return SGEMM_EMU_ERR_NULL;
    if (threads != 256 && threads != 512 && threads != 1024) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (item_elems == 0 || item_elems % 4 != 0 || item_elems >= (int64_t(1) << 31))
        return SGEMM_EMU_ERR_UNSUPPORTED;
    if (!aligned16(A) || !aligned16(B) || !aligned16(C)) return SGEMM_EMU_ERR_UNSUPPORTED;
    if (items > INT64_MAX / item_elems) return SGEMM_EMU_ERR_DIM;
    const Extent ea = extent(A, items, 1, item_elems, item_elems, item_elems);
    const Extent eb = extent(B, items, 1, item_elems, item_elems, item_elems);
    const Extent ec = extent(C, items, 1, item_elems, item_elems, item_elems);
    if (!all_ok({ea, eb, ec})) return SGEMM_EMU_ERR_DIM;
    if (overlap(ec, ea) || overlap(ec, eb)) return SGEMM_EMU_ERR_ALIAS;
    hipError_t e = sgemm_emu::launch_stream_probe(items, item_elems, A, B, C, threads, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

int sgemm_emu_mfma_probe(int m, int n, int k, const float* A, int lda, const float* B, int ldb,
                         float* C, int ldc, hipStream_t stream) {
    if (m < 0 || n < 0 || k < 0) return SGEMM_EMU_ERR_DIM;
    if (m == 0 || n == 0) return SGEMM_EMU_OK;
    if (k == 0 || m % 128 != 0 || n % 256 != 0 || k % 32 != 0) return SGEMM_EMU_ERR_UNSUPPORTED;
    if ((int64_t)(m / 128) * (n / 256) > ((int64_t)1 << 31) / 512 - 1) return SGEMM_EMU_ERR_DIM;
    if (lda < 32 || ldb < n || ldc < n) return SGEMM_EMU_ERR_LD;
    if (A == nullptr || B == nullptr || C == nullptr) return SGEMM_EMU_ERR_NULL;
    const Extent ea = extent(A, 1, m, 32, lda, 0);
    const Extent eb = extent(B, 1, 32, n, ldb, 0);
    const Extent ec = extent(C, 1, m, n, ldc, 0);
    if (!all_ok({ea, eb, ec})) return SGEMM_EMU_ERR_DIM;
    if (overlap(ec, ea) || overlap(ec, eb)) return SGEMM_EMU_ERR_ALIAS;
    hipError_t e = sgemm_emu::launch_mfma_probe(m, n, k, A, lda, B, ldb, C, ldc, stream);
    return e == hipSuccess ? SGEMM_EMU_OK : hip_fail(e);
}

const char* sgemm_emu_strerror(int code) {
    switch (code) {
        case SGEMM_EMU_OK: return "success";
        case SGEMM_EMU_ERR_DIM: return "negative or out-of-range size";
        case SGEMM_EMU_ERR_LD: return "leading dimension too small";
        case SGEMM_EMU_ERR_NULL: return "null pointer with nonzero work";
        case SGEMM_EMU_ERR_STRIDE: return "negative batch stride or overlapping output items";
        case SGEMM_EMU_ERR_ALIAS: return "output overlaps an input";
        case SGEMM_EMU_ERR_UNSUPPORTED: return "unsupported size or shape";
        case SGEMM_EMU_ERR_HIP: return "HIP runtime error";
        case SGEMM_EMU_ERR_POLICY: return "invalid or unavailable policy";
        default: return "unknown status code";
    }
}

int sgemm_emu_last_hip_error(void) { return g_last_hip_error; }

}  // extern "C"
