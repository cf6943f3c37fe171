/*
 * sgemm_emu.h -- C ABI of the single-precision-emulating GEMM library for
 * AMD Instinct MI355X (gfx950).
 *
 * Method (Ootomo & Yokota, "Reducing shared memory footprint to leverage high
 * throughput on Tensor Cores and its flexible API extension library",
 * Sec. 4.4): every FP32 operand element x is split into two fp16 values
 *     hi = toFP16(x),   lo = toFP16((x - toFP32(hi)) * 2^11)
 * (round to nearest even), and the product is formed from three fp16 matrix
 * products with FP32 accumulation,
 *     C = hiA.hiB + (loA.hiB + hiA.loB) / 2^11      (eq. corr-5),
 * with the two correction products accumulated apart from the main one.  The
 * split is done in registers, so no fp16 copy of A or B is ever written to
 * device memory or kept in LDS in addition to the FP32 data.
 *
 * Conventions shared by all entry points:
 *   - Matrices are row-major FP32; "ld" is the distance in elements between
 *     the starts of consecutive rows.
 *   - Matrix pointers are DEVICE pointers owned by the caller.  The library
 *     allocates no device memory and keeps no pointer after returning.
 *   - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *     without waiting; buffers must stay valid until the stream reaches it.
 *   - Inputs are expected to satisfy |x| <= 65504 (the fp16 range of hi);
 *     outside that range, or for NaN/Inf, the result is unspecified.
 *   - Every argument is validated before anything is enqueued.  On an error
 *     nothing is launched and a negative code is returned; the functions
 *     never throw and never abort.
 *   - Calls may be captured in a HIP graph (stream capture): a call only
 *     launches kernels on the given stream; it allocates nothing, records no
 *     memset and does not synchronize.
 *   - All functions are thread-safe: the library's only mutable global state
 *     is the last HIP error code, kept per thread, and the number of
 *     workgroups of a kernel that fit on a device, computed on first use and
 *     kept in atomics.
 */
#ifndef SGEMM_EMU_H
#define SGEMM_EMU_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- Status codes ------------------------------------------------------ */
#define SGEMM_EMU_OK 0
#define SGEMM_EMU_ERR_DIM (-1)         /* negative m, n, k, batch or ncols    */
#define SGEMM_EMU_ERR_LD (-2)          /* leading dimension too small          */
#define SGEMM_EMU_ERR_NULL (-3)        /* NULL pointer with nonzero work       */
#define SGEMM_EMU_ERR_STRIDE (-4)      /* negative stride, C items overlap, or
                                          an operand's span (strides and ld)
                                          runs past the end of the address
                                          space                               */
#define SGEMM_EMU_ERR_ALIAS (-5)       /* C overlaps A or B (or u)             */
#define SGEMM_EMU_ERR_UNSUPPORTED (-6) /* size outside what an entry supports  */
#define SGEMM_EMU_ERR_HIP (-7)         /* the HIP runtime reported an error    */
#define SGEMM_EMU_ERR_POLICY (-8)      /* unknown policy value                 */

/* Element strides between consecutive batch items of A, B and C.  A zero
 * stride for A or B reuses (broadcasts) one matrix for every item; C's stride
 * must keep items apart (stride.c >= (m-1)*ldc + n when batch > 1). */
typedef struct {
    int64_t a, b, c;
} sgemm_emu_stride_t;

/*
 * Batched emulated SGEMM (Sec. 4.4; batched form of Sec. 4.4.2):
 *   for t in [0, batch):  C_t := A_t . B_t
 * with A_t = A + t*stride.a (m x k, row-major, lda >= max(1, k)),
 *      B_t = B + t*stride.b (k x n, row-major, ldb >= max(1, n)),
 *      C_t = C + t*stride.c (m x n, row-major, ldc >= max(1, n)).
 * C is overwritten (no alpha/beta).  m = 0, n = 0 or batch = 0 is a no-op;
 * k = 0 stores zeros.  Pointers need no particular alignment; 16-byte aligned
 * bases with ld and strides multiples of 4 take the vector-load path.
 * Errors: SGEMM_EMU_ERR_DIM, _LD, _NULL, _STRIDE, _ALIAS, _HIP.
 */
int sgemm_emu_batched(int m, int n, int k,
                      const float* A, int lda,
                      const float* B, int ldb,
                      float* C, int ldc,
                      int batch, sgemm_emu_stride_t stride,
                      hipStream_t stream);

/* Policy of the emulated product, after the paper's policy-based design
 * (Sec. 4.4): the instruction shape and tiling, whether error correction is
 * applied, and where the split happens.
 *
 * flow:
 *   SGEMM_EMU_FLOW_AUTO   library choice: SPLIT on full tiles when a
 *                         full-tile kernel applies (see
 *                         sgemm_emu_resolve_policy): 128x256 when k >= 1024
 *                         and batch * m * n >= 2048 * 2048, else 256x128,
 *                         else 128x128.  Otherwise, for m and n above 1024
 *                         with 16-byte aligned A and B rows, k >= 32, at
 *                         least 2^35 multiply-adds (batch m n k) and the
 *                         REG flow's conditions met, the first of 128x256
 *                         (when it is preferred as above) and 256x128 whose
 *                         whole tiles cover at least 95% of C and number at
 *                         least 256 (batch included):
 *                         that interior (and k rounded down to a multiple
 *                         of 32) runs on the full-tile kernel, the
 *                         remaining k is added to it in place, and the edge
 *                         strips run on the REG flow with 64 x 64 tiles, one
 *                         launch after another on the stream.  Otherwise
 *                         REG whenever its conditions hold: tile 64x64 for
 *                         m, n <= 64, else 128x128, else (B rows without
 *                         vector loads, below 2^35 multiply-adds) 64x64.
 *                         Otherwise SPLIT on the general kernel.
 *   SGEMM_EMU_FLOW_SPLIT  FP32 tiles are split in registers between the
 *                         global load and the LDS store; LDS holds hi and lo
 *                         (the same 4 bytes per element as FP32) and the
 *                         waves read ready operand vectors.
 *   SGEMM_EMU_FLOW_DIRECT FP32 tiles in LDS; every wave reads FP32 and
 *                         splits its own fragments in registers (the data
 *                         flow of the paper's extension library, Fig. 6
 *                         bottom).
 *   SGEMM_EMU_FLOW_STAGED FP32 tiles in LDS; every wave converts its part to
 *                         hi/lo, writes them back to LDS and reloads them as
 *                         fragments (the flow forced by a load-only fragment
 *                         API, Fig. 6 top).  Measurement only: three LDS
 *                         passes per element instead of one.
 *   SGEMM_EMU_FLOW_REG    no LDS: every wave loads its operand elements from
 *                         global memory straight into registers, splits them
 *                         there and runs its MFMAs (fragments built without
 *                         shared memory, Sec. 4.2); no barriers, so all waves
 *                         stream independently.  For HBM-bound batches of
 *                         small products.  Needs 16-byte aligned A rows
 *                         (A 16-byte aligned, lda and stride.a multiples of
 *                         4, lda < 2^23, ldb < 2^25) and, for tile 128x128,
 *                         B vectors of 4 (B 16-byte aligned, ldb, stride.b
 *                         and n multiples of 4) or else of 2 (8-byte
 *                         aligned, even); tiles 64x64 and 128x128 only.
 *                         Otherwise SGEMM_EMU_ERR_POLICY.
 * ec:   1 = error correction (3 products), 0 = hi.hi only (the comparison
 *       without correction: accuracy and cost).
 * tile: 0 = automatic, or one of SGEMM_EMU_TILE_*.  With flow AUTO the
 *       tile follows the flow the library picks.  With a named flow, AUTO
 *       picks a tile that flow has: REG 64x64 when m, n <= 64, else 128x128
 *       where its B vectors allow it, else 64x64; DIRECT and STAGED 64x64
 *       when m, n <= 64, else 128x128; SPLIT by shape (64x64 when m, n <= 64,
 *       256x128 for many 256-row tiles, else 128x128).
 */
#define SGEMM_EMU_FLOW_AUTO 0
#define SGEMM_EMU_FLOW_SPLIT 1
#define SGEMM_EMU_FLOW_DIRECT 2
#define SGEMM_EMU_FLOW_STAGED 3
#define SGEMM_EMU_FLOW_REG 4

#define SGEMM_EMU_TILE_AUTO 0
#define SGEMM_EMU_TILE_64x64 1   /* 4 waves of 32x32 (LDS flows: k-chunk 32) */
#define SGEMM_EMU_TILE_128x128 2 /* 4 waves of 64x64 (LDS flows: k-chunk 32) */
#define SGEMM_EMU_TILE_256x128 3 /* 8 waves of 64x64, k-chunk 32; LDS flows  */
#define SGEMM_EMU_TILE_128x256 4 /* 8 waves of 64x64, k-chunk 32; split flow,
                                    full tiles only                          */

typedef struct {
    int flow;
    int ec;
    int tile;
} sgemm_emu_policy_t;

/* sgemm_emu_batched with an explicit policy (NULL = automatic, with error
 * correction).  Extra error: SGEMM_EMU_ERR_POLICY. */
int sgemm_emu_batched_ex(int m, int n, int k,
                         const float* A, int lda,
                         const float* B, int ldb,
                         float* C, int ldc,
                         int batch, sgemm_emu_stride_t stride,
                         const sgemm_emu_policy_t* policy,
                         hipStream_t stream);

/* The policy sgemm_emu_batched_ex would run for these arguments, with AUTO
 * flow and tile replaced by the library's choice (ec is copied), and, if
 * `kernel` is not NULL, the name of the kernel it would launch (a static
 * string; "" for an empty problem).  A host-only query: no HIP call,
 * nothing is enqueued.  Same validation and errors as sgemm_emu_batched_ex,
 * plus SGEMM_EMU_ERR_NULL for a NULL out; for an empty problem (nothing
 * would run) out receives the policy unresolved.
 * With error correction, the split flow with tile 128x128, 256x128 or
 * 128x256, and the direct and staged flows with tile 128x128, run a
 * pipelined full-tile kernel when m and n are multiples of the tile, k is a
 * positive multiple of 32, A and B rows are 16-byte aligned and a chunk's
 * byte offsets stay below 2^31 ((rows of the tile x lda + 32) x 4 < 2^31
 * and (32 ldb + columns of the tile) x 4 < 2^31: lda below about 2^29 /
 * tile rows, ldb below about 2^24); otherwise the general LDS kernel (128x256
 * has none: SGEMM_EMU_ERR_POLICY).  Without error correction (ec = 0, for
 * measuring what the correction costs), the split flow with tile 128x128
 * or 128x256 runs the same full-tile kernel under the same conditions, and
 * AUTO picks among those two tiles; the decomposition of large ragged
 * products is made only with error correction. */
int sgemm_emu_resolve_policy(int m, int n, int k,
                             const float* A, int lda,
                             const float* B, int ldb,
                             float* C, int ldc,
                             int batch, sgemm_emu_stride_t stride,
                             const sgemm_emu_policy_t* policy,
                             sgemm_emu_policy_t* out,
                             const char** kernel);

/*
 * Work distribution of the GEMM kernels, computed on the host by the same
 * functions the kernels run (no GPU is touched): which task each workgroup
 * takes and which tile of an item each task is.  These decide that every
 * output tile is computed exactly once, so they are exposed to be checked.
 *
 * sgemm_emu_xcd_order: task_of_workgroup[b] for b in [0, grid) is the task
 *   workgroup b of a grid of `grid` workgroups takes first (the full-tile
 *   and register-flow kernels take only that task; the persistent kernels
 *   take it and every grid-th task after it).  Workgroups are dispatched
 *   round-robin over the 8 XCDs; the numbering gives each XCD one contiguous
 *   range of task ids.  grid >= 1; task_of_workgroup holds grid ints
 *   (caller-owned host memory).
 * sgemm_emu_tile_order: for task t in [0, tiles_m * tiles_n) of one batch
 *   item, tile_row[t] and tile_col[t] are the tile's row and column in the
 *   tiles_m x tiles_n grid of output tiles (groups of 8 tile rows, column by
 *   column within a group).  tiles_m, tiles_n >= 1 and their product below
 *   2^31; each array holds tiles_m * tiles_n ints (caller-owned host
 *   memory).
 * sgemm_emu_block_order: the same for a launch of one item on the 128 x 256
 *   full-tile kernel when tiles_m and tiles_n are multiples of 16 (e.g. the
 *   8192 x 8192 product, 64 x 32 tiles): the 256 tasks the device runs at
 *   once form one 16 x 16 block of tiles (each XCD an 8 x 4 part), blocks
 *   taken down the columns, so that the XCDs share A rows and B columns in
 *   the last-level cache.  SGEMM_EMU_ERR_DIM for grids that are not
 *   multiples of 16 (those keep the grouped order).
 * All three return SGEMM_EMU_OK, SGEMM_EMU_ERR_DIM for sizes out of range, or
 * SGEMM_EMU_ERR_NULL for a NULL array.
 */
int sgemm_emu_xcd_order(int grid, int* task_of_workgroup);
int sgemm_emu_tile_order(int tiles_m, int tiles_n, int* tile_row, int* tile_col);
int sgemm_emu_block_order(int tiles_m, int tiles_n, int* tile_row, int* tile_col);

/*
 * Batched multiply-accumulate in emulated FP32 with transposable operands:
 *   for t in [0, batch):  D_t := op(A_t) . op(B_t) + C_t
 * the matrix-multiply-accumulate of a fragment API (Sec. 2.3.1) computed by
 * the method of Sec. 4.4 through the library's fragment interface
 * (mfmae/wmma_tcec.hpp; the kernel is written with its load_matrix_sync,
 * mma_sync and store_matrix_sync).  op(A) is m x k, op(B) is k x n.
 *   op_a: SGEMM_EMU_OP_N  A_t is stored m x k row-major, lda >= max(1, k)
 *         SGEMM_EMU_OP_T  A_t is stored as its transpose, k x m row-major
 *                         (A column-major), lda >= max(1, m)
 *   op_b: SGEMM_EMU_OP_N  B_t stored k x n row-major, ldb >= max(1, n)
 *         SGEMM_EMU_OP_T  B_t stored n x k row-major, ldb >= max(1, k)
 *   layout_cd: SGEMM_EMU_ROW_MAJOR  C_t and D_t are m x n row-major,
 *                                   ldc, ldd >= max(1, n)
 *              SGEMM_EMU_COL_MAJOR  stored as n x m row-major,
 *                                   ldc, ldd >= max(1, m)
 * A_t = A + t*stride.a, B_t = B + t*stride.b, C_t = C + t*stride.c,
 * D_t = D + t*stride.d.  C may be NULL (then D := op(A).op(B)); C == D with
 * ldc == ldd and stride.c == stride.d accumulates in place; any other
 * overlap of D with A, B or C is an error.  k = 0 gives D := C (or 0).
 * shape selects the instruction (MFMAE_SHAPE_16x16x32 or
 * MFMAE_SHAPE_32x32x16), ec the policy: 1 = error correction (3 products),
 * 0 = hi.hi only.  16-byte accesses are used along each operand's contiguous
 * direction when its base is 16-byte aligned and its ld and stride are
 * multiples of 4; any alignment is accepted.  Supported: m, n, k < 2^30
 * (else SGEMM_EMU_ERR_UNSUPPORTED).
 * Errors: SGEMM_EMU_ERR_DIM, _LD, _NULL (A or B NULL with k > 0, D NULL),
 * _STRIDE, _ALIAS, _POLICY (op, layout, shape or ec out of range),
 * _UNSUPPORTED, _HIP.
 */
#define SGEMM_EMU_OP_N 0
#define SGEMM_EMU_OP_T 1
#define SGEMM_EMU_ROW_MAJOR 0
#define SGEMM_EMU_COL_MAJOR 1

typedef struct {
    int64_t a, b, c, d;
} sgemm_emu_stride4_t;

int sgemm_emu_batched_acc(int op_a, int op_b, int layout_cd,
                          int m, int n, int k,
                          const float* A, int lda,
                          const float* B, int ldb,
                          const float* C, int ldc,
                          float* D, int ldd,
                          int batch, sgemm_emu_stride4_t stride,
                          int shape, int ec, hipStream_t stream);

/*
 * Batched Householder application with the reflector built in registers
 * (Sec. 4.2.1, eq. householder, read as H = I - 2 u u^T):
 *   for t in [0, batch):  C_t := (I - 2 u_t u_t^T) . B_t
 * u_t = u + t*stride_u (n FP32 values), B_t = B + t*stride_b (n x ncols,
 * row-major, ldb >= max(1, ncols)), C_t = C + t*stride_c (n x ncols, ldc >=
 * max(1, ncols)).  Each entry of H is formed as fmaf(-2 u_i, u_j, delta_ij)
 * directly in the operand registers and then split as above; H is never
 * stored.  u is used as given (it is not normalised).
 * Supported: n == 64 and ldb < 2^27 (else SGEMM_EMU_ERR_UNSUPPORTED).
 * Errors: SGEMM_EMU_ERR_DIM, _LD, _NULL, _STRIDE, _ALIAS, _UNSUPPORTED, _HIP.
 */
int householder_emu_batched(int n, const float* u, int64_t stride_u,
                            const float* B, int ldb, int64_t stride_b, int ncols,
                            float* C, int ldc, int64_t stride_c,
                            int batch, hipStream_t stream);

/* householder_emu_batched with a choice of how the reflector's fragments are
 * built (the comparison of Sec. 4.2.1):
 *   SGEMM_EMU_HOUSEHOLDER_RULE  in registers by foreach_ij (as above);
 *   SGEMM_EMU_HOUSEHOLDER_LDS   baseline: every entry of H is formed once,
 *                               split and written to LDS (16 KiB per wave),
 *                               and the fragments are loaded from there.
 * Both form the same entries and give bit-identical results.  Extra error:
 * SGEMM_EMU_ERR_POLICY for an unknown mode. */
#define SGEMM_EMU_HOUSEHOLDER_RULE 0
#define SGEMM_EMU_HOUSEHOLDER_LDS 1

int householder_emu_batched_ex(int n, const float* u, int64_t stride_u,
                               const float* B, int ldb, int64_t stride_b, int ncols,
                               float* C, int ldc, int64_t stride_c,
                               int batch, int mode, hipStream_t stream);

/*
 * Batched Givens rotation with the rotation matrix built in registers
 * (Sec. 4.3.1):
 *   for t in [0, batch):  C_t := G(i, j, theta_t) . B_t
 * where G(i, j, theta) is the n x n identity except G_ii = G_jj = c,
 * G_ij = -s and G_ji = s, with c = cos theta_t and s = sin theta_t given as
 * c_t = c[t*stride_cs], s_t = s[t*stride_cs] (FP32, used as given: c^2 + s^2
 * need not be 1).  B_t = B + t*stride_b (n x ncols, row-major, ldb >=
 * max(1, ncols)), C_t = C + t*stride_c (n x ncols, ldc >= max(1, ncols)).
 * The plane (i, j) is the same for every item; 0 <= i, j < n, i != j.
 * The product is formed densely with the emulated FP32 method, as for
 * sgemm_emu_batched, with G's operand fragments built without memory
 * traffic.  mode selects how (Sec. 4.3.1 compares these):
 *   SGEMM_EMU_GIVENS_AUTO      EMBEDDED when (i, j) has a compiled
 *                              instance, else MAP.
 *   SGEMM_EMU_GIVENS_MAP       fragments zero-filled, then 1, c, s and -s
 *                              set through the element map with (i, j)
 *                              passed as kernel arguments.
 *   SGEMM_EMU_GIVENS_EMBEDDED  as MAP with (i, j) fixed at compile time;
 *                              compiled for n = 64 and (i, j) in
 *                              {(5,37), (37,5), (0,1), (31,32), (62,63)};
 *                              other planes give SGEMM_EMU_ERR_UNSUPPORTED.
 *   SGEMM_EMU_GIVENS_LDS       baseline: each wave writes G to LDS and
 *                              loads its fragments from there.
 * Supported: n == 64 and ldb < 2^27 (else SGEMM_EMU_ERR_UNSUPPORTED).
 * Errors: SGEMM_EMU_ERR_DIM (also i or j out of range or i == j), _LD,
 * _NULL, _STRIDE, _ALIAS (C overlaps B, c or s), _UNSUPPORTED, _POLICY
 * (unknown mode), _HIP.
 */
#define SGEMM_EMU_GIVENS_AUTO 0
#define SGEMM_EMU_GIVENS_MAP 1
#define SGEMM_EMU_GIVENS_EMBEDDED 2
#define SGEMM_EMU_GIVENS_LDS 3

int givens_emu_batched(int n, int i, int j,
                       const float* c, const float* s, int64_t stride_cs,
                       const float* B, int ldb, int64_t stride_b, int ncols,
                       float* C, int ldc, int64_t stride_c,
                       int batch, int mode, hipStream_t stream);

/*
 * Batched inclusive scan through a rule-built matrix (Sec. 4.1, eq.
 * scan-mat): for every row r in [0, rows),
 *   Y[r][j] := sum_{i <= j} X[r][i],   j in [0, len)
 * computed with the upper-triangular all-ones matrix U (u_ij = 1 for
 * i <= j), whose operand fragments are generated from that rule with
 * foreach_ij, in emulated FP32 (Sec. 4.4): each block of 1024 values is
 * taken as 32 segments of 32, scanned within segments by one product with
 * U's 32 x 32 block, and the segments and blocks are chained by FP32 running
 * totals.  X: rows x len, row stride ldx >= max(1, len); Y likewise with
 * ldy.  Y may be X itself (ldy == ldx) for an in-place scan; any other
 * overlap is an error.  Rows are independent; a wavefront scans 8 rows, so
 * parallelism comes from the number of rows.  Rows of a multiple of 1024
 * values with 16-byte aligned X and Y rows take 16-byte accesses.  Any
 * number of rows: more than 268,435,424 take several launches.
 * Errors: SGEMM_EMU_ERR_DIM, _LD (also when rows x ld runs past the end of
 * the address space), _NULL, _ALIAS, _HIP.
 */
int sgemm_emu_scan(int64_t rows, int len, const float* X, int64_t ldx,
                   float* Y, int64_t ldy, hipStream_t stream);

/*
 * The split of Sec. 4.4 (eqs. corr-1/corr-2) applied elementwise on the
 * device: hi[i], lo[i] receive the binary16 bit patterns of
 * toFP16(x[i]) and toFP16((x[i] - toFP32(hi)) * 2^11).  count >= 0; x, hi
 * and lo are device pointers of count elements and must not overlap.
 * form selects the device function that splits, so that each form the
 * kernels use can be checked bit for bit:
 *   SGEMM_EMU_SPLIT_SCALAR  one value at a time (rule-built entries, the
 *                           B operand of the Householder and Givens
 *                           kernels, single values at tile edges)
 *   SGEMM_EMU_SPLIT_PAIR    two values at a time, hi converted as a packed
 *                           pair (B staging of the full-tile kernel, the
 *                           general kernel's staging)
 *   SGEMM_EMU_SPLIT_EIGHT   eight consecutive values into one operand vector
 *                           (A staging of the full-tile kernel, the per-wave
 *                           split of the direct and staged flows, the
 *                           register-direct flow, the fragment loads, the
 *                           scan, the Householder baseline's entries)
 * Values past the last whole pair or group of eight are split one at a
 * time.  Errors: SGEMM_EMU_ERR_DIM (also when count elements run past the
 * end of the address space), _NULL, _ALIAS, SGEMM_EMU_ERR_POLICY (form
 * unknown), _HIP.
 */
#define SGEMM_EMU_SPLIT_SCALAR 0
#define SGEMM_EMU_SPLIT_PAIR 1
#define SGEMM_EMU_SPLIT_EIGHT 2
int sgemm_emu_split(int64_t count, const float* x, uint16_t* hi, uint16_t* lo, int form,
                    hipStream_t stream);

/* ---- Fragment maps (Sec. 2.3.2, 4.2, 4.3) ------------------------------
 * shape: MFMAE_SHAPE_16x16x32 (v_mfma_f32_16x16x32_f16) or
 *        MFMAE_SHAPE_32x32x16 (v_mfma_f32_32x32x16_f16)
 * use:   MFMAE_USE_A (M x K), MFMAE_USE_B (K x N), MFMAE_USE_ACC (M x N)
 * Host-only table queries: no HIP call is made. */
#define MFMAE_SHAPE_16x16x32 0
#define MFMAE_SHAPE_32x32x16 1
#define MFMAE_USE_A 0
#define MFMAE_USE_B 1
#define MFMAE_USE_ACC 2

/* Elements per lane for (shape, use), or SGEMM_EMU_ERR_UNSUPPORTED. */
int mfmae_num_elements(int shape, int use);

/* Matrix position (i, j) -> lane (0..63) and element index holding it
 * (the paper's `map`, Sec. 4.3).  Errors: _UNSUPPORTED, _DIM (out of range),
 * _NULL. */
int mfmae_map(int shape, int use, int i, int j, int* lane, int* elem);

/* For one lane, the matrix position of each of its elements (the index part
 * of the paper's `foreach_ij`, Sec. 4.2): i_out[e], j_out[e] for
 * e < mfmae_num_elements(shape, use).  Errors: _UNSUPPORTED, _DIM, _NULL. */
int mfmae_foreach(int shape, int use, int lane, int* i_out, int* j_out);

/* Run ONE fp16 MFMA of the given shape on one wavefront with operands given
 * lane by lane (the register-level counterpart of the paper's mapping probe,
 * Sec. 2.3.2): a[lane*8 + e], b[lane*8 + e] are binary16 bit patterns of
 * element e of that lane's A and B operand, the accumulator starts at zero,
 * and d[lane*n + e] receives element e of the lane's result (n = 4 for
 * 16x16x32, 16 for 32x32x16).  Device pointers.
 * Errors: _UNSUPPORTED, _NULL, _HIP. */
int mfmae_mma_probe(int shape, const uint16_t* a, const uint16_t* b, float* d,
                    hipStream_t stream);

/* ---- Measurement references -----------------------------------------------
 * The memory traffic of a batched product without its arithmetic: for
 * t < items, C_t := A_t + B_t elementwise over item_elems floats, one
 * workgroup of `threads` threads per item (256, 512 or 1024), 16-byte loads
 * of A and B and nontemporal 16-byte stores of C.  With the item sizes of a
 * batched workload (A, B, C of m k, k n, m n floats) it moves the same bytes
 * as the product in the same per-item pattern, so its rate is the HBM rate
 * that access pattern reaches on the device.  A, B, C are device pointers
 * to items * item_elems floats each, 16-byte aligned, C not overlapping A
 * or B; item_elems is a positive multiple of 4 below 2^31.
 * Errors: _DIM, _NULL, _UNSUPPORTED (threads, alignment or item_elems),
 * _ALIAS, _HIP. */
int sgemm_emu_stream_probe(int64_t items, int64_t item_elems, const float* A, const float* B,
                           float* C, int threads, hipStream_t stream);

/* The arithmetic of the full-tile kernel without its data movement (the
 * three products of Sec. 4.4 alone): on the m x n output, in 128 x 256 tiles
 * with the same grid, task order, waves and MFMA sequence as the full-tile
 * kernel, the operand fragments of the first k chunk (A[i][0..31],
 * B[0..31][j]) are split once and held in registers, and the k loop runs
 * the k / 32 chunks' products on them with no global loads, split or LDS
 * traffic.  C := (k / 32) * (the emulated product of that chunk), written
 * as the kernel writes C.  Its rate (2 m n k / time) is the rate the
 * matrix units reach for these products at the clock the device holds
 * under them.  m a multiple of 128, n of 256, k a positive multiple of 32;
 * lda >= 32, ldb >= n, ldc >= n; A, B, C device pointers (only the first 32
 * columns of A and the first 32 rows of B are read); C must not overlap
 * them.  m = 0 or n = 0: no-op.
 * Errors: _DIM, _UNSUPPORTED (sizes not multiples), _LD, _NULL, _ALIAS, _HIP. */
int sgemm_emu_mfma_probe(int m, int n, int k, const float* A, int lda, const float* B, int ldb,
                         float* C, int ldc, hipStream_t stream);

/* ---- Diagnostics ------------------------------------------------------- */
/* Static text for a status code. */
const char* sgemm_emu_strerror(int code);
/* The hipError_t behind the calling thread's last SGEMM_EMU_ERR_HIP (0 if
 * none). */
int sgemm_emu_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SGEMM_EMU_H */
