/*
 * Oracle for single-precision-emulating GEMM on fp16 matrix units.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no header, helper or table with the HIP
 * path.
 *
 * Everything here is deliberately plain: one output element at a time, the
 * sum over k in ascending order, no blocking and no reordering.  OpenMP only
 * distributes independent output rows over threads; it never changes the
 * arithmetic of any element.
 *
 * Contents and the passage of the paper each follows:
 *   - oracle_f32_to_f16 / oracle_f16_to_f32: the conversions toFP16 and
 *     toFP32 used by the split (Sec. 4.4, eqs. corr-1..corr-4), written out
 *     from the IEEE-754 binary16 definition with round-to-nearest-even.
 *   - oracle_split: A_F16 = toFP16(A), dA_F16 = toFP16((A - toFP32(A_F16)) * 2^11)
 *     (Sec. 4.4, eqs. corr-1 and corr-2; the same rule for B, corr-3/corr-4).
 *   - oracle_gemm: for C = A*B (Sec. 2.2) the plain FP64 product of the FP32
 *     inputs, the normaliser sum_k |a||b|, the plain FP32 product as a
 *     sequential fmaf chain (the FP32 SIMT computation the method is
 *     compared with, Sec. 4.4 and 4.4.2), and the method-exact model
 *     A_F16 B_F16 + (dA_F16 B_F16 + A_F16 dB_F16) / 2^11 summed in FP64
 *     (Sec. 4.4, eq. corr-5).
 *   - oracle_gemm_acc: the accumulate form D = A*B + C0 of a fragment API
 *     (Sec. 2.3.1, Sec. 4.4), the same quantities with C0 as every sum's start.
 *   - oracle_scan: inclusive prefix sums of each row, the product a^T U with
 *     the upper-triangular all-ones U of Sec. 4.1 (eq. scan-mat, rule
 *     u-rule), written as running sums.
 *   - oracle_householder: H = I - 2 u u^T built explicitly and applied to
 *     B (Sec. 4.2.1, eq. householder, read as an outer product).
 *   - oracle_givens: the rotation G(i, j, theta) of Sec. 4.3.1 (identity
 *     except G_ii = G_jj = c, G_ij = -s, G_ji = s) built explicitly and
 *     applied to B, with c and s given as FP32 values.
 *
 * Compile with -ffp-contract=off so that only the explicit fmaf/fma calls
 * fuse.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads an OpenMP region of the oracle uses (1 without OpenMP). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---------------------------------------------------------------------- */
/* binary16 conversions from the IEEE-754 definition                       */
/* ---------------------------------------------------------------------- */

/* Round the FP32 value x to the nearest binary16 value, ties to even.
 * binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Normal values have 11 significant bits; below 2^-14 the grid is fixed at
 * 2^-24 (gradual underflow).  A value whose rounded magnitude would exceed
 * the largest finite binary16 (65504) becomes infinity. */
uint16_t oracle_f32_to_f16(float x)
{
    uint32_t b;
    memcpy(&b, &x, 4);
    uint16_t sign = (uint16_t)((b >> 16) & 0x8000u);
    uint32_t e = (b >> 23) & 0xffu;
    uint32_t f = b & 0x7fffffu;

    if (e == 0xffu) /* infinity or NaN */
        return (uint16_t)(sign | 0x7c00u | (f ? 0x200u : 0u));

    /* |x| = M * 2^E exactly, M an integer. */
    uint64_t M;
    int E;
    int log2x; /* floor(log2 |x|), only meaningful for M != 0 */
    if (e == 0) {
        if (f == 0)
            return sign; /* signed zero */
        M = f;
        E = -149;
        log2x = -127; /* any FP32 subnormal is far below 2^-14 */
    } else {
        M = 0x800000u | f;
        E = (int)e - 150;
        log2x = (int)e - 127;
    }

    /* Spacing of the binary16 grid around |x|: 2^S. */
    int S = (log2x >= -14) ? log2x - 10 : -24;
    int shift = S - E; /* >= 0 for every finite FP32 input */

    uint64_t q;
    if (shift <= 0) {
        q = M << (-shift);
    } else if (shift > 40) {
        q = 0; /* far below half of the smallest grid step */
    } else {
        uint64_t rem = M & ((1ull << shift) - 1);
        uint64_t half = 1ull << (shift - 1);
        q = M >> shift;
        if (rem > half || (rem == half && (q & 1u)))
            q += 1;
    }

    /* value = q * 2^S; re-encode. */
    if (q == 0)
        return sign;
    if (S == -24 && q < 1024)
        return (uint16_t)(sign | q); /* subnormal */
    if (q == 2048) { /* rounding carried into the next binade */
        q = 1024;
        S += 1;
    }
    int biased = S + 25; /* exponent of q*2^S with q in [1024,2048) */
    if (biased >= 31)
        return (uint16_t)(sign | 0x7c00u); /* overflow */
    return (uint16_t)(sign | ((uint32_t)biased << 10) | (uint32_t)(q - 1024));
}

/* Exact binary16 -> FP32 (every binary16 value is representable). */
float oracle_f16_to_f32(uint16_t h)
{
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    uint32_t e = (h >> 10) & 0x1fu;
    uint32_t f = h & 0x3ffu;
    float mag;
    if (e == 0x1fu) {
        uint32_t b = sign | 0x7f800000u | (f << 13);
        float r;
        memcpy(&r, &b, 4);
        return r;
    }
    if (e == 0)
        mag = ldexpf((float)f, -24);
    else
        mag = ldexpf((float)(1024u + f), (int)e - 25);
    return sign ? -mag : mag;
}

/* The split of Sec. 4.4, eqs. corr-1/corr-2:
 *   hi = toFP16(x)
 *   lo = toFP16((x - toFP32(hi)) * 2^11)
 * For |x| <= 65504 the subtraction and the scaling are exact in FP32, so the
 * only roundings are the two toFP16 conversions. */
void oracle_split(int64_t n, const float *x, uint16_t *hi, uint16_t *lo)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint16_t h = oracle_f32_to_f16(x[i]);
        float r = (x[i] - oracle_f16_to_f32(h)) * 2048.0f;
        hi[i] = h;
        lo[i] = oracle_f32_to_f16(r);
    }
}

/* ---------------------------------------------------------------------- */
/* GEMM: C = A * B per batch item, one output element at a time            */
/* ---------------------------------------------------------------------- */

/* Row-major operands with leading dimensions, batch strides in elements.
 * Any output pointer may be NULL, in which case it is not computed.
 *   C64[b,i,j] = sum_k (double)A[b,i,k] * (double)B[b,k,j]   (k ascending)
 *   N64[b,i,j] = sum_k |A[b,i,k]| * |B[b,k,j]|              (FP64)
 *   C32[b,i,j]: c = 0; for k ascending: c = fmaf(A, B, c)
 *   CM [b,i,j] = sum_k [ hiA hiB + (loA hiB + hiA loB) * 2^-11 ]  (FP64)
 * Output strides: ldc per row, sc per batch item.  */
void oracle_gemm(int batch, int m, int n, int k,
                 const float *A, int64_t lda, int64_t sa,
                 const float *B, int64_t ldb, int64_t sb,
                 double *C64, double *N64, float *C32, double *CM,
                 int64_t ldc, int64_t sc)
{
    int64_t rows = (int64_t)batch * m;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r) {
        int64_t b = r / m, i = r % m;
        const float *a = A + b * sa + i * lda;
        const float *bb = B + b * sb;
        for (int j = 0; j < n; ++j) {
            double s64 = 0.0, nrm = 0.0, sm = 0.0;
            float s32 = 0.0f;
            for (int kk = 0; kk < k; ++kk) {
                float av = a[kk];
                float bv = bb[(int64_t)kk * ldb + j];
                if (C64)
                    s64 += (double)av * (double)bv;
                if (N64)
                    nrm += fabs((double)av) * fabs((double)bv);
                if (C32)
                    s32 = fmaf(av, bv, s32);
                if (CM) {
                    uint16_t ha = oracle_f32_to_f16(av);
                    uint16_t hb = oracle_f32_to_f16(bv);
                    double ah = oracle_f16_to_f32(ha);
                    double bh = oracle_f16_to_f32(hb);
                    double al = oracle_f16_to_f32(oracle_f32_to_f16(
                        (av - (float)ah) * 2048.0f));
                    double bl = oracle_f16_to_f32(oracle_f32_to_f16(
                        (bv - (float)bh) * 2048.0f));
                    sm += ah * bh + (al * bh + ah * bl) / 2048.0;
                }
            }
            int64_t o = b * sc + i * ldc + j;
            if (C64)
                C64[o] = s64;
            if (N64)
                N64[o] = nrm;
            if (C32)
                C32[o] = s32;
            if (CM)
                CM[o] = sm;
        }
    }
}

/* Accumulate form D = A * B + C0 (the matrix-multiply-accumulate of a
 * fragment API, Sec. 2.3.1 and Sec. 4.4): the same four quantities as
 * oracle_gemm with C0 as the starting value of every sum,
 *   C64 = C0 + sum_k A B          (FP64, C0 first, then k ascending)
 *   N64 = |C0| + sum_k |A| |B|
 *   C32: c = C0; for k ascending: c = fmaf(A, B, c)
 *   CM  = C0 + sum_k [ hiA hiB + (loA hiB + hiA loB) * 2^-11 ]  (FP64)
 * C0 has row stride ldc0 and item stride sc0; outputs ldd and sd. */
void oracle_gemm_acc(int batch, int m, int n, int k,
                     const float *A, int64_t lda, int64_t sa,
                     const float *B, int64_t ldb, int64_t sb,
                     const float *C0, int64_t ldc0, int64_t sc0,
                     double *C64, double *N64, float *C32, double *CM,
                     int64_t ldd, int64_t sd)
{
    int64_t rows = (int64_t)batch * m;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r) {
        int64_t b = r / m, i = r % m;
        const float *a = A + b * sa + i * lda;
        const float *bb = B + b * sb;
        const float *c0 = C0 + b * sc0 + i * ldc0;
        for (int j = 0; j < n; ++j) {
            float cv = c0[j];
            double s64 = cv, nrm = fabs((double)cv), sm = cv;
            float s32 = cv;
            for (int kk = 0; kk < k; ++kk) {
                float av = a[kk];
                float bv = bb[(int64_t)kk * ldb + j];
                s64 += (double)av * (double)bv;
                nrm += fabs((double)av) * fabs((double)bv);
                s32 = fmaf(av, bv, s32);
                if (CM) {
                    uint16_t ha = oracle_f32_to_f16(av);
                    uint16_t hb = oracle_f32_to_f16(bv);
                    double ah = oracle_f16_to_f32(ha);
                    double bh = oracle_f16_to_f32(hb);
                    double al = oracle_f16_to_f32(oracle_f32_to_f16(
                        (av - (float)ah) * 2048.0f));
                    double bl = oracle_f16_to_f32(oracle_f32_to_f16(
                        (bv - (float)bh) * 2048.0f));
                    sm += ah * bh + (al * bh + ah * bl) / 2048.0;
                }
            }
            int64_t o = b * sd + i * ldd + j;
            if (C64)
                C64[o] = s64;
            if (N64)
                N64[o] = nrm;
            if (C32)
                C32[o] = s32;
            if (CM)
                CM[o] = sm;
        }
    }
}

/* Sampled form for large problems: output s is the dot product of
 * arow[s*k .. s*k+k) and bcol[s*k .. s*k+k), with the same four quantities
 * as oracle_gemm. */
void oracle_dots(int64_t nsamp, int k, const float *arow, const float *bcol,
                 double *C64, double *N64, float *C32, double *CM)
{
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t s = 0; s < nsamp; ++s) {
        oracle_gemm(1, 1, 1, k, arow + s * k, k, 0, bcol + s * k, 1, 0,
                    C64 ? C64 + s : 0, N64 ? N64 + s : 0,
                    C32 ? C32 + s : 0, CM ? CM + s : 0, 1, 0);
    }
}

/* ---------------------------------------------------------------------- */
/* Householder: C = (I - 2 u u^T) B, H formed explicitly (Sec. 4.2.1)      */
/* ---------------------------------------------------------------------- */

/* H in FP32 with one rounding per entry: fmaf(-2 u_i, u_j, delta_ij).
 * (-2 u_i is exact.)  H is n x n row-major. */
void oracle_householder_h32(int n, const float *u, float *H)
{
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j)
            H[(int64_t)i * n + j] = fmaf(-2.0f * u[i], u[j], i == j ? 1.0f : 0.0f);
}

/* H in FP64: delta_ij - 2 u_i u_j (the product is exact in FP64). */
void oracle_householder_h64(int n, const float *u, double *H)
{
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j)
            H[(int64_t)i * n + j] = (i == j ? 1.0 : 0.0) - 2.0 * (double)u[i] * (double)u[j];
}

/* Batched application.  Per item b: u_b (n), B_b (n x ncols, ldb), outputs
 * n x ncols with row stride ldc and item stride sc:
 *   C64 = H64 B, N64 = |H64| |B|, C32 = fmaf chain of H32 B,
 *   CM  = method-exact model of the emulated product H32 * B.
 * Only items listed in `items` (nitems of them) are computed; output slot t
 * receives item items[t]. */
void oracle_householder(int n, int ncols, int nitems, const int64_t *items,
                        const float *u, int64_t su,
                        const float *B, int64_t ldb, int64_t sb,
                        double *C64, double *N64, float *C32, double *CM,
                        int64_t ldc, int64_t sc)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < nitems; ++t) {
        int64_t b = items[t];
        const float *ub = u + b * su;
        const float *Bb = B + b * sb;
        for (int i = 0; i < n; ++i) {
            for (int j = 0; j < ncols; ++j) {
                double s64 = 0.0, nrm = 0.0, sm = 0.0;
                float s32 = 0.0f;
                for (int kk = 0; kk < n; ++kk) {
                    double h64 = (i == kk ? 1.0 : 0.0) - 2.0 * (double)ub[i] * (double)ub[kk];
                    float h32 = fmaf(-2.0f * ub[i], ub[kk], i == kk ? 1.0f : 0.0f);
                    float bv = Bb[(int64_t)kk * ldb + j];
                    s64 += h64 * (double)bv;
                    nrm += fabs(h64) * fabs((double)bv);
                    s32 = fmaf(h32, bv, s32);
                    if (CM) {
                        uint16_t ha = oracle_f32_to_f16(h32);
                        uint16_t hb = oracle_f32_to_f16(bv);
                        double ah = oracle_f16_to_f32(ha);
                        double bh = oracle_f16_to_f32(hb);
                        double al = oracle_f16_to_f32(oracle_f32_to_f16(
                            (h32 - (float)ah) * 2048.0f));
                        double bl = oracle_f16_to_f32(oracle_f32_to_f16(
                            (bv - (float)bh) * 2048.0f));
                        sm += ah * bh + (al * bh + ah * bl) / 2048.0;
                    }
                }
                int64_t o = (int64_t)t * sc + (int64_t)i * ldc + j;
                if (C64)
                    C64[o] = s64;
                if (N64)
                    N64[o] = nrm;
                if (C32)
                    C32[o] = s32;
                if (CM)
                    CM[o] = sm;
            }
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Givens rotation: C = G(i, j, theta) B, G formed explicitly (Sec. 4.3.1) */
/* ---------------------------------------------------------------------- */

/* Entry (r, q) of the n x n rotation in the (i, j) plane: the identity
 * except G_ii = G_jj = c, G_ij = -s, G_ji = s.  Every entry is one of the
 * FP32 values 0, 1, c, s, -s, so the FP32 and FP64 matrices are equal. */
static float givens_entry(int r, int q, int i, int j, float c, float s)
{
    if ((r == i && q == i) || (r == j && q == j))
        return c;
    if (r == i && q == j)
        return -s;
    if (r == j && q == i)
        return s;
    return r == q ? 1.0f : 0.0f;
}

void oracle_givens_matrix(int n, int i, int j, float c, float s, float *G)
{
    for (int r = 0; r < n; ++r)
        for (int q = 0; q < n; ++q)
            G[(int64_t)r * n + q] = givens_entry(r, q, i, j, c, s);
}

/* Batched application.  Per item b: c_b = c[b * scs], s_b = s[b * scs],
 * B_b (n x ncols, ldb, item stride sb); outputs n x ncols with row stride
 * ldc and item stride sc:
 *   C64 = G B, N64 = |G| |B|, C32 = fmaf chain of G B (k ascending),
 *   CM  = method-exact model of the emulated product G * B.
 * Only items listed in `items` are computed; output slot t receives item
 * items[t]. */
void oracle_givens(int n, int gi, int gj, int ncols, int nitems, const int64_t *items,
                   const float *c, const float *s, int64_t scs,
                   const float *B, int64_t ldb, int64_t sb,
                   double *C64, double *N64, float *C32, double *CM,
                   int64_t ldc, int64_t sc)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int t = 0; t < nitems; ++t) {
        int64_t b = items[t];
        float cb = c[b * scs], sbv = s[b * scs];
        const float *Bb = B + b * sb;
        for (int i = 0; i < n; ++i) {
            for (int j = 0; j < ncols; ++j) {
                double s64 = 0.0, nrm = 0.0, sm = 0.0;
                float s32 = 0.0f;
                for (int kk = 0; kk < n; ++kk) {
                    float g = givens_entry(i, kk, gi, gj, cb, sbv);
                    float bv = Bb[(int64_t)kk * ldb + j];
                    s64 += (double)g * (double)bv;
                    nrm += fabs((double)g) * fabs((double)bv);
                    s32 = fmaf(g, bv, s32);
                    if (CM) {
                        uint16_t ha = oracle_f32_to_f16(g);
                        uint16_t hb = oracle_f32_to_f16(bv);
                        double ah = oracle_f16_to_f32(ha);
                        double bh = oracle_f16_to_f32(hb);
                        double al = oracle_f16_to_f32(oracle_f32_to_f16(
                            (g - (float)ah) * 2048.0f));
                        double bl = oracle_f16_to_f32(oracle_f32_to_f16(
                            (bv - (float)bh) * 2048.0f));
                        sm += ah * bh + (al * bh + ah * bl) / 2048.0;
                    }
                }
                int64_t o = (int64_t)t * sc + (int64_t)i * ldc + j;
                if (C64)
                    C64[o] = s64;
                if (N64)
                    N64[o] = nrm;
                if (C32)
                    C32[o] = s32;
                if (CM)
                    CM[o] = sm;
            }
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Scan: y_j = sum_{i <= j} x_i per row (Sec. 4.1, eq. scan-mat)           */
/* ---------------------------------------------------------------------- */

/* Row r of X (len values, row stride ldx) gives row r of each output (row
 * stride ldy):
 *   Y64 = running FP64 sum, N64 = running sum of |x|, Y32 = running FP32
 *   sum (one rounded addition per element, left to right), YM = running
 *   FP64 sum of the split values hi + lo 2^-11 (the method model of x . U:
 *   every entry of U is 1 or 0, whose lo parts are 0). */
void oracle_scan(int64_t rows, int len, const float *X, int64_t ldx,
                 double *Y64, double *N64, float *Y32, double *YM, int64_t ldy)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t r = 0; r < rows; ++r) {
        const float *x = X + r * ldx;
        double s64 = 0.0, nrm = 0.0, sm = 0.0;
        float s32 = 0.0f;
        for (int j = 0; j < len; ++j) {
            float v = x[j];
            s64 += (double)v;
            nrm += fabs((double)v);
            s32 = s32 + v;
            uint16_t h = oracle_f32_to_f16(v);
            double vh = oracle_f16_to_f32(h);
            double vl = oracle_f16_to_f32(oracle_f32_to_f16((v - (float)vh) * 2048.0f));
            sm += vh + vl / 2048.0;
            int64_t o = r * ldy + j;
            if (Y64)
                Y64[o] = s64;
            if (N64)
                N64[o] = nrm;
            if (Y32)
                Y32[o] = s32;
            if (YM)
                YM[o] = sm;
        }
    }
}
