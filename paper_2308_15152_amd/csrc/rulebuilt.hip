// Batched products with a rule-built left operand, n = 64, in emulated FP32
// (Sec. 4.4).  The 64 x 64 left matrix is never read from memory: its MFMA
// A-operand fragments are built in registers from a rule.
//
//   Householder (Sec. 4.2.1, eq. householder; foreach_ij of Sec. 4.2):
//     C = (I - 2 u u^T) B.  For every A-operand element it holds, a lane
//     evaluates h_ij = fmaf(-2 u_i, u_j, delta_ij) and splits it into hi/lo.
//     Per 16-wide k step one foreach_ij over the A-operand map fills both
//     32-row blocks (the index computation is shared by the two fragments,
//     and -2 u_i of the lane's rows is computed once), which is what keeps
//     rule-built fragments cheaper than a trip through memory.  The baseline
//     forms every entry once into LDS and loads the fragments from there.
//   Givens (Sec. 4.3.1; map of Sec. 4.3):
//     C = G(i, j, theta) B with G the identity except G_ii = G_jj = c,
//     G_ij = -s, G_ji = s.  The fragments are filled with zeros and the
//     nonzero entries are set through map(): (row, col) -> (lane, element).
//     With (i, j) kernel arguments the lane and element of c and s are found
//     at run time (a compare and select per element the lane holds); with
//     (i, j) embedded at compile time every map() folds to a constant.  The
//     baseline writes G to LDS and loads the fragments from there.
//
// One wavefront handles one batch item and up to 64 columns of B.  B is
// read straight from global memory into the B-operand registers.  When rows
// allow 8-byte accesses the two 32-column blocks interleave their columns,
// so for a fixed k the 32 lanes of a half-wave read one 256-byte row segment
// with one 8-byte load each (and C is written the same way); otherwise lane
// l holds column l % 32 of each block (128-byte segments).  The kernels are
// bound by HBM traffic (B read once, C written once).
#include "internal.h"
#include "mfmae/frag.hpp"
#include "mfmae/tcec.hpp"
#include "sgemm_emu.h"

namespace sgemm_emu {

using mfmae::f32x16_t;
using mfmae::half8_t;
using mfmae::Shape32;
using mfmae::Use;

namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
using FragA = mfmae::fragment<Shape32, Use::A, _Float16>;

struct RuleParams {
    int ncols;
    // Householder: u_b = u + b su (64 values)
    const float* u;
    int64_t su;
    // Givens: c_b = c[b scs], s_b = s[b scs]; rotation plane (gi, gj)
    const float* c;
    const float* s;
    int64_t scs;
    int gi, gj;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int batch;      // items of this launch
    int64_t item0;  // first item of this launch
};

constexpr int kWaves = 4;  // waves (tasks) per workgroup

// ---------------------------------------------------------------------------
// Left-operand builders.  build(s, hh, hl) produces the hi and lo fragments
// of rows 32 tm .. 32 tm + 31, columns (k) 16 s .. 16 s + 15 of the 64 x 64
// left matrix, for tm = 0, 1.
// ---------------------------------------------------------------------------

struct HouseholderRule {
    // u arrives in one coalesced load, u_l in lane l; the entries the map
    // asks for are read from the lane that holds them (cross-lane reads, no
    // memory access), so building H adds no vector-memory instructions
    float ulane;
    float urow[2];  // -2 u_i of the lane's row in each 32-row block

    __device__ void init(const RuleParams& p, int64_t item, unsigned char*) {
        ulane = p.u[item * p.su + (threadIdx.x & 63)];
        mfmae::foreach_ij<FragA>([&](int e, int i, int) {
            if (e == 0) {
                urow[0] = -2.0f * __shfl(ulane, i);
                urow[1] = -2.0f * __shfl(ulane, 32 + i);
            }
        });
    }

    __device__ void build(int s, half8_t (&hh)[2], half8_t (&hl)[2]) const {
        mfmae::foreach_ij<FragA>([&](int e, int i, int jj) {
            const int gj = 16 * s + jj;
            const float uj = __shfl(ulane, gj);
#pragma unroll
            for (int tm = 0; tm < 2; ++tm) {
                const float h = __builtin_fmaf(urow[tm], uj, (32 * tm + i) == gj ? 1.0f : 0.0f);
                _Float16 vh, vl;
                mfmae::tcec::split_rounded(h, vh, vl);
                hh[tm][e] = vh;
                hl[tm][e] = vl;
            }
        });
    }
};

// Set element (r, q) of the 64 x 64 matrix held as fragments f[tm] (rows
// 32 tm .., columns 16 s ..) to v, if it falls in k step s: the lane that
// map() names writes element `elem` of fragment r / 32.  With r and q
// compile-time constants every test folds away but the lane compare.
__device__ inline void set_entry(FragA (&f)[2], int s, int r, int q, _Float16 v) {
    if ((q >> 4) != s) return;
    int lane, elem;
    mfmae::map<FragA>(lane, elem, r & 31, q & 15);
    if ((int)(threadIdx.x & 63) != lane) return;
    const int tm = r >> 5;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < FragA::num_elements; ++e)
            if (t == tm && e == elem) f[t].x[e] = v;
}

// Givens rotation through map().  EMBED: the plane (I, J) is a compile-time
// constant; otherwise it comes from the kernel arguments.
template <bool EMBED, int I, int J>
struct GivensMapRule {
    int gi, gj;
    _Float16 ch, cl, sh, sl, nsh, nsl;  // hi/lo of c, s and -s

    __device__ void init(const RuleParams& p, int64_t item, unsigned char*) {
        gi = EMBED ? I : p.gi;
        gj = EMBED ? J : p.gj;
        const float c = p.c[item * p.scs];
        const float s = p.s[item * p.scs];
        mfmae::tcec::split(c, ch, cl);
        mfmae::tcec::split(s, sh, sl);
        mfmae::tcec::split(-s, nsh, nsl);
    }

    __device__ void build(int s, half8_t (&hh)[2], half8_t (&hl)[2]) const {
        FragA fh[2], fl[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            mfmae::fill(fh[t], (_Float16)0.0f);
            mfmae::fill(fl[t], (_Float16)0.0f);
        }
        // ones on the part of the diagonal in this k step (hi 1, lo 0)
#pragma unroll
        for (int d = 0; d < 16; ++d) set_entry(fh, s, 16 * s + d, 16 * s + d, (_Float16)1.0f);
        // the rotation entries (c overrides the diagonal one)
        set_entry(fh, s, gi, gi, ch);
        set_entry(fl, s, gi, gi, cl);
        set_entry(fh, s, gj, gj, ch);
        set_entry(fl, s, gj, gj, cl);
        set_entry(fh, s, gi, gj, nsh);
        set_entry(fl, s, gi, gj, nsl);
        set_entry(fh, s, gj, gi, sh);
        set_entry(fl, s, gj, gi, sl);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            hh[t] = mfmae::pack(fh[t]);
            hl[t] = mfmae::pack(fl[t]);
        }
    }
};

// Baselines: the left matrix is written to the wave's own 16 KiB of LDS
// (hi and lo planes) and the fragments are loaded from there, as a fragment
// API without rule-built fragments requires.  Rows of 64 halves (128 bytes,
// 8 pieces of 8 halves); piece p of row r is stored at position
// p ^ ((r ^ (r >> 3)) & 7), so that the 32 rows a fragment load touches
// spread over all banks.
struct LdsOperand {
    unsigned char* hi;  // [64 rows][128 bytes]
    unsigned char* lo;

    __device__ static int off(int r, int p) { return r * 128 + 16 * (p ^ ((r ^ (r >> 3)) & 7)); }

    __device__ void bind(unsigned char* lds) {
        hi = lds;
        lo = lds + 64 * 128;
    }

    __device__ void build(int s, half8_t (&hh)[2], half8_t (&hl)[2]) const {
        const int l = threadIdx.x & 63;
        const int p = 2 * s + (l >> 5);  // k = 16 s + 8 (l / 32) + e
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const int o = off(32 * tm + (l & 31), p);
            hh[tm] = *reinterpret_cast<const half8_t*>(hi + o);
            hl[tm] = *reinterpret_cast<const half8_t*>(lo + o);
        }
    }
};

// Givens baseline: zero both planes, then lane r writes G_rr (c at i and j,
// else 1) and lanes 0 and 1 the two off-diagonal entries.
struct GivensLdsRule : LdsOperand {
    __device__ void init(const RuleParams& p, int64_t item, unsigned char* lds) {
        const int l = threadIdx.x & 63;
        bind(lds);
        const float c = p.c[item * p.scs];
        const float s = p.s[item * p.scs];
        // zero both planes: 64 rows x 8 pieces, 8 pieces per lane
        const half8_t z = {};
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int piece = 64 * t + l;
            *reinterpret_cast<half8_t*>(hi + off(piece >> 3, piece & 7)) = z;
            *reinterpret_cast<half8_t*>(lo + off(piece >> 3, piece & 7)) = z;
        }
        // A wave's LDS accesses complete in the order they are issued; the
        // fences keep the compiler from reordering the zeros, these entries
        // and the loads in build().
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        auto put = [&](int r, int q, float v) {
            _Float16 vh, vl;
            mfmae::tcec::split(v, vh, vl);
            const int o = off(r, q >> 3) + 2 * (q & 7);
            *reinterpret_cast<_Float16*>(hi + o) = vh;
            *reinterpret_cast<_Float16*>(lo + o) = vl;
        };
        put(l, l, (l == p.gi || l == p.gj) ? c : 1.0f);
        if (l == 0) put(p.gi, p.gj, -s);
        if (l == 1) put(p.gj, p.gi, s);
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
};

// Householder baseline: every entry h_ij = fmaf(-2 u_i, u_j, delta_ij) is
// formed once, split, and written to LDS; lane l forms 8 pieces of 8
// entries (rows (64 t + l) / 8, t = 0..7).
struct HouseholderLdsRule : LdsOperand {
    __device__ void init(const RuleParams& p, int64_t item, unsigned char* lds) {
        const int l = threadIdx.x & 63;
        bind(lds);
        // u as in the register-built rule: one coalesced load, entries read
        // from the lane that holds them
        const float ulane = p.u[item * p.su + l];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int piece = 64 * t + l;
            const int r = piece >> 3, q0 = 8 * (piece & 7);
            const float ur = -2.0f * __shfl(ulane, r);
            float h[8];
#pragma unroll
            for (int v = 0; v < 8; ++v)
                h[v] = mfmae::tcec::as_fp32(
                    __builtin_fmaf(ur, __shfl(ulane, q0 + v), (r == q0 + v) ? 1.0f : 0.0f));
            half8_t vh, vl;
            mfmae::tcec::split8(h, vh, vl);
            *reinterpret_cast<half8_t*>(hi + off(r, piece & 7)) = vh;
            *reinterpret_cast<half8_t*>(lo + off(r, piece & 7)) = vl;
        }
        // the fragment loads in build() read what other lanes wrote
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
};

// ---------------------------------------------------------------------------
// The common body: one wave = one item and one group of 64 columns.
// PAIR: the two 32-column blocks interleave their columns (column j of
// block cb is c0 + 2 j + cb), so one 8-byte load of a B row and one 8-byte
// store of a C row serve both blocks; needs 8-byte aligned, even-length B
// and C rows.  Otherwise block cb holds columns c0 + 32 cb + j.
// ---------------------------------------------------------------------------
template <class Rule, bool PAIR>
__device__ inline void rule64_body(const RuleParams& p, unsigned char* lds) {
    // wave index as a wave-uniform (scalar) value, so that the per-item base
    // pointers below live in SGPRs and loads use scalar-base addressing
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    const int64_t task = (int64_t)blockIdx.x * kWaves + wave;
    const int ngroups = (p.ncols + 63) / 64;
    const int64_t local = task / ngroups;
    const int c0 = (int)(task - local * ngroups) * 64;
    if (local >= p.batch) return;  // whole wave; the kernels have no barrier
    const int64_t item = local + p.item0;

    const float* __restrict__ Bi = p.B + item * p.sb;
    float* __restrict__ Ci = p.C + item * p.sc;

    Rule rule;
    rule.init(p, item, lds);

    const int j = l & 31;
    // first column of this lane in block 0, and whether it (and, paired,
    // its neighbour) lies inside B
    const int col0 = PAIR ? c0 + 2 * j : c0 + j;
    const bool ok0 = col0 < p.ncols;
    const bool ok1 = PAIR ? ok0 : col0 + 32 < p.ncols;

    f32x16_t acc[2][2], cor[2][2];
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                acc[tm][cb][e] = 0.0f;
                cor[tm][cb][e] = 0.0f;
            }

#pragma unroll
    for (int s = 0; s < 4; ++s) {
        // B operands of this 16-wide k step for both column blocks: lane l
        // holds rows 16 s + 8 (l / 32) + e; the row start of (s, e) is
        // wave-uniform and the lane part is a 32-bit offset.
        half8_t bh[2], bl[2];
        const int lane_off = 8 * (l >> 5) * (int)p.ldb + col0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float* rowp = Bi + (int64_t)(16 * s + e) * p.ldb;
            float x[2];
            if constexpr (PAIR) {
                f32x2 v = {0.0f, 0.0f};
                if (ok0) v = *reinterpret_cast<const f32x2*>(rowp + lane_off);
                x[0] = v[0];
                x[1] = v[1];
            } else {
                x[0] = ok0 ? rowp[lane_off] : 0.0f;
                x[1] = ok1 ? rowp[lane_off + 32] : 0.0f;
            }
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                _Float16 vh, vl;
                mfmae::tcec::split(x[cb], vh, vl);
                bh[cb][e] = vh;
                bl[cb][e] = vl;
            }
        }
        half8_t hh[2], hl[2];
        rule.build(s, hh, hl);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                acc[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hh[tm], bh[cb], acc[tm][cb],
                                                                     0, 0, 0);
                cor[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hl[tm], bh[cb], cor[tm][cb],
                                                                     0, 0, 0);
                cor[tm][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hh[tm], bl[cb], cor[tm][cb],
                                                                     0, 0, 0);
            }
    }

    // C = main + corr * 2^-11; element e of a block is row
    // 8 (e / 4) + 4 (l / 32) + e % 4 of it.
#pragma unroll
    for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int row = 32 * tm + mfmae::layout<Shape32, Use::Acc>::row(l, e);
            float v[2];
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
                v[cb] = __builtin_fmaf(cor[tm][cb][e], mfmae::tcec::kLoScaleInv, acc[tm][cb][e]);
            float* dst = Ci + (int64_t)row * p.ldc + col0;
            if constexpr (PAIR) {
                if (ok0) *reinterpret_cast<f32x2*>(dst) = f32x2{v[0], v[1]};
            } else {
                if (ok0) dst[0] = v[0];
                if (ok1) dst[32] = v[1];
            }
        }
}

template <bool PAIR>
__global__ __launch_bounds__(64 * kWaves, 2) void householder64_kernel(RuleParams p) {
    rule64_body<HouseholderRule, PAIR>(p, nullptr);
}

template <bool PAIR>
__global__ __launch_bounds__(64 * kWaves, 2) void householder64_lds_kernel(RuleParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[kWaves][2 * 64 * 128];
    rule64_body<HouseholderLdsRule, PAIR>(p, lds[threadIdx.x >> 6]);
}

template <bool EMBED, int I, int J, bool PAIR>
__global__ __launch_bounds__(64 * kWaves, 2) void givens64_kernel(RuleParams p) {
    rule64_body<GivensMapRule<EMBED, I, J>, PAIR>(p, nullptr);
}

template <bool PAIR>
__global__ __launch_bounds__(64 * kWaves, 2) void givens64_lds_kernel(RuleParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[kWaves][2 * 64 * 128];
    rule64_body<GivensLdsRule, PAIR>(p, lds[threadIdx.x >> 6]);
}

// Launch `kernel` over the batch in pieces below 2^31 work-items (the
// dispatch packet counts work-items in 32 bits).
template <class K>
hipError_t launch_rule(K kernel, RuleParams p, int64_t batch, hipStream_t stream) {
    const int64_t ngroups = (p.ncols + 63) / 64;
    const int64_t max_blocks = (int64_t(1) << 31) / (64 * kWaves) - 1;
    const int64_t items_per_launch = max_blocks * kWaves / ngroups;
    if (items_per_launch == 0) return hipErrorInvalidConfiguration;
    for (int64_t i0 = 0; i0 < batch; i0 += items_per_launch) {
        const int64_t items = batch - i0 < items_per_launch ? batch - i0 : items_per_launch;
        p.batch = (int)items;
        p.item0 = i0;
        const int64_t blocks = (items * ngroups + kWaves - 1) / kWaves;
        hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(64 * kWaves), 0, stream, p);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

bool pairs_ok(const float* B, int64_t ldb, int64_t sb, const float* C, int64_t ldc, int64_t sc,
              int ncols) {
    return ((uintptr_t)B % 8 == 0) && ((uintptr_t)C % 8 == 0) && ldb % 2 == 0 && ldc % 2 == 0 &&
           sb % 2 == 0 && sc % 2 == 0 && ncols % 2 == 0;
}

// The rotation planes (i, j) with a compile-time instance of the Givens
// kernel.
#define SGEMM_EMU_GIVENS_PLANES(X) X(5, 37) X(37, 5) X(0, 1) X(31, 32) X(62, 63)

template <bool PAIR>
hipError_t launch_givens_embedded(const RuleParams& p, int64_t batch, hipStream_t stream) {
#define SGEMM_EMU_GIVENS_CASE(I, J) \
    if (p.gi == I && p.gj == J) return launch_rule(givens64_kernel<true, I, J, PAIR>, p, batch, stream);
    SGEMM_EMU_GIVENS_PLANES(SGEMM_EMU_GIVENS_CASE)
#undef SGEMM_EMU_GIVENS_CASE
    return hipErrorInvalidValue;
}

}  // namespace

bool givens_embedded(int i, int j) {
#define SGEMM_EMU_GIVENS_TEST(I, J) \
    if (i == I && j == J) return true;
    SGEMM_EMU_GIVENS_PLANES(SGEMM_EMU_GIVENS_TEST)
#undef SGEMM_EMU_GIVENS_TEST
    return false;
}

hipError_t launch_householder64(const HouseholderArgs& a, hipStream_t stream) {
    RuleParams p{};
    p.ncols = a.ncols;
    p.u = a.u;
    p.su = a.su;
    p.B = a.B;
    p.ldb = a.ldb;
    p.sb = a.sb;
    p.C = a.C;
    p.ldc = a.ldc;
    p.sc = a.sc;
    const bool pair = pairs_ok(a.B, a.ldb, a.sb, a.C, a.ldc, a.sc, a.ncols);
    if (a.mode == SGEMM_EMU_HOUSEHOLDER_LDS)
        return pair ? launch_rule(householder64_lds_kernel<true>, p, a.batch, stream)
                    : launch_rule(householder64_lds_kernel<false>, p, a.batch, stream);
    return pair ? launch_rule(householder64_kernel<true>, p, a.batch, stream)
                : launch_rule(householder64_kernel<false>, p, a.batch, stream);
}

hipError_t launch_givens64(const GivensArgs& a, hipStream_t stream) {
    RuleParams p{};
    p.ncols = a.ncols;
    p.c = a.c;
    p.s = a.s;
    p.scs = a.scs;
    p.gi = a.i;
    p.gj = a.j;
    p.B = a.B;
    p.ldb = a.ldb;
    p.sb = a.sb;
    p.C = a.C;
    p.ldc = a.ldc;
    p.sc = a.sc;
    const bool pair = pairs_ok(a.B, a.ldb, a.sb, a.C, a.ldc, a.sc, a.ncols);
    switch (a.mode) {
        case SGEMM_EMU_GIVENS_EMBEDDED:
            return pair ? launch_givens_embedded<true>(p, a.batch, stream)
                        : launch_givens_embedded<false>(p, a.batch, stream);
        case SGEMM_EMU_GIVENS_LDS:
            return pair ? launch_rule(givens64_lds_kernel<true>, p, a.batch, stream)
                        : launch_rule(givens64_lds_kernel<false>, p, a.batch, stream);
        default:
            return pair ? launch_rule(givens64_kernel<false, 0, 0, true>, p, a.batch, stream)
                        : launch_rule(givens64_kernel<false, 0, 0, false>, p, a.batch, stream);
    }
}

}  // namespace sgemm_emu
