// Work distribution shared by the batched GEMM kernels: kernel parameters,
// the persistent task walk and the XCD-aware numbering of workgroups.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace sgemm_emu {

constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

struct KParams {
    int m, n, k;
    const float* A;
    int64_t lda, sa;
    const float* B;
    int64_t ldb, sb;
    float* C;
    int64_t ldc, sc;
    int tiles_m, tiles_n;
    int ntasks;       // (items of this launch) x (tiles per item)
    int item0;        // first batch item of this launch
    int vec_a, vec_b;
    int xcd_remap;    // 1 if gridDim.x is a multiple of 8
};

// ---------------------------------------------------------------------------
// Work distribution.
//
// The grid is persistent: about as many workgroups as fit on the GPU at
// once, each walking the task list (task = one BM x BN tile of one item)
// with a stride of gridDim.x, and streaming k chunks back to back across
// task boundaries so that the loads of a task's first chunk overlap the
// previous task's last chunk and its stores.
//
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Renumbering workgroup b to (b % 8) * (G / 8) + b / 8 makes the tasks
// that run at the same time on one XCD a contiguous range of task ids, so
// tiles that share A rows and B columns share an L2.  Within an item, tiles
// are ordered in groups of GROUP_M tile rows so that consecutive tiles reuse
// the same B columns.
// ---------------------------------------------------------------------------
__device__ inline int first_task(const KParams& p) {
    int b = blockIdx.x;
    if (p.xcd_remap) {
        const int per = gridDim.x >> 3;
        b = (b & 7) * per + (b >> 3);
    }
    return b;
}

// Task of workgroup b in a grid of G workgroups.  Workgroups are dispatched
// round-robin over the 8 XCDs, so b runs on XCD b % 8 as that XCD's
// (b / 8)-th workgroup; numbering them so that every XCD receives one
// contiguous range of task ids keeps the tiles of one item, which share A
// rows and B columns, in one L2.  A bijection of [0, G) for any G.
__device__ inline int xcd_task(int b, int G) {
    const int x = b & 7, i = b >> 3;
    const int q = G >> 3, r = G & 7;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

struct TaskPos {
    const float* A;  // item base pointers
    const float* B;
    float* C;
    int m0, n0;      // tile origin
};

template <int BM, int BN>
__device__ inline TaskPos task_pos(const KParams& p, int task) {
    const int tiles = p.tiles_m * p.tiles_n;
    const int item = task / tiles;
    const int t = task - item * tiles;
    constexpr int GROUP_M = 8;
    const int group_size = GROUP_M * p.tiles_n;
    const int g = t / group_size;
    const int first_m = g * GROUP_M;
    const int gm = min(p.tiles_m - first_m, GROUP_M);
    const int r = t - g * group_size;
    const int64_t it = (int64_t)item + p.item0;
    TaskPos q;
    q.A = p.A + it * p.sa;
    q.B = p.B + it * p.sb;
    q.C = p.C + it * p.sc;
    q.m0 = (first_m + r % gm) * BM;
    q.n0 = (r / gm) * BN;
    return q;
}

}  // namespace sgemm_emu
