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

// Task of workgroup b in a grid of G workgroups.  Workgroups are dispatched
// round-robin over the 8 XCDs, so b runs on XCD b % 8 as that XCD's
// (b / 8)-th workgroup; numbering them so that every XCD receives one
// contiguous range of task ids keeps the tiles of one item, which share A
// rows and B columns, in one L2.  A bijection of [0, G) for any G >= 1: XCD
// x < G mod 8 receives floor(G / 8) + 1 ids, the others floor(G / 8).
__host__ __device__ inline int xcd_task(int b, int G) {
    const int x = b & 7, i = b >> 3;
    const int q = G >> 3, r = G & 7;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

// Tile (row, column) of the t-th task of one item in a grid of tiles_m x
// tiles_n tiles.  Tiles are taken in groups of GROUP_M tile rows (the last
// group may hold fewer), column by column within a group, so that the
// workgroups running at the same time on one XCD share B columns as well as
// A rows.  A bijection of [0, tiles_m tiles_n) onto the tile grid.
constexpr int GROUP_M = 8;

struct TileRC {
    int tm, tn;
};

__host__ __device__ inline TileRC grouped_tile(int t, int tiles_m, int tiles_n) {
    const int group_size = GROUP_M * tiles_n;
    const int grp = t / group_size;
    const int first_m = grp * GROUP_M;
    const int rest = tiles_m - first_m;
    const int gm = rest < GROUP_M ? rest : GROUP_M;
    const int r = t - grp * group_size;
    return {first_m + r % gm, r / gm};
}

// Tile order for one large product on the 128 x 256 tile (one item per
// launch, tiles_m and tiles_n multiples of 16): the 256 tasks the device
// runs at the same time -- 32 on each of the 8 XCDs, one workgroup per CU --
// form one 16 x 16 block of tiles, each XCD an 8 x 4 part of it, so that the
// XCDs share A rows (four each) and B columns (two each) in the last-level
// cache, not only within their own L2.  Task t of XCD x = t / (G / 8) (the
// numbering of xcd_task) is the s-th of that XCD, s = t mod (G / 8); block
// s / 32, taken down the columns of blocks, position s mod 32 in the XCD's
// part.  A bijection of [0, tiles_m tiles_n) onto the tile grid.
__host__ __device__ inline bool block_order_applies(int tiles_m, int tiles_n, int ntasks) {
    return tiles_m % 16 == 0 && tiles_n % 16 == 0 && (int64_t)tiles_m * tiles_n == ntasks;
}

__host__ __device__ inline TileRC block_tile(int t, int tiles_m, int tiles_n) {
    const int per_xcd = tiles_m * tiles_n / 8;  // a multiple of 32
    const int x = t / per_xcd, s = t - x * per_xcd;
    const int w = s >> 5, i = s & 31;
    const int blocks_m = tiles_m / 16;
    const int bm = w % blocks_m, bn = w / blocks_m;
    return {16 * bm + 8 * (x & 1) + (i & 7), 16 * bn + 4 * (x >> 1) + (i >> 3)};
}

// The persistent kernels: workgroup b of G walks tasks xcd_task(b, G) + i G.
__device__ inline int first_task(const KParams& p) { return xcd_task(blockIdx.x, gridDim.x); }

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
    const TileRC rc = grouped_tile(task - item * tiles, p.tiles_m, p.tiles_n);
    const int64_t it = (int64_t)item + p.item0;
    TaskPos q;
    q.A = p.A + it * p.sa;
    q.B = p.B + it * p.sb;
    q.C = p.C + it * p.sc;
    q.m0 = rc.tm * BM;
    q.n0 = rc.tn * BN;
    return q;
}

}  // namespace sgemm_emu
