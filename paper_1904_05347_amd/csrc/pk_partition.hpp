// pk_partition.hpp -- the integer maps that distribute the output tiles and
// the (tile, K-block) iterations of one launch over its work-groups (Section
// 3.1.1: the blocks of C are independent panel products, and a block's K
// range is a sum of K-block products, so any partition of either is exact).
// Plain integer arithmetic, compiled for the host as well as the device, so
// the CPU tests exercise the very functions the kernels call.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pk {

// Tile (tm, tn) of logical tile t, in column strips of group_m tile-rows (so
// that concurrently running tiles share A and B panels).
__host__ __device__ inline void tile_of_ints(int tiles_m, int tiles_n, int group_m, int t, int &tm, int &tn)
{
    const int group = group_m * tiles_n;
    const int gid = t / group;
    const int first_m = gid * group_m;
    const int gsz = tiles_m - first_m < group_m ? tiles_m - first_m : group_m;
    const int in_group = t - gid * group;
    tm = first_m + in_group % gsz;
    tn = in_group / gsz;
}

// Logical tile of work-group pid when work-groups are dealt to the xcds
// XCDs round-robin (pid % xcds): each XCD receives a contiguous run of
// logical tiles, whose panels then stay in its own L2.  A permutation of
// 0 .. num-1.
__host__ __device__ inline int xcd_tile(int pid, int num, int xcds)
{
    if (xcds <= 1) return pid;
    const int q = num / xcds, r = num % xcds;
    const int x = pid % xcds, loc = pid / xcds;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + loc;
}

// Stream-K: the T = tiles * nkb iterations split evenly over G work-groups;
// logical work-group g owns [start(g), start(g+1)).
struct StreamK {
    int T, G, nkb;

    __host__ __device__ int start(int g) const { return (int)(((int64_t)g * T) / G); }
    // the work-group whose range holds iteration i: the largest g with start(g) <= i
    __host__ __device__ int owner(int i) const { return (int)(((int64_t)(i + 1) * G + T - 1) / T) - 1; }
    // partial-tile slot of work-group g for tile t: 2g for its range's first
    // tile, 2g + 1 for its last (a range cuts at most those two)
    __host__ __device__ int slot(int g, int t) const { return start(g) / nkb == t ? 2 * g : 2 * g + 1; }
};

// Logical stream-K work-group of work-group b (dealt round-robin to xcds
// XCDs): each XCD gets a contiguous share of the ranges, so the tiles one
// XCD works on are neighbours.  A permutation of 0 .. G-1 when G % xcds == 0.
__host__ __device__ inline int sk_logical(int b, int G, int xcds)
{
    return (xcds > 1 && G % xcds == 0) ? (b % xcds) * (G / xcds) + b / xcds : b;
}

}  // namespace pk
