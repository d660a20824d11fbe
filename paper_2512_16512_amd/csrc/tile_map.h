// Workgroup -> output-tile mapping shared by the kernel families.
//
// The grid is one workgroup per output tile (the parallelized outer
// strip-mine of M and N).  Two run-time reorderings are applied to the
// workgroup id before it is turned into tile coordinates:
//
// 1. XCD remap.  The MI355X dispatcher hands workgroups to its 8 XCDs
//    round-robin (id % 8), and each XCD has a private L2.  Renumbering so
//    that XCD x receives one contiguous band of ids makes the tiles that run
//    together on one XCD neighbours in the tile order, so they share A and B
//    panels in that XCD's L2.
// 2. Raster (interchange of the two parallel tile loops): row-major,
//    column-major, or grouped bands of `g` tile-rows walked column by column
//    (so consecutive ids reuse the same few A row-panels and sweep B).
#pragma once

#include <hip/hip_runtime.h>

namespace xtc {

__device__ __forceinline__ void tile_coords(int bid, int G, int tiles_m, int tiles_n,
                                            int raster, int xcd_remap, int &tm, int &tn) {
    if (xcd_remap && G >= 8) {
        const int x = bid & 7, q = G >> 3, rem = G & 7;
        bid = x * q + (x < rem ? x : rem) + (bid >> 3);
    }
    if (raster == 1) {
        tm = bid % tiles_m;
        tn = bid / tiles_m;
    } else if (raster >= 2) {
        // a group taller than the grid is the whole grid (also keeps
        // raster * tiles_n within the tile count)
        const int rg = raster < tiles_m ? raster : tiles_m;
        const int per = rg * tiles_n;
        const int grp = bid / per;
        const int first = grp * rg;
        const int left = tiles_m - first;
        const int gsz = left < rg ? left : rg;
        const int r = bid - grp * per;
        tm = first + r % gsz;
        tn = r / gsz;
    } else {
        tm = bid / tiles_n;
        tn = bid % tiles_n;
    }
}

}  // namespace xtc
