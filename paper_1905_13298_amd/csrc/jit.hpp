// Kernel arguments shared by the weight-specialised kernel template and its
// launcher. The generated code itself reads none of them: the template's
// prologue turns them into per-lane offsets in fixed registers.
#pragma once

#include <cstdint>

#include "fastdiv.hpp"

namespace ds {

struct JitArgs {
    const int32_t *x;
    int32_t *y;
    const int32_t *residual;  // NULL when the layer adds none
    int x_bytes, y_bytes;
    int xshift;               // log2 of the bytes of an x element: 2 int32, 1 int16, 0 int8
    int NQ, OHOW, OW, H, W, C, K, HW, sh, sw, ph, pw;
    int ybase, ynst, yrst, ycst;  // output (n, oh, ow) of channel 0 at y[ybase + n*ynst + oh*yrst + ow*ycst]
    int tiles_p;              // pixel tiles (workgroups) per segment
    int group_tiles;          // pixel tiles that run all segments before the next tiles
    int nseg;
    int wsplit_log2;          // waves per 64 pixels: 1, 2, 4, 8 or 16, each a share of the reduction
    int pgroups_log2;         // groups of 64 pixels per workgroup: 1, 2 or 4
    int tile_major;           // block order: 0 grouped, 1 tile-major, 2 XCD-local tile-major
    FastDiv div_ohow, div_ow;
};

}  // namespace ds
