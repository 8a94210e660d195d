// Template of the weight-specialised ConvShift kernels.
//
// The paper (Section 6) proposes compiling the shift kernels at run time. With
// the weights known, every shift amount and sign becomes part of the
// instruction stream: for each reduction element j (input channel, tap) a
// lane loads its input value x, forms each right shift x >> s that the 64
// output channels of a segment use there once, and each non-zero weight is one
// v_add_u32 or v_sub_u32 of that shifted value into its channel's accumulator;
// zero weights cost nothing.
//
// This file is compiled to assembly when the library is built. The kernel
// below computes, per lane, what the generated code needs (the byte offsets of
// the lane's taps in x, or an offset past the end of x for taps in the
// padding; the byte offset of its output pixel in y) and hands them over in
// fixed registers at the JITBODY marker. At run time the generator replaces
// the marker with a jump, through a table, to the code of this wave's segment
// (up to 64 output channels and a range of input channels), assembled from
// generated machine words; each segment ends the wave itself. Register use of
// the generated code (the clobbers below): v14..v95 (v16, v17 the shifted
// values, v18..v81 the accumulators, v82..v95 the loads in flight), s28..s31;
// 96 VGPRs in all, so that 5 waves fit on a SIMD. Layers that read x at one
// tap per element (1 x 1 windows, and wider windows through a zero-padded copy
// of x, where the tap is an offset in the instruction) run the second entry
// point, which hands over only the first tap: v5..v12 hold 8 loads in flight,
// v14, v15 the shifted values and v16..v79 the accumulators; 80 VGPRs, 6
// waves per SIMD.
//
// A workgroup covers P groups of 64 pixels (P = 1, 2 or 4) with W waves each
// (the wave split, W = 1, 2, 4, 8 or 16; P * W <= 16 waves). Without a wave
// split each wave covers its 64 pixels with the whole reduction of its
// segment. With a split (grids too small to fill the chip otherwise), the W
// waves of a pixel group each run a contiguous share of the reduction in code
// of their own; they add their partial sums into LDS, which the prologue
// zeroes, and after a barrier each finishes its share of the segment's
// channels. The P waves running one share's code (one per pixel group) share
// its instruction fetch on their CU. v3 holds the lane's LDS byte offset:
// (pixel group in the workgroup) * 16 KiB + lane * 4, channel j at j * 256
// above it.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "jit.hpp"

using ds::JitArgs;

template <bool kOneTap>
__device__ __forceinline__ void jit_conv(const JitArgs &p)
{
    extern __shared__ int32_t red[];  // wave split: [pixel groups][64 channels][64 lanes]
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wl = p.wsplit_log2;
    const int pg = wave >> wl, share = wave & ((1 << wl) - 1);  // pixel group, reduction share
    // Block order: groups of `group_tiles` pixel tiles (the last group may be
    // smaller); within a group, the segments one after the other, and within a
    // segment the group's tiles, so that the inputs of a few pixel tiles stay in
    // L2 while the segments go by. Tile-major (small grids): all segments of a
    // tile, then the next tile, so that the blocks resident on one CU (block b
    // and b + 256 k at the start) run the same segment's code. The grid is
    // exactly tiles_p * nseg blocks.
    const int b = blockIdx.x;
    int sg, tile;
    if (p.tile_major == 2 && b < (p.tiles_p >> 3) * 8 * p.nseg) {
        // XCD-local tile-major: workgroups are dealt to the 8 XCDs in turn
        // (block b to XCD b % 8), so whole rows of 8 tiles map tile 8 i + x to
        // XCD x: every segment of a tile then runs on one XCD and reads the
        // tile's input through that XCD's L2 only. The tiles of the last,
        // partial row (the rest of the grid) take the plain tile-major order.
        const int j = b >> 3;
        const int row = j / p.nseg;
        sg = j - row * p.nseg;
        tile = row * 8 + (b & 7);
    } else if (p.tile_major) {
        tile = b / p.nseg;
        sg = b - tile * p.nseg;
    } else {
        const int per_group = p.group_tiles * p.nseg;
        const int grp = b / per_group, r = b - grp * per_group;
        const int gsize = min(p.group_tiles, p.tiles_p - grp * p.group_tiles);
        sg = r / gsize;
        tile = grp * p.group_tiles + (r - sg * gsize);
    }
    const int seg = __builtin_amdgcn_readfirstlane((sg << wl) + share);
    const int q = ((tile << p.pgroups_log2) + pg) * 64 + lane;
    const int lds = pg * 16384 + lane * 4;
    if (wl > 0) {
        // Each wave zeroes 64 >> wl channels of its pixel group's partial sums.
        const int per = 64 >> wl;
        for (int j = 0; j < per; ++j) red[(pg * 64 + share * per + j) * 64 + lane] = 0;
        __syncthreads();
    }
    const int kOOB = int(0x80000000u);
    int yoff = kOOB;
    int t0 = kOOB, t1 = kOOB, t2 = kOOB, t3 = kOOB, t4 = kOOB, t5 = kOOB, t6 = kOOB, t7 = kOOB,
        t8 = kOOB;
    if (tile < p.tiles_p && q < p.NQ) {
        const int n = ds::fdiv(q, p.div_ohow);
        const int pix = q - n * p.OHOW;
        const int oh = ds::fdiv(pix, p.div_ow);
        const int ow = pix - oh * p.OW;
        yoff = (p.ybase + n * p.ynst + oh * p.yrst + ow * p.ycst) * 4;
        const int ih0 = oh * p.sh - p.ph, iw0 = ow * p.sw - p.pw, base = n * p.C * p.HW;
        // Taps of a 3 x 3 window (r, s) = (t / 3, t % 3); a 1 x 1 layer uses t0 only.
        auto off = [&](int rr, int ss) {
            const int ih = ih0 + rr, iw = iw0 + ss;
            return (ih >= 0 && ih < p.H && iw >= 0 && iw < p.W) ? (base + ih * p.W + iw) << p.xshift : kOOB;
        };
        t0 = off(0, 0);
        if (!kOneTap) {
            t1 = off(0, 1); t2 = off(0, 2);
            t3 = off(1, 0); t4 = off(1, 1); t5 = off(1, 2);
            t6 = off(2, 0); t7 = off(2, 1); t8 = off(2, 2);
        }
    }
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(p.x), short(0), p.x_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(p.y, short(0), p.y_bytes,
                                                                        0x00020000);
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(p.residual), short(0), p.residual ? p.y_bytes : 0, 0x00020000);
    if constexpr (kOneTap) {
        asm volatile("; JITBODY"
                     :
                     : "{s[20:23]}"(xr), "{s[24:27]}"(yr), "{s[36:39]}"(rr), "{s19}"(seg), "{v3}"(lds),
                       "{v4}"(t0), "{v13}"(yoff)
                     : "memory", "v5", "v6", "v7", "v8", "v9", "v10", "v11", "v12", "v14", "v15",
                       "v16", "v17", "v18", "v19", "v20", "v21", "v22", "v23", "v24", "v25", "v26",
                       "v27", "v28", "v29", "v30", "v31", "v32", "v33", "v34", "v35", "v36", "v37",
                       "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45", "v46", "v47", "v48",
                       "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59",
                       "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70",
                       "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "s28", "s29",
                       "s30", "s31");
    } else {
        asm volatile("; JITBODY"
                     :
                     : "{s[20:23]}"(xr), "{s[24:27]}"(yr), "{s[36:39]}"(rr), "{s19}"(seg), "{v3}"(lds),
                       "{v4}"(t0), "{v5}"(t1), "{v6}"(t2), "{v7}"(t3), "{v8}"(t4), "{v9}"(t5),
                       "{v10}"(t6), "{v11}"(t7), "{v12}"(t8), "{v13}"(yoff)
                     : "memory", "v14", "v15", "v16", "v17", "v18", "v19", "v20", "v21", "v22", "v23",
                       "v24", "v25", "v26", "v27", "v28", "v29", "v30", "v31", "v32", "v33", "v34",
                       "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45",
                       "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56",
                       "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67",
                       "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78",
                       "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89",
                       "v90", "v91", "v92", "v93", "v94", "v95", "s28", "s29", "s30", "s31");
    }
}

// Layers with up to 3 x 3 taps per element: 96 VGPRs, 5 waves per SIMD.
// Workgroups of 256 threads, or 512 / 1024 with a wave split of 8 / 16.
extern "C" __global__ void __launch_bounds__(1024) ds_jit_conv_template(const JitArgs p)
{
    jit_conv<false>(p);
}

// Layers with one tap per element: 80 VGPRs, 6 waves per SIMD.
extern "C" __global__ void __launch_bounds__(1024) ds_jit_conv_one_tap_template(const JitArgs p)
{
    jit_conv<true>(p);
}
