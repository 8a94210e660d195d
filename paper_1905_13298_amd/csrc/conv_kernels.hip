// Kernels of the shift operators for CDNA4 (gfx950) and the host code that
// plans and launches them.
//
// The computation (DeepShift Section 3, Eqs. 1-3, Figure 1a) is an implicit
// GEMM over output pixels q = (n, oh, ow) and output channels k with the
// reduction j = (c, r, s):
//     y[k][q] = init[k] + sum_j  term(X[j][q], code[k][j])        (mod 2^32)
// where X[j][q] is the input value under tap j of pixel q (0 in the padding).
//
// Shift-accumulate in two VALU instructions. Each code is decoded once per
// call into a word d with the shift amount in bits 0-4 (31 for a zero weight)
// and bit 31 set for a negative weight. With m = d >> 31 (0 or -1):
//     acc += (x >> (d & 31)) ^ m          -> v_ashrrev_i32 + v_xad_u32
// For a negative weight (x >> s) ^ -1 = -(x >> s) - 1, so init[k] adds back
// one per negative non-zero weight of row k (negcount). For x >= 0 a zero
// weight gives (x >> 31) ^ 0 = 0. When a staged chunk holds a negative x the
// kernel switches to three instructions, ((x >> s) & z) ^ m with z = 0 for
// zero weights, which is exact for every int32.
//
// Work decomposition. Lanes map to output pixels and each wave owns TN output
// channels, so a weight is the same for all 64 lanes: it lives in scalar
// registers (s_load from the decoded buffer, mask by s_ashr), and the inner
// loop has no branch on sign or zero. A workgroup is 4 waves covering
// 4*TN channels and P = 64*TM pixels; the input values the tile needs are
// staged in LDS one chunk of CC input channels at a time and shared by the
// four waves. Integer addition modulo 2^32 is associative, so split-K
// partial sums (int32 atomics) and any reduction order are bit-exact.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <mutex>

#include "conv_plan.hpp"

namespace ds {

int forced_variant()
{
    static const int v = [] {
        const char *e = std::getenv("DS_FORCE_VARIANT");
        if (!e || !*e) return -1;
        return std::atoi(e);
    }();
    return v;
}

// ---------------------------------------------------------------------------
// Division by a launch-constant divisor for dividends below 2^31
// (round-up multiplier method of Granlund and Montgomery, 1994).

struct FastDiv {
    uint32_t d, m, l;
};

static FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{d, uint32_t(m), l};
}

__device__ __forceinline__ int fdiv(int n, const FastDiv &f)
{
    return int((__umulhi(uint32_t(n), f.m) + uint32_t(n)) >> f.l);
}

// ---------------------------------------------------------------------------
// Scratch memory: stream-ordered allocations from one pool per device that
// keeps freed memory for reuse.

static hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t st)
{
    static std::mutex mu;
    static hipMemPool_t pools[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    {
        std::lock_guard<std::mutex> lock(mu);
        if (!pools[dev]) {
            hipMemPoolProps props = {};
            props.allocType = hipMemAllocationTypePinned;
            props.location.type = hipMemLocationTypeDevice;
            props.location.id = dev;
            hipMemPool_t pool;
            e = hipMemPoolCreate(&pool, &props);
            if (e != hipSuccess) return e;
            uint64_t keep = UINT64_MAX;
            e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
            if (e != hipSuccess) return e;
            pools[dev] = pool;
        }
    }
    return hipMallocFromPoolAsync(p, bytes, pools[dev], st);
}

// ---------------------------------------------------------------------------
// One thread per output element, codes read straight from the packed words.
// Used for shapes the tiled kernel does not cover and as a second opinion in
// the tests.

template <Inner OP>
__global__ void __launch_bounds__(256)
conv_direct_kernel(const int32_t *__restrict__ x, const uint32_t *__restrict__ wp,
                   const int32_t *__restrict__ wi, const int32_t *__restrict__ bias,
                   int32_t *__restrict__ y, ConvGeom g, int wpr)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int ow = int(idx % g.ow);
        int64_t t = idx / g.ow;
        const int oh = int(t % g.oh);
        t /= g.oh;
        const int k = int(t % g.k);
        const int n = int(t / g.k);
        uint32_t acc = bias ? uint32_t(bias[k]) : 0u;
        for (int c = 0; c < g.c; ++c)
            for (int r = 0; r < g.r; ++r) {
                const int ih = oh * g.sh - g.ph + r;
                if (ih < 0 || ih >= g.h) continue;
                for (int s = 0; s < g.s; ++s) {
                    const int iw = ow * g.sw - g.pw + s;
                    if (iw < 0 || iw >= g.w) continue;
                    const int32_t xv = x[(int64_t(n * g.c + c) * g.h + ih) * g.w + iw];
                    const int j = (c * g.r + r) * g.s + s;
                    if constexpr (OP == Inner::Shift) {
                        const uint32_t code = (wp[int64_t(k) * wpr + j / 6] >> (5 * (j % 6))) & 31u;
                        const int sh = int(code & 15u);
                        if (sh == 15) continue;
                        const uint32_t tv = uint32_t(xv >> sh);
                        acc += (code & 16u) ? 0u - tv : tv;
                    } else {
                        acc += uint32_t(xv) * uint32_t(wi[int64_t(k) * g.crs + j]);
                    }
                }
            }
        y[idx] = int32_t(acc);
    }
}

// ---------------------------------------------------------------------------
// Preparation: decoded weights wd[kg][j][TN] (k = kg*TN + t) and init[k].
// Rows k >= K and taps j >= C*R*S (the padding up to whole chunks) become
// zero weights.

template <Inner OP, int TN>
__global__ void __launch_bounds__(256)
prep_weights_kernel(const uint32_t *__restrict__ wp, const int32_t *__restrict__ wi, int K,
                    int CRS, int wpr, int Jpad, int Kpad, int32_t *__restrict__ wd)
{
    const int64_t total = int64_t(Kpad) * Jpad;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int t = int(idx % TN);
        const int64_t rest = idx / TN;
        const int j = int(rest % Jpad);
        const int k = int(rest / Jpad) * TN + t;
        int32_t v;
        if (k < K && j < CRS) {
            if constexpr (OP == Inner::Shift) {
                const uint32_t code = (wp[int64_t(k) * wpr + j / 6] >> (5 * (j % 6))) & 31u;
                const uint32_t sh = code & 15u;
                v = sh == 15u ? 31 : int32_t(sh | ((code >> 4) << 31));
            } else {
                v = wi[int64_t(k) * CRS + j];
            }
        } else {
            v = OP == Inner::Shift ? 31 : 0;
        }
        wd[idx] = v;
    }
}

// init[k] = bias[k] + negcount[k] (shift) or bias[k] (multiply); one wave per row.
template <Inner OP>
__global__ void __launch_bounds__(256)
prep_init_kernel(const uint32_t *__restrict__ wp, const int32_t *__restrict__ bias, int K,
                 int CRS, int wpr, int Kpad, int32_t *__restrict__ init)
{
    const int k = blockIdx.x * 4 + int(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (k >= Kpad) return;
    uint32_t cnt = 0;
    if (OP == Inner::Shift && k < K) {
        for (int wdx = lane; wdx < wpr; wdx += 64) {
            const uint32_t word = wp[int64_t(k) * wpr + wdx];
            for (int j = 0; j < 6; ++j) {
                const uint32_t code = (word >> (5 * j)) & 31u;
                const bool live = wdx * 6 + j < CRS;
                cnt += (live && (code & 16u) && (code & 15u) != 15u) ? 1u : 0u;
            }
        }
    }
    for (int off = 32; off > 0; off >>= 1) cnt += uint32_t(__shfl_xor(int(cnt), off));
    if (lane == 0)
        init[k] = k < K ? int32_t((bias ? uint32_t(bias[k]) : 0u) + cnt) : 0;
}

// y[n][k][q] = init[k]: the starting value when split-K partial sums are added atomically.
__global__ void __launch_bounds__(256)
fill_init_kernel(const int32_t *__restrict__ init, int32_t *__restrict__ y, int64_t total,
                 int K, int OHOW)
{
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x)
        y[idx] = init[(idx / OHOW) % K];
}

// ---------------------------------------------------------------------------
// Tiled kernel.

enum StageMode : int {
    MODE_WINDOW = 0,    // r x s window with padding: LDS holds padded input rows
    MODE_POINT = 1,     // 1x1, no padding, NCHW: LDS holds X[c][q] (lanes load pixels)
    MODE_ROWMAJOR = 2,  // h = w = 1 (LinearShift): LDS holds X[c][q] (lanes load features)
};

struct TiledParams {
    int N, C, H, W, K, R, S, sh, sw, ph, pw, OH, OW;
    int OHOW, NQ, HW;
    int Jpad;           // decoded row length (chunks * CC * R * S)
    int VH, IWP;        // padded input height / width (window mode)
    int slots_max;      // LDS rows per channel (window mode)
    int tiles_p, tiles_k, chunks_per_split, nchunks;
    int atomic_out;     // split-K: add partial sums atomically into y
    FastDiv div_ohow, div_ow, div_vh;
};

// acc[i][t] += term(xv[i], d[t]) for one tap j and TN channels.
template <Inner OP, bool SIGNED, int TM, int TN>
__device__ __forceinline__ void sac_step(uint32_t (&acc)[TM][TN], const int32_t (&xv)[TM],
                                         const int32_t *__restrict__ wrow)
{
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int32_t d = wrow[t];
        if constexpr (OP == Inner::Mul) {
#pragma unroll
            for (int i = 0; i < TM; ++i) acc[i][t] += uint32_t(xv[i]) * uint32_t(d);
        } else {
            const uint32_t m = uint32_t(d >> 31);
            const int sh = d & 31;
            if constexpr (SIGNED) {
                const uint32_t z = sh == 31 ? 0u : ~0u;
#pragma unroll
                for (int i = 0; i < TM; ++i) acc[i][t] += (uint32_t(xv[i] >> sh) & z) ^ m;
            } else {
#pragma unroll
                for (int i = 0; i < TM; ++i) acc[i][t] += uint32_t(xv[i] >> sh) ^ m;
            }
        }
    }
}

template <Inner OP, bool SIGNED, int TM, int TN, int CC, int SK>
__device__ __forceinline__ void compute_window(uint32_t (&acc)[TM][TN], const int32_t *lds,
                                               const int (&base)[TM],
                                               const int32_t *__restrict__ wk, int R,
                                               int slots_max, int IWP)
{
    for (int c = 0; c < CC; ++c) {
        for (int r = 0; r < R; ++r) {
            const int rowoff = (c * slots_max + r) * IWP;
            int addr[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i) addr[i] = base[i] + rowoff;
#pragma unroll
            for (int s = 0; s < SK; ++s) {
                int32_t xv[TM];
#pragma unroll
                for (int i = 0; i < TM; ++i) xv[i] = lds[addr[i] + s];
                sac_step<OP, SIGNED, TM, TN>(acc, xv, wk + s * TN);
            }
            wk += SK * TN;
        }
    }
}

template <Inner OP, bool SIGNED, int TM, int TN, int CC, int PL>
__device__ __forceinline__ void compute_point(uint32_t (&acc)[TM][TN], const int32_t *lds,
                                              int lane, const int32_t *__restrict__ wk)
{
#pragma unroll
    for (int c = 0; c < CC; ++c) {
        int32_t xv[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) xv[i] = lds[c * PL + i * 64 + lane];
        sac_step<OP, SIGNED, TM, TN>(acc, xv, wk + c * TN);
    }
}

template <Inner OP, int MODE, int TM, int TN, int CC, int SK>
__global__ void __launch_bounds__(256)
tiled_kernel(const int32_t *__restrict__ x, const int32_t *__restrict__ wd,
             const int32_t *__restrict__ init, int32_t *__restrict__ y, const TiledParams p)
{
    extern __shared__ int32_t lds[];
    __shared__ int sflag[2];
    constexpr int P = 64 * TM;
    constexpr int PL = MODE == MODE_ROWMAJOR ? P + 1 : P;  // odd stride: transposed writes
    const int tid = threadIdx.x, lane = tid & 63;
    // The wave index is the same for all lanes of a wave; saying so lets every
    // quantity derived from it (this wave's channels, its weight rows) live in
    // scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // Block order: consecutive tiles on one XCD (blocks are dealt to the 8 XCDs
    // round-robin) share a pixel tile, so its input stays in that XCD's L2.
    const int G = gridDim.x, b = blockIdx.x;
    const int per = G >> 3, rem = G & 7, xcd = b & 7, loc = b >> 3;
    const int id = xcd < rem ? xcd * (per + 1) + loc : rem * (per + 1) + (xcd - rem) * per + loc;
    const int ct = id % p.tiles_k;
    const int rest = id / p.tiles_k;
    const int pt = rest % p.tiles_p;
    const int z = rest / p.tiles_p;

    const int q0 = pt * P;
    const int kw = ct * 4 * TN + wave * TN;  // first output channel of this wave
    const int32_t *__restrict__ wrow = wd + size_t(kw / TN) * p.Jpad * TN;

    // Per-lane output pixels q = q0 + i*64 + lane.
    int yoff[TM], base[TM], goff[TM];
    int vbase = 0, slots = 0;
    if constexpr (MODE == MODE_WINDOW) {
        const int n0 = fdiv(q0, p.div_ohow);
        const int oh0 = fdiv(q0 - n0 * p.OHOW, p.div_ow);
        vbase = n0 * p.VH + oh0 * p.sh;
        const int ql = min(q0 + P, p.NQ) - 1;
        const int nl = fdiv(ql, p.div_ohow);
        const int ohl = fdiv(ql - nl * p.OHOW, p.div_ow);
        slots = nl * p.VH + ohl * p.sh + p.R - vbase;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int q = q0 + i * 64 + lane;
        yoff[i] = -1;
        base[i] = 0;
        goff[i] = -1;
        if (q < p.NQ) {
            const int n = fdiv(q, p.div_ohow);
            const int pix = q - n * p.OHOW;
            const int oh = fdiv(pix, p.div_ow);
            const int ow = pix - oh * p.OW;
            yoff[i] = n * p.K * p.OHOW + pix;
            if constexpr (MODE == MODE_WINDOW)
                base[i] = (n * p.VH + oh * p.sh - vbase) * p.IWP + ow * p.sw;
            if constexpr (MODE == MODE_POINT)
                goff[i] = n * p.C * p.HW + oh * p.sh * p.W + ow * p.sw;
        }
    }

    uint32_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t) acc[i][t] = 0u;

    const int ch_begin = z * p.chunks_per_split;
    const int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);
    if (tid == 0) sflag[0] = sflag[1] = 0;

    for (int ch = ch_begin; ch < ch_end; ++ch) {
        const int c0 = ch * CC;
        int32_t neg = 0;
        __syncthreads();  // the previous chunk is no longer being read

        if constexpr (MODE == MODE_WINDOW) {
            const int JJ = (p.IWP + 63) >> 6;
            for (int c = 0; c < CC; ++c) {
                const int cc = c0 + c;
                for (int jj = 0; jj < JJ; ++jj) {
                    const int u = lane + 64 * jj;
                    const int iw = u - p.pw;
                    const bool colok = u < p.IWP && iw >= 0 && iw < p.W;
                    for (int s0 = wave; s0 < slots; s0 += 32) {
                        int32_t v[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int slot = s0 + 4 * e;
                            v[e] = 0;
                            if (slot < slots && cc < p.C) {
                                const int vv = vbase + slot;
                                const int n = fdiv(vv, p.div_vh);
                                const int ih = vv - n * p.VH - p.ph;
                                if (ih >= 0 && ih < p.H && colok)
                                    v[e] = x[(n * p.C + cc) * p.HW + ih * p.W + iw];
                            }
                        }
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int slot = s0 + 4 * e;
                            if (slot < slots && u < p.IWP) {
                                lds[(c * p.slots_max + slot) * p.IWP + u] = v[e];
                                neg |= v[e];
                            }
                        }
                    }
                }
            }
        } else if constexpr (MODE == MODE_POINT) {
            constexpr int CW = CC / 4;
            int32_t v[TM][CW];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int cw = 0; cw < CW; ++cw) {
                    const int cc = c0 + wave + 4 * cw;
                    v[i][cw] = (goff[i] >= 0 && cc < p.C) ? x[goff[i] + cc * p.HW] : 0;
                }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int cw = 0; cw < CW; ++cw) {
                    lds[(wave + 4 * cw) * PL + i * 64 + lane] = v[i][cw];
                    neg |= v[i][cw];
                }
        } else {  // MODE_ROWMAJOR: lanes cover CC consecutive features of 64/CC rows
            constexpr int RPW = 64 / CC;        // rows per wave instruction
            constexpr int RR = P / (4 * RPW);   // rounds per thread
            const int cl = lane % CC, rs = lane / CC;
            const int cc = c0 + cl;
            int32_t v[RR];
#pragma unroll
            for (int rr = 0; rr < RR; ++rr) {
                const int q = q0 + rr * 4 * RPW + wave * RPW + rs;
                v[rr] = (q < p.NQ && cc < p.C) ? x[q * p.C + cc] : 0;
            }
#pragma unroll
            for (int rr = 0; rr < RR; ++rr) {
                lds[cl * PL + rr * 4 * RPW + wave * RPW + rs] = v[rr];
                neg |= v[rr];
            }
        }
        if constexpr (OP == Inner::Shift) {
            if (neg < 0) sflag[ch & 1] = 1;  // a negative input in this chunk
        }
        __syncthreads();
        const bool sgn = OP == Inner::Shift && sflag[ch & 1] != 0;
        if (tid == 0) sflag[(ch + 1) & 1] = 0;  // read by nobody until the next barrier

        const int32_t *__restrict__ wk =
            wrow + size_t(c0) * (MODE == MODE_WINDOW ? p.R * SK : 1) * TN;
        if constexpr (MODE == MODE_WINDOW) {
            if (sgn)
                compute_window<OP, true, TM, TN, CC, SK>(acc, lds, base, wk, p.R, p.slots_max, p.IWP);
            else
                compute_window<OP, false, TM, TN, CC, SK>(acc, lds, base, wk, p.R, p.slots_max, p.IWP);
        } else {
            if (sgn)
                compute_point<OP, true, TM, TN, CC, PL>(acc, lds, lane, wk);
            else
                compute_point<OP, false, TM, TN, CC, PL>(acc, lds, lane, wk);
        }
    }

    // Epilogue: y[n][k][pix] for this wave's channels; lanes store consecutive pixels.
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int k = kw + t;
        if (k >= p.K) continue;
        const uint32_t ini = p.atomic_out ? 0u : uint32_t(init[k]);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if (yoff[i] < 0) continue;
            const int o = yoff[i] + k * p.OHOW;
            if (p.atomic_out)
                atomicAdd(reinterpret_cast<unsigned int *>(y) + o, acc[i][t]);
            else
                y[o] = int32_t(acc[i][t] + ini);
        }
    }
}

// ---------------------------------------------------------------------------
// Planning and launch.

constexpr int kTN = 8;          // output channels per wave (scalar weights per tap)
constexpr int kLdsLimit = 64 * 1024;
constexpr int kTargetBlocks = 512;  // at least two workgroups per CU (256 CUs)

template <Inner OP, int MODE, int TM, int TN, int CC, int SK>
static hipError_t launch_tiled(const TiledParams &p, int grid, size_t lds_bytes,
                               const int32_t *x, const int32_t *wd, const int32_t *init,
                               int32_t *y, hipStream_t st)
{
    hipLaunchKernelGGL((tiled_kernel<OP, MODE, TM, TN, CC, SK>), dim3(grid), dim3(256), lds_bytes,
                       st, x, wd, init, y, p);
    return hipGetLastError();
}

struct Variant {
    int mode, tm, cc, sk;
};

template <Inner OP>
static hipError_t dispatch_tiled(const Variant &v, const TiledParams &p, int grid, size_t lds,
                                 const int32_t *x, const int32_t *wd, const int32_t *init,
                                 int32_t *y, hipStream_t st)
{
#define DS_CASE(M, TM, CC, SK)                                                               \
    if (v.mode == M && v.tm == TM && v.cc == CC && v.sk == SK)                               \
        return launch_tiled<OP, M, TM, kTN, CC, SK>(p, grid, lds, x, wd, init, y, st);
    DS_CASE(MODE_ROWMAJOR, 4, 16, 1)
    DS_CASE(MODE_POINT, 8, 8, 1)
    DS_CASE(MODE_WINDOW, 8, 8, 3)
    DS_CASE(MODE_WINDOW, 8, 4, 3)
    DS_CASE(MODE_WINDOW, 8, 2, 3)
    DS_CASE(MODE_WINDOW, 8, 4, 1)
    DS_CASE(MODE_WINDOW, 8, 2, 1)
    DS_CASE(MODE_WINDOW, 8, 4, 2)
    DS_CASE(MODE_WINDOW, 8, 2, 2)
    DS_CASE(MODE_WINDOW, 8, 4, 5)
    DS_CASE(MODE_WINDOW, 8, 2, 5)
    DS_CASE(MODE_WINDOW, 4, 4, 7)
    DS_CASE(MODE_WINDOW, 4, 2, 7)
#undef DS_CASE
    return hipErrorInvalidValue;
}

// Largest LDS row count per channel over all pixel tiles of the window mode.
static int window_slots_max(const ConvGeom &g, int P, int VH)
{
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow, OHOW = int64_t(g.oh) * g.ow;
    int best = 0;
    for (int64_t q0 = 0; q0 < NQ; q0 += P) {
        const int64_t ql = std::min(q0 + P, NQ) - 1;
        const int64_t v0 = (q0 / OHOW) * VH + ((q0 % OHOW) / g.ow) * g.sh;
        const int64_t vl = (ql / OHOW) * VH + ((ql % OHOW) / g.ow) * g.sh + g.r;
        best = int(std::max<int64_t>(best, vl - v0));
    }
    return best;
}

static hipError_t run_direct(const ConvGeom &g, const int32_t *x, const uint32_t *wp,
                             const int32_t *wi, const int32_t *bias, int32_t *y, Inner op,
                             hipStream_t st)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    const int grid = int(std::min<int64_t>((total + 255) / 256, 1 << 20));
    const int wpr = (g.crs + 5) / 6;
    if (op == Inner::Shift)
        hipLaunchKernelGGL(conv_direct_kernel<Inner::Shift>, dim3(grid), dim3(256), 0, st, x, wp,
                           wi, bias, y, g, wpr);
    else
        hipLaunchKernelGGL(conv_direct_kernel<Inner::Mul>, dim3(grid), dim3(256), 0, st, x, wp,
                           wi, bias, y, g, wpr);
    return hipGetLastError();
}

hipError_t run_conv(const ConvGeom &g, const int32_t *x, const uint32_t *wp, const int32_t *wi,
                    const int32_t *bias, int32_t *y, Inner op, hipStream_t st)
{
    const bool rowmajor = g.h == 1 && g.w == 1 && g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0;
    const bool point = !rowmajor && g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0;
    const int VH = g.h + 2 * g.ph, IWP = g.w + 2 * g.pw;

    Variant v{-1, 0, 0, 0};
    int slots_max = 0;
    size_t lds = 0;
    if (rowmajor) {
        v = Variant{MODE_ROWMAJOR, 4, 16, 1};
        lds = size_t(16) * (64 * 4 + 1) * 4;
    } else if (point) {
        v = Variant{MODE_POINT, 8, 8, 1};
        lds = size_t(8) * 64 * 8 * 4;
    } else if (g.s == 1 || g.s == 2 || g.s == 3 || g.s == 5 || g.s == 7) {
        const int tm = g.s == 7 ? 4 : 8;
        slots_max = window_slots_max(g, 64 * tm, VH);
        const int per_c = slots_max * IWP * 4;
        const int cc_opts[3] = {8, 4, 2};
        for (int cc : cc_opts) {
            if (cc == 8 && g.s != 3) continue;
            if (size_t(cc) * per_c <= size_t(kLdsLimit)) {
                v = Variant{MODE_WINDOW, tm, cc, g.s};
                lds = size_t(cc) * per_c;
                break;
            }
        }
    }
    const int fv = forced_variant();
    if (v.mode < 0 || fv == 0) return run_direct(g, x, wp, wi, bias, y, op, st);

    const int P = 64 * v.tm;
    const int RS = g.r * g.s;
    const int nchunks = (g.c + v.cc - 1) / v.cc;
    const int Jpad = nchunks * v.cc * RS;
    const int tiles_k = (g.k + 4 * kTN - 1) / (4 * kTN);
    const int Kpad = tiles_k * 4 * kTN;
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow;
    const int tiles_p = int((NQ + P - 1) / P);
    int splits = 1;
    const int64_t g0 = int64_t(tiles_p) * tiles_k;
    if (g0 < kTargetBlocks) splits = int(std::min<int64_t>(nchunks, (kTargetBlocks + g0 - 1) / g0));
    const int cps = (nchunks + splits - 1) / splits;
    splits = (nchunks + cps - 1) / cps;
    const int64_t grid = g0 * splits;
    if (grid > INT32_MAX) return hipErrorInvalidValue;

    TiledParams p;
    p.N = g.n; p.C = g.c; p.H = g.h; p.W = g.w; p.K = g.k; p.R = g.r; p.S = g.s;
    p.sh = g.sh; p.sw = g.sw; p.ph = g.ph; p.pw = g.pw; p.OH = g.oh; p.OW = g.ow;
    p.OHOW = g.oh * g.ow; p.NQ = int(NQ); p.HW = g.h * g.w;
    p.Jpad = Jpad; p.VH = VH; p.IWP = IWP; p.slots_max = slots_max;
    p.tiles_p = tiles_p; p.tiles_k = tiles_k; p.chunks_per_split = cps; p.nchunks = nchunks;
    p.atomic_out = splits > 1;
    p.div_ohow = make_fastdiv(uint32_t(p.OHOW));
    p.div_ow = make_fastdiv(uint32_t(g.ow));
    p.div_vh = make_fastdiv(uint32_t(VH));

    // Scratch: init[Kpad] then wd[Kpad][Jpad].
    const size_t init_bytes = (size_t(Kpad) * 4 + 255) & ~size_t(255);
    const size_t bytes = init_bytes + size_t(Kpad) * Jpad * 4;
    void *scratch = nullptr;
    hipError_t e = scratch_alloc(&scratch, bytes, st);
    if (e != hipSuccess) return e;
    int32_t *init = static_cast<int32_t *>(scratch);
    int32_t *wd = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) + init_bytes);
    const int wpr = (g.crs + 5) / 6;

    const int64_t pw_total = int64_t(Kpad) * Jpad;
    const int pgrid = int(std::min<int64_t>((pw_total + 255) / 256, 8192));
    if (op == Inner::Shift) {
        hipLaunchKernelGGL((prep_weights_kernel<Inner::Shift, kTN>), dim3(pgrid), dim3(256), 0, st,
                           wp, wi, g.k, g.crs, wpr, Jpad, Kpad, wd);
        hipLaunchKernelGGL(prep_init_kernel<Inner::Shift>, dim3((Kpad + 3) / 4), dim3(256), 0, st,
                           wp, bias, g.k, g.crs, wpr, Kpad, init);
    } else {
        hipLaunchKernelGGL((prep_weights_kernel<Inner::Mul, kTN>), dim3(pgrid), dim3(256), 0, st,
                           wp, wi, g.k, g.crs, wpr, Jpad, Kpad, wd);
        hipLaunchKernelGGL(prep_init_kernel<Inner::Mul>, dim3((Kpad + 3) / 4), dim3(256), 0, st,
                           wp, bias, g.k, g.crs, wpr, Kpad, init);
    }
    e = hipGetLastError();
    if (e == hipSuccess && p.atomic_out) {
        const int64_t total = int64_t(g.n) * g.k * p.OHOW;
        const int fgrid = int(std::min<int64_t>((total + 255) / 256, 8192));
        hipLaunchKernelGGL(fill_init_kernel, dim3(fgrid), dim3(256), 0, st, init, y, total, g.k,
                           p.OHOW);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        e = op == Inner::Shift
                ? dispatch_tiled<Inner::Shift>(v, p, int(grid), lds, x, wd, init, y, st)
                : dispatch_tiled<Inner::Mul>(v, p, int(grid), lds, x, wd, init, y, st);
    }
    const hipError_t ef = hipFreeAsync(scratch, st);
    return e != hipSuccess ? e : ef;
}

}  // namespace ds
