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
#include <cstdio>
#include <cstdlib>
#include <type_traits>

#include "conv_plan.hpp"
#include "fastdiv.hpp"
#include "tuning.hpp"

namespace ds {

int forced_variant() { return tuning(kForceVariant); }

static bool rows_path(const ConvGeom &g, const OutMap &map, const Padded &pad);

// ---------------------------------------------------------------------------
// Scratch memory: stream-ordered allocations from the device's default memory
// pool (hipMallocAsync), freed in stream order (hipFreeAsync) once the call's
// kernels are enqueued. The library keeps no pool and no allocation of its own:
// with the runtime's default release threshold of the default pool, freed
// scratch goes back to the driver at the caller's next synchronisation, and
// calls enqueued back to back reuse it in the meantime.

hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t st)
{
    return hipMallocAsync(p, bytes, st);
}

// ---------------------------------------------------------------------------
// One thread per output element, codes read straight from the packed words.
// Used for shapes the tiled kernel does not cover and as a second opinion in
// the tests.

template <Inner OP>
__global__ void __launch_bounds__(256)
conv_direct_kernel(const int32_t *__restrict__ x, const uint32_t *__restrict__ wp,
                   const int32_t *__restrict__ wi, const int32_t *__restrict__ bias,
                   int32_t *__restrict__ y, ConvGeom g, int wpr, CodeFmt fmt)
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
                        const uint32_t code = fmt.at(wp + int64_t(k) * wpr, j);
                        const int sh = int(code & 15u);
                        if (sh == 15) continue;
                        const uint32_t tv = uint32_t(xv >> sh);
                        acc += (code & 16u) ? 0u - tv : tv;
                    } else if constexpr (OP == Inner::Mul24) {
                        acc += mul24(xv, wi[int64_t(k) * g.crs + j]);
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
// zero weights. init[k] adds back the one that each negative weight's
// complement (x >> s) ^ -1 = -(x >> s) - 1 leaves out.

// One launch, two roles: blocks [0, wblocks) decode weights (grid-stride over
// wd), the remaining blocks compute init, one wave per row k.
template <Inner OP, int TN>
__global__ void __launch_bounds__(256)
prep_kernel(const uint32_t *__restrict__ wp, const int32_t *__restrict__ wi,
            const int32_t *__restrict__ bias, int K, int CRS, int wpr, int Jpad, int Kpad,
            int wblocks, int32_t *__restrict__ wd, int32_t *__restrict__ init, CodeFmt fmt)
{
    if (int(blockIdx.x) < wblocks) {
        const int64_t total = int64_t(Kpad) * Jpad;
        for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
             idx += int64_t(wblocks) * blockDim.x) {
            const int t = int(idx % TN);
            const int64_t rest = idx / TN;
            const int j = int(rest % Jpad);
            const int k = int(rest / Jpad) * TN + t;
            int32_t v;
            if (k < K && j < CRS) {
                if constexpr (OP == Inner::Shift) {
                    const uint32_t code = fmt.at(wp + int64_t(k) * wpr, j);
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
        return;
    }
    // init[k] = bias[k] + negcount[k] (shift) or bias[k] (multiply)
    const int k = (int(blockIdx.x) - wblocks) * 4 + int(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (k >= Kpad) return;
    uint32_t cnt = 0;
    if (OP == Inner::Shift && k < K) {
        const uint32_t *row = wp + int64_t(k) * wpr;
        for (int wdx = lane; wdx < wpr; wdx += 64) {
            for (int j = 0; j < fmt.per_word; ++j) {
                const int col = wdx * fmt.per_word + j;
                if (col >= CRS) break;
                const uint32_t code = fmt.at(row, col);
                cnt += ((code & 16u) && (code & 15u) != 15u) ? 1u : 0u;
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

// The same for fewer than 2^31 elements and a 16-byte aligned y: 32-bit
// multiply-shift division instead of the 64-bit divide (which made the pass three
// times slower than its stores), and four consecutive elements per lane in one
// 16-byte store (a plane boundary may fall between them). The total % 4 last
// elements are written by the first lanes of the grid.
__global__ void __launch_bounds__(256)
fill_init32_kernel(const int32_t *__restrict__ init, int32_t *__restrict__ y, int total,
                   FastDiv div_ohow, FastDiv div_k)
{
    const int quads = total >> 2;
    const int first = int(blockIdx.x) * 256 + int(threadIdx.x);
    auto at = [&](int idx) {
        const int plane = fdiv(idx, div_ohow);
        return init[plane - fdiv(plane, div_k) * int(div_k.d)];
    };
    for (int qd = first; qd < quads; qd += int(gridDim.x) * 256) {
        const int idx = qd * 4;
        reinterpret_cast<int4 *>(y)[qd] = make_int4(at(idx), at(idx + 1), at(idx + 2), at(idx + 3));
    }
    if (first < (total & 3)) y[quads * 4 + first] = at(quads * 4 + first);
}

// y[map(n, k, oh, ow)] = init[k] (0 without init) over a problem's output grid
// (fewer than 2^31 elements; flat index split with multiply-shift division).
__global__ void __launch_bounds__(256)
fill_mapped_kernel(const int32_t *__restrict__ init, int32_t *__restrict__ y, int total,
                   FastDiv div_ow, FastDiv div_oh, FastDiv div_k, OutMap m)
{
    for (int idx = int(blockIdx.x) * 256 + int(threadIdx.x); idx < total; idx += int(gridDim.x) * 256) {
        const int t = fdiv(idx, div_ow), ow = idx - t * int(div_ow.d);
        const int u = fdiv(t, div_oh), oh = t - u * int(div_oh.d);
        const int n = fdiv(u, div_k), k = u - n * int(div_k.d);
        y[m.base + int64_t(n) * m.nstride + int64_t(k) * m.kstride + int64_t(oh) * m.rstride +
          int64_t(ow) * m.cstride] = init ? init[k] : 0;
    }
}

// y[map(n, k, oh, ow)] = src[((n * K + k) * OH + oh) * OW + ow]: a dense result
// scattered into its place (fewer than 2^31 elements).
__global__ void __launch_bounds__(256)
copy_mapped_kernel(const int32_t *__restrict__ src, int32_t *__restrict__ y, int total,
                   FastDiv div_ow, FastDiv div_oh, FastDiv div_k, OutMap m)
{
    for (int idx = int(blockIdx.x) * 256 + int(threadIdx.x); idx < total; idx += int(gridDim.x) * 256) {
        const int t = fdiv(idx, div_ow), ow = idx - t * int(div_ow.d);
        const int u = fdiv(t, div_oh), oh = t - u * int(div_oh.d);
        const int n = fdiv(u, div_k), k = u - n * int(div_k.d);
        y[m.base + int64_t(n) * m.nstride + int64_t(k) * m.kstride + int64_t(oh) * m.rstride +
          int64_t(ow) * m.cstride] = src[idx];
    }
}

// y[0 .. count) = 0, 16 bytes per store (y 16-byte aligned, count a multiple of 4).
__global__ void __launch_bounds__(256) fill_zero_kernel(int4 *__restrict__ y, int64_t count4)
{
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < count4; i += int64_t(gridDim.x) * 256)
        y[i] = make_int4(0, 0, 0, 0);
}

__global__ void __launch_bounds__(256) fill_zero_scalar_kernel(int32_t *__restrict__ y, int64_t count)
{
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < count; i += int64_t(gridDim.x) * 256)
        y[i] = 0;
}

// xp[p][i][j] = x[p][i - ph][j - pw] where that lies inside x, else 0: planes of
// h x w copied into zero-padded planes of xh x xw (which may also crop).
template <typename T>
__global__ void __launch_bounds__(256)
pad_planes_kernel(const T *__restrict__ x, int32_t *__restrict__ xp, int total, int h,
                  int w, int ph, int pw, FastDiv div_xw, FastDiv div_xh)
{
    for (int idx = int(blockIdx.x) * 256 + int(threadIdx.x); idx < total; idx += int(gridDim.x) * 256) {
        const int t = fdiv(idx, div_xw), j = idx - t * int(div_xw.d);
        const int pl = fdiv(t, div_xh), i = t - pl * int(div_xh.d);
        const int ii = i - ph, jj = j - pw;
        xp[idx] = (unsigned(ii) < unsigned(h) && unsigned(jj) < unsigned(w))
                      ? int32_t(x[(int64_t(pl) * h + ii) * w + jj])
                      : 0;
    }
}

// The same into a 16-byte aligned xp: four consecutive elements per lane (a row
// or plane boundary may fall between them) in one 16-byte store; the total % 4
// last elements are written by the first lanes of the grid.
template <typename T>
__global__ void __launch_bounds__(256)
pad_planes4_kernel(const T *__restrict__ x, int32_t *__restrict__ xp, int total, int h, int w,
                   int ph, int pw, FastDiv div_xw, FastDiv div_xh)
{
    auto at = [&](int idx) {
        const int t = fdiv(idx, div_xw), j = idx - t * int(div_xw.d);
        const int pl = fdiv(t, div_xh), i = t - pl * int(div_xh.d);
        const int ii = i - ph, jj = j - pw;
        return (unsigned(ii) < unsigned(h) && unsigned(jj) < unsigned(w))
                   ? int32_t(x[(int64_t(pl) * h + ii) * w + jj])
                   : 0;
    };
    const int quads = total >> 2;
    const int first = int(blockIdx.x) * 256 + int(threadIdx.x);
    for (int qd = first; qd < quads; qd += int(gridDim.x) * 256) {
        const int idx = qd * 4;
        reinterpret_cast<int4 *>(xp)[qd] = make_int4(at(idx), at(idx + 1), at(idx + 2), at(idx + 3));
    }
    if (first < (total & 3)) xp[quads * 4 + first] = at(quads * 4 + first);
}

// The epilogue on one output value v of channel k at flat index o.
__device__ __forceinline__ uint32_t apply_epilogue(uint32_t v, int k, int64_t o, const Epilogue &e)
{
    if (e.mul) {
        const int64_t t = (int64_t(int32_t(v)) * e.mul[k]) >> e.mul_shift;  // arithmetic: floor
        v = uint32_t(t) + (e.add ? uint32_t(e.add[k]) : 0u);
    }
    if (e.res) v += uint32_t(e.res[o]);
    if (e.relu && int32_t(v) < 0) v = 0u;
    return v;
}

// The epilogue as a pass of its own over y [N][K][P], where it cannot run in the
// producing kernel's registers (split-K partial sums, transposed outputs, the
// one-thread-per-output kernel).
__global__ void __launch_bounds__(256)
epilogue_kernel(int32_t *__restrict__ y, int64_t total, int K, int P, const Epilogue e)
{
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int k = int((idx / P) % K);
        y[idx] = int32_t(apply_epilogue(uint32_t(y[idx]), k, idx, e));
    }
}

// xt[c][b] = x[b][c] for a row-major x [rows][cols]: 64 x 64 tiles through LDS,
// so that both the reads and the writes are coalesced.
__global__ void __launch_bounds__(256)
transpose_kernel(const int32_t *__restrict__ x, int32_t *__restrict__ xt, int rows, int cols)
{
    __shared__ int32_t tile[64][65];
    const int tiles_c = (cols + 63) / 64;
    const int c0 = int(blockIdx.x % tiles_c) * 64, r0 = int(blockIdx.x / tiles_c) * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        if (r < rows && c < cols) tile[i][tx] = x[int64_t(r) * cols + c];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int c = c0 + i, r = r0 + tx;
        if (c < cols && r < rows) xt[int64_t(c) * rows + r] = tile[tx][i];
    }
}

// ---------------------------------------------------------------------------
// Tiled kernel.
//
// Staging. Each chunk of CC input channels is copied from HBM straight into
// LDS with buffer loads that write LDS (buffer_load_dword ... lds): one
// instruction moves 64 consecutive LDS words, lane l supplying the word at
// its own global offset. Lanes whose element lies in the zero padding, past
// the last pixel or past the input get an offset beyond the buffer's size,
// and the hardware returns 0 for them; channels past C use a buffer of size
// 0. The LDS holds two chunks: while chunk t is computed, chunk t+1 is in
// flight, and one barrier per chunk hands the buffers over.
//
// Sign check. After its copies land, each wave ORs the words it brought in
// and publishes whether any was negative; the barrier makes the four flags
// visible, and the chunk takes the two-instruction path when all are clear.

enum StageMode : int {
    MODE_WINDOW = 0,  // r x s taps with padding: LDS holds padded input rows of the tile
    MODE_POINT = 1,   // 1x1 taps, no padding: LDS holds X[c][q]; covers LinearShift (h = w = 1)
};

constexpr uint32_t kOOB = 0x80000000u;       // buffer offset past every valid input byte
constexpr int kRsrcWord3 = 0x00020000;       // raw buffer, 32-bit data (gfx9 family)

struct TiledParams {
    int N, C, H, W, K, R, S, sh, sw, ph, pw, OH, OW;
    int OHOW, NQ, HW;
    int Jpad;           // decoded row length (chunks * CC * R * S)
    int VH, IWP;        // padded input height / width (window mode)
    int PLANE;          // LDS words per channel per chunk (window mode, multiple of 64)
    int tiles_p, tiles_k, chunks_per_split, nchunks;
    int atomic_out;     // split-K: add partial sums atomically into y
    int fuse_epi;       // apply the epilogue in the kernel (not split, not transposed)
    // Output placement: y[ybase + n*ynst + k*ykst + oh*yrst + ow*ycst] (see OutMap).
    int ybase, ynst, ykst, yrst, ycst;
    Epilogue epi;
    int x_bytes;        // size of x in bytes (< 2^31)
    FastDiv div_ohow, div_ow, div_vh, div_iwp;
};

typedef __attribute__((address_space(3))) void *lds_ptr_t;

__device__ __forceinline__ void copy_to_lds(__amdgpu_buffer_rsrc_t r, int32_t *dst, uint32_t voff,
                                            uint32_t soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)dst, 4, voff, soff, 0, 0);
}

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
        } else if constexpr (OP == Inner::Mul24) {
#pragma unroll
            for (int i = 0; i < TM; ++i) acc[i][t] += mul24(xv[i], d);
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
__device__ __forceinline__ void compute_window(uint32_t (&acc)[TM][TN], const int32_t *buf,
                                               const int (&base)[TM],
                                               const int32_t *__restrict__ wk, int R, int PLANE,
                                               int IWP)
{
    for (int c = 0; c < CC; ++c) {
        for (int r = 0; r < R; ++r) {
            const int rowoff = c * PLANE + r * IWP;
            int addr[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i) addr[i] = base[i] + rowoff;
#pragma unroll
            for (int s = 0; s < SK; ++s) {
                int32_t xv[TM];
#pragma unroll
                for (int i = 0; i < TM; ++i) xv[i] = buf[addr[i] + s];
                sac_step<OP, SIGNED, TM, TN>(acc, xv, wk + s * TN);
            }
            wk += SK * TN;
        }
    }
}

template <Inner OP, bool SIGNED, int TM, int TN, int CC>
__device__ __forceinline__ void compute_point(uint32_t (&acc)[TM][TN], const int32_t *buf,
                                              int lane, const int32_t *__restrict__ wk)
{
    constexpr int P = 64 * TM;
#pragma unroll
    for (int c = 0; c < CC; ++c) {
        int32_t xv[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) xv[i] = buf[c * P + i * 64 + lane];
        sac_step<OP, SIGNED, TM, TN>(acc, xv, wk + c * TN);
    }
}

// GW: copy segments (64 LDS words) per wave and channel, window mode.
template <Inner OP, int MODE, int TM, int TN, int CC, int SK, int GW>
__global__ void __launch_bounds__(256)
tiled_kernel(const int32_t *__restrict__ x, const int32_t *__restrict__ wd,
             const int32_t *__restrict__ init, int32_t *__restrict__ y, const TiledParams p)
{
    extern __shared__ int32_t lds[];
    __shared__ int neg_flag[2][4];
    constexpr int P = 64 * TM;
    constexpr int NV = MODE == MODE_WINDOW ? GW : TM;   // staging offsets per lane
    const int tid = threadIdx.x, lane = tid & 63;
    // The wave index is the same for all lanes of a wave; saying so lets every
    // quantity derived from it (this wave's channels, its weight rows, its copy
    // segments) live in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int BUF = MODE == MODE_WINDOW ? CC * p.PLANE : CC * P;

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

    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(x), short(0), p.x_bytes, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t zr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(x), short(0), 0, kRsrcWord3);

    // Per-lane output pixels q = q0 + i*64 + lane, and the staging offsets.
    int yoff[TM], base[TM];
    uint32_t voff[NV];
    int vbase = 0, nseg = 0;
    if constexpr (MODE == MODE_WINDOW) {
        const int n0 = fdiv(q0, p.div_ohow);
        const int oh0 = fdiv(q0 - n0 * p.OHOW, p.div_ow);
        vbase = n0 * p.VH + oh0 * p.sh;
        const int ql = min(q0 + P, p.NQ) - 1;
        const int nl = fdiv(ql, p.div_ohow);
        const int ohl = fdiv(ql - nl * p.OHOW, p.div_ow);
        const int live = (nl * p.VH + ohl * p.sh + p.R - vbase) * p.IWP;  // words per channel
        nseg = (live + 63) >> 6;
#pragma unroll
        for (int g = 0; g < GW; ++g) {
            const int e = (wave + 4 * g) * 64 + lane;
            voff[g] = kOOB;
            if (e < live) {
                const int slot = fdiv(e, p.div_iwp);
                const int iw = e - slot * p.IWP - p.pw;
                const int vv = vbase + slot;
                const int n = fdiv(vv, p.div_vh);
                const int ih = vv - n * p.VH - p.ph;
                if (ih >= 0 && ih < p.H && iw >= 0 && iw < p.W)
                    voff[g] = uint32_t(((n * p.C) * p.HW + ih * p.W + iw) * 4);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int q = q0 + i * 64 + lane;
        yoff[i] = -1;
        base[i] = 0;
        if constexpr (MODE == MODE_POINT) voff[i] = kOOB;
        if (q < p.NQ) {
            const int n = fdiv(q, p.div_ohow);
            const int pix = q - n * p.OHOW;
            const int oh = fdiv(pix, p.div_ow);
            const int ow = pix - oh * p.OW;
            yoff[i] = p.ybase + n * p.ynst + oh * p.yrst + ow * p.ycst;
            if constexpr (MODE == MODE_WINDOW)
                base[i] = (n * p.VH + oh * p.sh - vbase) * p.IWP + ow * p.sw;
            if constexpr (MODE == MODE_POINT)
                voff[i] = uint32_t((n * p.C * p.HW + oh * p.sh * p.W + ow * p.sw) * 4);
        }
    }

    // Copies of one chunk into LDS buffer `bf`: this wave's share.
    auto issue = [&](int ch, int bf) {
        int32_t *dst = lds + bf * BUF;
        if constexpr (MODE == MODE_WINDOW) {
            for (int c = 0; c < CC; ++c) {
                const int cc = ch * CC + c;
                const __amdgpu_buffer_rsrc_t r = cc < p.C ? xr : zr;
                const uint32_t soff = cc < p.C ? uint32_t(cc * p.HW * 4) : 0u;
#pragma unroll
                for (int g = 0; g < GW; ++g) {
                    const int seg = wave + 4 * g;
                    if (seg < nseg) copy_to_lds(r, dst + c * p.PLANE + seg * 64, voff[g], soff);
                }
            }
        } else {
#pragma unroll
            for (int cw = 0; cw < CC / 4; ++cw) {
                const int c = wave + 4 * cw;
                const int cc = ch * CC + c;
                const __amdgpu_buffer_rsrc_t r = cc < p.C ? xr : zr;
                const uint32_t soff = cc < p.C ? uint32_t(cc * p.HW * 4) : 0u;
#pragma unroll
                for (int i = 0; i < TM; ++i) copy_to_lds(r, dst + c * P + i * 64, voff[i], soff);
            }
        }
    };
    // Wait for this wave's copies into buffer `bf`; with `publish`, also tell the
    // other waves whether any word it brought in is negative.
    auto land = [&](int bf, bool publish) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (!publish) return;
        const int32_t *src = lds + bf * BUF;
        int32_t o = 0;
        if constexpr (MODE == MODE_WINDOW) {
            for (int c = 0; c < CC; ++c)
#pragma unroll
                for (int g = 0; g < GW; ++g) {
                    const int seg = wave + 4 * g;
                    if (seg < nseg) o |= src[c * p.PLANE + seg * 64 + lane];
                }
        } else {
#pragma unroll
            for (int cw = 0; cw < CC / 4; ++cw)
#pragma unroll
                for (int i = 0; i < TM; ++i) o |= src[(wave + 4 * cw) * P + i * 64 + lane];
        }
        const bool any = __any(o < 0);
        if (lane == 0) neg_flag[bf][wave] = any ? 1 : 0;
    };

    uint32_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t) acc[i][t] = 0u;

    auto compute = [&](auto signed_tag, int ch, int bf) {
        constexpr bool SG = decltype(signed_tag)::value;
        const int32_t *buf = lds + bf * BUF;
        const int32_t *__restrict__ wk =
            wrow + size_t(ch * CC) * (MODE == MODE_WINDOW ? p.R * SK : 1) * TN;
        if constexpr (MODE == MODE_WINDOW)
            compute_window<OP, SG, TM, TN, CC, SK>(acc, buf, base, wk, p.R, p.PLANE, p.IWP);
        else
            compute_point<OP, SG, TM, TN, CC>(acc, buf, lane, wk);
    };

    const int ch_begin = z * p.chunks_per_split;
    const int ch_end = min(p.nchunks, ch_begin + p.chunks_per_split);
    constexpr bool SHIFT = OP == Inner::Shift;

    // Two phases, so that neither chunk loop chooses between compute paths:
    // chunks take the two-instruction form until one holds a negative input,
    // and every chunk from there on takes the three-instruction form.
    issue(ch_begin, 0);
    land(0, SHIFT);
    __syncthreads();
    int ch = ch_begin;
    if constexpr (SHIFT) {
        for (; ch < ch_end; ++ch) {
            const int bf = (ch - ch_begin) & 1;
            if (neg_flag[bf][0] | neg_flag[bf][1] | neg_flag[bf][2] | neg_flag[bf][3]) break;
            const bool more = ch + 1 < ch_end;
            if (more) issue(ch + 1, bf ^ 1);
            compute(std::false_type{}, ch, bf);
            if (more) land(bf ^ 1, true);
            __syncthreads();
        }
    }
    for (; ch < ch_end; ++ch) {
        const int bf = (ch - ch_begin) & 1;
        const bool more = ch + 1 < ch_end;
        if (more) issue(ch + 1, bf ^ 1);
        compute(std::integral_constant<bool, SHIFT>{}, ch, bf);
        if (more) land(bf ^ 1, false);
        __syncthreads();
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
            const int o = yoff[i] + k * p.ykst;
            if (p.atomic_out)
                atomicAdd(reinterpret_cast<unsigned int *>(y) + o, acc[i][t]);
            else if (p.fuse_epi)
                y[o] = int32_t(apply_epilogue(acc[i][t] + ini, k, o, p.epi));
            else
                y[o] = int32_t(acc[i][t] + ini);
        }
    }
}

// ---------------------------------------------------------------------------
// Planning and launch.

constexpr int kTN = 8;              // output channels per wave (scalar weights per tap)
constexpr int kLdsLimit = 64 * 1024;
constexpr int kFullGrid = 3000;     // workgroups that keep 256 CUs busy without a split
constexpr int kSplitGrid = 4096;    // workgroups to aim for when splitting (16 per CU)

struct Variant {
    int mode, tm, cc, sk, gw;
};

// The compiled instances. Window mode: GW copy segments per wave cover planes of
// up to 4*GW*64 words per channel.
static const Variant kVariants[] = {
    {MODE_POINT, 8, 8, 1, 0},  {MODE_POINT, 4, 8, 1, 0},
    {MODE_WINDOW, 8, 4, 3, 8}, {MODE_WINDOW, 8, 2, 3, 8}, {MODE_WINDOW, 4, 4, 3, 8},
    {MODE_WINDOW, 4, 2, 3, 8}, {MODE_WINDOW, 4, 1, 3, 16},
    {MODE_WINDOW, 4, 2, 7, 24}, {MODE_WINDOW, 4, 1, 7, 24},
    {MODE_WINDOW, 4, 2, 1, 16}, {MODE_WINDOW, 4, 2, 2, 16}, {MODE_WINDOW, 4, 2, 5, 16},
    {MODE_WINDOW, 4, 1, 5, 24},
    // 4 taps per row: the 4-tap stride phases of a 7 x 7 / 2 layer's input gradient
    {MODE_WINDOW, 4, 2, 4, 16}, {MODE_WINDOW, 4, 1, 4, 24},
};

template <Inner OP, int MODE, int TM, int CC, int SK, int GW>
static hipError_t launch_tiled(const TiledParams &p, int grid, size_t lds, const int32_t *x,
                               const int32_t *wd, const int32_t *init, int32_t *y, hipStream_t st)
{
    hipLaunchKernelGGL((tiled_kernel<OP, MODE, TM, kTN, CC, SK, GW>), dim3(grid), dim3(256), lds,
                       st, x, wd, init, y, p);
    return hipGetLastError();
}

template <Inner OP>
static hipError_t dispatch_tiled(const Variant &v, const TiledParams &p, int grid, size_t lds,
                                 const int32_t *x, const int32_t *wd, const int32_t *init,
                                 int32_t *y, hipStream_t st)
{
#define DS_CASE(M, TM, CC, SK, GW)                                                           \
    if (v.mode == M && v.tm == TM && v.cc == CC && v.sk == SK && v.gw == GW)                 \
        return launch_tiled<OP, M, TM, CC, SK, GW>(p, grid, lds, x, wd, init, y, st);
    DS_CASE(MODE_POINT, 8, 8, 1, 0)
    DS_CASE(MODE_POINT, 4, 8, 1, 0)
    DS_CASE(MODE_WINDOW, 8, 4, 3, 8)
    DS_CASE(MODE_WINDOW, 8, 2, 3, 8)
    DS_CASE(MODE_WINDOW, 4, 4, 3, 8)
    DS_CASE(MODE_WINDOW, 4, 2, 3, 8)
    DS_CASE(MODE_WINDOW, 4, 1, 3, 16)
    DS_CASE(MODE_WINDOW, 4, 2, 7, 24)
    DS_CASE(MODE_WINDOW, 4, 1, 7, 24)
    DS_CASE(MODE_WINDOW, 4, 2, 1, 16)
    DS_CASE(MODE_WINDOW, 4, 2, 2, 16)
    DS_CASE(MODE_WINDOW, 4, 2, 5, 16)
    DS_CASE(MODE_WINDOW, 4, 1, 5, 24)
    DS_CASE(MODE_WINDOW, 4, 2, 4, 16)
    DS_CASE(MODE_WINDOW, 4, 1, 4, 24)
#undef DS_CASE
    return hipErrorInvalidValue;
}

// Largest number of padded input rows (per channel) any pixel tile of P
// output pixels needs in window mode.
static int window_rows_max(const ConvGeom &g, int P, int VH)
{
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow, OHOW = int64_t(g.oh) * g.ow;
    int64_t best = 0;
    for (int64_t q0 = 0; q0 < NQ; q0 += P) {
        const int64_t ql = std::min(q0 + P, NQ) - 1;
        const int64_t v0 = (q0 / OHOW) * VH + ((q0 % OHOW) / g.ow) * g.sh;
        const int64_t vl = (ql / OHOW) * VH + ((ql % OHOW) / g.ow) * g.sh + g.r;
        best = std::max(best, vl - v0);
    }
    return int(best);
}

static hipError_t run_direct(const ConvGeom &g, const int32_t *x, const uint32_t *wp,
                             const int32_t *wi, const int32_t *bias, int32_t *y, Inner op,
                             hipStream_t st)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    const int grid = int(std::min<int64_t>((total + 255) / 256, 1 << 20));
    const int wpr = int(row_words_bits(g.crs, g.bits));
    if (op == Inner::Shift)
        hipLaunchKernelGGL(conv_direct_kernel<Inner::Shift>, dim3(grid), dim3(256), 0, st, x, wp,
                           wi, bias, y, g, wpr, code_fmt(g.bits));
    else if (op == Inner::Mul)
        hipLaunchKernelGGL(conv_direct_kernel<Inner::Mul>, dim3(grid), dim3(256), 0, st, x, wp,
                           wi, bias, y, g, wpr, code_fmt(g.bits));
    else
        hipLaunchKernelGGL(conv_direct_kernel<Inner::Mul24>, dim3(grid), dim3(256), 0, st, x, wp,
                           wi, bias, y, g, wpr, code_fmt(g.bits));
    return hipGetLastError();
}

// Padded input extents of the window mode for g.
static void padded_dims(const ConvGeom &g, const Padded &pad, int &VH, int &IWP)
{
    VH = pad.vh > 0 ? pad.vh : g.h + 2 * g.ph;
    IWP = pad.iwp > 0 ? pad.iwp : g.w + 2 * g.pw;
}

// Picks the tiled instance for a problem: v.mode < 0 when none fits.
static Variant choose_variant(const ConvGeom &g, const Padded &pad, int &plane, size_t &lds)
{
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow;
    // Pointwise staging reads input pixel (oh*sh, ow*sw) with no bounds check of its
    // own, so the output grid must stay inside the input (always so for a 1x1
    // window without padding and the usual output size).
    const bool point = g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0 &&
                       g.oh <= (g.h - 1) / g.sh + 1 && g.ow <= (g.w - 1) / g.sw + 1 &&
                       pad.vh <= 0 && pad.iwp <= 0;
    plane = 0;
    lds = 0;
    const int fv = forced_variant();
    if (point) {
        const int tm = fv == 8 && NQ > 256 ? 8 : 4;
        lds = size_t(2) * 8 * 64 * tm * 4;
        return Variant{MODE_POINT, tm, 8, 1, 0};
    }
    int VH = 0, IWP = 0;
    padded_dims(g, pad, VH, IWP);
    const int order[2][2] = {{4, 8}, {8, 4}};
    for (int tm : order[fv == 8 ? 1 : 0]) {
        const int rows = window_rows_max(g, 64 * tm, VH);
        const int64_t live = int64_t(rows) * IWP;
        const int pl = int((live + 63) / 64 * 64);
        // Among the instances that fit, take the one that pads the fewest input
        // channels up to whole chunks, then the largest chunk; prefer leaving LDS
        // room for several workgroups per CU.
        for (int budget : {48 * 1024, kLdsLimit}) {
            const Variant *best = nullptr;
            int best_pad = 0;
            for (const Variant &v : kVariants) {
                if (v.mode != MODE_WINDOW || v.tm != tm || v.sk != g.s) continue;
                if (live > int64_t(4) * v.gw * 64) continue;
                if (size_t(2) * v.cc * pl * 4 > size_t(budget)) continue;
                const int pad = (g.c + v.cc - 1) / v.cc * v.cc - g.c;
                if (!best || pad < best_pad || (pad == best_pad && v.cc > best->cc)) {
                    best = &v;
                    best_pad = pad;
                }
            }
            if (best) {
                plane = pl;
                lds = size_t(2) * best->cc * pl * 4;
                return *best;
            }
        }
    }
    return Variant{-1, 0, 0, 0, 0};
}

// Split-K factor and chunks per split for a tiled launch.
static void plan_splits(const ConvGeom &g, const Variant &v, int &tiles_p, int &tiles_k,
                        int &nchunks, int &splits, int &cps)
{
    const int P = 64 * v.tm;
    nchunks = (g.c + v.cc - 1) / v.cc;
    tiles_k = (g.k + 4 * kTN - 1) / (4 * kTN);
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow;
    tiles_p = int((NQ + P - 1) / P);
    // Split the reduction when the tiles alone are too few to keep every CU at
    // full residency for most of the kernel (measured on MI355X: grids of
    // fewer than ~3000 workgroups lose 10-30 %; about 16 workgroups per CU
    // recovers it), keeping at least four chunks per split unless the grid is
    // so small that latency, not throughput, decides.
    const int64_t g0 = int64_t(tiles_p) * tiles_k;
    splits = 1;
    if (g0 < kFullGrid) {
        const int64_t want = (kSplitGrid + g0 - 1) / g0;
        const int64_t cap = g0 >= 64 ? nchunks / 4 : nchunks;  // tiny grids: any split
        splits = int(std::max<int64_t>(1, std::min<int64_t>(want, cap)));
    }
    cps = (nchunks + splits - 1) / splits;
    splits = (nchunks + cps - 1) / cps;
}

static bool use_direct(const ConvGeom &g, const Variant &v)
{
    const int64_t x_bytes = int64_t(g.n) * g.c * g.h * g.w * 4;
    return v.mode < 0 || x_bytes >= (int64_t(1) << 31) || forced_variant() == 0;
}

bool tiled_fits(const ConvGeom &g, const Padded &pad)
{
    int plane = 0;
    size_t lds = 0;
    const Variant v = choose_variant(g, pad, plane, lds);
    return !use_direct(g, v);
}

// A problem on 1 x 1 inputs with 1 x 1 taps (LinearShift, x [n][c]) runs on the
// transposed input x^T [c][n] as one image of width n, so that the copies into
// LDS read consecutive words, and produces y^T [k][n], whose stores (and
// split-K atomics) are consecutive too; a transpose then gives y [n][k].
static ConvGeom tiled_geometry(const ConvGeom &g, bool &rowmajor)
{
    rowmajor = g.h == 1 && g.w == 1 && g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0;
    if (!rowmajor) return g;
    ConvGeom t = g;
    t.n = 1;
    t.h = 1;
    t.w = g.n;
    t.sh = t.sw = 1;
    t.oh = 1;
    t.ow = g.n;
    return t;
}

void describe_conv(const ConvGeom &g0, char *buf, size_t len)
{
    if (rows_path(g0, OutMap(), Padded())) {
        snprintf(buf, len, "rows");
        return;
    }
    bool rowmajor = false;
    const ConvGeom g = tiled_geometry(g0, rowmajor);
    int plane = 0;
    size_t lds = 0;
    const Variant v = choose_variant(g, Padded(), plane, lds);
    if (use_direct(g, v)) {
        snprintf(buf, len, "direct");
        return;
    }
    int tiles_p, tiles_k, nchunks, splits, cps;
    plan_splits(g, v, tiles_p, tiles_k, nchunks, splits, cps);
    if (v.mode == MODE_POINT)
        snprintf(buf, len, "tiled point%s tm%d cc%d splits%d", rowmajor ? " transposed" : "", v.tm,
                 v.cc, splits);
    else
        snprintf(buf, len, "tiled window tm%d cc%d s%d gw%d splits%d", v.tm, v.cc, v.sk, v.gw,
                 splits);
}

// The epilogue as its own pass over y (see epilogue_kernel).
hipError_t run_fill_init(const ConvGeom &g, const int32_t *init, int32_t *y, hipStream_t st)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    if (total <= 0) return hipSuccess;
    if (total <= INT32_MAX && reinterpret_cast<uintptr_t>(y) % 16 == 0) {
        const int grid = int(std::min<int64_t>((total / 4 + 255) / 256, 4096));
        hipLaunchKernelGGL(fill_init32_kernel, dim3(std::max(grid, 1)), dim3(256), 0, st, init, y,
                           int(total), make_fastdiv(uint32_t(g.oh * g.ow)), make_fastdiv(uint32_t(g.k)));
    } else {
        const int grid = int(std::min<int64_t>((total + 255) / 256, 8192));
        hipLaunchKernelGGL(fill_init_kernel, dim3(grid), dim3(256), 0, st, init, y, total, g.k,
                           g.oh * g.ow);
    }
    return hipGetLastError();
}

hipError_t run_fill_mapped(const ConvGeom &g, const int32_t *init, int32_t *y, const OutMap &map,
                           hipStream_t st)
{
    if (map.dense() && init) return run_fill_init(g, init, y, st);
    OutMap m = map;
    if (m.dense()) {
        m.kstride = g.oh * g.ow;
        m.nstride = g.k * m.kstride;
        m.rstride = g.ow;
        m.cstride = 1;
    }
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    if (total <= 0) return hipSuccess;
    if (total > INT32_MAX) return hipErrorInvalidValue;
    const int grid = int(std::min<int64_t>((total + 255) / 256, 8192));
    hipLaunchKernelGGL(fill_mapped_kernel, dim3(grid), dim3(256), 0, st, init, y, int(total),
                       make_fastdiv(uint32_t(g.ow)), make_fastdiv(uint32_t(g.oh)),
                       make_fastdiv(uint32_t(g.k)), m);
    return hipGetLastError();
}

hipError_t run_copy_mapped(const ConvGeom &g, const int32_t *src, int32_t *y, const OutMap &map,
                           hipStream_t st)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    if (total <= 0) return hipSuccess;
    if (total > INT32_MAX || map.dense()) return hipErrorInvalidValue;
    const int grid = int(std::min<int64_t>((total + 255) / 256, 8192));
    hipLaunchKernelGGL(copy_mapped_kernel, dim3(grid), dim3(256), 0, st, src, y, int(total),
                       make_fastdiv(uint32_t(g.ow)), make_fastdiv(uint32_t(g.oh)),
                       make_fastdiv(uint32_t(g.k)), map);
    return hipGetLastError();
}

hipError_t run_fill_zero(int32_t *y, int64_t count, hipStream_t st)
{
    if (count <= 0) return hipSuccess;
    // The 16-byte-aligned body in vector stores, the few elements around it one by one.
    const int64_t head = std::min<int64_t>(count, ((16 - int64_t(reinterpret_cast<uintptr_t>(y) & 15)) & 15) / 4);
    const int64_t body4 = (count - head) / 4;
    const int64_t tail = count - head - body4 * 4;
    if (reinterpret_cast<uintptr_t>(y) & 3) return hipErrorInvalidValue;
    if (head)
        hipLaunchKernelGGL(fill_zero_scalar_kernel, dim3(1), dim3(256), 0, st, y, head);
    if (body4)
        hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned(std::min<int64_t>((body4 + 255) / 256, 8192))),
                           dim3(256), 0, st, reinterpret_cast<int4 *>(y + head), body4);
    if (tail)
        hipLaunchKernelGGL(fill_zero_scalar_kernel, dim3(1), dim3(256), 0, st, y + head + body4 * 4, tail);
    return hipGetLastError();
}

hipError_t run_pad_planes(const void *x, int32_t *xp, int64_t planes, int h, int w, int ph,
                          int pw, int xh, int xw, hipStream_t st, int xbytes)
{
    const int64_t total = planes * xh * xw;
    if (total <= 0) return hipSuccess;
    if (total > INT32_MAX || h <= 0 || w <= 0) return hipErrorInvalidValue;
    const FastDiv dxw = make_fastdiv(uint32_t(xw)), dxh = make_fastdiv(uint32_t(xh));
    if (reinterpret_cast<uintptr_t>(xp) % 16 == 0) {
        const int grid = std::max(1, int(std::min<int64_t>((total / 4 + 255) / 256, 4096)));
        if (xbytes == 2)
            hipLaunchKernelGGL(pad_planes4_kernel<int16_t>, dim3(grid), dim3(256), 0, st,
                               static_cast<const int16_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
        else if (xbytes == 1)
            hipLaunchKernelGGL(pad_planes4_kernel<int8_t>, dim3(grid), dim3(256), 0, st,
                               static_cast<const int8_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
        else
            hipLaunchKernelGGL(pad_planes4_kernel<int32_t>, dim3(grid), dim3(256), 0, st,
                               static_cast<const int32_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
        return hipGetLastError();
    }
    const int grid = int(std::min<int64_t>((total + 255) / 256, 8192));
    if (xbytes == 2)
        hipLaunchKernelGGL(pad_planes_kernel<int16_t>, dim3(grid), dim3(256), 0, st,
                           static_cast<const int16_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
    else if (xbytes == 1)
        hipLaunchKernelGGL(pad_planes_kernel<int8_t>, dim3(grid), dim3(256), 0, st,
                           static_cast<const int8_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
    else
        hipLaunchKernelGGL(pad_planes_kernel<int32_t>, dim3(grid), dim3(256), 0, st,
                           static_cast<const int32_t *>(x), xp, int(total), h, w, ph, pw, dxw, dxh);
    return hipGetLastError();
}

hipError_t run_epilogue(const ConvGeom &g, int32_t *y, const Epilogue &epi, hipStream_t st)
{
    const int64_t total = int64_t(g.n) * g.k * g.oh * g.ow;
    const int grid = int(std::min<int64_t>((total + 255) / 256, 8192));
    hipLaunchKernelGGL(epilogue_kernel, dim3(grid), dim3(256), 0, st, y, total, g.k, g.oh * g.ow,
                       epi);
    return hipGetLastError();
}

// Everything run_conv decides for a problem before it enqueues work: the kernel,
// the split of the reduction and the scratch the call needs. Shared by run_conv
// and conv_scratch_bytes, so that a caller-supplied workspace is sized exactly
// as the launch uses it.
struct ConvLayout {
    ConvGeom g;           // the problem the tiled kernel sees (x^T for row-major inputs)
    bool mapped = false, rowmajor = false, direct = false, via_dense = false;
    Variant v{};
    int plane = 0;
    size_t lds = 0;
    int tiles_p = 0, tiles_k = 0, nchunks = 0, splits = 0, cps = 0, Jpad = 0, Kpad = 0;
    int64_t grid = 0;
    size_t init_bytes = 0, wd_bytes = 0, xt_bytes = 0, yt_bytes = 0;
    size_t scratch_bytes() const { return init_bytes + wd_bytes + xt_bytes + yt_bytes; }
};

// ---------------------------------------------------------------------------
// Small-batch LinearShift (a 1 x 1 problem on 1 x 1 inputs with fewer than 256
// rows): lanes own output channels instead of batch rows, so that a few rows do
// not leave the tiled kernel's 256-row tiles almost empty (at batch 1 it uses
// one lane in 256). A workgroup of 16 waves covers 64 output channels and up to
// 8 batch rows; its waves split the reduction into 16 contiguous ranges of
// packed words and add their partial sums in LDS. Each lane decodes its own
// channel's codes (a 64-byte line of its row holds 96 five-bit codes) and reads
// the inputs as wave-uniform scalars. Per term: the shifted input, masked to 0
// for a zero weight, xor'ed with the sign mask and added; the +1 that turns
// ~t into -t is added once per negative weight as a count. The multiplication
// operators run in the same tiling with int32 weights (the comparison kernel).
constexpr int kRowsWaves = 16;

struct RowsArgs {
    const uint32_t *wp;   // packed codes [K][wpr] (Shift)
    const int32_t *wi;    // int32 weights [K][C] (Mul, Mul24)
    const int32_t *bias;  // [K] or NULL
    int32_t *y;           // [B][K]
    int B, C, K, wpr;
    Epilogue epi;
};

// ROWS batch rows per workgroup (1, 2, 4 or 8: the smallest power of two that
// covers the batch, up to 8); BITS-bit codes, 32 / BITS per word. Rows past
// the batch read the last row again and are not stored, so the inner loops have
// no branch; inputs past the last column are read at the last column, under
// zero codes (packed rows are padded with them). The reduction runs in chunks
// of 8 packed words: each lane loads its row's 8 words and the wave stages the
// chunk's inputs of its ROWS rows in LDS (coalesced loads, all issued
// together), then reads them back as broadcasts. gridDim.z > 1 splits the
// reduction over that many workgroups per block of channels and rows, whose
// sums meet in y through int32 atomics after a fill pass (no epilogue then).
constexpr int kRowsWords = 8;

template <Inner OP, int ROWS, int BITS>
__global__ void __launch_bounds__(1024)
linear_rows_kernel(const int32_t *__restrict__ x, const RowsArgs a)
{
    constexpr int PER = OP == Inner::Shift ? 32 / BITS : 1;  // reduction columns per unit
    constexpr int U = OP == Inner::Shift ? kRowsWords : 64;  // units per chunk
    constexpr int E = U * PER;                               // columns per chunk
    __shared__ uint32_t part[kRowsWaves][ROWS][64];
    __shared__ int32_t xbuf[kRowsWaves][ROWS][E];
    // A chunk's packed words of the wave's 64 weight rows, loaded 8 rows of U
    // consecutive words per instruction (lanes U words apart would touch 64 cache
    // lines per load) and read back row by row (odd row pitch: no bank conflicts).
    __shared__ uint32_t wbuf[OP == Inner::Shift ? kRowsWaves : 1][64][U + 1];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int k = int(blockIdx.x) * 64 + lane;
    const int kc = min(k, a.K - 1);  // lanes past K compute a copy of the last channel, not stored
    const int b0 = int(blockIdx.y) * ROWS;
    const int nb = min(ROWS, a.B - b0);
    const int nsplit = int(gridDim.z), part_i = int(blockIdx.z);
    uint32_t acc[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) acc[r] = 0u;
    uint32_t ncount = 0u;
    // This wave's share [u0, u1) of the units (packed words, or input columns for
    // the multiplication operators): part part_i of nsplit, then 1/16 of it.
    const int units = OP == Inner::Shift ? a.wpr : a.C;
    const int p0 = int(int64_t(units) * part_i / nsplit), p1 = int(int64_t(units) * (part_i + 1) / nsplit);
    const int u0 = p0 + int(int64_t(p1 - p0) * wave / kRowsWaves);
    const int u1 = p0 + int(int64_t(p1 - p0) * (wave + 1) / kRowsWaves);
    const CodeFmt fmt{BITS, 32 / BITS};
    if constexpr (OP == Inner::Shift) {
        // Each chunk's weight words and inputs are loaded into registers, then
        // staged through LDS: the weight words 8 rows of U consecutive words per
        // load instruction (lanes U words apart would touch 64 cache lines per
        // load), read back row by row. With one batch row per workgroup (the least
        // arithmetic per load) they are loaded one chunk ahead, so that their
        // latency overlaps the previous chunk's arithmetic: on MI355X 25088 ->
        // 4096 at batch 1 ran in 41.6 instead of 45.9 us, while the multi-row
        // tilings ran 1-4 % slower that way (fewer waves fit their registers).
        constexpr bool kAhead = ROWS == 1;
        constexpr int XE = (E + 63) / 64;  // input columns per lane and row
        uint32_t nw[U];
        int32_t nx[ROWS][XE];
        auto fetch = [&](int uc) {
#pragma unroll
            for (int i = 0; i < U; ++i) {
                const int e = i * 64 + lane, rr = e / U, ww = e % U;
                const int kr = min(int(blockIdx.x) * 64 + rr, a.K - 1);
                nw[i] = a.wp[int64_t(kr) * a.wpr + min(uc + ww, u1 - 1)];
            }
            const int cb = uc * PER;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int32_t *xrow = x + int64_t(b0 + min(r, nb - 1)) * a.C;
#pragma unroll
                for (int t = 0; t < XE; ++t) {
                    const int e = lane + 64 * t;
                    if (e < E) nx[r][t] = xrow[min(cb + e, a.C - 1)];
                }
            }
        };
        if (kAhead && u0 < u1) fetch(u0);
        for (int uc = u0; uc < u1; uc += U) {
            if (!kAhead) fetch(uc);
#pragma unroll
            for (int i = 0; i < U; ++i) {
                const int e = i * 64 + lane;
                wbuf[wave][e / U][e % U] = nw[i];
            }
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int t = 0; t < XE; ++t)
                    if (lane + 64 * t < E) xbuf[wave][r][lane + 64 * t] = nx[r][t];
            // Written and read back by the same wave, whose LDS accesses run in
            // order; the wave barrier keeps the compiler from moving the reads up.
            __builtin_amdgcn_wave_barrier();
            uint32_t wv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) wv[u] = wbuf[wave][lane][u];
            if (kAhead && uc + U < u1) fetch(uc + U);
            const int un = min(U, u1 - uc);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (u >= un) break;
#pragma unroll
                for (int j = 0; j < PER; ++j) {
                    const uint32_t code = fmt.canonical((wv[u] >> (BITS * j)) & ((1u << BITS) - 1u));
                    const int sh = int(code & 15u);
                    int32_t z = sh == 15 ? 0 : -1;                 // zero weight: the term is 0
                    uint32_t neg = (code & 16u) ? uint32_t(z) : 0u;  // negative: ~t, the +1 counted
                    ncount += neg & 1u;
                    // Kept in registers as masks (an and and a xor per term, not selects).
                    asm volatile("" : "+v"(z), "+v"(neg));
#pragma unroll
                    for (int r = 0; r < ROWS; ++r)
                        acc[r] += uint32_t((xbuf[wave][r][u * PER + j] & z) >> sh) ^ neg;
                }
            }
            // The next chunk overwrites wbuf and xbuf after these reads (in order).
            __builtin_amdgcn_wave_barrier();
        }
    } else {
        for (int uc = u0; uc < u1; uc += U) {
            const int cb = uc * PER;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int32_t *xrow = x + int64_t(b0 + min(r, nb - 1)) * a.C;
#pragma unroll
                for (int e = lane; e < E; e += 64) xbuf[wave][r][e] = xrow[min(cb + e, a.C - 1)];
            }
            // (LDS is written and read back by the same wave: in order, no barrier;
            // the wave barrier keeps the compiler from moving the reads up.)
            __builtin_amdgcn_wave_barrier();
            const int un = min(U, u1 - uc);
            const int32_t *wrow = a.wi + int64_t(kc) * a.C;
            for (int u = 0; u < un; ++u) {
                const int32_t w = wrow[uc + u];
#pragma unroll
                for (int r = 0; r < ROWS; ++r) {
                    const int32_t xv = xbuf[wave][r][u];
                    acc[r] += OP == Inner::Mul ? uint32_t(xv) * uint32_t(w) : mul24(xv, w);
                }
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r) part[wave][r][lane] = acc[r] + ncount;
    __syncthreads();
    // Wave r finishes batch row b0 + r: the 16 partial sums, then bias and
    // epilogue, or (split) an atomic add into y, which holds the bias.
    if (wave < nb && k < a.K) {
        uint32_t v = 0u;
        for (int q = 0; q < kRowsWaves; ++q) v += part[q][wave][lane];
        const int64_t o = int64_t(b0 + wave) * a.K + k;
        if (nsplit > 1) {
            atomicAdd(reinterpret_cast<unsigned int *>(a.y + o), v);
        } else {
            v += a.bias ? uint32_t(a.bias[k]) : 0u;
            a.y[o] = int32_t(apply_epilogue(v, k, o, a.epi));
        }
    }
}

template <Inner OP, int ROWS>
static void launch_rows(dim3 grid, const int32_t *x, const RowsArgs &a, int bits, hipStream_t st)
{
    const dim3 block(64 * kRowsWaves);
    if constexpr (OP != Inner::Shift) {
        hipLaunchKernelGGL((linear_rows_kernel<OP, ROWS, 5>), grid, block, 0, st, x, a);
    } else if (bits == 5) {
        hipLaunchKernelGGL((linear_rows_kernel<OP, ROWS, 5>), grid, block, 0, st, x, a);
    } else if (bits == 4) {
        hipLaunchKernelGGL((linear_rows_kernel<OP, ROWS, 4>), grid, block, 0, st, x, a);
    } else if (bits == 3) {
        hipLaunchKernelGGL((linear_rows_kernel<OP, ROWS, 3>), grid, block, 0, st, x, a);
    } else {
        hipLaunchKernelGGL((linear_rows_kernel<OP, ROWS, 2>), grid, block, 0, st, x, a);
    }
}

// Workgroups per block of the small-batch kernel: fewer than 256 workgroups of
// 16 waves leave CUs idle and each wave a long walk along its weight rows, so the
// reduction is split over up to 8 workgroups per block (each wave keeping at
// least 4 units: a split adds a fill pass, which a shorter reduction does not
// repay), when there is no epilogue.
static int rows_splits(int64_t blocks, int units, bool may_split)
{
    int splits = 1;
    if (may_split)
        while (splits < 8 && blocks * splits < 256 && units / (kRowsWaves * splits * 2) >= 4) splits *= 2;
    return splits;
}

// Batch rows per workgroup (1, 2, 4 or 8, at most the batch): the one with the
// least estimated time, rounds of 256 workgroups (one 1024-thread workgroup per
// CU) times each workgroup's work, (1.5 + rows) / parts (a code's decode costs
// about 1.5 times a row's term). More rows share each decoded code, fewer give
// more workgroups. The measured best on MI355X (graph replays), which this
// picks: 2048 -> 1000 with 8 rows at batch 32-128 (12.3, 19.5, 31.9 us against
// 13.7, 20.5, 34.1 with 4), with 4 at batch 16 and 192 (9.2 against 12.1 with
// 8; 48.1 against 61.3: 384 workgroups of 8 rows fill the chip one and a half
// times), with 2 at batch 8 (7.7 us); 512 -> 1000 at batch 32 with 2 (6.2 us
// against 10.4 with 8); 256 -> 128 at batch 8 with 1 (3.8 us against 6.5 with
// 8). The DS_ROWS_BATCH override is for measurements.
static int rows_per_block(const ConvGeom &g, int units, bool may_split)
{
    const int forced = tuning(kRowsBatch);
    if (forced == 1 || forced == 2 || forced == 4 || forced == 8) return forced;
    const int64_t kg = (g.k + 63) / 64;
    int best = 1;
    double best_cost = 0.0;
    for (int rows = 1; rows <= 8 && rows <= g.n; rows *= 2) {
        const int64_t blocks = kg * ((g.n + rows - 1) / rows);
        const int splits = rows_splits(blocks, units, may_split);
        const int64_t rounds = std::max<int64_t>(1, (blocks * splits + 255) / 256);
        const double cost = double(rounds) * (1.5 + rows) / splits;
        if (rows == 1 || cost <= best_cost) {
            best = rows;
            best_cost = cost;
        }
    }
    return best;
}

template <Inner OP>
static void launch_rows_op(const ConvGeom &g, const int32_t *x, const RowsArgs &a, int rows, int splits,
                           hipStream_t st)
{
    const dim3 grid(unsigned((g.k + 63) / 64), unsigned((g.n + rows - 1) / rows), unsigned(splits));
    if (rows == 8) launch_rows<OP, 8>(grid, x, a, g.bits, st);
    else if (rows == 4) launch_rows<OP, 4>(grid, x, a, g.bits, st);
    else if (rows == 2) launch_rows<OP, 2>(grid, x, a, g.bits, st);
    else launch_rows<OP, 1>(grid, x, a, g.bits, st);
}

// Whether a problem takes the small-batch LinearShift kernel: 1 x 1 taps on
// 1 x 1 inputs, dense output, fewer than 256 rows, no forced variant.
static bool rows_path(const ConvGeom &g, const OutMap &map, const Padded &pad)
{
    return g.h == 1 && g.w == 1 && g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0 && map.dense() &&
           pad.vh == 0 && pad.iwp == 0 && g.n < 256 && forced_variant() < 0;
}

static hipError_t run_rows(const ConvGeom &g, const int32_t *x, const uint32_t *wp, const int32_t *wi,
                           const int32_t *bias, int32_t *y, Inner op, hipStream_t st, const Epilogue &epi)
{
    const int units = op == Inner::Shift ? int(row_words_bits(g.c, g.bits)) : g.c;
    const int rows = rows_per_block(g, units, !epi.any());
    const int64_t blocks = int64_t((g.k + 63) / 64) * ((g.n + rows - 1) / rows);
    const int splits = rows_splits(blocks, units, !epi.any());
    if (splits > 1) {
        const hipError_t e = bias ? run_fill_init(g, bias, y, st) : run_fill_zero(y, int64_t(g.n) * g.k, st);
        if (e != hipSuccess) return e;
    }
    RowsArgs a;
    a.wp = wp;
    a.wi = wi;
    a.bias = bias;
    a.y = y;
    a.B = g.n;
    a.C = g.c;
    a.K = g.k;
    a.wpr = int(row_words_bits(g.c, g.bits));
    a.epi = epi;
    if (op == Inner::Shift) launch_rows_op<Inner::Shift>(g, x, a, rows, splits, st);
    else if (op == Inner::Mul) launch_rows_op<Inner::Mul>(g, x, a, rows, splits, st);
    else launch_rows_op<Inner::Mul24>(g, x, a, rows, splits, st);
    return hipGetLastError();
}

static ConvLayout conv_layout(const ConvGeom &g0, const OutMap &map, const Padded &pad)
{
    ConvLayout L;
    // A strided output map or custom padded extents come only from the
    // input-gradient phases: tiled kernel, no epilogue, no transposition.
    L.mapped = !map.dense() || pad.vh > 0 || pad.iwp > 0;
    L.g = L.mapped ? g0 : tiled_geometry(g0, L.rowmajor);
    const ConvGeom &g = L.g;
    L.v = choose_variant(g, pad, L.plane, L.lds);
    L.direct = use_direct(g, L.v);
    if (L.direct) return L;
    plan_splits(g, L.v, L.tiles_p, L.tiles_k, L.nchunks, L.splits, L.cps);
    L.Jpad = L.nchunks * L.v.cc * g.r * g.s;
    L.Kpad = L.tiles_k * 4 * kTN;
    L.grid = int64_t(L.tiles_p) * L.tiles_k * L.splits;
    // Split partial sums meet through int32 atomics; through a strided output map
    // those land on scattered addresses, so a split mapped problem accumulates into
    // a dense buffer that is scattered into place afterwards.
    L.via_dense = L.mapped && L.splits > 1;
    // Scratch: init[Kpad], wd[Kpad][Jpad], x^T for row-major inputs, y^T (row-major) or
    // the dense partial sums (split mapped problems).
    const int64_t x_bytes = int64_t(g.n) * g.c * g.h * g.w * 4;
    L.init_bytes = (size_t(L.Kpad) * 4 + 255) & ~size_t(255);
    L.wd_bytes = (size_t(L.Kpad) * L.Jpad * 4 + 255) & ~size_t(255);
    L.xt_bytes = L.rowmajor ? (size_t(x_bytes) + 255) & ~size_t(255) : 0;
    L.yt_bytes = L.rowmajor ? size_t(g0.n) * g0.k * 4
               : L.via_dense ? size_t(g.n) * g.k * g.oh * g.ow * 4 : 0;
    return L;
}

size_t conv_scratch_bytes(const ConvGeom &g0, const OutMap &map, const Padded &pad)
{
    if (rows_path(g0, map, pad)) return 0;
    const ConvLayout L = conv_layout(g0, map, pad);
    return L.direct ? 0 : L.scratch_bytes();
}

hipError_t run_conv(const ConvGeom &g0, const int32_t *x, const uint32_t *wp, const int32_t *wi,
                    const int32_t *bias, int32_t *y, Inner op, hipStream_t st, const Epilogue &epi,
                    const OutMap &map, const Padded &pad, const Workspace &ws)
{
    if (rows_path(g0, map, pad)) return run_rows(g0, x, wp, wi, bias, y, op, st, epi);
    const ConvLayout L = conv_layout(g0, map, pad);
    const ConvGeom &g = L.g;
    const bool mapped = L.mapped, rowmajor = L.rowmajor;
    if (L.direct) {
        if (mapped) return hipErrorInvalidValue;
        const hipError_t e = run_direct(g0, x, wp, wi, bias, y, op, st);
        return e == hipSuccess && epi.any() ? run_epilogue(g0, y, epi, st) : e;
    }
    if (mapped && epi.any()) return hipErrorInvalidValue;
    if (L.grid > INT32_MAX) return hipErrorInvalidValue;
    const Variant &v = L.v;
    const int64_t x_bytes = int64_t(g.n) * g.c * g.h * g.w * 4;
    const int64_t NQ = int64_t(g.n) * g.oh * g.ow;

    TiledParams p;
    p.N = g.n; p.C = g.c; p.H = g.h; p.W = g.w; p.K = g.k; p.R = g.r; p.S = g.s;
    p.sh = g.sh; p.sw = g.sw; p.ph = g.ph; p.pw = g.pw; p.OH = g.oh; p.OW = g.ow;
    p.OHOW = g.oh * g.ow; p.NQ = int(NQ); p.HW = g.h * g.w;
    p.Jpad = L.Jpad; p.PLANE = L.plane;
    padded_dims(g, pad, p.VH, p.IWP);
    const OutMap m = map.dense() ? OutMap{0, g.k * g.oh * g.ow, g.oh * g.ow, g.ow, 1} : map;
    p.ybase = int(m.base); p.ynst = m.nstride; p.ykst = m.kstride; p.yrst = m.rstride; p.ycst = m.cstride;
    p.tiles_p = L.tiles_p; p.tiles_k = L.tiles_k; p.chunks_per_split = L.cps; p.nchunks = L.nchunks;
    p.atomic_out = L.splits > 1;
    p.fuse_epi = epi.any() && !p.atomic_out && !rowmajor;
    p.epi = epi;
    p.x_bytes = int(x_bytes);
    p.div_ohow = make_fastdiv(uint32_t(p.OHOW));
    p.div_ow = make_fastdiv(uint32_t(g.ow));
    p.div_vh = make_fastdiv(uint32_t(p.VH));
    p.div_iwp = make_fastdiv(uint32_t(p.IWP));
    if (L.via_dense) {
        const OutMap d{0, g.k * g.oh * g.ow, g.oh * g.ow, g.ow, 1};
        p.ybase = 0; p.ynst = d.nstride; p.ykst = d.kstride; p.yrst = d.rstride; p.ycst = d.cstride;
    }
    // Scratch from the caller's workspace when one is given (every byte of it that
    // the call reads is written first in the call: nothing needs clearing), else
    // from the stream-ordered pool.
    const size_t bytes = L.scratch_bytes();
    void *scratch = nullptr;
    hipError_t e = hipSuccess;
    if (ws.ptr) {
        if (bytes > ws.bytes) return hipErrorInvalidValue;
        scratch = ws.ptr;
    } else {
        e = scratch_alloc(&scratch, bytes, st);
        if (e != hipSuccess) return e;
    }
    int32_t *init = static_cast<int32_t *>(scratch);
    int32_t *wd = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) + L.init_bytes);
    const int32_t *xin = x;
    int32_t *yout = y;
    if (L.via_dense)
        yout = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) + L.init_bytes + L.wd_bytes);
    if (rowmajor) {
        yout = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) + L.init_bytes + L.wd_bytes +
                                           L.xt_bytes);
        int32_t *xt = reinterpret_cast<int32_t *>(static_cast<char *>(scratch) + L.init_bytes + L.wd_bytes);
        const int64_t tiles = int64_t((g0.c + 63) / 64) * ((g0.n + 63) / 64);
        hipLaunchKernelGGL(transpose_kernel, dim3(unsigned(tiles)), dim3(256), 0, st, x, xt, g0.n,
                           g0.c);
        xin = xt;
    }
    const int wpr = int(row_words_bits(g.crs, g.bits));
    const int Kpad = L.Kpad, Jpad = L.Jpad;
    const int64_t pw_total = int64_t(Kpad) * Jpad;
    const int wblocks = int(std::min<int64_t>((pw_total + 255) / 256, 4096));
    const int pgrid = wblocks + (Kpad + 3) / 4;
    if (op == Inner::Shift)
        hipLaunchKernelGGL((prep_kernel<Inner::Shift, kTN>), dim3(pgrid), dim3(256), 0, st, wp, wi,
                           bias, g.k, g.crs, wpr, Jpad, Kpad, wblocks, wd, init, code_fmt(g.bits));
    else  // both multiply operators copy the int32 weights
        hipLaunchKernelGGL((prep_kernel<Inner::Mul, kTN>), dim3(pgrid), dim3(256), 0, st, wp, wi,
                           bias, g.k, g.crs, wpr, Jpad, Kpad, wblocks, wd, init, code_fmt(g.bits));
    e = hipGetLastError();
    if (e == hipSuccess && p.atomic_out) e = run_fill_mapped(g, init, yout, L.via_dense ? OutMap() : map, st);
    if (e == hipSuccess) {
        e = op == Inner::Shift ? dispatch_tiled<Inner::Shift>(v, p, int(L.grid), L.lds, xin, wd, init, yout, st)
            : op == Inner::Mul ? dispatch_tiled<Inner::Mul>(v, p, int(L.grid), L.lds, xin, wd, init, yout, st)
                               : dispatch_tiled<Inner::Mul24>(v, p, int(L.grid), L.lds, xin, wd, init, yout, st);
    }
    if (e == hipSuccess && L.via_dense) e = run_copy_mapped(g, yout, y, map, st);
    if (e == hipSuccess && rowmajor) {
        const int64_t tiles = int64_t((g0.n + 63) / 64) * ((g0.k + 63) / 64);
        hipLaunchKernelGGL(transpose_kernel, dim3(unsigned(tiles)), dim3(256), 0, st, yout, y, g0.k,
                           g0.n);
        e = hipGetLastError();
    }
    if (e == hipSuccess && epi.any() && !p.fuse_epi) e = run_epilogue(g0, y, epi, st);
    if (ws.ptr) return e;
    const hipError_t ef = hipFreeAsync(scratch, st);
    return e != hipSuccess ? e : ef;
}

}  // namespace ds
