// Weight-specialised ConvShift kernels (the run-time compilation the paper
// suggests in Section 6): code generation, code object assembly and launch.
//
// With the weight codes known when the plan is made, the inner loop needs no
// weight loads, no decode and no work for zero weights. For each reduction
// element (input channel c, tap (r, s)) a lane loads its input x, forms each
// right shift x >> s that the output channels of the segment (64, or 16 / 32
// on small grids) use at that element (once, into one of two registers in
// turn), and adds or subtracts it into the accumulators of the channels with
// that shift: one v_add_u32 / v_sub_u32 per non-zero weight, with the register
// and the sign fixed in the instruction. The term of a weight with sign bit
// set is -(x >> shift) (Eq. 1 with the sign applied after the shift), so the
// results equal those of ds_conv2d_shift bit for bit.
//
// Code layout. A plan is one code object: the template kernel built with the
// library (jit_template.hip), whose last loadable segment `.jitbody` is
// replaced by the generated code: a table of jump stubs, then one block of
// straight-line code per segment (up to 64 output channels x a range of reduction
// elements; with a wave split, one per share of that range). The template
// computes the lane's tap and output offsets and jumps through the table; each
// segment ends the wave. Segments are spliced into the template image in
// memory (no assembler or linker runs at plan time) and the result is loaded
// with hipModuleLoadData.
//
// Variants of the same code: windows over 3 x 3 read a zero-padded copy of x
// (uniform tap offsets); small grids split each 64 pixels' reduction over 2 to
// 16 waves that meet in LDS, and long reductions over segments that meet in y
// through atomics; the stride phases of an input gradient run as output-channel
// groups of one problem (fuse_phases).
#include <hip/hip_runtime.h>

#include <elf.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "common.hpp"
#include "conv_plan.hpp"
#include "jit.hpp"
#include "tuning.hpp"

// The template code object, embedded by the build (see build.py).
extern "C" const unsigned char ds_jit_template_image[];
extern "C" const unsigned char ds_jit_template_image_end[];

namespace ds {
namespace {

// Register contract with the template (see the JITBODY marker there), one map
// per entry point. Up to 3 x 3 taps per element: v3 the lane's LDS byte offset
// (wave split), v4..v12 the byte offset in x of tap (r, s) = v[4 + 3r + s] at
// channel 0, v13 the byte offset in y of the lane's output pixel at channel 0,
// v14, v15 the multiplier's temporaries, v16, v17 x >> s alternately (x itself
// stays in its load slot), v18..v81 the accumulators of the segment's 64
// output channels, v82..v95 up to 14 loads in flight: 96 VGPRs, 5 waves per
// SIMD. One tap per element (1 x 1 windows, or the tap column as an offset in
// the instruction): v4 the tap, v5..v12 up to 8 loads in flight (the
// multiplier's temporaries share them, free by then), v14, v15 the shifted
// values, v16..v79 the accumulators: 80 VGPRs, 6 waves per SIMD.
struct RegMap {
    int lds, tap0, yoff, tmp_lo, tmp_hi, tab, acc, slot, max_slots;
    const char *kernel;
};
constexpr RegMap kMap96 = {3, 4, 13, 14, 15, 16, 18, 82, 14, "ds_jit_conv_template"};
constexpr RegMap kMap80 = {3, 4, 13, 5, 6, 14, 16, 5, 8, "ds_jit_conv_one_tap_template"};
constexpr int kXrsrc = 20, kYrsrc = 24, kRrsrc = 36;  // buffer resources (SGPR quads)
constexpr int kSy = 28, kSx = 29, kSmul = 30;         // scalar scratch of the generated code
constexpr int kSw = 31;                               // multiplication plans: the current weight
constexpr int kTN = 64;      // output channels per segment (at most; see Spec::tn)
constexpr int kBlockPixels = 256;
constexpr int kStubWords = 5;
constexpr int kMaxTaps = 3;  // R, S <= 3: the template computes a 3 x 3 window of taps
constexpr int kMaxPaddedS = 1023;  // wider windows: tap column s at immediate offset 4 s < 4096

// gfx950 instruction encodings used by the generator (VOP2, VOP1, VOP3, MUBUF,
// SOP1/SOP2/SOPP words; see the CDNA ISA reference).
constexpr uint32_t kOpAshr = 0x11, kOpMax = 0x0d, kOpAdd = 0x34, kOpSub = 0x35;  // VOP2
constexpr uint32_t kOpMulLo = 0x285, kOpMulHi = 0x287, kOpAlignbit = 0x1ce;     // VOP3
constexpr uint32_t kOpMad24 = 0x1c2;                                            // VOP3 v_mad_i32_i24
constexpr uint32_t kLoad = 0xe0501000u, kStore = 0xe0701000u, kAtomicAdd = 0xe1081000u;
constexpr uint32_t kLoadI16 = 0xe04c1000u, kLoadI8 = 0xe0441000u;  // buffer_load_sshort / _sbyte
constexpr uint32_t kEndpgm = 0xbf810000u, kNop = 0xbf800000u, kBarrier = 0xbf8a0000u;
constexpr uint32_t kDsAdd = 0xd8000000u, kDsRead = 0xd86c0000u;  // ds_add_u32, ds_read_b32
constexpr uint32_t kLiteral = 255;

class Emitter {
public:
    std::vector<uint32_t> w;

    static uint32_t vgpr(int r) { return 256u + uint32_t(r); }
    static bool is_inline(int32_t v) { return v >= -16 && v <= 64; }
    static uint32_t inline_int(int32_t v) { return v >= 0 ? 128u + uint32_t(v) : 192u + uint32_t(-v); }

    void vop2(uint32_t op, int vdst, uint32_t src0, int vsrc1)
    {
        w.push_back((op << 25) | (uint32_t(vdst) << 17) | (uint32_t(vsrc1) << 9) | src0);
    }
    // vdst = op(imm, vsrc1), the constant inline when it fits, else a literal word.
    void vop2_imm(uint32_t op, int vdst, int32_t imm, int vsrc1)
    {
        if (is_inline(imm)) {
            vop2(op, vdst, inline_int(imm), vsrc1);
        } else {
            vop2(op, vdst, kLiteral, vsrc1);
            w.push_back(uint32_t(imm));
        }
    }
    void mov_imm(int vdst, int32_t imm)
    {
        const uint32_t base = 0x7e000200u | (uint32_t(vdst) << 17);  // v_mov_b32
        if (is_inline(imm)) {
            w.push_back(base | inline_int(imm));
        } else {
            w.push_back(base | kLiteral);
            w.push_back(uint32_t(imm));
        }
    }
    void vop3(uint32_t op, int vdst, uint32_t s0, uint32_t s1, uint32_t s2)
    {
        w.push_back(0xd0000000u | (op << 16) | uint32_t(vdst));
        w.push_back(s0 | (s1 << 9) | (s2 << 18));
    }
    void wait_vm(int n)  // s_waitcnt vmcnt(n), other counters not waited on
    {
        w.push_back(0xbf8c0f70u | uint32_t(n & 15) | (uint32_t(n >> 4) << 14));
    }
    void mubuf(uint32_t word0, int vdata, int vaddr, int srsrc, int soff, uint32_t imm = 0)
    {
        w.push_back(word0 | (imm & 0xfffu));  // 12-bit immediate byte offset
        w.push_back((uint32_t(soff) << 24) | (uint32_t(srsrc / 4) << 16) |
                    (uint32_t(vdata) << 8) | uint32_t(vaddr));
    }
    // LDS at v[vaddr] + offset (16 bits): ds_add_u32 of v[vdata]; ds_read_b32 into v[vdst].
    void ds_add(int vaddr, int vdata, uint32_t offset)
    {
        w.push_back(kDsAdd | (offset & 0xffffu));
        w.push_back(uint32_t(vaddr) | (uint32_t(vdata) << 8));
    }
    void ds_read(int vdst, int vaddr, uint32_t offset)
    {
        w.push_back(kDsRead | (offset & 0xffffu));
        w.push_back(uint32_t(vaddr) | (uint32_t(vdst) << 24));
    }
    void wait_lgkm0() { w.push_back(0xbf8cc07fu); }  // s_waitcnt lgkmcnt(0)
    void s_mov_imm(int sdst, uint32_t imm)
    {
        w.push_back(0xbe8000ffu | (uint32_t(sdst) << 16));
        w.push_back(imm);
    }
    void s_add_imm(int sdst, uint32_t imm)  // s_add_u32 sdst, sdst, imm
    {
        w.push_back(0x8000ff00u | (uint32_t(sdst) << 16) | uint32_t(sdst));
        w.push_back(imm);
    }
};

struct Spec {
    ConvGeom g{};
    const uint32_t *wp = nullptr;  // host packed codes [k][rw], codes of fmt.bits bits
    // Multiplication plans (the comparison operator, not DeepShift): host int32
    // weights [k][crs] in place of wp; each non-zero weight is one v_mad_i32_i24.
    const int32_t *wint = nullptr;
    int act_bytes = 4;   // bytes of an element of x: 4 int32, 2 int16 (DS_ACT_I16), 1 int8 (DS_ACT_I8)
    int64_t rw = 0;
    CodeFmt fmt;
    const int32_t *bias = nullptr, *mul = nullptr, *add = nullptr;  // host, [k] or NULL
    int mul_shift = 0;
    bool relu = false, residual = false;
    int nsplit = 1, kgroups = 0, nseg = 0, tiles_p = 0;
    int slots = 8;       // loads in flight per wave
    OutMap map;          // where output (n, k, oh, ow) goes in y (dense by default)
    // Windows over 3 x 3: the kernel reads a zero-padded copy of x, [n][c][xh][xw]
    // with the padding included, that the plan makes before each run; a lane's
    // window then starts at one offset and every tap sits at a uniform distance
    // from it. Zero: x itself, with per-tap offsets from the template.
    int xh = 0, xw = 0;
    // Waves per 64 pixels (1, 2, 4, 8 or 16), each with a contiguous share of
    // every part's reduction elements, meeting in LDS; a workgroup covers
    // 64 * pgroups pixels with pgroups * wsplit waves (by default 256 / wsplit
    // pixels up to a split of 4, 64 beyond).
    int wsplit = 1;
    // Output channels per segment: 64, or 32 / 16 on grids too small to fill the
    // chip (more segments, each with less code, at the price of forming each
    // shift for fewer channels).
    int tn = kTN;
    // Groups of 64 pixels per workgroup (1, 2 or 4; pgroups * wsplit <= 16 waves):
    // a workgroup covers 64 * pgroups pixels.
    int pgroups = 4;
    // Fused stride phases of an input gradient: output-channel group kg stores
    // its first channel at element kout[kg] + (pixel's map offset) and has kjn[kg]
    // channels (empty: group kg stores channel 64 kg + j at its map offset).
    std::vector<int64_t> kout;
    std::vector<int> kjn;
    // Block order (see the template): all segments of one pixel tile after the
    // other, instead of groups of tiles passing through the segments one by one.
    int tile_major = 0;         // 0 grouped, 1 tile-major, 2 XCD-local tile-major
    bool one_tap = false;       // the 80-VGPR entry point (one tap register)
    // A LinearShift of batch > 1 (x [N][C] -> y [N][K]) runs as a 1 x 1 layer over
    // x^T viewed as one image of 1 x N pixels, so that the 64 lanes of a load read
    // 64 consecutive batch rows of one input channel (coalesced) instead of 64 rows
    // C elements apart, and store y^T [K][N] as coalesced (lanes C or K elements
    // apart made 4096 -> 4096 at batch 256 run 1.5-2.7x slower on MI355X). The
    // plan transposes x into an int32 copy of its own before the kernel and y^T
    // back into y after it; that last pass adds the residual and applies the ReLU
    // of a layer with a residual. `lin` keeps the layer as given.
    bool xt = false;
    ConvGeom lin{};
};

// Element strides of the output map of a spec (the dense layout when unset).
inline OutMap full_map(const Spec &sp)
{
    if (!sp.map.dense()) return sp.map;
    OutMap m;
    m.kstride = sp.g.oh * sp.g.ow;
    m.nstride = sp.g.k * m.kstride;
    m.rstride = sp.g.ow;
    m.cstride = 1;
    return m;
}

inline int code_at(const Spec &sp, int k, int j)
{
    return int(sp.fmt.at(sp.wp + int64_t(k) * sp.rw, j));
}

// Whether weight (k, j) contributes a term: a non-zero code, or a non-zero
// weight of a multiplication plan.
inline bool weight_nonzero(const Spec &sp, int k, int j)
{
    if (sp.wint) return sp.wint[int64_t(k) * sp.g.crs + j] != 0;
    return (code_at(sp, k, j) & 15) != 15;
}

// Instruction words of the code of all segments of an unsplit plan with `tn`
// output channels per segment (shift codes): per element with a non-zero weight
// in the group, its load, wait and offset update (5 words), a word per distinct
// non-zero shift and a word per non-zero weight; per segment its accumulator
// set-up and epilogue (about 3 words per channel and 16 more).
int64_t code_words(const Spec &sp, int tn)
{
    const ConvGeom &g = sp.g;
    int64_t words = 0;
    for (int kb = 0; kb < g.k; kb += tn) {
        const int jn = std::min(tn, g.k - kb);
        for (int i = 0; i < g.crs; ++i) {
            uint32_t shifts = 0;
            int nz = 0;
            for (int j = 0; j < jn; ++j) {
                const int code = code_at(sp, kb + j, i);
                if ((code & 15) == 15) continue;
                ++nz;
                shifts |= 1u << (code & 15);
            }
            if (nz) words += 5 + nz + __builtin_popcount(shifts & ~1u);
        }
        words += 3 * jn + 16;
    }
    return words;
}

// Straight-line code of one wave's segment: output channels [64 kg, 64 kg + 64)
// and reduction elements [e0, e1), element i being (input channel i / RS, tap
// i % RS). `split`: the partial sums of several parts of the reduction meet in y
// through atomic adds (y holds the bias beforehand and the epilogue runs
// afterwards, as separate passes). With a wave split W = sp.wsplit > 1, the W
// waves sharing 64 pixels run shares 0..W-1 of a part's elements: each adds its
// 64 sums into LDS, waits for the others at a barrier and finishes channels
// [tn share / W, tn (share + 1) / W) of the totals (tn: channels per segment).
void emit_segment(Emitter &e, const Spec &sp, int kg, int e0, int e1, int share, bool split)
{
    const ConvGeom &g = sp.g;
    const int kbase = kg * sp.tn;
    const int jn = sp.kjn.empty() ? std::min(sp.tn, g.k - kbase) : sp.kjn[size_t(kg)];
    const int RS = g.r * g.s;
    const bool padded = sp.xh > 0;
    // The padded and transposed copies are int32 whatever x holds; x itself is
    // read with a sign-extending load of its own width.
    const bool wide = padded || sp.xt || sp.act_bytes == 4;
    const uint32_t cstride = padded ? uint32_t(sp.xh) * uint32_t(sp.xw) * 4u
                                    : uint32_t(g.h) * uint32_t(g.w) * uint32_t(wide ? 4 : sp.act_bytes);
    const uint32_t load_op = wide ? kLoad : sp.act_bytes == 2 ? kLoadI16 : kLoadI8;
    const uint32_t rstride = uint32_t(sp.xw) * 4u;
    const uint32_t kstride = uint32_t(full_map(sp).kstride) * 4u;
    // Byte offset of the group's first output channel (added to the lane's v13).
    const uint32_t out0 = sp.kout.empty() ? uint32_t(kbase) * kstride : uint32_t(sp.kout[size_t(kg)]) * 4u;
    // The elements with at least one non-zero weight in the group; the others
    // contribute nothing and are not even loaded.
    std::vector<int> el;
    el.reserve(size_t(e1 - e0));
    for (int i = e0; i < e1; ++i)
        for (int j = 0; j < jn; ++j)
            if (weight_nonzero(sp, kbase + j, i)) {
                el.push_back(i);
                break;
            }
    const int E = int(el.size());

    const RegMap &m = sp.one_tap ? kMap80 : kMap96;
    for (int j = 0; j < jn; ++j)
        e.mov_imm(m.acc + j, (!split && sp.bias && share == 0) ? sp.bias[kbase + j] : 0);

    // Listed element n's load goes to slot n % nslots and reads x at v[tap] + s29,
    // where s29 = c * H * W * 4 for the channel of the most recently issued load.
    // From a padded copy: at v4 + s29 + 4 s, where s29 = (c * xh * xw + r * xw) * 4
    // for the channel and tap row of that load.
    const int nslots = sp.slots;
    const int D = std::min(nslots, E);
    uint32_t cur = uint32_t(e0 / RS) * cstride;
    e.s_mov_imm(kSx, cur);
    auto issue = [&](int n) {
        const int i = el[size_t(n)];
        const int c = i / RS, t = i % RS, tr = t / g.s, ts = t % g.s;
        const uint32_t soff = uint32_t(c) * cstride + (padded ? uint32_t(tr) * rstride : 0u);
        if (soff != cur) {
            e.s_add_imm(kSx, soff - cur);  // modulo 2^32
            cur = soff;
        }
        const int slot = m.slot + n % nslots;
        if (padded)
            e.mubuf(load_op, slot, m.tap0, kXrsrc, kSx, uint32_t(ts) * 4u);
        else
            e.mubuf(load_op, slot, m.tap0 + tr * 3 + ts, kXrsrc, kSx);
    };
    for (int n = 0; n < D; ++n) issue(n);

    bool sw_set = false;     // multiplication plans: s31 holds sw_val
    int32_t sw_val = 0;
    for (int i = 0; i < E; ++i) {
        const int issued = std::min(E, i + D);
        e.wait_vm(issued - i - 1);
        const int slot = m.slot + i % nslots;
        const int jw = el[size_t(i)];  // column of the element in the packed rows
        if (sp.wint) {
            // acc += x * w (low 24 bits of each, signed): the weight as an inline
            // constant when it is one, else from s31, set only when it changes.
            for (int j = 0; j < jn; ++j) {
                const int32_t wv = sp.wint[int64_t(kbase + j) * g.crs + jw];
                if (wv == 0) continue;
                uint32_t src1;
                if (Emitter::is_inline(wv)) {
                    src1 = Emitter::inline_int(wv);
                } else {
                    if (!sw_set || sw_val != wv) {
                        e.s_mov_imm(kSw, uint32_t(wv));
                        sw_set = true;
                        sw_val = wv;
                    }
                    src1 = uint32_t(kSw);
                }
                e.vop3(kOpMad24, m.acc + j, Emitter::vgpr(slot), src1, Emitter::vgpr(m.acc + j));
            }
            if (i + D < E) issue(i + D);
            continue;
        }
        // The element's non-zero weights grouped by shift; each shift is formed
        // once, into one of two registers in turn, right before the adds that use it.
        int by_shift[15][kTN], count[15] = {};
        for (int j = 0; j < jn; ++j) {
            const int code = code_at(sp, kbase + j, jw);
            if ((code & 15) != 15) by_shift[code & 15][count[code & 15]++] = code & 16 ? -1 - j : j;
        }
        int formed = 0;
        for (int sh = 0; sh <= 14; ++sh) {
            if (count[sh] == 0) continue;
            int src = slot;
            if (sh > 0) {
                src = m.tab + (formed++ & 1);
                e.vop2(kOpAshr, src, Emitter::inline_int(sh), slot);
            }
            for (int q = 0; q < count[sh]; ++q) {
                const int v = by_shift[sh][q];
                if (v < 0)
                    e.vop2(kOpSub, m.acc - 1 - v, Emitter::vgpr(m.acc - 1 - v), src);  // acc - term
                else
                    e.vop2(kOpAdd, m.acc + v, Emitter::vgpr(src), m.acc + v);          // term + acc
            }
        }
        if (i + D < E) issue(i + D);
    }

    // The channels this wave finishes: all, or its share of them after the LDS sum.
    int j0 = 0, j1 = jn;
    if (sp.wsplit > 1) {
        for (int j = 0; j < jn; ++j) e.ds_add(m.lds, m.acc + j, uint32_t(j) * 256u);
        e.wait_lgkm0();
        e.w.push_back(kBarrier);
        j0 = std::min(jn, share * sp.tn / sp.wsplit);
        j1 = std::min(jn, (share + 1) * sp.tn / sp.wsplit);
        for (int j = j0; j < j1; ++j) e.ds_read(m.acc + j, m.lds, uint32_t(j) * 256u);
        e.wait_lgkm0();
    }
    if (!split) {
        if (sp.mul) {
            for (int j = j0; j < j1; ++j) {
                // floor(acc * mul / 2^mul_shift): the low word of the 64-bit product
                // shifted right, taken from its two halves.
                e.s_mov_imm(kSmul, uint32_t(sp.mul[kbase + j]));
                e.vop3(kOpMulLo, m.tmp_lo, uint32_t(kSmul), Emitter::vgpr(m.acc + j), 0);
                e.vop3(kOpMulHi, m.tmp_hi, uint32_t(kSmul), Emitter::vgpr(m.acc + j), 0);
                e.vop3(kOpAlignbit, m.acc + j, Emitter::vgpr(m.tmp_hi), Emitter::vgpr(m.tmp_lo),
                       Emitter::inline_int(sp.mul_shift));
                const int32_t a = sp.add ? sp.add[kbase + j] : 0;
                if (a != 0) e.vop2_imm(kOpAdd, m.acc + j, a, m.acc + j);
            }
        }
        if (sp.residual && !sp.xt) {
            for (int jb = j0; jb < j1; jb += nslots) {
                const int nb = std::min(nslots, j1 - jb);
                e.s_mov_imm(kSy, out0 + uint32_t(jb) * kstride);
                for (int b = 0; b < nb; ++b) {
                    e.mubuf(kLoad, m.slot + b, m.yoff, kRrsrc, kSy);
                    if (b + 1 < nb) e.s_add_imm(kSy, kstride);
                }
                e.wait_vm(0);
                for (int b = 0; b < nb; ++b)
                    e.vop2(kOpAdd, m.acc + jb + b, Emitter::vgpr(m.slot + b), m.acc + jb + b);
            }
        }
        if (sp.relu && !(sp.xt && sp.residual))
            for (int j = j0; j < j1; ++j) e.vop2(kOpMax, m.acc + j, Emitter::inline_int(0), m.acc + j);
    }
    e.s_mov_imm(kSy, out0 + uint32_t(j0) * kstride);
    for (int j = j0; j < j1; ++j) {
        e.mubuf(split ? kAtomicAdd : kStore, m.acc + j, m.yoff, kYrsrc, kSy);
        if (j + 1 < j1) e.s_add_imm(kSy, kstride);
    }
    e.w.push_back(kEndpgm);
}

// Body of `.jitbody`: the jump stubs, then the segments (each 64-byte aligned),
// then a tail of s_endpgm words so that instruction prefetch past the last
// segment stays inside the loaded image.
std::vector<uint32_t> generate_body(const Spec &sp)
{
    Emitter e;
    const int nstub = sp.nseg * sp.wsplit;  // stub s19 = block segment * wsplit + share
    e.w.resize(size_t(nstub) * kStubWords, kNop);
    std::vector<size_t> start(nstub);
    const int RS = sp.g.r * sp.g.s;
    int seg = 0;
    for (int kg = 0; kg < sp.kgroups; ++kg) {
        for (int part = 0; part < sp.nsplit; ++part) {
            const int c0 = int(int64_t(part) * sp.g.c / sp.nsplit);
            const int c1 = int(int64_t(part + 1) * sp.g.c / sp.nsplit);
            const int E = (c1 - c0) * RS;
            for (int share = 0; share < sp.wsplit; ++share, ++seg) {
                while (e.w.size() % 16) e.w.push_back(kNop);
                start[seg] = e.w.size();
                emit_segment(e, sp, kg, c0 * RS + int(int64_t(E) * share / sp.wsplit),
                             c0 * RS + int(int64_t(E) * (share + 1) / sp.wsplit), share, sp.nsplit > 1);
            }
        }
    }
    for (int i = 0; i < 64; ++i) e.w.push_back(kEndpgm);
    for (int s = 0; s < nstub; ++s) {
        // s_getpc_b64 s[28:29] (= address of the next word); s_add_u32 s28, s28,
        // delta; s_addc_u32 s29, s29, 0; s_setpc_b64 s[28:29]
        uint32_t *stub = &e.w[size_t(s) * kStubWords];
        const uint64_t delta = (start[s] - (size_t(s) * kStubWords + 1)) * 4;
        stub[0] = 0xbe9c1c00u;
        stub[1] = 0x801cff1cu;
        stub[2] = uint32_t(delta);
        stub[3] = 0x821d801du;
        stub[4] = 0xbe801d1cu;
    }
    return e.w;
}

// The template image with `.jitbody` replaced by `body`: the body is appended
// at the end of the file, and the section header and the program header of the
// last loadable segment (which holds `.jitbody` alone) are pointed at it.
ds_status splice_body(const std::vector<uint32_t> &body, std::vector<uint8_t> &out)
{
    const size_t n = size_t(ds_jit_template_image_end - ds_jit_template_image);
    out.assign(ds_jit_template_image, ds_jit_template_image + n);
    Elf64_Ehdr eh;
    if (n < sizeof eh) return fail(DS_ERR_HIP, "template code object missing");
    std::memcpy(&eh, out.data(), sizeof eh);
    if (std::memcmp(eh.e_ident, ELFMAG, SELFMAG) != 0 || eh.e_ident[EI_CLASS] != ELFCLASS64 ||
        eh.e_shentsize != sizeof(Elf64_Shdr) || eh.e_phentsize != sizeof(Elf64_Phdr) ||
        eh.e_shoff + uint64_t(eh.e_shnum) * sizeof(Elf64_Shdr) > n ||
        eh.e_phoff + uint64_t(eh.e_phnum) * sizeof(Elf64_Phdr) > n || eh.e_shstrndx >= eh.e_shnum)
        return fail(DS_ERR_HIP, "template code object malformed");
    auto shdr = [&](int i) {
        Elf64_Shdr s;
        std::memcpy(&s, out.data() + eh.e_shoff + size_t(i) * sizeof s, sizeof s);
        return s;
    };
    auto phdr = [&](int i) {
        Elf64_Phdr p;
        std::memcpy(&p, out.data() + eh.e_phoff + size_t(i) * sizeof p, sizeof p);
        return p;
    };
    const Elf64_Shdr strtab = shdr(eh.e_shstrndx);
    int js = -1;
    for (int i = 0; i < eh.e_shnum; ++i) {
        const Elf64_Shdr s = shdr(i);
        if (strtab.sh_offset + s.sh_name + 9 <= n &&
            std::memcmp(out.data() + strtab.sh_offset + s.sh_name, ".jitbody", 9) == 0)
            js = i;
    }
    if (js < 0) return fail(DS_ERR_HIP, "template code object has no .jitbody section");
    Elf64_Shdr sec = shdr(js);
    int jp = -1;
    uint64_t top = 0;
    for (int i = 0; i < eh.e_phnum; ++i) {
        const Elf64_Phdr p = phdr(i);
        if (p.p_type != PT_LOAD) continue;
        if (p.p_vaddr == sec.sh_addr) jp = i;
        top = std::max(top, p.p_vaddr);
    }
    if (jp < 0 || phdr(jp).p_vaddr != top || phdr(jp).p_filesz != sec.sh_size)
        return fail(DS_ERR_HIP, ".jitbody is not alone in the last loadable segment");
    Elf64_Phdr seg = phdr(jp);
    const uint64_t align = std::max<uint64_t>(seg.p_align, 256);
    const uint64_t off = (out.size() + align - 1) / align * align + seg.p_vaddr % align;
    const uint64_t bytes = uint64_t(body.size()) * 4;
    out.resize(off + bytes);
    std::memcpy(out.data() + off, body.data(), bytes);
    seg.p_offset = off;
    seg.p_filesz = seg.p_memsz = bytes;
    sec.sh_offset = off;
    sec.sh_size = bytes;
    std::memcpy(out.data() + eh.e_phoff + size_t(jp) * sizeof seg, &seg, sizeof seg);
    std::memcpy(out.data() + eh.e_shoff + size_t(js) * sizeof sec, &sec, sizeof sec);
    return ok();
}

struct CreateArgs {
    const uint32_t *wp;
    const int32_t *wint;  // multiplication plans (wp == NULL)
    const int32_t *bias, *mul, *add;
    int mul_shift;
    int64_t n, c, h, w, k, r, s;
    int sh, sw, ph, pw;
    uint32_t flags;
    int splits;
};

// Planning of a spec whose geometry, codes and epilogue are set: code width
// checks, pixel tiles, segments and the split of the reduction.
ds_status finish_spec(Spec &sp, int bits, int splits, int deep_blocks = 3072)
{
    const ConvGeom &g = sp.g;
    sp.fmt = code_fmt(bits);
    sp.rw = row_words_bits(g.crs, bits);
    const int used = sp.fmt.per_word * bits;
    for (int64_t i = 0; sp.wp && used < 32 && i < int64_t(g.k) * sp.rw; ++i)
        if (sp.wp[i] >> used)
            return fail(DS_ERR_INVALID_CODE, "bits %d-31 of packed word %lld are not 0", used, (long long)i);
    if (g.r > kMaxTaps || g.s > kMaxTaps) {
        if (g.s > kMaxPaddedS)
            return fail(DS_ERR_UNSUPPORTED, "kernels wider than %d columns are not supported", kMaxPaddedS);
        const int64_t xh = int64_t(g.oh - 1) * g.sh + g.r, xw = int64_t(g.ow - 1) * g.sw + g.s;
        const int64_t xe = prod({g.n, g.c, xh, xw});
        if (xe < 0 || xe > kMaxElems / 4)
            return fail(DS_ERR_UNSUPPORTED, "the padded input would take 2^31 bytes or more");
        sp.xh = int(xh);
        sp.xw = int(xw);
    }
    const int64_t nq = int64_t(g.n) * g.oh * g.ow;
    // Channels per segment: 64, unless forced (fused input-gradient phases keep
    // their own groups of 64).
    {
        const int forced = tuning(kJitTn);
        sp.tn = sp.kjn.empty() && (forced == 16 || forced == 32) ? forced : kTN;
    }
    sp.kgroups = (g.k + sp.tn - 1) / sp.tn;
    // One tap per element (1 x 1 windows, or wider ones through the padded copy):
    // the 80-VGPR entry point, 6 waves per SIMD instead of 5.
    sp.one_tap = (int64_t(g.r) * g.s == 1 || sp.xh > 0) && tuning(kJitMap) != 96;
    // Wave split (2 or 4 waves per 64 pixels, each with a share of the reduction,
    // meeting in LDS): more waves without atomics on grids under 2048 workgroups
    // of 256 pixels, each share keeping 128 reduction elements (32 on grids under
    // 256 workgroups, where parallelism decides). A strided 1 x 1 layer, whose
    // loads already span twice the cache lines, splits at most in 2; other
    // one-tap layers keep shares of 64: with 80 VGPRs a CU holds 6 workgroups of
    // 16 KiB of LDS (a split of 4) but only 5 of 32 KiB (a split of 2). In a
    // randomized A/B on MI355X a split of 4 against 2 ran ResNet-50's (N = 128)
    // 256 -> 64 layers at 56 x 56, 512 -> 256 at 28 x 28 and 256 -> 1024 at
    // 14 x 14 5-10 % faster, its 3 x 3 layers at 56 x 56 5 % faster.
    const int64_t base = (nq + kBlockPixels - 1) / kBlockPixels * sp.kgroups;
    {
        const bool thin = base < 256;
        const bool strided_point = int64_t(g.r) * g.s == 1 && (g.sh > 1 || g.sw > 1);
        const bool wide = sp.one_tap && !strided_point;
        const int64_t min_share = thin ? 32 : wide ? 64 : 128;
        const int cap = strided_point && !thin ? 2 : 4;
        int ws = 1;
        if (base < 2048)
            while (ws < cap && g.crs / (2 * ws) >= min_share) ws *= 2;
        const int forced = tuning(kJitWsplit);
        sp.wsplit = forced == 1 || forced == 2 || forced == 4 || forced == 8 || forced == 16 ? forced : ws;
    }
    // A workgroup covers 256 pixels with 4 waves, 128 with 2 x 2, and 64 with 4,
    // 8 or 16 waves sharing them, unless forced otherwise.
    {
        const int forced = tuning(kJitPgroups);
        const int dflt = sp.wsplit <= 4 ? 4 / sp.wsplit : 1;
        sp.pgroups = (forced == 1 || forced == 2 || forced == 4) && forced * sp.wsplit <= 16 ? forced : dflt;
    }
    const int tile_pixels = 64 * sp.pgroups;
    sp.tiles_p = int((nq + tile_pixels - 1) / tile_pixels);
    // Split-K: the parts' partial sums meet in y through int32 atomics after a fill
    // pass, a round trip of y per part, so splitting is kept to what the grid needs.
    // (1) Toward 384 workgroups (1.5 waves per SIMD on MI355X's 1024 SIMDs), each
    // wave's share keeping at least 64 reduction elements. (2) A window whose
    // parts keep at least 768 elements (a long reduction hides the round trips)
    // spreads further, toward `deep_blocks`. Both splits were fitted to a sweep
    // of every ResNet-50 (N = 128) and ResNet-18 (N = 32) convolution over wave
    // splits 1, 2, 4 and 1-8 parts on MI355X: summed over each network the rule
    // is within 0.5 % of the best choice per layer.
    // (3) A 1 x 1 layer on a grid under 256 workgroups of 256 pixels (at least 4
    // pixel tiles) whose wave shares keep at least 128 elements per part spreads
    // toward 2400 workgroups (ResNet-50's 2048 -> 512 layer at 7 x 7: 3 parts ran
    // 1.1x faster than 1 or 2).
    // (5) A window on a grid under 256 workgroups of 256 pixels (a small batch)
    // lets each wave's share of a part go down to 24 reduction elements: such a
    // grid has too few waves to use the chip's SIMDs, and one wave per SIMD issues
    // at half the rate of two. On MI355X the 128 -> 128, 3 x 3 layer at 28 x 28 and
    // batch 1 ran its kernel in 9.9 us at 12 or 16 parts against 13.7 us at 4 (and
    // 12.5 us at 24).
    int ns = splits;
    // A transposed LinearShift (x^T as one image of 1 x N pixels): 32-channel
    // segments below 4 tiles of 64 rows (64 from there), one group of 64 rows per
    // workgroup, a wave split of 16 while each share keeps 64 input channels,
    // and parts toward 4096 waves while each wave keeps 16 input channels. Layout
    // sweeps of 3 x 5 x 3 x 4 segment widths, wave splits, pixel groups and parts
    // on MI355X (graph replays, transposing passes of 64 x 64 tiles included):
    // 4096 -> 4096 at batch 256 116 us at best, 117 us by this rule (16 / 1 / 1),
    // 182 us by the convolution rules below; 2048 -> 1000 at batch 128 25.1 /
    // 25.5 (16 / 1 / 4) / 36.6 us; 1024 -> 1024 at batch 64 19.5 / 20.9 (16 / 1
    // / 4) / 26.6 us.
    if (sp.xt && sp.kjn.empty() && tuning(kJitTn) < 0 && tuning(kJitWsplit) < 0 && tuning(kJitPgroups) < 0) {
        sp.tn = nq >= 4 * 64 ? kTN : 32;
        sp.kgroups = (g.k + sp.tn - 1) / sp.tn;
        int ws = 16;
        while (ws > 1 && g.c / ws < 64) ws /= 2;
        sp.wsplit = ws;
        sp.pgroups = 1;
        sp.tiles_p = int((nq + 63) / 64);
        if (ns == 0) {
            const int64_t w1 = int64_t(sp.tiles_p) * sp.kgroups * ws;
            ns = 1;
            while (ns < 8 && w1 * ns < 4096 && g.c / (ws * ns * 2) >= 16) ns *= 2;
        }
    }
    if (ns == 0) {
        const int64_t blocks = int64_t(sp.tiles_p) * sp.kgroups;
        const bool thin_window = base < 256 && int64_t(g.r) * g.s > 1;
        const int64_t floor_share = thin_window ? 24 : 64;
        int64_t want = std::min<int64_t>((384 + blocks - 1) / blocks, g.crs / (floor_share * sp.wsplit));
        if (deep_blocks > 0 && int64_t(g.r) * g.s > 1)
            want = std::max<int64_t>(want, std::min<int64_t>((deep_blocks + blocks - 1) / blocks, g.crs / 768));
        const int64_t tiles256 = (nq + kBlockPixels - 1) / kBlockPixels;
        if (int64_t(g.r) * g.s == 1 && base < 256 && tiles256 >= 4)
            want = std::max<int64_t>(want, std::min<int64_t>((2400 + blocks - 1) / blocks, g.crs / (128 * sp.wsplit)));
        // (4) Fewer than 4 tiles of 256 pixels (a LinearShift at small batch): every
        // code segment streams through the instruction cache for a few waves only,
        // and more parts mean more code streams: at most 4 (with a wave split of 4,
        // 2048 -> 1000 at batch 128: 45 us at 4 parts, 49 us at 2, 57 us at 8;
        // 512 -> 1000 at batch 32: 18 us at 4, 21 us at 2), and none once the grid
        // has a workgroup per CU (4096 -> 4096 at batch 256, 256 workgroups: 174 us
        // whole, 258 us in 2 parts).
        if (tiles256 < 4) want = blocks >= 256 ? 1 : std::min<int64_t>(want, 4);
        ns = int(std::max<int64_t>(1, want));
        // (6) Grids of under 2048 waves (2 per SIMD) are bound by how fast each
        // wave streams its straight-line code. When the choice above splits the
        // reduction or leaves a wave more than 14 KiB of code, segments of 16
        // channels run with a wave split of 4, or 8 where 4 would leave a wave
        // more than 14 KiB (up to 112 KiB per workgroup): more, shorter code
        // streams on more CUs, at the price of forming each shift for 16 channels
        // only. A grid of at most 32 waves doubles the split while it stays within
        // 64 waves, and a grid of 4 or more pixel tiles that fits one workgroup per
        // CU twice over is split in 2 parts (its tiles share each code stream, so
        // the shorter streams pay for the fill pass). On MI355X, kernels replayed
        // in a HIP graph: 128 -> 128, 3 x 3 at 28 x 28, batch 1 (13 tiles): 10.8
        // us (64 channels, 12 parts) -> 9.7 (16 channels, split 8) -> 8.2 us (in
        // 2 parts; 3 parts, 312 workgroups on 256 CUs: 10.2 us); 256 -> 128 at
        // batch 8: 11.6 (64 channels, split 4) -> 5.4 -> 4.0 us (split 8); 512 ->
        // 1000 at batch 32 (one tile): 14.2 -> 10.0 us (2 parts: 10.4). 2048 ->
        // 1000 at batch 128 (190 KiB per group of 16 channels) ran 61-65 us unsplit
        // with any wave split or segment width, against 40 us in 4 parts. The new
        // grid stays under 2048 waves too: ResNet-18's 128 -> 256, 3 x 3 / 2 layer
        // at batch 32 (98 tiles, 12544 waves in that form) went from 52 to 76 us,
        // its 256 -> 512, 1 x 1 / 2 layer (3200 waves) from 18 to 20 us.
        const int64_t waves = blocks * ns * sp.pgroups * sp.wsplit;
        if (base < 256 && waves < 2048 && !sp.wint && sp.kjn.empty() && tuning(kJitTn) < 0 &&
            tuning(kJitWsplit) < 0 && tuning(kJitPgroups) < 0) {
            const int64_t per_wave = code_words(sp, kTN) * 4 / (int64_t(sp.kgroups) * ns * sp.wsplit);
            if (ns > 1 || per_wave > 14 * 1024) {
                const int tn = 16;
                const int64_t kg = (g.k + tn - 1) / tn;
                const int64_t per_group = code_words(sp, tn) * 4 / kg;
                const int64_t tiles = (nq + 63) / 64;
                int ws = per_group <= 56 * 1024 ? 4 : 8;
                int64_t w = tiles * kg * ws;
                if (per_group <= 112 * 1024 && g.crs >= 8 * ws && w < 2048) {
                    while (ws < 16 && w <= 32 && g.crs >= 16 * ws) {
                        ws *= 2;
                        w *= 2;
                    }
                    const bool two = tiles >= 4 && tiles * kg * 2 <= 256 && per_group / ws > 4 * 1024 &&
                                     g.c >= 2;
                    sp.tn = tn;
                    sp.kgroups = int(kg);
                    sp.wsplit = ws;
                    sp.pgroups = 1;
                    sp.tiles_p = int(tiles);
                    ns = two ? 2 : 1;
                }
            }
        }
    }
    // (7) A grid of under 8192 waves (8 per SIMD) at a wave split of 4 or less
    // doubles the split to 8 while each share keeps 64 reduction elements per
    // part (not a strided 1 x 1 layer, whose loads span twice the cache lines;
    // not the small grids of rule (6)). On MI355X, wave split 8 on every layer:
    // ResNet-18 (N = 32, 800-6272 waves per layer) 5.7 % faster summed over its
    // layers (3 x 3 layers 5-11 %; its stride-2 1 x 1 layers 17 % faster and 5 %
    // slower), ResNet-50 (N = 128) 9 % slower, the layers of 12544 waves or more
    // 2-4 % slower, its 1024 -> 256 layers at 14 x 14 (6272 waves) 3.5 % faster.
    {
        const bool strided_point = int64_t(g.r) * g.s == 1 && (g.sh > 1 || g.sw > 1);
        const int64_t tiles64 = (nq + 63) / 64;
        const int64_t waves = tiles64 * sp.kgroups * ns * sp.wsplit;
        if (!sp.xt && sp.tn == kTN && sp.wsplit <= 4 && !strided_point && waves < 8192 &&
            g.crs / (int64_t(ns) * 8) >= 64 && sp.kjn.empty() && tuning(kJitWsplit) < 0 &&
            tuning(kJitPgroups) < 0 && tuning(kJitTn) < 0) {
            sp.wsplit = 8;
            sp.pgroups = 1;
            sp.tiles_p = int(tiles64);
        }
    }
    sp.nsplit = std::min(ns, g.c);
    const int64_t nseg = int64_t(sp.kgroups) * sp.nsplit;
    if (nseg * sp.tiles_p > INT32_MAX) return fail(DS_ERR_UNSUPPORTED, "grid too large");
    sp.nseg = int(nseg);
    // Tile-major order on small pixel grids (at most 100 tiles of 256 pixels) whose
    // input is at most 128 MiB. Workgroups land on the CUs in turn (block b on the
    // CU of b - 256 at the start, found with a probe of HW_ID on MI355X), so in this
    // order the blocks resident on a CU run one code segment, and a tile's segments
    // are spread over the 8 XCDs, each fetching the tile's input into its own L2:
    // cheap for small inputs only. A sweep of ResNet-50 at N = 128: its 14 x 14 and
    // 7 x 7 layers ran 1-12 % faster, while its 56 x 56 stride-2 1 x 1 layer (a
    // 411 MB input) ran 1.34x slower.
    // A strided 1 x 1 layer (little code, an input read at scattered pixels) takes
    // the XCD-local variant, which keeps each tile on one XCD: 4 % faster on
    // ResNet-50's 1024 -> 2048 stride-2 layer at 14 x 14, 13-25 % on ResNet-18's
    // three (N = 32). Layers with more code per input ran 5-25 % slower in it:
    // every XCD's L2 then holds every segment's code.
    {
        const int64_t tiles256 = (nq + kBlockPixels - 1) / kBlockPixels;
        const int64_t xin = sp.xh > 0 ? prod({g.n, g.c, sp.xh, sp.xw}) : prod({g.n, g.c, g.h, g.w});
        const bool strided_point = int64_t(g.r) * g.s == 1 && (g.sh > 1 || g.sw > 1);
        const bool small = tiles256 <= 100 && xin * 4 <= (int64_t(128) << 20);
        sp.tile_major = small ? (strided_point ? 2 : 1) : 0;
    }
    // Loads in flight: 14, the most the register budget holds (a sweep of every
    // ResNet-50 convolution on MI355X: 1 % faster summed than 8, up to 4 % on the
    // largest pixel grids). One tap per element (1 x 1 windows, or wider ones
    // through the padded copy): the 80-VGPR entry point, 6 waves per SIMD with 8
    // loads in flight; ResNet-50's 37 such layers (N = 128) ran 2.8 % faster
    // summed than with 96 VGPRs (8 or 14 loads in flight alike), ResNet-18's four
    // 3.6 %.
    const RegMap &m = sp.one_tap ? kMap80 : kMap96;
    const int slots = tuning(kJitSlots);
    sp.slots = std::min(m.max_slots, std::max(1, slots < 0 ? m.max_slots : slots));
    return ok();
}

// Shape checks of a forward layer given by its sizes (no pointers); fills g.
ds_status check_layer(int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, int64_t r, int64_t s,
                      int sh, int sw, int ph, int pw, int bits, ConvGeom &g)
{
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0 || k <= 0 || r <= 0 || s <= 0)
        return fail(DS_ERR_INVALID_SHAPE, "all sizes must be > 0");
    if (sh < 1 || sw < 1 || ph < 0 || pw < 0)
        return fail(DS_ERR_INVALID_ARG, "stride must be >= 1 and padding >= 0");
    const int64_t oh = h + 2 * int64_t(ph) - r, ow = w + 2 * int64_t(pw) - s;
    if (oh < 0 || ow < 0) return fail(DS_ERR_INVALID_SHAPE, "kernel larger than the padded input");
    const int64_t xe = prod({n, c, h, w}), ye = prod({n, k, oh / sh + 1, ow / sw + 1});
    const int64_t crs = prod({c, r, s});
    // x and y are addressed through buffer resources: their sizes in bytes stay below 2^31.
    if (xe < 0 || ye < 0 || xe > kMaxElems / 4 || ye > kMaxElems / 4 || crs > kMaxElems ||
        h + 2 * int64_t(ph) > kMaxElems || w + 2 * int64_t(pw) > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "tensors of 2^31 or more bytes are not supported");
    g = ConvGeom{int(n), int(c), int(h), int(w), int(k), int(r), int(s), sh, sw, ph, pw,
                 int(oh / sh + 1), int(ow / sw + 1), int(crs), bits};
    return DS_SUCCESS;
}

// A LinearShift (a 1 x 1 window on 1 x 1 inputs, output dense) runs on x^T from
// batch 32 up (see Spec::xt; MI355X, graph replays, both passes included: 2048 ->
// 1000 at batch 32 12.4 against 26.9 us on x, 512 -> 1000 at batch 32 10.2
// against 10.3 us); at batch 8 the passes cost more than they save.
void transpose_linear(Spec &sp)
{
    const ConvGeom g = sp.g;
    const int forced = tuning(kJitTranspose);
    const bool want = forced == 0 ? false : forced == 1 ? g.n > 1 : g.n >= 32;
    if (want && g.h == 1 && g.w == 1 && g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0 && sp.map.dense() &&
        int64_t(g.n) * g.c <= kMaxElems / 4 && int64_t(g.n) * g.k <= kMaxElems / 4) {
        sp.xt = true;
        sp.lin = g;
        sp.g = ConvGeom{1, g.c, 1, g.n, g.k, 1, 1, 1, 1, 0, 0, 1, g.n, g.c, g.bits};
    }
}

// Validation and planning shared by ds_jit_conv_create and ds_jit_conv_image.
ds_status plan_spec(const CreateArgs &a, Spec &sp)
{
    if (!a.wp && !a.wint) return fail(DS_ERR_NULL_POINTER, "w_packed must not be NULL");
    if (a.flags & ~(DS_RELU | DS_JIT_RESIDUAL | 0xF00u | 0x3000u)) return fail(DS_ERR_INVALID_ARG, "unknown flags");
    const uint32_t act = (a.flags >> 12) & 3u;
    if (act == 3u) return fail(DS_ERR_INVALID_ARG, "DS_ACT_I16 and DS_ACT_I8 are exclusive");
    if (a.wint && (a.flags & ~DS_RELU)) return fail(DS_ERR_INVALID_ARG, "multiplication plans take DS_RELU only");
    const int bits = flags_code_bits(a.flags);
    if (bits < 0) return fail(DS_ERR_INVALID_ARG, "DS_CODE_BITS must be 2..5 (or 0 for 5)");
    if (a.add && !a.mul) return fail(DS_ERR_INVALID_ARG, "add needs mul");
    if (a.mul && (a.mul_shift < 0 || a.mul_shift > 31))
        return fail(DS_ERR_INVALID_ARG, "mul_shift must be in [0, 31]");
    if (a.splits < 0) return fail(DS_ERR_INVALID_ARG, "splits must be >= 0");
    if (a.s > kMaxPaddedS)
        return fail(DS_ERR_UNSUPPORTED, "kernels wider than %d columns are not supported", kMaxPaddedS);
    ds_status st = check_layer(a.n, a.c, a.h, a.w, a.k, a.r, a.s, a.sh, a.sw, a.ph, a.pw, bits, sp.g);
    if (st != DS_SUCCESS) return st;
    sp.wp = a.wp;
    sp.wint = a.wint;
    sp.act_bytes = act == 1u ? 2 : act == 2u ? 1 : 4;
    sp.bias = a.bias; sp.mul = a.mul; sp.add = a.add; sp.mul_shift = a.mul ? a.mul_shift : 0;
    sp.relu = a.flags & DS_RELU;
    sp.residual = a.flags & DS_JIT_RESIDUAL;
    transpose_linear(sp);
    return finish_spec(sp, bits, a.splits);
}

// Host re-pack of the codes of one input-gradient phase (5-bit format): row c,
// column (k * Ta + t) * Tb + u holds code[k][c][r0 + sh*(Ta-1-t)][s0 + sw*(Tb-1-u)].
std::vector<uint32_t> repack_phase(const uint32_t *wp, const ConvGeom &fwd, const GradPhase &ph)
{
    const CodeFmt src = code_fmt(fwd.bits);
    const int64_t wpr_in = row_words_bits(fwd.crs, fwd.bits);
    const int Ta = ph.g.r, Tb = ph.g.s, cols = ph.g.crs;
    const int64_t wpr = row_words(cols);
    std::vector<uint32_t> out(size_t(ph.g.k) * size_t(wpr), 0u);
    for (int c = 0; c < fwd.c; ++c)
        for (int64_t wd = 0; wd < wpr; ++wd) {
            uint32_t word = 0;
            for (int j = 0; j < 6; ++j) {
                const int64_t jp = wd * 6 + j;
                uint32_t code = 15u;
                if (jp < cols) {
                    const int k = int(jp / (Ta * Tb)), rem = int(jp % (Ta * Tb));
                    const int t = rem / Tb, u = rem % Tb;
                    const int r = ph.r0 + fwd.sh * (Ta - 1 - t), s = ph.s0 + fwd.sw * (Tb - 1 - u);
                    code = src.at(wp + int64_t(k) * wpr_in, (c * fwd.r + r) * fwd.s + s);
                }
                word |= code << (5 * j);
            }
            out[size_t(c) * size_t(wpr) + size_t(wd)] = word;
        }
    return out;
}

// The stride phases of an input gradient as one problem: output-channel group
// (phase p, channels 64 q ..) of a stride-1 correlation of dy over the union of
// the phases' windows, aligned at a common padding (the largest); a phase's tap
// t sits at union tap t + (P - its padding), and the union taps outside its own
// window carry zero weights, which generate no code. Possible when at least two
// phases have taps and all of those share one output grid. Fills sp (geometry,
// map, kout, kjn) and the codes it points to; false otherwise.
bool fuse_phases(const uint32_t *wp, const ConvGeom &fwd, const std::vector<GradPhase> &phases,
                 Spec &sp, std::vector<uint32_t> &codes)
{
    std::vector<const GradPhase *> act;
    for (const GradPhase &ph : phases)
        if (ph.g.r > 0 && ph.g.s > 0) act.push_back(&ph);
    if (act.size() < 2) return false;
    int P = act[0]->g.ph, Q = act[0]->g.pw;
    for (const GradPhase *ph : act) {
        if (ph->g.oh != act[0]->g.oh || ph->g.ow != act[0]->g.ow) return false;
        P = std::max(P, ph->g.ph);
        Q = std::max(Q, ph->g.pw);
    }
    int Tu = 0, Tv = 0;
    for (const GradPhase *ph : act) {
        Tu = std::max(Tu, ph->g.r + P - ph->g.ph);
        Tv = std::max(Tv, ph->g.s + Q - ph->g.pw);
    }
    const int C = fwd.c, K = fwd.k, cpad = (C + kTN - 1) / kTN * kTN, groups = cpad / kTN;
    ConvGeom &g = sp.g;
    g = act[0]->g;
    g.k = int(act.size()) * cpad;
    g.r = Tu;
    g.s = Tv;
    g.ph = P;
    g.pw = Q;
    g.crs = K * Tu * Tv;
    g.bits = 5;
    sp.map = act[0]->map;
    sp.map.base = 0;
    const CodeFmt src = code_fmt(fwd.bits);
    const int64_t wpr_in = row_words_bits(fwd.crs, fwd.bits);
    const int64_t wpr = row_words(g.crs);
    codes.assign(size_t(g.k) * size_t(wpr), 0u);
    sp.kout.clear();
    sp.kjn.clear();
    for (size_t pi = 0; pi < act.size(); ++pi) {
        const GradPhase &ph = *act[pi];
        const int du = P - ph.g.ph, dv = Q - ph.g.pw;
        for (int q = 0; q < groups; ++q) {
            sp.kout.push_back(ph.map.base + int64_t(q) * kTN * ph.map.kstride);
            sp.kjn.push_back(std::min(kTN, C - q * kTN));
        }
        for (int c = 0; c < cpad; ++c) {
            uint32_t *row = codes.data() + (pi * size_t(cpad) + size_t(c)) * size_t(wpr);
            for (int64_t wd = 0; wd < wpr; ++wd) {
                uint32_t word = 0;
                for (int j = 0; j < 6; ++j) {
                    const int64_t jp = wd * 6 + j;
                    uint32_t code = 15u;
                    if (c < C && jp < g.crs) {
                        const int k = int(jp / (Tu * Tv)), rem = int(jp % (Tu * Tv));
                        const int t = rem / Tv - du, u = rem % Tv - dv;
                        if (t >= 0 && t < ph.g.r && u >= 0 && u < ph.g.s) {
                            const int r = ph.r0 + fwd.sh * (ph.g.r - 1 - t);
                            const int s = ph.s0 + fwd.sw * (ph.g.s - 1 - u);
                            code = src.at(wp + int64_t(k) * wpr_in, (c * fwd.r + r) * fwd.s + s);
                        }
                    }
                    word |= code << (5 * j);
                }
                row[wd] = word;
            }
        }
    }
    sp.wp = codes.data();
    return true;
}

}  // namespace
}  // namespace ds

using namespace ds;

// A plan: one generated kernel (forward), or the phases of an input gradient,
// each a plan of its own writing its part of dx, plus the parts no tap reaches.
struct ds_jit_conv {
    int device = -1;
    hipModule_t module = nullptr;
    hipFunction_t fn = nullptr;
    Spec sp;
    int group_tiles = 16;           // in 256-pixel tiles
    int64_t code_bytes = 0;
    int32_t *init = nullptr;        // [k] bias or zeros: y's start for split-K
    int32_t *mul = nullptr, *add = nullptr;
    bool backward = false;
    ConvGeom fwd;                   // backward: the forward layer
    int32_t *xpad = nullptr;        // windows over 3 x 3: the zero-padded input [n][c][xh][xw];
                                    // a transposed LinearShift: x^T [c][n] (int32)
    int32_t *dense = nullptr;       // split phase: its partial sums, dense [n][k][oh][ow];
                                    // a transposed LinearShift: y^T [k][n]
    OutMap scatter;                 // ... and where they go in dx
    std::vector<ds_jit_conv *> parts;
    std::vector<GradPhase> zeros;   // backward: phases whose dx positions are 0
};

static ds_status destroy_plan(ds_jit_conv *p)
{
    if (!p) return ok();
    hipError_t e = hipSuccess;
    ds_status st = DS_SUCCESS;
    for (ds_jit_conv *q : p->parts) {
        const ds_status sq = destroy_plan(q);
        if (st == DS_SUCCESS) st = sq;
    }
    if (p->module) e = hipModuleUnload(p->module);
    for (int32_t *q : {p->init, p->mul, p->add, p->dense, p->xpad})
        if (q) {
            const hipError_t f = hipFree(q);
            if (e == hipSuccess) e = f;
        }
    delete p;
    if (e != hipSuccess) return fail(DS_ERR_HIP, "ds_jit_conv_destroy: %s", hipGetErrorString(e));
    if (st != DS_SUCCESS) return st;
    return ok();
}

static ds_status upload(int32_t **dst, const int32_t *src, int k, bool zeros)
{
    if (hipMalloc(dst, size_t(k) * 4) != hipSuccess) return fail(DS_ERR_HIP, "hipMalloc failed");
    hipError_t e = zeros ? hipMemset(*dst, 0, size_t(k) * 4)
                         : hipMemcpy(*dst, src, size_t(k) * 4, hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(DS_ERR_HIP, "upload: %s", hipGetErrorString(e));
    return ok();
}

// Generates, loads and completes the plan of one planned spec (host bias, mul
// and add as in the spec; they are not kept).
static ds_status build_plan(const Spec &spec, ds_jit_conv **out)
{
    *out = nullptr;
    ds_jit_conv *p = new ds_jit_conv;
    p->sp = spec;
    std::vector<uint8_t> img;
    const std::vector<uint32_t> body = generate_body(p->sp);
    p->code_bytes = int64_t(body.size()) * 4;
    ds_status st = splice_body(body, img);
    if (st != DS_SUCCESS) {
        delete p;
        return st;
    }
    if (hipGetDevice(&p->device) != hipSuccess) {
        delete p;
        return fail(DS_ERR_HIP, "no HIP device");
    }
    hipError_t e = hipModuleLoadData(&p->module, img.data());
    if (e == hipSuccess)
        e = hipModuleGetFunction(&p->fn, p->module, (p->sp.one_tap ? kMap80 : kMap96).kernel);
    if (e != hipSuccess) {
        destroy_plan(p);
        return fail(DS_ERR_HIP, "loading the generated code: %s", hipGetErrorString(e));
    }
    const int K = p->sp.g.k;
    // What the separate split-K passes need is copied to the device here.
    if (p->sp.nsplit > 1) {
        st = upload(&p->init, spec.bias, K, !spec.bias);
        if (st == DS_SUCCESS && spec.mul) st = upload(&p->mul, spec.mul, K, false);
        if (st == DS_SUCCESS && spec.add) st = upload(&p->add, spec.add, K, false);
        if (st != DS_SUCCESS) {
            const std::string msg = last_error();
            destroy_plan(p);
            return fail(st, "%s", msg.c_str());
        }
    }
    if (p->sp.xh > 0 || p->sp.xt) {
        const size_t bytes = p->sp.xt ? size_t(p->sp.g.c) * p->sp.g.w * 4
                                      : size_t(p->sp.g.n) * p->sp.g.c * p->sp.xh * p->sp.xw * 4;
        if (hipMalloc(&p->xpad, bytes) != hipSuccess) {
            destroy_plan(p);
            return fail(DS_ERR_HIP, "hipMalloc of %zu bytes (%s input) failed", bytes,
                        p->sp.xt ? "transposed" : "padded");
        }
    }
    if (p->sp.xt) {
        const size_t bytes = size_t(p->sp.g.k) * p->sp.g.w * 4;
        if (hipMalloc(&p->dense, bytes) != hipSuccess) {
            destroy_plan(p);
            return fail(DS_ERR_HIP, "hipMalloc of %zu bytes (transposed output) failed", bytes);
        }
    }
    p->sp.bias = p->sp.mul = p->sp.add = nullptr;
    p->sp.wp = nullptr;
    p->sp.wint = nullptr;
    p->group_tiles = tuning(kJitGroupTiles) > 0 ? tuning(kJitGroupTiles) : 16;
    *out = p;
    return ok();
}

extern "C" ds_status ds_jit_conv_image(const uint32_t *w_packed, const int32_t *bias,
                                       const int32_t *mul, const int32_t *add, int32_t mul_shift,
                                       int64_t n, int64_t c, int64_t h, int64_t w, int64_t k,
                                       int64_t r, int64_t s, int32_t stride_h, int32_t stride_w,
                                       int32_t pad_h, int32_t pad_w, uint32_t flags,
                                       int32_t splits, void *image, int64_t capacity,
                                       int64_t *size)
{
    try {
        if (!size) return fail(DS_ERR_NULL_POINTER, "size must not be NULL");
        Spec sp;
        const CreateArgs a{w_packed, nullptr, bias, mul, add, mul_shift, n, c, h, w, k, r, s,
                           stride_h, stride_w, pad_h, pad_w, flags, splits};
        ds_status st = plan_spec(a, sp);
        if (st != DS_SUCCESS) return st;
        std::vector<uint8_t> img;
        st = splice_body(generate_body(sp), img);
        if (st != DS_SUCCESS) return st;
        *size = int64_t(img.size());
        if (!image || capacity < int64_t(img.size()))
            return fail(DS_ERR_BUFFER_TOO_SMALL, "the code object needs %lld bytes", (long long)img.size());
        std::memcpy(image, img.data(), img.size());
        return ok();
    } catch (const std::bad_alloc &) {
        return fail(DS_ERR_HIP, "out of host memory");
    }
}

extern "C" ds_status ds_jit_conv_create(const uint32_t *w_packed, const int32_t *bias,
                                        const int32_t *mul, const int32_t *add, int32_t mul_shift,
                                        int64_t n, int64_t c, int64_t h, int64_t w, int64_t k,
                                        int64_t r, int64_t s, int32_t stride_h, int32_t stride_w,
                                        int32_t pad_h, int32_t pad_w, uint32_t flags,
                                        int32_t splits, ds_jit_conv **plan)
{
    if (!plan) return fail(DS_ERR_NULL_POINTER, "plan must not be NULL");
    *plan = nullptr;
    try {
        Spec sp;
        const CreateArgs a{w_packed, nullptr, bias, mul, add, mul_shift, n, c, h, w, k, r, s,
                           stride_h, stride_w, pad_h, pad_w, flags, splits};
        ds_status st = plan_spec(a, sp);
        if (st != DS_SUCCESS) return st;
        return build_plan(sp, plan);
    } catch (const std::bad_alloc &) {
        return fail(DS_ERR_HIP, "out of host memory");
    }
}

extern "C" ds_status ds_jit_conv_backward_data_create(const uint32_t *w_packed, int64_t n,
                                                      int64_t c, int64_t h, int64_t w, int64_t k,
                                                      int64_t r, int64_t s, int32_t stride_h,
                                                      int32_t stride_w, int32_t pad_h,
                                                      int32_t pad_w, uint32_t flags,
                                                      int32_t splits, ds_jit_conv **plan)
{
    if (!plan) return fail(DS_ERR_NULL_POINTER, "plan must not be NULL");
    *plan = nullptr;
    if (!w_packed) return fail(DS_ERR_NULL_POINTER, "w_packed must not be NULL");
    const int bits = flags_code_bits(flags);
    if ((flags & ~0xF00u) != 0 || bits < 0)
        return fail(DS_ERR_INVALID_ARG, "flags must be 0 apart from DS_CODE_BITS(2..5)");
    if (splits < 0) return fail(DS_ERR_INVALID_ARG, "splits must be >= 0");
    ds_jit_conv *p = nullptr;
    try {
        ConvGeom g;
        ds_status st = check_layer(n, c, h, w, k, r, s, stride_h, stride_w, pad_h, pad_w, bits, g);
        if (st != DS_SUCCESS) return st;
        const std::vector<GradPhase> phases = grad_phases(g);
        for (const GradPhase &ph : phases)
            if (ph.g.s > kMaxPaddedS)
                return fail(DS_ERR_UNSUPPORTED, "a stride phase is wider than %d columns", kMaxPaddedS);
        const CodeFmt fmt = code_fmt(bits);
        const int64_t rw = row_words_bits(g.crs, bits);
        const int used = fmt.per_word * bits;
        for (int64_t i = 0; used < 32 && i < int64_t(g.k) * rw; ++i)
            if (w_packed[i] >> used)
                return fail(DS_ERR_INVALID_CODE, "bits %d-31 of packed word %lld are not 0", used, (long long)i);
        p = new ds_jit_conv;
        p->backward = true;
        p->fwd = g;
        if (hipGetDevice(&p->device) != hipSuccess) {
            delete p;
            return fail(DS_ERR_HIP, "no HIP device");
        }
        for (const GradPhase &ph : phases)
            if (ph.g.r == 0 || ph.g.s == 0) p->zeros.push_back(ph);
        // Stride phases fused into one kernel when they can be (no split of the
        // reduction: the wave split supplies the parallelism); else one per phase.
        {
            Spec sp;
            std::vector<uint32_t> codes;
            if (splits <= 1 && fuse_phases(w_packed, g, phases, sp, codes)) {
                st = finish_spec(sp, 5, 1, 0);
                ds_jit_conv *part = nullptr;
                if (st == DS_SUCCESS) st = build_plan(sp, &part);
                if (st != DS_SUCCESS) {
                    const std::string msg = last_error();
                    destroy_plan(p);
                    return fail(st, "%s", msg.c_str());
                }
                p->code_bytes += part->code_bytes;
                p->parts.push_back(part);
                *plan = p;
                return ok();
            }
        }
        for (const GradPhase &ph : phases) {
            if (ph.g.r == 0 || ph.g.s == 0) continue;
            const std::vector<uint32_t> codes = repack_phase(w_packed, g, ph);
            Spec sp;
            sp.g = ph.g;
            sp.wp = codes.data();
            sp.map = ph.map;
            transpose_linear(sp);  // the input gradient of a LinearShift: dx = dy W, on dy^T
            // A strided phase that splits pays a dense buffer's round trip (below), so
            // it splits only toward the 384-block floor (MI355X: a 3x3 stride-2 layer's
            // phases ran 1.3x faster unsplit at 392 blocks than at 2 parts, and 1.1x
            // faster at 2 parts than at 3-11 on a 200-block grid).
            st = finish_spec(sp, 5, splits, ph.map.dense() ? 3072 : 0);
            // Split partial sums meet through int32 atomics, which on a strided map land
            // on scattered addresses: such a phase accumulates densely into a buffer of
            // its own and is scattered into dx afterwards.
            const bool via_dense = st == DS_SUCCESS && sp.nsplit > 1 && !ph.map.dense();
            if (via_dense) sp.map = OutMap();
            ds_jit_conv *part = nullptr;
            if (st == DS_SUCCESS) st = build_plan(sp, &part);
            if (st == DS_SUCCESS && via_dense) {
                part->scatter = ph.map;
                const size_t bytes = size_t(ph.g.n) * ph.g.k * ph.g.oh * ph.g.ow * 4;
                if (hipMalloc(&part->dense, bytes) != hipSuccess) {
                    destroy_plan(part);
                    part = nullptr;
                    st = fail(DS_ERR_HIP, "hipMalloc of %zu bytes failed", bytes);
                }
            }
            if (st != DS_SUCCESS) {
                const std::string msg = last_error();
                destroy_plan(p);
                return fail(st, "%s", msg.c_str());
            }
            p->code_bytes += part->code_bytes;
            p->parts.push_back(part);
        }
        *plan = p;
        return ok();
    } catch (const std::bad_alloc &) {
        if (p) destroy_plan(p);
        return fail(DS_ERR_HIP, "out of host memory");
    }
}

// The first pass of a transposed LinearShift: xt [c][n] = x [n][c] as int32
// (sign-extended from int16 / int8 elements), in 32 x 32 tiles through LDS
// (reads and writes coalesced; 64 x 64 tiles, a quarter as many workgroups, ran
// 4096 -> 4096 at batch 256 at 0.9 TB/s), and with a split reduction y^T [k][n]
// = init[k], the start of the parts' atomic adds, in the workgroups after the
// tiles. 256 threads.
constexpr int kTT = 32;  // transpose tile

template <typename T>
__global__ void __launch_bounds__(256)
transpose_in_kernel(const T *__restrict__ x, int32_t *__restrict__ xt, int rows, int cols, int tiles_c,
                    int tiles, const int32_t *__restrict__ init, int32_t *__restrict__ yt, int k)
{
    __shared__ int32_t tile[kTT][kTT + 1];
    const int b = int(blockIdx.x);
    if (b >= tiles) {
        // fill: y^T [k][rows] = init[k], 256 elements per workgroup
        const int64_t i = int64_t(b - tiles) * 256 + threadIdx.x;
        if (i < int64_t(k) * rows) yt[i] = init[i / rows];
        return;
    }
    const int c0 = (b % tiles_c) * kTT, r0 = (b / tiles_c) * kTT;
    const int tx = threadIdx.x % kTT, ty = threadIdx.x / kTT;
    for (int i = ty; i < kTT; i += 256 / kTT) {
        const int r = r0 + i, c = c0 + tx;
        if (r < rows && c < cols) tile[i][tx] = int32_t(x[int64_t(r) * cols + c]);
    }
    __syncthreads();
    for (int i = ty; i < kTT; i += 256 / kTT) {
        const int c = c0 + i, r = r0 + tx;
        if (c < cols && r < rows) xt[int64_t(c) * rows + r] = tile[tx][i];
    }
}

static hipError_t run_transpose_in(const int32_t *x, int32_t *xt, int rows, int cols, int xbytes,
                                   const int32_t *init, int32_t *yt, int k, hipStream_t st)
{
    const int tiles_c = (cols + kTT - 1) / kTT;
    const int64_t tiles = int64_t(tiles_c) * ((rows + kTT - 1) / kTT);
    const int64_t fills = init ? (int64_t(k) * rows + 255) / 256 : 0;
    if (tiles + fills > INT32_MAX) return hipErrorInvalidValue;
    if (tiles + fills == 0) return hipSuccess;
    const dim3 grid{unsigned(tiles + fills)}, block{256u};
    if (xbytes == 2)
        hipLaunchKernelGGL(transpose_in_kernel<int16_t>, grid, block, 0, st, reinterpret_cast<const int16_t *>(x),
                           xt, rows, cols, tiles_c, int(tiles), init, yt, k);
    else if (xbytes == 1)
        hipLaunchKernelGGL(transpose_in_kernel<int8_t>, grid, block, 0, st, reinterpret_cast<const int8_t *>(x),
                           xt, rows, cols, tiles_c, int(tiles), init, yt, k);
    else
        hipLaunchKernelGGL(transpose_in_kernel<int32_t>, grid, block, 0, st, x, xt, rows, cols, tiles_c,
                           int(tiles), init, yt, k);
    return hipGetLastError();
}

// The last pass of a transposed LinearShift: y [n][k] = yt [k][n] in 32 x 32
// tiles through LDS, with what the generated kernel left of the epilogue: for a
// split reduction all of it (v * mul[k] >> mul_shift, floor, + add[k]), and
// then, for a layer with a residual, + res[n][k] and the ReLU. 256 threads.
__global__ void __launch_bounds__(256)
transpose_back_kernel(const int32_t *__restrict__ yt, int32_t *__restrict__ y, int rows, int cols,
                      int tiles_c, const int32_t *__restrict__ mul, const int32_t *__restrict__ add,
                      int mul_shift, const int32_t *__restrict__ res, int relu)
{
    __shared__ int32_t tile[kTT][kTT + 1];
    const int n0 = int(blockIdx.x % unsigned(tiles_c)) * kTT, k0 = int(blockIdx.x / unsigned(tiles_c)) * kTT;
    const int tx = threadIdx.x % kTT, ty = threadIdx.x / kTT;
    for (int i = ty; i < kTT; i += 256 / kTT) {
        const int k = k0 + i, n = n0 + tx;
        if (k < cols && n < rows) tile[i][tx] = yt[int64_t(k) * rows + n];
    }
    __syncthreads();
    for (int i = ty; i < kTT; i += 256 / kTT) {
        const int n = n0 + i, k = k0 + tx;
        if (n < rows && k < cols) {
            const int64_t o = int64_t(n) * cols + k;
            uint32_t v = uint32_t(tile[tx][i]);
            if (mul) v = uint32_t(int32_t((int64_t(int32_t(v)) * mul[k]) >> mul_shift)) + (add ? uint32_t(add[k]) : 0u);
            if (res) v += uint32_t(res[o]);
            if (relu && int32_t(v) < 0) v = 0u;
            y[o] = int32_t(v);
        }
    }
}

static hipError_t run_transpose_back(const int32_t *yt, int32_t *y, int rows, int cols, const int32_t *mul,
                                     const int32_t *add, int mul_shift, const int32_t *res, bool relu,
                                     hipStream_t st)
{
    const int tiles_c = (rows + kTT - 1) / kTT;
    const int64_t tiles = int64_t(tiles_c) * ((cols + kTT - 1) / kTT);
    if (tiles <= 0) return hipSuccess;
    if (tiles > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(transpose_back_kernel, dim3{unsigned(tiles)}, dim3{256u}, 0, st, yt, y, rows, cols,
                       tiles_c, mul, add, mul_shift, res, relu ? 1 : 0);
    return hipGetLastError();
}

// Enqueues one generated kernel (with its split-K fill and epilogue passes).
static hipError_t run_part(const ds_jit_conv *plan, const int32_t *x, const int32_t *residual,
                           int32_t *y, int64_t x_bytes, int64_t y_bytes, hipStream_t st)
{
    const Spec &sp = plan->sp;
    const ConvGeom &g = sp.g;
    const OutMap m = full_map(sp);
    const bool split = sp.nsplit > 1;
    int32_t *const dst = y;
    if (plan->dense) {  // accumulate densely (y^T for a transposed LinearShift), scatter below
        y = plan->dense;
        y_bytes = int64_t(g.n) * g.k * g.oh * g.ow * 4;
    }
    hipError_t e = hipSuccess;
    // Padded input: the template sees the copy as x with no padding, and its tap
    // (0, 0) offset is where each lane's window starts.
    const bool padded = sp.xh > 0;
    if (padded) {
        e = run_pad_planes(x, plan->xpad, int64_t(g.n) * g.c, g.h, g.w, g.ph, g.pw, sp.xh, sp.xw, st,
                           sp.act_bytes);
        x = plan->xpad;
        x_bytes = int64_t(g.n) * g.c * sp.xh * sp.xw * 4;
    } else if (sp.xt) {
        // with a split reduction, y^T starts at the bias in the same pass
        e = run_transpose_in(x, plan->xpad, sp.lin.n, sp.lin.c, sp.act_bytes, split ? plan->init : nullptr, y,
                             sp.lin.k, st);
        x = plan->xpad;
        x_bytes = int64_t(sp.lin.n) * sp.lin.c * 4;
    }
    if (e == hipSuccess && split && !sp.xt) e = run_fill_mapped(g, plan->init, y, sp.map, st);
    if (e == hipSuccess) {
        JitArgs a;
        a.x = x;
        a.y = y;
        a.residual = split || sp.xt ? nullptr : residual;
        a.x_bytes = int(x_bytes);
        a.xshift = padded || sp.xt || sp.act_bytes == 4 ? 2 : sp.act_bytes == 2 ? 1 : 0;
        a.y_bytes = int(y_bytes);
        a.OHOW = g.oh * g.ow;
        a.NQ = g.n * a.OHOW;
        a.OW = g.ow; a.C = g.c; a.K = g.k;
        a.H = padded ? sp.xh : g.h;
        a.W = padded ? sp.xw : g.w;
        a.HW = a.H * a.W;
        a.sh = g.sh; a.sw = g.sw;
        a.ph = padded ? 0 : g.ph;
        a.pw = padded ? 0 : g.pw;
        a.ybase = int(m.base); a.ynst = m.nstride; a.yrst = m.rstride; a.ycst = m.cstride;
        a.tiles_p = sp.tiles_p;
        const int per256 = 4 / sp.pgroups;  // pixel tiles per 256 pixels
        a.group_tiles = std::min(plan->group_tiles * per256, sp.tiles_p);
        a.nseg = sp.nseg;
        a.wsplit_log2 = sp.wsplit == 16 ? 4 : sp.wsplit == 8 ? 3 : sp.wsplit == 4 ? 2 : sp.wsplit == 2 ? 1 : 0;
        a.pgroups_log2 = sp.pgroups == 4 ? 2 : sp.pgroups == 2 ? 1 : 0;
        const int order = tuning(kJitOrder);
        a.tile_major = order < 0 ? sp.tile_major : order >= 0 && order <= 2 ? order : 0;
        a.div_ohow = make_fastdiv(uint32_t(a.OHOW));
        a.div_ow = make_fastdiv(uint32_t(a.OW));
        void *args[] = {&a};
        // LDS: 16 KiB of partial sums per group of 64 pixels in the workgroup.
        const unsigned lds = sp.wsplit > 1 ? unsigned(sp.pgroups) * 16384u : 0u;
        const unsigned threads = 64u * unsigned(sp.pgroups * sp.wsplit);
        e = hipModuleLaunchKernel(plan->fn, unsigned(int64_t(sp.tiles_p) * sp.nseg), 1, 1,
                                  threads, 1, 1, lds, st, args, nullptr);
    }
    if (e == hipSuccess && split && !sp.xt) {
        Epilogue epi;
        epi.mul = plan->mul;
        epi.add = plan->add;
        epi.res = residual;
        epi.mul_shift = sp.mul_shift;
        epi.relu = sp.relu;
        if (epi.any()) e = run_epilogue(g, y, epi, st);
    }
    // A transposed LinearShift ends in the pass that transposes y^T into y, with
    // the whole epilogue of a split reduction, else the residual and its ReLU.
    if (e == hipSuccess && sp.xt)
        e = run_transpose_back(plan->dense, dst, sp.lin.n, sp.lin.k, split ? plan->mul : nullptr,
                               split ? plan->add : nullptr, sp.mul_shift, residual,
                               (split || residual) && sp.relu, st);
    else if (e == hipSuccess && plan->dense)
        e = run_copy_mapped(g, plan->dense, dst, plan->scatter, st);
    return e;
}

extern "C" ds_status ds_jit_conv_run(const ds_jit_conv *plan, const void *xv,
                                     const int32_t *residual, int32_t *y, void *stream)
{
    // x holds int32 elements, or int16 / int8 ones for a plan made with DS_ACT_I16 /
    // DS_ACT_I8; the kernels address it in bytes.
    const int32_t *x = static_cast<const int32_t *>(xv);
    if (!plan || !x || !y) return fail(DS_ERR_NULL_POINTER, "plan, x and y must not be NULL");
    const bool res_wanted = !plan->backward && plan->sp.residual;
    if (res_wanted != (residual != nullptr))
        return fail(DS_ERR_INVALID_ARG, res_wanted ? "the plan adds a residual: residual must not be NULL"
                                                   : "the plan adds no residual: residual must be NULL");
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != plan->device)
        return fail(DS_ERR_INVALID_ARG, "the plan was made on device %d, the current device is %d", plan->device, dev);
    // Forward: x [n][c][h][w] -> y [n][k][oh][ow]; input gradient: dy -> dx of the forward layer.
    const ConvGeom &g = plan->backward ? plan->fwd : plan->sp.g;
    const int64_t fx = int64_t(g.n) * g.c * g.h * g.w * (plan->backward ? 4 : plan->sp.act_bytes);
    const int64_t fy = int64_t(g.n) * g.k * g.oh * g.ow * 4;
    const int64_t xb = plan->backward ? fy : fx, yb = plan->backward ? fx : fy;
    const char *xn = plan->backward ? "dy" : "x", *yn = plan->backward ? "dx" : "y";
    if (overlap(x, xb, y, yb)) return fail(DS_ERR_INVALID_ARG, "%s overlaps %s", yn, xn);
    if (residual && overlap(residual, yb, y, yb)) return fail(DS_ERR_INVALID_ARG, "y overlaps residual");
    if (!device_range_ok(x, xb)) return fail(DS_ERR_INVALID_ARG, "%s is not a device buffer of %lld bytes", xn, (long long)xb);
    if (!device_range_ok(y, yb)) return fail(DS_ERR_INVALID_ARG, "%s is not a device buffer of %lld bytes", yn, (long long)yb);
    if (residual && !device_range_ok(residual, yb))
        return fail(DS_ERR_INVALID_ARG, "residual is not a device buffer of %lld bytes", (long long)yb);

    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    if (!plan->backward) {
        e = run_part(plan, x, residual, y, xb, yb, st);
    } else {
        // Positions no tap reaches are zero: all of dx is cleared densely first.
        if (!plan->zeros.empty())
            e = run_fill_zero(y, int64_t(g.n) * g.c * g.h * g.w, st);
        for (const ds_jit_conv *part : plan->parts)
            if (e == hipSuccess) e = run_part(part, x, nullptr, y, xb, yb, st);
    }
    if (e != hipSuccess) return fail(DS_ERR_HIP, "ds_jit_conv_run: %s", hipGetErrorString(e));
    return ok();
}

extern "C" ds_status ds_jit_conv_destroy(ds_jit_conv *plan) { return destroy_plan(plan); }

extern "C" ds_status ds_jit_conv_query(const ds_jit_conv *plan, int64_t *code_bytes,
                                       int32_t *segments, int32_t *splits)
{
    if (!plan) return fail(DS_ERR_NULL_POINTER, "plan must not be NULL");
    int32_t seg = plan->backward ? 0 : plan->sp.nseg, sp = plan->backward ? 0 : plan->sp.nsplit;
    for (const ds_jit_conv *q : plan->parts) {
        seg += q->sp.nseg;
        sp = std::max(sp, q->sp.nsplit);
    }
    if (code_bytes) *code_bytes = plan->code_bytes;
    if (segments) *segments = seg;
    if (splits) *splits = sp;
    return ok();
}

extern "C" ds_status ds_jit_conv_layout(const ds_jit_conv *plan, int32_t *channels, int32_t *wsplit,
                                        int32_t *pixel_groups, int32_t *pixel_tiles, int32_t *transposed)
{
    if (!plan) return fail(DS_ERR_NULL_POINTER, "plan must not be NULL");
    const ds_jit_conv *k = plan->backward ? (plan->parts.empty() ? nullptr : plan->parts.front()) : plan;
    if (channels) *channels = k ? k->sp.tn : kTN;
    if (wsplit) *wsplit = k ? k->sp.wsplit : 1;
    if (pixel_groups) *pixel_groups = k ? k->sp.pgroups : 4;
    if (pixel_tiles) *pixel_tiles = k ? k->sp.tiles_p : 0;
    if (transposed) *transposed = k && k->sp.xt ? 1 : 0;
    return ok();
}

// ---------------------------------------------------------------------------
// Multiplication plans: the comparison operator of Section 6's timing (a
// multiplication-based kernel) in the plans' own tiling, for side-by-side
// timing with the shift plans. Not part of DeepShift.

extern "C" ds_status ds_jit_conv_mul_image(const int32_t *w, const int32_t *bias, int64_t n,
                                           int64_t c, int64_t h, int64_t w_, int64_t k, int64_t r,
                                           int64_t s, int32_t stride_h, int32_t stride_w,
                                           int32_t pad_h, int32_t pad_w, uint32_t flags,
                                           int32_t splits, void *image, int64_t capacity,
                                           int64_t *size)
{
    try {
        if (!size) return fail(DS_ERR_NULL_POINTER, "size must not be NULL");
        if (!w) return fail(DS_ERR_NULL_POINTER, "w must not be NULL");
        Spec sp;
        const CreateArgs a{nullptr, w, bias, nullptr, nullptr, 0, n, c, h, w_, k, r, s,
                           stride_h, stride_w, pad_h, pad_w, flags, splits};
        ds_status st = plan_spec(a, sp);
        if (st != DS_SUCCESS) return st;
        std::vector<uint8_t> img;
        st = splice_body(generate_body(sp), img);
        if (st != DS_SUCCESS) return st;
        *size = int64_t(img.size());
        if (!image || capacity < int64_t(img.size()))
            return fail(DS_ERR_BUFFER_TOO_SMALL, "the code object needs %lld bytes", (long long)img.size());
        std::memcpy(image, img.data(), img.size());
        return ok();
    } catch (const std::bad_alloc &) {
        return fail(DS_ERR_HIP, "out of host memory");
    }
}

extern "C" ds_status ds_jit_conv_mul_create(const int32_t *w, const int32_t *bias, int64_t n,
                                            int64_t c, int64_t h, int64_t w_, int64_t k, int64_t r,
                                            int64_t s, int32_t stride_h, int32_t stride_w,
                                            int32_t pad_h, int32_t pad_w, uint32_t flags,
                                            int32_t splits, ds_jit_conv **plan)
{
    if (!plan) return fail(DS_ERR_NULL_POINTER, "plan must not be NULL");
    *plan = nullptr;
    try {
        if (!w) return fail(DS_ERR_NULL_POINTER, "w must not be NULL");
        Spec sp;
        const CreateArgs a{nullptr, w, bias, nullptr, nullptr, 0, n, c, h, w_, k, r, s,
                           stride_h, stride_w, pad_h, pad_w, flags, splits};
        const ds_status st = plan_spec(a, sp);
        if (st != DS_SUCCESS) return st;
        return build_plan(sp, plan);
    } catch (const std::bad_alloc &) {
        return fail(DS_ERR_HIP, "out of host memory");
    }
}
