// Host-side entry points: the packed weight formats (DeepShift Section 4: one
// sign bit and a 4-bit shift per weight; Section 5's shorter shift ranges in 4,
// 3 or 2 bits) and status reporting.
//
// Packed layout of b-bit codes: floor(32 / b) codes per uint32 word, code j in
// bits [b*j, b*j + b), unused top bits zero, each row padded to whole words
// with the zero code. A b-bit code is the sign in its top bit and the shift
// code below, all ones meaning a zero weight; for b = 5 it is the canonical
// code (six per word, bits 30-31 zero, zero weight = shift code 15).
#include <cstring>
#include <string>

#include "common.hpp"

namespace ds {
std::string &last_error()
{
    static thread_local std::string msg;
    return msg;
}
}  // namespace ds

using namespace ds;

extern "C" int64_t ds_packed_row_words(int64_t cols) { return row_words(cols); }

extern "C" int64_t ds_packed_row_words_bits(int64_t cols, int32_t bits)
{
    if (bits < 2 || bits > 5) return -1;
    return row_words_bits(cols, bits);
}

extern "C" ds_status ds_pack_shift_weights_bits(const uint8_t *codes, int64_t rows, int64_t cols,
                                                int32_t bits, uint32_t *packed,
                                                int64_t packed_words)
{
    if (!codes || !packed) return fail(DS_ERR_NULL_POINTER, "pack: NULL pointer");
    if (bits < 2 || bits > 5) return fail(DS_ERR_INVALID_ARG, "pack: bits must be in [2, 5]");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "pack: rows and cols must be > 0");
    const int per = 32 / bits;
    const uint32_t zero = (1u << (bits - 1)) - 1u;  // the all-ones shift field
    const int64_t wpr = row_words_bits(cols, bits);
    const int64_t need = prod({rows, wpr});
    if (need < 0 || prod({rows, cols}) < 0 || cols > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "pack: size overflow");
    if (packed_words < need)
        return fail(DS_ERR_BUFFER_TOO_SMALL, "pack: need %lld words, have %lld",
                    (long long)need, (long long)packed_words);
    // Validate every code before writing anything.
    for (int64_t i = 0; i < rows * cols; ++i) {
        const unsigned code = codes[i], sh = code & 15u;
        if (code > 31)
            return fail(DS_ERR_INVALID_CODE, "pack: code %u at index %lld is >= 32", code, (long long)i);
        if (sh != 15u && sh >= zero)
            return fail(DS_ERR_INVALID_CODE, "pack: code %u at index %lld needs more than %d bits",
                        code, (long long)i, int(bits));
    }
    for (int64_t r = 0; r < rows; ++r) {
        const uint8_t *row = codes + r * cols;
        uint32_t *out = packed + r * wpr;
        for (int64_t wd = 0; wd < wpr; ++wd) {
            uint32_t word = 0;
            for (int j = 0; j < per; ++j) {
                const int64_t col = wd * per + j;
                uint32_t raw = zero;                      // padding: a zero weight
                if (col < cols) {
                    const uint32_t code = row[col], sh = code & 15u;
                    raw = ((code >> 4) << (bits - 1)) | (sh == 15u ? zero : sh);
                }
                word |= raw << (bits * j);
            }
            out[wd] = word;
        }
    }
    return ok();
}

extern "C" ds_status ds_unpack_shift_weights_bits(const uint32_t *packed, int64_t rows,
                                                  int64_t cols, int32_t bits, uint8_t *codes,
                                                  int64_t codes_len)
{
    if (!codes || !packed) return fail(DS_ERR_NULL_POINTER, "unpack: NULL pointer");
    if (bits < 2 || bits > 5) return fail(DS_ERR_INVALID_ARG, "unpack: bits must be in [2, 5]");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "unpack: rows and cols must be > 0");
    const int per = 32 / bits;
    const int64_t wpr = row_words_bits(cols, bits);
    const int64_t need = prod({rows, cols});
    if (need < 0 || prod({rows, wpr}) < 0 || cols > kMaxElems)
        return fail(DS_ERR_UNSUPPORTED, "unpack: size overflow");
    if (codes_len < need)
        return fail(DS_ERR_BUFFER_TOO_SMALL, "unpack: need %lld bytes, have %lld",
                    (long long)need, (long long)codes_len);
    const int used = per * bits;
    for (int64_t i = 0; used < 32 && i < rows * wpr; ++i)
        if (packed[i] >> used)
            return fail(DS_ERR_INVALID_CODE, "unpack: word %lld has bits %d-31 set", (long long)i, used);
    const CodeFmt fmt = code_fmt(bits);
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t col = 0; col < cols; ++col)
            codes[r * cols + col] = uint8_t(fmt.at(packed + r * wpr, int(col)));
    return ok();
}

extern "C" ds_status ds_pack_shift_weights(const uint8_t *codes, int64_t rows, int64_t cols,
                                           uint32_t *packed, int64_t packed_words)
{
    return ds_pack_shift_weights_bits(codes, rows, cols, 5, packed, packed_words);
}

extern "C" ds_status ds_unpack_shift_weights(const uint32_t *packed, int64_t rows, int64_t cols,
                                             uint8_t *codes, int64_t codes_len)
{
    return ds_unpack_shift_weights_bits(packed, rows, cols, 5, codes, codes_len);
}

extern "C" const char *ds_status_string(ds_status st)
{
    switch (st) {
    case DS_SUCCESS: return "success";
    case DS_ERR_NULL_POINTER: return "null pointer";
    case DS_ERR_INVALID_SHAPE: return "invalid shape";
    case DS_ERR_INVALID_ARG: return "invalid argument";
    case DS_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case DS_ERR_INVALID_CODE: return "invalid weight code";
    case DS_ERR_HIP: return "HIP runtime error";
    case DS_ERR_UNSUPPORTED: return "unsupported size";
    case DS_STATUS_MAX_: break;
    }
    return "unknown status";
}

extern "C" const char *ds_last_error_message(void) { return last_error().c_str(); }
