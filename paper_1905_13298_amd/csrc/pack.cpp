// Host-side entry points: the 5-bit weight format (DeepShift Section 4: one
// sign bit and a 4-bit shift per weight) and status reporting.
//
// Packed layout: six codes per uint32 word, code j in bits [5j, 5j + 5),
// bits 30-31 zero, each row padded to whole words with code 15 (zero weight).
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

extern "C" ds_status ds_pack_shift_weights(const uint8_t *codes, int64_t rows, int64_t cols,
                                           uint32_t *packed, int64_t packed_words)
{
    if (!codes || !packed) return fail(DS_ERR_NULL_POINTER, "pack: NULL pointer");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "pack: rows and cols must be > 0");
    const int64_t wpr = row_words(cols);
    const int64_t need = prod({rows, wpr});
    if (need < 0 || prod({rows, cols}) < 0) return fail(DS_ERR_UNSUPPORTED, "pack: size overflow");
    if (packed_words < need)
        return fail(DS_ERR_BUFFER_TOO_SMALL, "pack: need %lld words, have %lld",
                    (long long)need, (long long)packed_words);
    // Validate every code before writing anything.
    for (int64_t i = 0; i < rows * cols; ++i)
        if (codes[i] > 31)
            return fail(DS_ERR_INVALID_CODE, "pack: code %u at index %lld is >= 32",
                        unsigned(codes[i]), (long long)i);
    for (int64_t r = 0; r < rows; ++r) {
        const uint8_t *row = codes + r * cols;
        uint32_t *out = packed + r * wpr;
        for (int64_t wd = 0; wd < wpr; ++wd) {
            uint32_t word = 0;
            for (int j = 0; j < 6; ++j) {
                const int64_t col = wd * 6 + j;
                const uint32_t code = col < cols ? row[col] : 15u;
                word |= code << (5 * j);
            }
            out[wd] = word;
        }
    }
    return ok();
}

extern "C" ds_status ds_unpack_shift_weights(const uint32_t *packed, int64_t rows, int64_t cols,
                                             uint8_t *codes, int64_t codes_len)
{
    if (!codes || !packed) return fail(DS_ERR_NULL_POINTER, "unpack: NULL pointer");
    if (rows <= 0 || cols <= 0) return fail(DS_ERR_INVALID_SHAPE, "unpack: rows and cols must be > 0");
    const int64_t wpr = row_words(cols);
    const int64_t need = prod({rows, cols});
    if (need < 0 || prod({rows, wpr}) < 0) return fail(DS_ERR_UNSUPPORTED, "unpack: size overflow");
    if (codes_len < need)
        return fail(DS_ERR_BUFFER_TOO_SMALL, "unpack: need %lld bytes, have %lld",
                    (long long)need, (long long)codes_len);
    for (int64_t i = 0; i < rows * wpr; ++i)
        if (packed[i] >> 30)
            return fail(DS_ERR_INVALID_CODE, "unpack: word %lld has bits 30-31 set", (long long)i);
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t col = 0; col < cols; ++col)
            codes[r * cols + col] =
                uint8_t((packed[r * wpr + col / 6] >> (5 * (col % 6))) & 31u);
    return ok();
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
    }
    return "unknown status";
}

extern "C" const char *ds_last_error_message(void) { return last_error().c_str(); }
