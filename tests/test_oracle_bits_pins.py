"""Pins for the b-bit packed weight codes (Section 5's shorter shift ranges), and
the library's packer against the oracle's.

Reading (also in the oracle): a b-bit code holds the sign in its top bit and the
shift code in the b-1 bits below, the all-ones shift code meaning a zero weight;
floor(32 / b) codes per word from bit 0 up; rows start on a new word and are
padded with the zero weight. The oracle's packer is pinned to

* a little-endian bit stream assembled with ``numpy.packbits`` (an independent
  route from codes to words);
* words derived by hand from the definition for b = 2, 3, 4;
* the 5-bit format itself at b = 5 (already pinned) and the round trip;
* the representable range: shift codes up to 2^(b-1) - 2, plus the zero weight.
"""
import numpy as np
import pytest

import oracle
from paper_1905_13298_amd import _native, ops

BITS = [2, 3, 4, 5]


def representable_codes(rng, shape, bits, zero_frac=0.15):
    ones = (1 << (bits - 1)) - 1
    sign = rng.integers(0, 2, shape)
    shift = rng.integers(0, ones, shape) if ones > 0 else np.zeros(shape, np.int64)
    shift[rng.random(shape) < zero_frac] = 15
    return (sign << 4 | shift).astype(np.uint8)


def bitstream_pack(codes, bits):
    rows, cols = codes.shape
    per = 32 // bits
    ones = (1 << (bits - 1)) - 1
    wpr = -(-cols // per)
    out = np.zeros((rows, wpr), np.uint32)
    for r in range(rows):
        stream = np.zeros(wpr * 32, np.uint8)
        for col in range(wpr * per):
            if col < cols:
                code = int(codes[r, col])
                field = ones if code & 15 == 15 else code & 15
                raw = (code >> 4 & 1) << (bits - 1) | field
            else:
                raw = ones
            base = (col // per) * 32 + (col % per) * bits
            for t in range(bits):
                stream[base + t] = raw >> t & 1
        out[r] = np.frombuffer(np.packbits(stream, bitorder="little").tobytes(), dtype="<u4")
    return out


@pytest.mark.parametrize("bits", BITS)
def test_pack_matches_bitstream(bits):
    rng = np.random.default_rng(bits)
    for cols in (1, 5, 32 // bits, 32 // bits + 1, 37, 64):
        codes = representable_codes(rng, (3, cols), bits)
        np.testing.assert_array_equal(oracle.pack_codes_bits(codes, bits), bitstream_pack(codes, bits))


def test_pack_literal_words():
    # 2 bits: +1, -1, zero, zero (sign set) -> fields 00, 10, 01, 11; padding 01
    assert oracle.pack_codes_bits(np.array([[0, 16, 15, 31]], np.uint8), 2)[0, 0] == 0x555555D8
    # 3 bits: +1/4, -1/2, zero, +1 -> 010, 101, 011, 000; padding 011 (bits 30-31 zero)
    assert oracle.pack_codes_bits(np.array([[2, 17, 15, 0]], np.uint8), 3)[0, 0] == 0x1B6DB0EA
    # 4 bits: +2^-6, -2^-6, zero, zero (sign set), +1/2, -1, +1, +1/8
    w = oracle.pack_codes_bits(np.array([[6, 22, 15, 31, 1, 16, 0, 3]], np.uint8), 4)
    assert w.shape == (1, 1) and w[0, 0] == 0x3081F7E6


def test_five_bits_is_the_default_format():
    rng = np.random.default_rng(9)
    codes = rng.integers(0, 32, (4, 29)).astype(np.uint8)
    np.testing.assert_array_equal(oracle.pack_codes_bits(codes, 5), oracle.pack_codes(codes))


@pytest.mark.parametrize("bits", BITS)
def test_round_trip_and_range(bits):
    rng = np.random.default_rng(20 + bits)
    codes = representable_codes(rng, (5, 41), bits)
    back = oracle.unpack_codes_bits(oracle.pack_codes_bits(codes, bits), 41, bits)
    np.testing.assert_array_equal(back, codes)
    ones = (1 << (bits - 1)) - 1
    if ones < 15:
        bad = codes.copy()
        bad[2, 7] = ones          # the first shift that does not fit
        assert oracle.pack_codes_bits(bad, bits) is None
        bad[2, 7] = 16 | ones
        assert oracle.pack_codes_bits(bad, bits) is None


@pytest.mark.parametrize("bits", BITS)
def test_library_pack_matches_oracle(bits):
    rng = np.random.default_rng(40 + bits)
    for rows, cols in ((1, 1), (7, 33), (16, 128), (3, 1000)):
        codes = representable_codes(rng, (rows, cols), bits)
        got = ops.pack_shift_weights(codes, bits=bits)
        np.testing.assert_array_equal(got, oracle.pack_codes_bits(codes, bits))
        assert got.shape[1] == ops.packed_row_words(cols, bits) == -(-cols // (32 // bits))
        np.testing.assert_array_equal(ops.unpack_shift_weights(got, cols, bits=bits), codes)


def test_library_rejects_codes_that_do_not_fit():
    lib = _native.lib()
    codes = np.array([[0, 1, 2]], np.uint8)       # shift codes 0..2: fit 3 bits, not 2 (only 0)
    out = np.full(4, 0xABCD, np.uint32)
    assert lib.ds_pack_shift_weights_bits(codes.ctypes.data, 1, 3, 3, out.ctypes.data, 4) == 0
    assert lib.ds_pack_shift_weights_bits(codes.ctypes.data, 1, 3, 2, out.ctypes.data, 4) == 5
    out[:] = 0xABCD
    assert lib.ds_pack_shift_weights_bits(codes.ctypes.data, 1, 3, 2, out.ctypes.data, 4) == 5
    assert np.all(out == 0xABCD)                     # nothing written
    assert lib.ds_pack_shift_weights_bits(codes.ctypes.data, 1, 3, 6, out.ctypes.data, 4) == 3
    assert lib.ds_pack_shift_weights_bits(codes.ctypes.data, 1, 3, 1, out.ctypes.data, 4) == 3
    assert lib.ds_packed_row_words_bits(10, 3) == 1 and lib.ds_packed_row_words_bits(11, 3) == 2
    assert lib.ds_packed_row_words_bits(10, 6) == -1
    # unused top bits of 3-bit words must be zero
    words = np.array([1 << 30], np.uint32)
    dst = np.zeros(10, np.uint8)
    assert lib.ds_unpack_shift_weights_bits(words.ctypes.data, 1, 10, 3, dst.ctypes.data, 10) == 5


def test_entry_points_validate_the_code_width():
    lib = _native.lib()
    fake = 0x10000
    # DS_CODE_BITS(6) and (1) are rejected before any device access
    for b in (1, 6, 15):
        assert lib.ds_linear_shift(fake, fake * 2, None, fake * 4, 2, 3, 4, 16, b << 8, None) == 3
        assert lib.ds_conv2d_shift_backward_data(fake, fake * 2, fake * 4, 1, 2, 6, 6, 3, 3, 3, 1, 1,
                                                 1, 1, 16, b << 8, None) == 3
    with pytest.raises(ValueError):
        ops.code_bits_flag(6)
    assert ops.code_bits_flag(5) == 0 and ops.code_bits_flag(3) == 3 << 8
