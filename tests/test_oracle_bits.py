"""Pins for the oracle's plain log2(G)-bit index stream (Sec. 3.1): the index
width the paper states for example group sizes, hand-written streams,
round trips, the byte count, and b = 8 being the byte array itself."""
import numpy as np
import pytest

import oracle


def test_index_width_is_plain_log2():
    # Sec. 3.1: G = 4 needs a 2-bit index (4 bits for the group's s = 2
    # weights); a group of G needs log2 G bits
    assert [oracle.index_width(G) for G in (1, 2, 3, 4, 5, 8, 16, 64, 256)] == [1, 1, 2, 2, 3, 3, 4, 6, 8]
    assert 2 * oracle.index_width(4) == 4


def test_hand_streams():
    # 2-bit entries 1, 2, 3, 0, 3: bits 01 10 11 00 11 from the low end -> 0b11_00_11_10_01
    assert oracle.index_bits(np.array([1, 2, 3, 0, 3], np.uint8), 2).tolist() == [0b1100111001]
    # 3-bit entries 0..7, then 5: 0 | 1<<3 | 2<<6 | ... | 7<<21 | 5<<24 fits one word
    want = sum(v << (3 * i) for i, v in enumerate(range(8))) | (5 << 24)
    assert oracle.index_bits(np.array(list(range(8)) + [5], np.uint8), 3).tolist() == [want]
    # 11 entries of 3 bits: the 11th straddles words 0 and 1 (bits 30..32)
    s = oracle.index_bits(np.array([0] * 10 + [7], np.uint8), 3)
    assert s.tolist() == [0b11 << 30, 0b1]
    # 4-bit entries: one nibble each, low nibble first
    assert oracle.index_bits(np.array([0xA, 0x3, 0xF], np.uint8), 4).tolist() == [0xF3A]


@pytest.mark.parametrize("G", [2, 3, 4, 6, 8, 16, 32, 64, 100, 256])
def test_round_trip_and_size(G):
    rng = np.random.default_rng(G)
    b = oracle.index_width(G)
    idx = rng.integers(0, G, size=1237).astype(np.uint8)
    s = oracle.index_bits(idx, b)
    assert s.size == (idx.size * b + 31) // 32
    np.testing.assert_array_equal(oracle.index_unbits(s, idx.size, b), idx)
    # bits past the last entry are zero
    tail = idx.size * b % 32
    if tail:
        assert int(s[-1]) >> tail == 0


def test_eight_bit_stream_is_the_byte_array():
    idx = np.random.default_rng(1).integers(0, 256, size=64).astype(np.uint8)
    np.testing.assert_array_equal(oracle.index_bits(idx, 8).view(np.uint8), idx)


def test_value_too_wide_is_rejected():
    with pytest.raises(ValueError):
        oracle.index_bits(np.array([4], np.uint8), 2)
