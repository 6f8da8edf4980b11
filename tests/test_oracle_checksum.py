"""Pins of the oracle's layer checksum, the consumer stand-in of the
layered load: XOR of the little-endian 64-bit words of one layer's piece of
a page, XOR'd with its scale word.  Closed forms on single bytes, locality
(only that layer of that page counts), linearity under XOR, and the scale
word's place."""
import numpy as np
import pytest

import oracle

L, P = 3, 5
SH = oracle.make_shape(P, L, 16, 1, 8, 1, True)  # 256-byte pieces, scales
PIECE = oracle.sizes(SH)["piece"]


def cs(cache, sc, layer, pages):
    return oracle.layer_checksum(SH, cache, sc, layer, np.asarray(pages, np.int32))


def zeros():
    return np.zeros((L, P, PIECE), np.uint8), np.zeros((L, P, 8), np.uint8)


def test_zero_pages_give_zero():
    c, s = zeros()
    assert (cs(c, s, 1, range(P)) == 0).all()


@pytest.mark.parametrize("off,val", [(0, 1), (7, 0x80), (8, 0xAB), (PIECE - 1, 0xFF), (13, 3)])
def test_a_single_byte_lands_at_its_little_endian_place(off, val):
    c, s = zeros()
    c[2, 4, off] = val
    got = cs(c, s, 2, [4])[0]
    assert int(got) == val << (8 * (off % 8))
    # the same byte in another layer or page does not count
    assert cs(c, s, 1, [4])[0] == 0 and cs(c, s, 2, [3])[0] == 0


def test_two_words_with_the_same_bytes_cancel():
    c, s = zeros()
    c[0, 0, 5] = 0x5A
    c[0, 0, 13] = 0x5A  # same place in the next word
    assert cs(c, s, 0, [0])[0] == 0


def test_scale_word_is_xored_in_little_endian():
    c, s = zeros()
    s[1, 2] = np.arange(1, 9, dtype=np.uint8)
    assert int(cs(c, s, 1, [2])[0]) == int.from_bytes(bytes(range(1, 9)), "little")


def test_linear_under_xor_and_local():
    r = np.random.default_rng(3)
    a = r.integers(0, 256, size=(L, P, PIECE), dtype=np.uint8)
    b = r.integers(0, 256, size=(L, P, PIECE), dtype=np.uint8)
    sa = r.integers(0, 256, size=(L, P, 8), dtype=np.uint8)
    sb = r.integers(0, 256, size=(L, P, 8), dtype=np.uint8)
    for layer in range(L):
        x = cs(a ^ b, sa ^ sb, layer, range(P))
        assert np.array_equal(x, cs(a, sa, layer, range(P)) ^ cs(b, sb, layer, range(P)))
    # changing everything outside (layer 1, page 3) leaves that checksum
    keep = cs(a, sa, 1, [3])[0]
    a2, sa2 = a.copy(), sa.copy()
    a2[0] ^= 0xFF
    a2[2] ^= 0x11
    a2[1, [0, 1, 2, 4]] ^= 0x3C
    sa2[[0, 2]] ^= 0x77
    assert cs(a2, sa2, 1, [3])[0] == keep
    # and the order of pages only orders the output
    assert np.array_equal(cs(a, sa, 2, [4, 0, 2]), cs(a, sa, 2, [0, 2, 4])[[2, 0, 1]])


def test_bad_arguments():
    c, s = zeros()
    with pytest.raises(oracle.OracleError):
        cs(c, s, L, [0])
    with pytest.raises(oracle.OracleError):
        cs(c, s, 0, [P])
