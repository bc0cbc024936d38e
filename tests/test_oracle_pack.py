"""Pins of the oracle's hardening and packing."""
import os

import numpy as np
import pytest

from oracle import gsq, pack

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_harden_is_numpy_argmax_with_lowest_index_ties():
    rng = np.random.default_rng(0)
    lg = rng.integers(-2, 3, (3, 5, 64, 4)).astype(np.float32)   # many exact ties
    codes = gsq.harden(lg)
    np.testing.assert_array_equal(codes, np.argmax(lg, -1))
    first = np.array([[[min(k for k in range(4) if row[k] == row.max()) for row in r] for r in b] for b in lg])
    np.testing.assert_array_equal(codes, first)


@pytest.mark.parametrize("K,gs", [(2, 128), (3, 128), (4, 64), (5, 128), (8, 128), (8, 16)])
def test_plain_pack_matches_numpy_packbits_and_round_trips(K, gs):
    rng = np.random.default_rng(K * 100 + gs)
    B, O, I = 2, 3, 256
    codes = rng.integers(0, K, (B, O, I)).astype(np.uint8)
    sc16 = rng.uniform(0.001, 0.1, (B, O, I // gs)).astype(np.float16)
    data = pack.pack_plain(codes, sc16, K, gs)
    b = pack.code_bits(K)
    assert data.size == pack.packed_size_plain(B, O, I, K, gs)
    bits = np.unpackbits(codes.reshape(-1, 1), axis=1, bitorder="little")[:, :b].reshape(-1)
    np.testing.assert_array_equal(data[: B * O * I * b // 8], np.packbits(bits, bitorder="little"))
    np.testing.assert_array_equal(data[B * O * I * b // 8:].view("<f2"), sc16.reshape(-1))
    c2, s2 = pack.unpack_plain(data, B, O, I, K, gs)
    np.testing.assert_array_equal(c2, codes)
    np.testing.assert_array_equal(s2.view(np.uint16), sc16.view(np.uint16))


def test_bits_per_parameter_match_table_1():
    """Tab. 1 lists GSQ at 3.13 / 2.13 bpp for 3 / 2-bit codes with 16-bit scales per 128."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "bpp_table1.txt")) if l.strip() and l[0] != "#"]
    for bits, K, gs, bpp in rows:
        K, gs = int(K), int(gs)
        n = 4096 * 4096
        size = pack.packed_size_plain(1, 4096, 4096, K, gs)
        assert pack.code_bits(K) == int(bits)
        assert f"{size * 8 / n + 1e-9:.2f}" == bpp


def test_superblock_pack_round_trip_and_size():
    rng = np.random.default_rng(7)
    B, O, I = 2, 3, 512
    codes = rng.integers(0, 8, (B, O, I)).astype(np.uint8)
    d = rng.uniform(1e-4, 1e-3, (B, O, I // 256)).astype(np.float16)
    sc = rng.integers(0, 64, (B, O, I // 16)).astype(np.uint8)
    data = pack.pack_superblock(codes, d, sc)
    assert data.size == pack.packed_size_superblock(B, O, I) == B * O * 2 * 110
    c2, d2, s2 = pack.unpack_superblock(data, B, O, I)
    np.testing.assert_array_equal(c2, codes)
    np.testing.assert_array_equal(s2, sc)
    np.testing.assert_array_equal(d2.view(np.uint16), d.view(np.uint16))
    # independent bit check of the first record's scale field
    bits = np.unpackbits(sc[0, 0, :16].reshape(-1, 1), axis=1, bitorder="little")[:, :6].reshape(-1)
    np.testing.assert_array_equal(data[2:14], np.packbits(bits, bitorder="little"))


def test_fp16_scales_round_to_nearest_even():
    s = np.array([1.0 + 2.0**-11, 1.0 + 3 * 2.0**-11, 65504.0, 2.0**-25], dtype=np.float32)
    h = gsq.scales_fp16(s)
    assert h[0] == np.float16(1.0) and h[1] == np.float16(1.0 + 2.0**-9) and h[2] == np.float16(65504)
    assert h[3] == np.float16(0.0)     # 2^-25 is the half-way point to the smallest subnormal: ties to even
