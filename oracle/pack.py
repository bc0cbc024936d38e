"""Bit-packing of hardened GSQ layers.  Test infrastructure only.

Two layouts, both written out bit by bit here.

Plain group-wise layout (symmetric b-bit codes plus one 16-bit scale per group,
the storage behind Tab. 1's bits-per-parameter figures b + 16/gs):
    b = ceil(log2 K) bits per code (K = 2 -> 1, 3..4 -> 2, 5..8 -> 3), code = level index;
    code section: one little-endian (LSB-first) bitstream over all coordinates
        in row-major order ((batch, row, column)), code of coordinate e at bits
        [e*b, e*b + b); since gs*b is a multiple of 8 every group starts on a
        byte boundary;
    scale section: float16 scales, row-major (batch, row, group), little endian,
        immediately after the code section.

Super-block layout (K-quant style, §4.4 / App. E keep the deployment format;
the exact bytes are ours): every 256 consecutive weights of a row form one
110-byte record
    [d: float16, 2 bytes][sc: 16 x 6-bit sub-block scales, LSB-first, 12 bytes]
    [codes: 256 x 3-bit, LSB-first, 96 bytes]
records in row-major order.

Base-3 layout (3-level grids, e.g. ternary, the 1.58-bit case of §3.1 and Tab. 1):
    code section: the codes t in {0, 1, 2} of all coordinates in row-major order,
        five per byte, byte n = sum_{j<5} t_{5n+j} 3^j (3^5 = 243 <= 256), the last
        byte completed with zero codes: ceil(N / 5) bytes, 1.6 bits per weight;
    scale section: as in the plain layout.
Tab. 1 books ternary GSQ at 1.71 bits per parameter, which is the entropy
log2(3) = 1.585 bits per code plus 16 bits per 128 weights; a byte-aligned base-3
format cannot reach log2(3), and 5 codes per byte (1.6 + 0.125 = 1.725) is within
1 % of it.

Pinned by numpy.packbits(bitorder="little") on the expanded bit array, pack /
unpack round trips, Python integer arithmetic for the base-3 bytes, and the
bits-per-parameter figures of Tab. 1.
"""
import numpy as np

SUPERBLOCK = 256
SUB = 16
SB_BYTES = 2 + 12 + 96


TRITS_PER_BYTE = 5


def code_bits(K):
    """ceil(log2 K) for 2 <= K <= 16."""
    return int(np.ceil(np.log2(K)))


def _bits_of(values, width):
    """Expand unsigned integers into their low ``width`` bits, LSB first, concatenated."""
    values = np.asarray(values, dtype=np.uint64).reshape(-1)
    out = np.zeros(values.size * width, dtype=np.uint8)
    for j in range(width):
        out[j::width] = ((values >> np.uint64(j)) & np.uint64(1)).astype(np.uint8)
    return out


def _bytes_of(bits):
    """Gather a bit array into bytes: byte n = sum_j bit[8n + j] << j."""
    bits = np.asarray(bits, dtype=np.uint8)
    assert bits.size % 8 == 0
    b = bits.reshape(-1, 8).astype(np.uint16)
    return (b << np.arange(8, dtype=np.uint16)).sum(axis=1).astype(np.uint8)


def _values_of(data, width, count):
    """Inverse of _bits_of after _bytes_of."""
    data = np.frombuffer(bytes(data), dtype=np.uint8)
    bits = ((data[:, None] >> np.arange(8, dtype=np.uint8)) & 1).reshape(-1)[: count * width]
    bits = bits.reshape(count, width).astype(np.uint64)
    return (bits << np.arange(width, dtype=np.uint64)).sum(axis=1)


def packed_size_plain(batch, O, I, K, gs):
    b = code_bits(K)
    return batch * O * I * b // 8 + 2 * batch * O * (I // gs)


def packed_size_superblock(batch, O, I):
    return batch * O * (I // SUPERBLOCK) * SB_BYTES


def pack_plain(codes, scales16, K, gs):
    """Plain layout: code bitstream followed by float16 scales (see module doc)."""
    b = code_bits(K)
    codes = np.asarray(codes, dtype=np.uint8).reshape(-1)
    assert (gs * b) % 8 == 0 and int(codes.max(initial=0)) < K
    body = _bytes_of(_bits_of(codes, b))
    sc = np.asarray(scales16, dtype=np.float16).reshape(-1).astype("<f2").view(np.uint8)
    return np.concatenate([body, sc])


def unpack_plain(data, batch, O, I, K, gs):
    b = code_bits(K)
    n = batch * O * I
    nb = n * b // 8
    data = np.asarray(data, dtype=np.uint8)
    codes = _values_of(data[:nb], b, n).astype(np.uint8).reshape(batch, O, I)
    scales = data[nb:].copy().view("<f2").astype(np.float16).reshape(batch, O, I // gs)
    return codes, scales


def pack_superblock(codes, d16, sc):
    """Super-block layout: per 256 weights, d (fp16) + 16 x 6-bit sc + 256 x 3-bit codes."""
    codes = np.asarray(codes, dtype=np.uint8).reshape(-1, SUPERBLOCK)
    sc = np.asarray(sc, dtype=np.uint8).reshape(-1, SUPERBLOCK // SUB)
    d = np.asarray(d16, dtype=np.float16).reshape(-1).astype("<f2").view(np.uint8).reshape(-1, 2)
    assert int(codes.max(initial=0)) < 8 and int(sc.max(initial=0)) < 64
    out = np.empty((codes.shape[0], SB_BYTES), dtype=np.uint8)
    for r in range(codes.shape[0]):
        out[r, 0:2] = d[r]
        out[r, 2:14] = _bytes_of(_bits_of(sc[r], 6))
        out[r, 14:110] = _bytes_of(_bits_of(codes[r], 3))
    return out.reshape(-1)


def unpack_superblock(data, batch, O, I):
    rec = np.asarray(data, dtype=np.uint8).reshape(-1, SB_BYTES)
    n = rec.shape[0]
    d = rec[:, 0:2].copy().view("<f2").astype(np.float16).reshape(batch, O, I // SUPERBLOCK)
    sc = np.stack([_values_of(rec[r, 2:14], 6, 16) for r in range(n)]).astype(np.uint8)
    codes = np.stack([_values_of(rec[r, 14:110], 3, 256) for r in range(n)]).astype(np.uint8)
    return codes.reshape(batch, O, I), d, sc.reshape(batch, O, I // SUB)


def packed_size_base3(batch, O, I, gs):
    n = batch * O * I
    return -(-n // TRITS_PER_BYTE) + 2 * batch * O * (I // gs)


def pack_base3(codes, scales16):
    """Base-3 layout: five codes per byte (see module doc), then float16 scales."""
    codes = np.asarray(codes, dtype=np.uint8).reshape(-1)
    assert int(codes.max(initial=0)) < 3
    n = codes.size
    padded = np.zeros(-(-n // TRITS_PER_BYTE) * TRITS_PER_BYTE, dtype=np.int64)
    padded[:n] = codes
    weights = 3 ** np.arange(TRITS_PER_BYTE, dtype=np.int64)
    body = (padded.reshape(-1, TRITS_PER_BYTE) * weights).sum(axis=1).astype(np.uint8)
    sc = np.asarray(scales16, dtype=np.float16).reshape(-1).astype("<f2").view(np.uint8)
    return np.concatenate([body, sc])


def unpack_base3(data, batch, O, I, gs):
    n = batch * O * I
    nb = -(-n // TRITS_PER_BYTE)
    data = np.asarray(data, dtype=np.uint8)
    body = data[:nb].astype(np.int64)
    trits = np.stack([(body // 3 ** j) % 3 for j in range(TRITS_PER_BYTE)], axis=1).reshape(-1)[:n]
    scales = data[nb:].copy().view("<f2").astype(np.float16).reshape(batch, O, I // gs)
    return trits.astype(np.uint8).reshape(batch, O, I), scales
