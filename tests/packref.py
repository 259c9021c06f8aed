"""Bit-level Python reference of the packed code layout (include/palq.h).

Written from the layout text, independently of the library: used to check
the bytes the device pack produces and to read device-packed buffers.
"""
import numpy as np


def store_bits(bits: int) -> int:
    """Bits a code takes in a row: 6-bit codes are stored one per byte."""
    return 8 if bits == 6 else bits


def row_bytes(codes: int, bits: int) -> int:
    if bits == 3:
        return 12 * ((codes + 31) // 32)
    return 4 * ((codes * store_bits(bits) + 31) // 32)


def b3_hi_pos(j: int) -> int:
    return 2 * (j & 15) + (j >> 4)


def pack_row(codes, bits: int) -> bytes:
    """One row of codes (ints; signed ones as two's complement) -> bytes."""
    codes = [int(c) & ((1 << bits) - 1) for c in codes]
    nb = row_bytes(len(codes), bits)
    if bits == 3:
        out = bytearray(nb)
        for ci in range(0, len(codes), 32):
            chunk = codes[ci:ci + 32] + [0] * (32 - len(codes[ci:ci + 32]))
            lo, hi = 0, 0
            for j, v in enumerate(chunk):
                lo |= (v & 3) << (2 * j)
                hi |= ((v >> 2) & 1) << b3_hi_pos(j)
            base = 12 * (ci // 32)
            out[base:base + 8] = lo.to_bytes(8, "little")
            out[base + 8:base + 12] = hi.to_bytes(4, "little")
        return bytes(out)
    v = 0
    for j, c in enumerate(codes):
        v |= c << (store_bits(bits) * j)
    return v.to_bytes(nb, "little")


def unpack_row(buf: bytes, n: int, bits: int, signed: bool):
    out = []
    if bits == 3:
        for j in range(n):
            base = 12 * (j // 32)
            jj = j % 32
            lo = int.from_bytes(buf[base:base + 8], "little")
            hi = int.from_bytes(buf[base + 8:base + 12], "little")
            out.append(((lo >> (2 * jj)) & 3) | (((hi >> b3_hi_pos(jj)) & 1) << 2))
    else:
        v = int.from_bytes(buf[:row_bytes(n, bits)], "little")
        out = [(v >> (store_bits(bits) * j)) & ((1 << bits) - 1) for j in range(n)]
    if signed:
        out = [c - (1 << bits) if c >= (1 << (bits - 1)) else c for c in out]
    return out


def pack(codes, groups: int, bits: int) -> np.ndarray:
    """codes [n, h, w, groups*cpg] -> uint8 array of the packed tensor."""
    codes = np.asarray(codes)
    n, h, w, c = codes.shape
    cpg = c // groups
    rows = codes.reshape(-1, cpg)
    rb = row_bytes(cpg, bits)
    out = np.zeros((rows.shape[0], rb), np.uint8)
    for i, r in enumerate(rows.tolist()):
        out[i] = np.frombuffer(pack_row(r, bits), np.uint8)
    return out.reshape(-1)


def unpack(buf, shape, groups: int, bits: int, signed: bool) -> np.ndarray:
    n, h, w, c = shape
    cpg = c // groups
    rb = row_bytes(cpg, bits)
    buf = np.asarray(buf, np.uint8).reshape(-1, rb)
    rows = [unpack_row(bytes(r), cpg, bits, signed) for r in buf]
    return np.array(rows, np.int64).reshape(n, h, w, c)
