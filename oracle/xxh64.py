"""Oracle: 64-bit xxHash (XXH64), the prefix-key hash of Appendix C.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper keys its KV store H by a deterministic 64-bit xxHash of the
tokenized shared prefix.  This is the published XXH64 algorithm (four 64-bit
accumulators over 32-byte stripes, then the tail in 8/4/1-byte steps, then the
avalanche), written in plain Python integers modulo 2^64.  Prefix keys hash the
token IDs as little-endian int32 with seed 0.
"""
import struct

_M = (1 << 64) - 1
P1 = 0x9E3779B185EBCA87
P2 = 0xC2B2AE3D27D4EB4F
P3 = 0x165667B19E3779F9
P4 = 0x85EBCA77C2B2AE63
P5 = 0x27D4EB2F165667C5


def _rotl(x, r):
    return ((x << r) | (x >> (64 - r))) & _M


def _round(acc, lane):
    acc = (acc + lane * P2) & _M
    acc = _rotl(acc, 31)
    return (acc * P1) & _M


def _merge(acc, v):
    acc ^= _round(0, v)
    return (acc * P1 + P4) & _M


def xxh64(data: bytes, seed: int = 0) -> int:
    n = len(data)
    p = 0
    if n >= 32:
        v1 = (seed + P1 + P2) & _M
        v2 = (seed + P2) & _M
        v3 = seed & _M
        v4 = (seed - P1) & _M
        while p + 32 <= n:
            a, b, c, d = struct.unpack_from("<4Q", data, p)
            v1, v2, v3, v4 = _round(v1, a), _round(v2, b), _round(v3, c), _round(v4, d)
            p += 32
        acc = (_rotl(v1, 1) + _rotl(v2, 7) + _rotl(v3, 12) + _rotl(v4, 18)) & _M
        for v in (v1, v2, v3, v4):
            acc = _merge(acc, v)
    else:
        acc = (seed + P5) & _M
    acc = (acc + n) & _M
    while p + 8 <= n:
        (k,) = struct.unpack_from("<Q", data, p)
        acc ^= _round(0, k)
        acc = (_rotl(acc, 27) * P1 + P4) & _M
        p += 8
    if p + 4 <= n:
        (k,) = struct.unpack_from("<I", data, p)
        acc ^= (k * P1) & _M
        acc = (_rotl(acc, 23) * P2 + P3) & _M
        p += 4
    while p < n:
        acc ^= (data[p] * P5) & _M
        acc = (_rotl(acc, 11) * P1) & _M
        p += 1
    acc ^= acc >> 33
    acc = (acc * P2) & _M
    acc ^= acc >> 29
    acc = (acc * P3) & _M
    acc ^= acc >> 32
    return acc


def prefix_key(token_ids) -> int:
    """Key of a shared prefix: XXH64 (seed 0) over the token IDs as LE int32."""
    data = b"".join(struct.pack("<i", int(t)) for t in token_ids)
    return xxh64(data, 0)
