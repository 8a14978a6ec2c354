"""A tiny pure-Python XXH64, written from the published algorithm description
(xxHash specification, XXH64 section), used only to pin the xxhash library
that the oracle calls. Slow; for short inputs only."""
M = (1 << 64) - 1
P1 = 0x9E3779B185EBCA87
P2 = 0xC2B2AE3D27D4EB4F
P3 = 0x165667B19E3779F9
P4 = 0x85EBCA77C2B2AE63
P5 = 0x27D4EB2F165667C5


def _rotl(x, r):
    return ((x << r) | (x >> (64 - r))) & M


def _round(acc, lane):
    acc = (acc + lane * P2) & M
    return (_rotl(acc, 31) * P1) & M


def _merge(acc, v):
    acc ^= _round(0, v)
    return (acc * P1 + P4) & M


def _u64(b, i):
    return int.from_bytes(b[i:i + 8], "little")


def xxh64(data: bytes, seed: int = 0) -> int:
    n = len(data)
    i = 0
    if n >= 32:
        v = [(seed + P1 + P2) & M, (seed + P2) & M, seed & M, (seed - P1) & M]
        while i + 32 <= n:
            for k in range(4):
                v[k] = _round(v[k], _u64(data, i + 8 * k))
            i += 32
        acc = (_rotl(v[0], 1) + _rotl(v[1], 7) + _rotl(v[2], 12) + _rotl(v[3], 18)) & M
        for k in range(4):
            acc = _merge(acc, v[k])
    else:
        acc = (seed + P5) & M
    acc = (acc + n) & M
    while i + 8 <= n:
        acc ^= _round(0, _u64(data, i))
        acc = (_rotl(acc, 27) * P1 + P4) & M
        i += 8
    if i + 4 <= n:
        acc ^= (int.from_bytes(data[i:i + 4], "little") * P1) & M
        acc = (_rotl(acc, 23) * P2 + P3) & M
        i += 4
    while i < n:
        acc ^= (data[i] * P5) & M
        acc = (_rotl(acc, 11) * P1) & M
        i += 1
    acc ^= acc >> 33
    acc = (acc * P2) & M
    acc ^= acc >> 29
    acc = (acc * P3) & M
    acc ^= acc >> 32
    return acc
