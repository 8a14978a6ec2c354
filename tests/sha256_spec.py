"""A tiny pure-Python SHA-256 written from FIPS 180-4 (Sec. 4.1.2 functions,
Sec. 4.2.2 constants, Sec. 5.1.1 padding, Sec. 5.3.3 initial value, Sec. 6.2.2
computation). Used only by the tests, to pin the hashlib SHA-256 the oracle
calls and to recompute key chains from explicitly assembled messages.

The round constants and the initial value are not typed in: they are derived
here as the standard defines them (the first 32 bits of the fractional parts
of the cube roots of the first 64 primes, and of the square roots of the
first 8 primes), with exact integer roots. Slow; for short inputs only."""
import math

M32 = 0xFFFFFFFF


def _primes(n):
    out, c = [], 2
    while len(out) < n:
        if all(c % p for p in out if p * p <= c):
            out.append(c)
        c += 1
    return out


def _icbrt(x):
    """floor(x ** (1/3)) for a non-negative integer x, exactly."""
    if x == 0:
        return 0
    r = 1 << ((x.bit_length() + 2) // 3)  # >= the root
    while True:
        s = (2 * r + x // (r * r)) // 3
        if s >= r:
            break
        r = s
    while r * r * r > x:
        r -= 1
    while (r + 1) ** 3 <= x:
        r += 1
    return r


# fractional bits: floor(root(p) * 2^32) mod 2^32 = floor(root(p * 2^(32 k))) mod 2^32
K = [_icbrt(p << 96) & M32 for p in _primes(64)]
H0 = [math.isqrt(p << 64) & M32 for p in _primes(8)]


def _rotr(x, n):
    return ((x >> n) | (x << (32 - n))) & M32


def _compress(h, block):
    w = [int.from_bytes(block[4 * i:4 * i + 4], "big") for i in range(16)]
    for t in range(16, 64):
        s0 = _rotr(w[t - 15], 7) ^ _rotr(w[t - 15], 18) ^ (w[t - 15] >> 3)
        s1 = _rotr(w[t - 2], 17) ^ _rotr(w[t - 2], 19) ^ (w[t - 2] >> 10)
        w.append((w[t - 16] + s0 + w[t - 7] + s1) & M32)
    a, b, c, d, e, f, g, hh = h
    for t in range(64):
        t1 = (hh + (_rotr(e, 6) ^ _rotr(e, 11) ^ _rotr(e, 25)) + ((e & f) ^ (~e & g)) + K[t] + w[t]) & M32
        t2 = ((_rotr(a, 2) ^ _rotr(a, 13) ^ _rotr(a, 22)) + ((a & b) ^ (a & c) ^ (b & c))) & M32
        a, b, c, d, e, f, g, hh = (t1 + t2) & M32, a, b, c, (d + t1) & M32, e, f, g
    return [(x + y) & M32 for x, y in zip(h, (a, b, c, d, e, f, g, hh))]


def sha256(data: bytes) -> bytes:
    data = bytes(data)
    bits = 8 * len(data)
    msg = data + b"\x80" + b"\x00" * ((55 - len(data)) % 64) + bits.to_bytes(8, "big")
    assert len(msg) % 64 == 0
    h = list(H0)
    for i in range(0, len(msg), 64):
        h = _compress(h, msg[i:i + 64])
    return b"".join(x.to_bytes(4, "big") for x in h)
