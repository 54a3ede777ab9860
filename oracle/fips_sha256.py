"""SHA-256 written out from FIPS 180-4, in plain Python.  TEST INFRASTRUCTURE ONLY.

Slow and obviously correct; used to pin the library routine (``hashlib``)
that the oracle calls.  Nothing here is typed in from a table: the round
constants and the initial hash value are computed from their definitions.

* K_t (FIPS 180-4 Sec. 4.2.2): the first 32 bits of the fractional parts of
  the cube roots of the first 64 primes.
* H^(0) (Sec. 5.3.3): the first 32 bits of the fractional parts of the square
  roots of the first 8 primes.
* Functions Ch, Maj, Sigma0, Sigma1, sigma0, sigma1 (Sec. 4.1.2), padding
  (Sec. 5.1.1), message schedule and compression (Sec. 6.2.2).
"""
from __future__ import annotations

MASK = 0xFFFFFFFF


def first_primes(n: int):
    out = []
    c = 2
    while len(out) < n:
        if all(c % p for p in out if p * p <= c):
            out.append(c)
        c += 1
    return out


def _iroot(v: int, k: int) -> int:
    """floor(v ** (1/k)) for a non-negative integer v, exactly."""
    if v < 2:
        return v
    x = 1 << ((v.bit_length() + k - 1) // k)  # an upper bound
    while True:
        y = ((k - 1) * x + v // x ** (k - 1)) // k
        if y >= x:
            break
        x = y
    while x ** k > v:
        x -= 1
    while (x + 1) ** k <= v:
        x += 1
    return x


def frac_bits(p: int, k: int, bits: int = 32) -> int:
    """First ``bits`` bits of the fractional part of p ** (1/k)."""
    # floor(p^(1/k) * 2^bits) = floor((p * 2^(k*bits))^(1/k))
    return _iroot(p << (k * bits), k) & ((1 << bits) - 1)


PRIMES = first_primes(64)
K = [frac_bits(p, 3) for p in PRIMES]
H0 = [frac_bits(p, 2) for p in PRIMES[:8]]


def rotr(x: int, n: int) -> int:
    return ((x >> n) | (x << (32 - n))) & MASK


def ch(x, y, z):
    return (x & y) ^ (~x & z) & MASK


def maj(x, y, z):
    return (x & y) ^ (x & z) ^ (y & z)


def big_sigma0(x):
    return rotr(x, 2) ^ rotr(x, 13) ^ rotr(x, 22)


def big_sigma1(x):
    return rotr(x, 6) ^ rotr(x, 11) ^ rotr(x, 25)


def small_sigma0(x):
    return rotr(x, 7) ^ rotr(x, 18) ^ (x >> 3)


def small_sigma1(x):
    return rotr(x, 17) ^ rotr(x, 19) ^ (x >> 10)


def pad(message: bytes) -> bytes:
    """Sec. 5.1.1: append bit 1, zeros to 448 mod 512, then the 64-bit length."""
    ell = 8 * len(message)
    kz = (448 - (ell + 1)) % 512
    return message + bytes([0x80]) + bytes((kz - 7) // 8) + ell.to_bytes(8, "big")


def compress(state, block: bytes):
    """One application of the compression function (Sec. 6.2.2) to a 64-byte block."""
    assert len(block) == 64
    W = [int.from_bytes(block[4 * t:4 * t + 4], "big") for t in range(16)]
    for t in range(16, 64):
        W.append((small_sigma1(W[t - 2]) + W[t - 7] + small_sigma0(W[t - 15]) + W[t - 16]) & MASK)
    a, b, c, d, e, f, g, h = state
    for t in range(64):
        T1 = (h + big_sigma1(e) + ch(e, f, g) + K[t] + W[t]) & MASK
        T2 = (big_sigma0(a) + maj(a, b, c)) & MASK
        h, g, f, e = g, f, e, (d + T1) & MASK
        d, c, b, a = c, b, a, (T1 + T2) & MASK
    return [(x + y) & MASK for x, y in zip(state, (a, b, c, d, e, f, g, h))]


def sha256(message: bytes) -> bytes:
    m = pad(bytes(message))
    state = list(H0)
    for i in range(0, len(m), 64):
        state = compress(state, m[i:i + 64])
    return b"".join(x.to_bytes(4, "big") for x in state)


class Sha256:
    """hashlib-style wrapper so the RFC 2104 construction can take it."""

    digest_size = 32
    block_size = 64

    def __init__(self, data: bytes = b""):
        self._buf = bytearray(data)

    def update(self, data: bytes):
        self._buf += data

    def digest(self) -> bytes:
        return sha256(bytes(self._buf))

    def hexdigest(self) -> str:
        return self.digest().hex()
