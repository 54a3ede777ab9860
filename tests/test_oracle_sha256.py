"""Pins for the oracle's SHA-256 and HMAC (CPU only).

The oracle calls ``hashlib.sha256`` and ``hmac`` (OpenSSL).  They are pinned
against implementations that share no code with OpenSSL:

* ``oracle.fips_sha256``: FIPS 180-4 written out in Python, with its round
  constants and initial hash value computed from the primes that define them;
* CPython's built-in ``_sha256`` module (its own C code, not OpenSSL);
* GNU coreutils ``sha256sum`` (gnulib's C code);
* HMAC: RFC 2104 written out (``oracle.rfc2104``) over the FIPS code, and the
  stdlib's pure-Python HMAC path over ``_sha256``.

The published FIPS 180-4 / RFC 4231 example vectors are not available in this
environment and are not typed in from memory.
"""
import hashlib
import hmac
import math
import shutil
import subprocess

import numpy as np
import pytest

from oracle import fips_sha256 as F
from oracle import rfc2104
from oracle import kvgov as O

try:
    import _sha256  # CPython's own SHA-256, independent of OpenSSL
except ImportError:  # pragma: no cover
    _sha256 = None

# message lengths around the padding boundaries (55/56 and 119/120 bytes
# decide whether the length field fits in the last block)
EDGE_LENGTHS = [0, 1, 3, 31, 32, 55, 56, 57, 63, 64, 65, 95, 96, 119, 120, 127, 128, 129, 191, 192, 300]


def _messages(seed=7):
    g = np.random.default_rng(seed)
    for L in EDGE_LENGTHS:
        yield g.integers(0, 256, size=L, dtype=np.uint8).tobytes()
    for L in g.integers(0, 400, size=20):
        yield g.integers(0, 256, size=int(L), dtype=np.uint8).tobytes()


def test_constants_follow_their_definition():
    """K_t and H0 from exact integer roots agree with a float evaluation of the
    same definition (cube / square roots of the first primes)."""
    assert F.PRIMES[:10] == [2, 3, 5, 7, 11, 13, 17, 19, 23, 29]
    assert len(F.PRIMES) == 64 and F.PRIMES[-1] == 311
    for p, k in zip(F.PRIMES, F.K):
        r = p ** (1.0 / 3.0)
        assert k == int((r - math.floor(r)) * 2 ** 32)
    for p, h in zip(F.PRIMES[:8], F.H0):
        r = math.sqrt(p)
        assert h == int((r - math.floor(r)) * 2 ** 32)
    # the integer root is exact at perfect powers and just below them
    assert F._iroot(27 << 96, 3) == 3 << 32
    assert F._iroot((27 << 96) - 1, 3) == (3 << 32) - 1


def test_padding_lengths():
    for L in EDGE_LENGTHS:
        m = F.pad(bytes(L))
        assert len(m) % 64 == 0
        assert m[L] == 0x80
        assert int.from_bytes(m[-8:], "big") == 8 * L
        # one block of padding is added only when the length does not fit
        assert len(m) == 64 * ((L + 8) // 64 + 1)


def test_fips_python_matches_hashlib():
    for m in _messages():
        assert F.sha256(m) == hashlib.sha256(m).digest(), len(m)


@pytest.mark.skipif(_sha256 is None, reason="CPython built without _sha256")
def test_hashlib_matches_builtin_sha256():
    for m in _messages(11):
        assert hashlib.sha256(m).digest() == _sha256.sha256(m).digest()


@pytest.mark.skipif(shutil.which("sha256sum") is None, reason="no coreutils sha256sum")
def test_hashlib_matches_coreutils():
    for m in list(_messages(13))[:12]:
        out = subprocess.run(["sha256sum"], input=m, capture_output=True, check=True).stdout
        assert out.split()[0].decode() == hashlib.sha256(m).hexdigest()


def test_multiblock_long_message():
    m = bytes(range(256)) * 9  # 2304 bytes, 37 blocks after padding
    assert F.sha256(m) == hashlib.sha256(m).digest()


@pytest.mark.parametrize("klen", [0, 1, 31, 32, 63, 64, 65, 131])
def test_hmac_rfc2104_matches_library(klen):
    g = np.random.default_rng(100 + klen)
    key = g.integers(0, 256, size=klen, dtype=np.uint8).tobytes()
    for mlen in (0, 16, 32, 55, 56, 100):
        msg = g.integers(0, 256, size=mlen, dtype=np.uint8).tobytes()
        ref = rfc2104.hmac(F.sha256, key, msg)
        assert hmac.new(key, msg, hashlib.sha256).digest() == ref
        if _sha256 is not None:
            # the stdlib's pure-Python HMAC path (digestmod without OpenSSL)
            assert hmac.new(key, msg, _sha256.sha256).digest() == ref


def test_oracle_salt_is_hmac_with_K_as_key():
    """sigma_p = HMAC_K(principal_id): K keys the MAC, the id is the message
    (Sec. 4.1); swapping them gives a different value."""
    g = np.random.default_rng(5)
    K = g.integers(0, 256, size=32, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, size=(4, 32), dtype=np.uint8)
    got = O.salts(K, ids)
    for pid, s in zip(ids, got):
        assert s == rfc2104.hmac(F.sha256, K, pid.tobytes())
        assert s != rfc2104.hmac(F.sha256, pid.tobytes(), K)
        assert len(s) == 32
