"""HMAC written out from RFC 2104, in plain Python.  TEST INFRASTRUCTURE ONLY.

HMAC(K, m) = H((K' xor opad) || H((K' xor ipad) || m)), where K' is K
zero-padded to the hash's block size (B = 64 bytes for SHA-256) after first
replacing K by H(K) when K is longer than B; ipad is the byte 0x36 and opad
the byte 0x5c repeated B times (RFC 2104 Sec. 2).  Used by the tests to pin
the library ``hmac`` module that the oracle's salt derivation calls.
"""
from __future__ import annotations

from typing import Callable

IPAD = 0x36
OPAD = 0x5C


def hmac(hash_fn: Callable[[bytes], bytes], key: bytes, message: bytes,
         block_size: int = 64) -> bytes:
    key = bytes(key)
    if len(key) > block_size:
        key = hash_fn(key)
    key = key + bytes(block_size - len(key))
    inner = hash_fn(bytes(k ^ IPAD for k in key) + bytes(message))
    return hash_fn(bytes(k ^ OPAD for k in key) + inner)
