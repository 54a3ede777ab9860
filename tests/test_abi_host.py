"""The C ABI without a GPU: the library loads, exports every declared call,
and rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2608_09225_amd import kvgov as K

HEADER = K.HEADER_PATH
pytestmark = pytest.mark.skipif(not os.path.exists(K.LIB_PATH),
                                reason="libkvgov.so not built")


def _declared():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvgov_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 13, names
    L = ctypes.CDLL(K.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    # and the binding covers exactly the declared calls
    assert sorted(K._SIGNATURES) == names


def test_header_constants_match_binding():
    c = K.header_constants()
    assert (c["KVGOV_NONE"], c["KVGOV_ROOT"], c["KVGOV_BOUNDARY"]) == (K.NONE, K.ROOT, K.BOUNDARY)
    assert c["KVGOV_BLOCK_SIZE"] == K.BLOCK == 16
    assert c["KVGOV_OK"] == 0
    codes = [v for k, v in c.items() if k.startswith("KVGOV_E_")]
    assert len(codes) == len(set(codes)) and all(v < 0 for v in codes)
    L = K.lib()
    for name, v in c.items():
        if name.startswith("KVGOV_E_"):
            assert K.strerror(v) != "unknown error code", name
    assert K.strerror(12345) == "unknown error code"
    assert L.kvgov_version() >> 16 == 1


def test_host_validation_returns_before_any_launch():
    c = K.header_constants()
    INVAL, UNSUP = c["KVGOV_E_INVAL"], c["KVGOV_E_UNSUPPORTED"]
    L = K.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    key = (ctypes.c_uint8 * 65)()
    kp = ctypes.cast(key, ctypes.c_void_p)
    # salts
    assert L.kvgov_salts(None, 32, fake, 32, 4, fake, None) == INVAL
    assert L.kvgov_salts(kp, 0, fake, 32, 4, fake, None) == INVAL
    assert L.kvgov_salts(kp, 65, fake, 32, 4, fake, None) == UNSUP
    assert L.kvgov_salts(kp, 32, fake, -1, 4, fake, None) == INVAL
    assert L.kvgov_salts(kp, 32, fake, 1025, 4, fake, None) == INVAL
    assert L.kvgov_salts(kp, 32, fake, 32, -1, fake, None) == INVAL
    assert L.kvgov_salts(kp, 32, fake, 32, 4, None, None) == INVAL
    assert L.kvgov_salts(kp, 32, None, 0, 0, None, None) == 0  # P == 0: nothing to do
    # block offsets
    assert L.kvgov_block_offsets(None, 4, 16, fake, fake, None) == INVAL
    assert L.kvgov_block_offsets(fake, -1, 16, fake, fake, None) == INVAL
    assert L.kvgov_block_offsets(fake, 4, 8, fake, fake, None) == UNSUP
    assert L.kvgov_block_offsets(fake, 4, 16, fake, None, None) == INVAL

    def chains(**kw):
        a = dict(tokens=fake, n_tokens=64, tok_offsets=fake, n=2, principal=fake, salts=fake,
                 P=4, mode=K.ROOT, boundary_tok=fake, block_size=16, blk_offsets=fake,
                 hashes=fake, n_blocks=4, status=fake, stream=None)
        a.update(kw)
        return L.kvgov_hash_chains(*a.values())

    def chains_noalloc(**kw):
        a = dict(tokens=fake, n_tokens=64, tok_offsets=fake, n=2, principal=fake, salts=fake,
                 P=4, mode=K.ROOT, boundary_tok=fake, block_size=16, blk_offsets=fake,
                 hashes=fake, n_blocks=4, status=fake, stream=None)
        a.update(kw)
        return L.kvgov_hash_chains_noalloc(*a.values())

    # the allocation-free variant: the size limit first, then the same checks
    big = c["KVGOV_NOALLOC_MAX_REQUESTS"] + 1
    assert chains_noalloc(n=big, tokens=None, status=None) == c["KVGOV_E_TOO_LARGE"]
    assert chains_noalloc(n=-1) == INVAL
    assert chains_noalloc(mode=3) == INVAL
    assert chains_noalloc(block_size=32) == UNSUP
    assert chains_noalloc(status=None) == INVAL
    assert chains_noalloc(tok_offsets=None) == INVAL
    assert chains_noalloc(n=0, tokens=None, hashes=None) == 0  # nothing to do

    assert chains(n=-1) == INVAL
    assert chains(mode=3) == INVAL
    assert chains(block_size=32) == UNSUP
    assert chains(status=None) == INVAL
    assert chains(tok_offsets=None) == INVAL
    assert chains(blk_offsets=None) == INVAL
    assert chains(principal=None) == INVAL
    assert chains(salts=None) == INVAL
    assert chains(P=0) == INVAL
    assert chains(mode=K.BOUNDARY, boundary_tok=None) == INVAL
    assert chains(tokens=ctypes.c_void_p(0x1002)) == INVAL  # misaligned
    assert chains(hashes=ctypes.c_void_p(0x1001)) == INVAL
    assert chains(n=0) == 0

    def resume(**kw):
        a = dict(tokens=fake, n_tokens=64, tok_offsets=fake, n=2, principal=fake, salts=fake,
                 P=4, mode=K.ROOT, boundary_tok=fake, block_size=16, start_block=fake,
                 parents=fake, blk_offsets=fake, hashes=fake, n_blocks=4, status=fake,
                 stream=None)
        a.update(kw)
        return L.kvgov_hash_chains_resume(*a.values())

    assert resume(start_block=None) == INVAL
    assert resume(parents=None) == INVAL
    assert resume(parents=ctypes.c_void_p(0x1002)) == INVAL  # misaligned
    assert resume(n=-1) == INVAL
    assert resume(mode=3) == INVAL
    assert resume(block_size=8) == UNSUP
    assert resume(status=None) == INVAL
    assert resume(P=0) == INVAL
    assert resume(n=0, start_block=None, parents=None) == 0
    assert L.kvgov_resume_offsets(fake, None, 4, 16, fake, fake, None) == INVAL
    assert L.kvgov_resume_offsets(None, fake, 4, 16, fake, fake, None) == INVAL
    assert L.kvgov_resume_offsets(fake, fake, 4, 8, fake, fake, None) == UNSUP
    assert L.kvgov_resume_offsets(fake, fake, -1, 16, fake, fake, None) == INVAL
    # cache
    h = ctypes.c_void_p()
    assert L.kvgov_cache_create(3, ctypes.byref(h)) == INVAL
    assert L.kvgov_cache_create(32, ctypes.byref(h)) == INVAL
    assert L.kvgov_cache_create(10, None) == INVAL
    n = ctypes.c_int64()
    assert L.kvgov_cache_insert(None, fake, fake, 1, 4, None, None) == INVAL
    assert L.kvgov_cache_lookup(None, fake, fake, 1, 4, fake, None) == INVAL
    assert L.kvgov_cache_admit(None, fake, fake, 1, 4, fake, fake, None, None) == INVAL
    assert L.kvgov_cache_set_recency(None, 1) == INVAL
    assert L.kvgov_cache_evict(None, 10, None, None) == INVAL
    assert L.kvgov_cache_erase(None, fake, 1, None, None) == INVAL
    # radix
    assert L.kvgov_radix_create(3, 10, ctypes.byref(h)) == INVAL
    assert L.kvgov_radix_create(10, 31, ctypes.byref(h)) == INVAL
    assert L.kvgov_radix_create(10, 10, None) == INVAL
    assert L.kvgov_radix_insert(None, fake, 64, fake, 2, fake, fake, 4, K.ROOT, fake, fake,
                                4, None) == INVAL
    assert L.kvgov_radix_match(None, fake, 64, fake, 2, fake, fake, 4, K.ROOT, fake, fake,
                               4, fake, None) == INVAL
    assert L.kvgov_radix_clear(None, None) == INVAL
    assert L.kvgov_radix_stats(None, ctypes.byref(n), ctypes.byref(n), None) == INVAL
    assert L.kvgov_radix_destroy(None) == 0
    assert L.kvgov_cache_clear(None, None) == INVAL
    assert L.kvgov_cache_count(None, ctypes.byref(n), None) == INVAL
    assert L.kvgov_cache_export(None, fake, 1, ctypes.byref(n), None) == INVAL
    assert L.kvgov_cache_slots(None, ctypes.byref(n)) == INVAL
    assert L.kvgov_cache_destroy(None) == 0


def test_binding_fails_loudly_without_gpu():
    """No silent CPU path: without a GPU the binding refuses CPU tensors."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises((ValueError, RuntimeError)):
        K.salts(b"k" * 32, torch.zeros((2, 32), dtype=torch.uint8))


def test_peaks_library_exports_and_validates():
    from paper_2608_09225_amd import peaks as P
    if not os.path.exists(P.LIB_PATH):
        pytest.skip("libkvgov_peaks.so not built")
    with open(P.HEADER_PATH) as f:
        text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(kvgov_\w+)\s*\(", text)))
    assert names == sorted(P._SIGNATURES)
    L = P.lib()
    inval = int(re.search(r"KVGOV_PEAK_E_INVAL\s+\((-?\d+)\)", text).group(1))
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    n = ctypes.c_int64()
    assert L.kvgov_peak_valu(None, 4, 4, ctypes.byref(n), None) == inval
    assert L.kvgov_peak_valu(fake, 0, 4, ctypes.byref(n), None) == inval
    assert L.kvgov_peak_gather(fake, 3, fake, 4, 4, ctypes.byref(n), None) == inval
    assert L.kvgov_peak_gather(fake, 0, fake, 4, 4, ctypes.byref(n), None) == inval
    assert L.kvgov_peak_gather(ctypes.c_void_p(0x1008), 16, fake, 4, 4, ctypes.byref(n),
                               None) == inval


def test_chain_kernel_timing_hook_host_rules():
    c = K.header_constants()
    L = K.lib()
    fake = ctypes.c_void_p(0x1000)  # never recorded: the chain call below fails first
    assert L.kvgov_time_next_chain_kernel(None, None) == 0
    assert L.kvgov_time_next_chain_kernel(fake, None) == c["KVGOV_E_INVAL"]
    assert L.kvgov_time_next_chain_kernel(None, fake) == c["KVGOV_E_INVAL"]
    try:
        assert L.kvgov_time_next_chain_kernel(fake, fake) == 0
        # a chain call takes the pending pair, whatever it returns
        assert L.kvgov_hash_chains(None, 0, None, -1, None, None, 0, 0, None, 16, None, None,
                                   0, fake, None) == c["KVGOV_E_INVAL"]
    finally:
        assert L.kvgov_time_next_chain_kernel(None, None) == 0
