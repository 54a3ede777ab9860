"""KVGov HMAC-keyed namespace isolation, hot path on MI355X (gfx950).

The hot path (per-principal HMAC-SHA256 salts, salted chained block hashes,
device-resident prefix-cache insert and longest-prefix lookup) is a C-ABI
shared library of hand-written HIP kernels (``csrc/``, header
``include/kvgov.h``); ``kvgov`` is its Python binding.
"""
from . import kvgov  # noqa: F401
from .kvgov import (NONE, ROOT, BOUNDARY, Cache, KvgovError, block_offsets,  # noqa: F401
                    hash_chains, salts)
