"""CPU oracle for the KVGov hot path.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The product path (the
``libkvgov`` C ABI and its Python binding) never calls it, and this package
imports nothing from the product path: the two share no code.

What it computes, each piece plainly and in the paper's order:

* ``salts``        sigma_p = HMAC-SHA256(K, principal_id)        (Sec. 4.1)
* ``chain``        h_0 = H(tokens_0), h_j = H(h_{j-1}, tokens_j)   (Sec. 2.1)
                   root salting h_0 = H(sigma_p || tokens_0)       (Sec. 4.1)
                   boundary salting at block k                     (Sec. 4.2)
* ``chain_from``   the same recurrence entered at block j0 from the parent
                   digest h_{j0-1} (Sec. 2.1; Sec. 5.7, multi-turn sessions)
* ``Table``        a set of block hashes; lookup returns the number of
                   leading blocks present, i.e. the first miss     (Sec. 2.1,
                   Table "tab:taxonomy", block prefix cache row);
                   admit = lookup-then-insert in request order
* ``Radix``        token sequences per tree (per principal, or shared);
                   match = longest shared token prefix (Table "tab:taxonomy",
                   radix-tree row; Sec. 3.5; Sec. 4.1 per-principal root)

SHA-256 and HMAC come from Python's ``hashlib``/``hmac`` (OpenSSL).  The
package also carries its own FIPS 180-4 SHA-256 and RFC 2104 HMAC in plain
Python (``fips_sha256``, ``rfc2104``), used by the tests to pin the library
routines; all pins are listed in the tests.
"""
from .kvgov import (NONE, ROOT, BOUNDARY, BLOCK, salts, block_bytes, chain, chain_from,
                    hash_chains, hash_chains_parallel, hash_chains_resume, Table, lookup_hits,
                    Radix, lcp_tokens)

__all__ = ["NONE", "ROOT", "BOUNDARY", "BLOCK", "salts", "block_bytes", "chain", "chain_from",
           "hash_chains", "hash_chains_parallel", "hash_chains_resume", "Table", "lookup_hits",
           "Radix", "lcp_tokens"]
