"""The KVGov hot path, computed plainly on the CPU.  TEST INFRASTRUCTURE ONLY.

Readings of the paper taken here (each also listed in the design notes):

* Salt (Sec. 4.1, first display): sigma_p = HMAC-SHA256 with key K (the
  server secret) over the principal id bytes; the full 32-byte output.
* Token bytes: a block of B = 16 tokens is the 64 bytes of its int32 ids in
  little-endian order, nothing else (the paper does not fix an encoding).
* H is SHA-256 and "H(x, y)" is the concatenation x || y, parent digest
  first, as raw 32 bytes (Sec. 2.1 display; Sec. 4.1 names SHA256).
* Unsalted root: h_0 = SHA256(T_0) with no seed (Sec. 2.1 display).
* Root salting: h_0 = SHA256(sigma_p || T_0), later blocks chained
  unchanged (Sec. 4.1 display).
* Boundary salting (Sec. 4.2 display): blocks j < k unsalted,
  h_k = SHA256(sigma_p || h_{k-1} || T_k), blocks after k chained.  k is
  given per request as a token offset, k = boundary_tok // B (Sec. 5.6: a
  prompt that first differs at token i keeps no block from floor(i/B) on); k = 0 has
  no parent and is SHA256(sigma_p || T_0), the root-salted case; k at or
  beyond the last full block salts nothing (Sec. 4.2 places root salting
  at one end of the range of boundaries).
* Only full blocks are hashed, inserted and probed; a trailing partial block
  is ignored (Sec. 2.1: matches are truncated to a block boundary).
* Lookup returns the index of the first block whose hash is not in the table
  (the number of leading blocks matched, Table "tab:taxonomy"), and does not
  change the table.  Insert is set union.
"""
from __future__ import annotations

import hashlib
import hmac
import multiprocessing as mp
import os
import struct
from typing import Iterable, List, Optional, Sequence

import numpy as np

NONE, ROOT, BOUNDARY = 0, 1, 2
BLOCK = 16
DIGEST = 32


def sha256(data: bytes) -> bytes:
    return hashlib.sha256(data).digest()


# ---------------------------------------------------------------------------
# a1: salts (Sec. 4.1)
# ---------------------------------------------------------------------------

def salt(K: bytes, principal_id: bytes) -> bytes:
    """sigma_p = HMAC_K(principal_id) with SHA-256 (Sec. 4.1; abstract)."""
    return hmac.new(bytes(K), bytes(principal_id), hashlib.sha256).digest()


def salts(K: bytes, principal_ids) -> List[bytes]:
    """One salt per row of ``principal_ids`` (uint8 [P, L] or a list of bytes)."""
    return [salt(K, bytes(np.asarray(pid, dtype=np.uint8).tobytes())
                 if not isinstance(pid, (bytes, bytearray)) else bytes(pid))
            for pid in principal_ids]


# ---------------------------------------------------------------------------
# a2 / a3: chained block hashes (Sec. 2.1, 4.1, 4.2)
# ---------------------------------------------------------------------------

def block_bytes(tokens: Sequence[int], j: int) -> bytes:
    """T_j: the 16 int32 token ids of block j, little-endian."""
    return struct.pack("<16i", *[int(t) for t in tokens[BLOCK * j:BLOCK * (j + 1)]])


def chain(tokens: Sequence[int], mode: int, salt_bytes: Optional[bytes] = None,
          boundary_tok: Optional[int] = None, hash_fn=sha256) -> List[bytes]:
    """Block hashes h_0 .. h_{n-1} of one request, n = len(tokens) // 16."""
    n_full = len(tokens) // BLOCK
    if mode == BOUNDARY:
        if boundary_tok is None or not 0 <= boundary_tok <= len(tokens):
            raise ValueError("boundary_tok outside [0, len]")
        k = boundary_tok // BLOCK
    elif mode in (NONE, ROOT):
        k = None
    else:
        raise ValueError("unknown mode")
    if mode != NONE and (salt_bytes is None or len(salt_bytes) != DIGEST):
        raise ValueError("salted modes need a 32-byte salt")
    out: List[bytes] = []
    prev = b""  # h_{-1} does not exist
    for j in range(n_full):
        salted = (mode == ROOT and j == 0) or (mode == BOUNDARY and j == k)
        msg = (salt_bytes if salted else b"") + prev + block_bytes(tokens, j)
        prev = hash_fn(msg)
        out.append(prev)
    return out


def chain_from(tokens: Sequence[int], start: int, parent: Optional[bytes], mode: int,
               salt_bytes: Optional[bytes] = None, boundary_tok: Optional[int] = None,
               hash_fn=sha256) -> List[bytes]:
    """Block hashes h_start .. h_{n-1} of one request given h_{start-1}.

    Sec. 2.1: each h_j is a function of h_{j-1}, T_j and (Sec. 4.1, 4.2) of
    sigma_p on the salted block only, so the recurrence can be entered at any
    block with its parent digest (Sec. 5.7: a later turn of a session
    extends the earlier turn's prompt exactly).  ``parent`` is ignored when
    start is 0; the salt of a block below ``start`` is already inside it."""
    n_full = len(tokens) // BLOCK
    if not 0 <= start <= n_full:
        raise ValueError("start outside [0, len // 16]")
    if start > 0 and (parent is None or len(parent) != DIGEST):
        raise ValueError("resuming needs the 32-byte parent digest")
    if mode == BOUNDARY:
        if boundary_tok is None or not 0 <= boundary_tok <= len(tokens):
            raise ValueError("boundary_tok outside [0, len]")
        k = boundary_tok // BLOCK
    elif mode in (NONE, ROOT):
        k = 0 if mode == ROOT else None
    else:
        raise ValueError("unknown mode")
    if mode != NONE and (salt_bytes is None or len(salt_bytes) != DIGEST):
        raise ValueError("salted modes need a 32-byte salt")
    out: List[bytes] = []
    h = bytes(parent) if start > 0 else b""
    for j in range(start, n_full):
        sigma = salt_bytes if (k is not None and j == k) else b""
        h = hash_fn(sigma + h + block_bytes(tokens, j))
        out.append(h)
    return out


def hash_chains_resume(tokens, tok_offsets, principal, salt_list, mode, start, parents,
                       boundary_tok=None) -> np.ndarray:
    """``chain_from`` over a ragged batch, in the flat layout of the C ABI:
    request r contributes rows for blocks start[r] .. len_r // 16 - 1."""
    tok_offsets, n = _check_batch(tokens, tok_offsets, principal, len(salt_list), mode,
                                  boundary_tok)
    out = []
    for r in range(n):
        a, b = int(tok_offsets[r]), int(tok_offsets[r + 1])
        s = salt_list[int(principal[r])] if mode != NONE else None
        bt = int(boundary_tok[r]) if mode == BOUNDARY else None
        par = bytes(np.asarray(parents[r], dtype=np.uint8).tobytes())
        out.extend(chain_from(tokens[a:b], int(start[r]), par, mode, s, bt))
    if not out:
        return np.zeros((0, DIGEST), dtype=np.uint8)
    return np.frombuffer(b"".join(out), dtype=np.uint8).reshape(-1, DIGEST)


def _check_batch(tokens, tok_offsets, principal, P, mode, boundary_tok):
    tok_offsets = np.asarray(tok_offsets, dtype=np.int64)
    n = tok_offsets.shape[0] - 1
    if n < 0 or np.any(np.diff(tok_offsets) < 0) or (n >= 0 and tok_offsets[0] < 0) \
            or tok_offsets[-1] > len(tokens):
        raise ValueError("bad offsets")
    if mode != NONE:
        principal = np.asarray(principal)
        if principal.shape[0] != n or np.any(principal < 0) or np.any(principal >= P):
            raise ValueError("bad principal")
    return tok_offsets, n


def hash_chains(tokens, tok_offsets, principal, salt_list, mode,
                boundary_tok=None, requests: Optional[Iterable[int]] = None) -> np.ndarray:
    """Chains of a ragged batch in the flat layout of the C ABI.

    Returns uint8 [sum_r len_r // 16, 32], request after request.  With
    ``requests`` given, only those requests are hashed (in that order)."""
    tok_offsets, n = _check_batch(tokens, tok_offsets, principal, len(salt_list), mode,
                                  boundary_tok)
    rows = range(n) if requests is None else requests
    out = []
    for r in rows:
        a, b = int(tok_offsets[r]), int(tok_offsets[r + 1])
        s = salt_list[int(principal[r])] if mode != NONE else None
        bt = int(boundary_tok[r]) if mode == BOUNDARY else None
        out.extend(chain(tokens[a:b], mode, s, bt))
    if not out:
        return np.zeros((0, DIGEST), dtype=np.uint8)
    return np.frombuffer(b"".join(out), dtype=np.uint8).reshape(-1, DIGEST)


_POOL_ARGS = None


def _pool_chunk(rng_):
    tokens, tok_offsets, principal, salt_list, mode, boundary_tok = _POOL_ARGS
    return hash_chains(tokens, tok_offsets, principal, salt_list, mode,
                       boundary_tok, requests=range(*rng_)).tobytes()


def hash_chains_parallel(tokens, tok_offsets, principal, salt_list, mode,
                         boundary_tok=None, processes: Optional[int] = None,
                         requests: Optional[Sequence[int]] = None) -> np.ndarray:
    """``hash_chains`` split over worker processes by request ranges.

    Same result, request order kept; ``requests`` (a contiguous range) limits
    the work to those requests."""
    global _POOL_ARGS
    tok_offsets = np.asarray(tok_offsets, dtype=np.int64)
    n = tok_offsets.shape[0] - 1
    lo, hi = (0, n) if requests is None else (int(requests[0]), int(requests[-1]) + 1)
    processes = processes or os.cpu_count() or 1
    step = max(1, (hi - lo + 4 * processes - 1) // (4 * processes))
    chunks = [(a, min(a + step, hi)) for a in range(lo, hi, step)]
    _POOL_ARGS = (tokens, tok_offsets, principal, salt_list, mode, boundary_tok)
    try:
        ctx = mp.get_context("fork")
        with ctx.Pool(processes) as pool:
            parts = pool.map(_pool_chunk, chunks)
    finally:
        _POOL_ARGS = None
    data = b"".join(parts)
    return np.frombuffer(data, dtype=np.uint8).reshape(-1, DIGEST)


# ---------------------------------------------------------------------------
# a4 / a5: the block prefix cache (Sec. 2.1; Table "tab:taxonomy")
# ---------------------------------------------------------------------------

def _keys(hashes: np.ndarray, lo: int = 0, hi: Optional[int] = None) -> List[bytes]:
    h = np.ascontiguousarray(hashes[lo:hi], dtype=np.uint8)
    raw = h.tobytes()
    return [raw[i:i + DIGEST] for i in range(0, len(raw), DIGEST)]


NO_DEPTH = 0xFFFFFFFF


class Table:
    """The cache as a set of 32-byte keys, with the recency state that
    maintenance uses (the paper is silent on maintenance; the readings here
    are listed in the design notes):

    * a clock that advances by one with every insert or admission call;
    * per key a stamp, the clock of the latest such call whose batch held
      it, and a depth, the smallest block position (row within its request)
      it had in that call;
    * evict(max_keys) keeps the largest set of whole rank classes, ranked by
      stamp (newest first) and then depth (shallowest first), that fits in
      max_keys.  A chain's earlier block always has a stamp at least that of
      a later block and a smaller depth, so the kept set stays prefix-closed;
    * erase(keys) removes exactly the given keys."""

    def __init__(self):
        self.keys = set()
        self.clock = 0
        self.stamp = {}
        self.depth = {}

    def _touch(self, hashes: np.ndarray, blk_offsets) -> None:
        self.clock += 1
        blk_offsets = np.asarray(blk_offsets, dtype=np.int64)
        pos = {}
        for r in range(blk_offsets.shape[0] - 1):
            a, b = int(blk_offsets[r]), int(blk_offsets[r + 1])
            for j, k in enumerate(_keys(hashes, a, b)):
                pos[k] = min(pos.get(k, NO_DEPTH), j)
        for k, j in pos.items():
            self.stamp[k] = self.clock
            self.depth[k] = j

    def insert(self, hashes: np.ndarray, blk_offsets=None) -> int:
        """T <- T u {every key of the batch}; returns how many were not in T.
        Without offsets the batch is one request."""
        if blk_offsets is not None:
            blk_offsets = np.asarray(blk_offsets, dtype=np.int64)
            lo, hi = int(blk_offsets[0]), int(blk_offsets[-1])
        else:
            lo, hi = 0, int(hashes.shape[0])
            blk_offsets = np.array([0, hi], dtype=np.int64)
        new = set(_keys(hashes, lo, hi)) - self.keys
        self.keys |= new
        self._touch(hashes, blk_offsets)
        return len(new)

    def rank(self, k: bytes):
        return (self.stamp.get(k, 0), -self.depth.get(k, NO_DEPTH))

    def evict(self, max_keys: int) -> int:
        """Keeps the top rank classes that fit in max_keys; returns the
        number of keys kept."""
        classes = {}
        for k in self.keys:
            classes.setdefault(self.rank(k), []).append(k)
        kept = set()
        for rk in sorted(classes, reverse=True):
            if len(kept) + len(classes[rk]) > max_keys:
                break
            kept |= set(classes[rk])
        self.erase_set(self.keys - kept)
        return len(kept)

    def erase_set(self, ks) -> int:
        gone = set(ks) & self.keys
        self.keys -= gone
        for k in gone:
            self.stamp.pop(k, None)
            self.depth.pop(k, None)
        return len(gone)

    def erase(self, hashes: np.ndarray) -> int:
        """T <- T minus the given keys; returns how many were in T."""
        return self.erase_set(_keys(hashes))

    def lookup(self, hashes: np.ndarray, blk_offsets) -> np.ndarray:
        """hit[r] = first j with h_j(r) not in T, or n_full(r) if none is missing."""
        return lookup_hits(self.keys, hashes, blk_offsets)

    def admit(self, hashes: np.ndarray, blk_offsets):
        """Requests in order, each looked up and then inserted (Sec. 2.1: a
        request reuses the longest cached block prefix, and the blocks it
        computes join the cache).  Returns (hits, new): hits[r] as ``lookup``
        against T as it stands when r comes, new[r] = distinct keys of r
        not yet in T; T then takes r's keys."""
        blk_offsets = np.asarray(blk_offsets, dtype=np.int64)
        n = blk_offsets.shape[0] - 1
        hits = np.zeros(n, dtype=np.int32)
        new = np.zeros(n, dtype=np.int32)
        for r in range(n):
            a, b = int(blk_offsets[r]), int(blk_offsets[r + 1])
            keys_r = _keys(hashes, a, b)
            hits[r] = lookup_hits(self.keys, hashes, blk_offsets, requests=[r])[0]
            fresh = set(keys_r) - self.keys
            new[r] = len(fresh)
            self.keys |= fresh
        self._touch(hashes, blk_offsets)
        return hits, new


def lookup_hits(keys: set, hashes: np.ndarray, blk_offsets,
                requests: Optional[Iterable[int]] = None) -> np.ndarray:
    blk_offsets = np.asarray(blk_offsets, dtype=np.int64)
    n = blk_offsets.shape[0] - 1
    rows = list(range(n)) if requests is None else list(requests)
    out = np.zeros(len(rows), dtype=np.int32)
    raw = np.ascontiguousarray(hashes, dtype=np.uint8)
    for i, r in enumerate(rows):
        a, b = int(blk_offsets[r]), int(blk_offsets[r + 1])
        j = 0
        while j < b - a and raw[a + j].tobytes() in keys:
            j += 1
        out[i] = j
    return out


# ---------------------------------------------------------------------------
# radix-tree prefix cache (Table "tab:taxonomy", radix-tree row; Sec. 3.5;
# Sec. 4.1: sigma_p as the root node gives each principal a disjoint tree)
# ---------------------------------------------------------------------------

def lcp_tokens(a: np.ndarray, b: np.ndarray) -> int:
    """Number of leading tokens a and b share."""
    n = min(len(a), len(b))
    if n == 0:
        return 0
    diff = np.nonzero(np.asarray(a[:n]) != np.asarray(b[:n]))[0]
    return int(diff[0]) if diff.size else n


class Radix:
    """Token sequences per tree: one tree per principal (root salting, keyed
    by the principal's salt, the tree's root) or one shared tree (unsalted).
    match(q) = max over the tree's sequences s of lcp_tokens(q, s)."""

    def __init__(self):
        self.trees = {}

    @staticmethod
    def _tree(mode: int, salt_bytes: Optional[bytes]):
        if mode == NONE:
            return b""
        if mode == ROOT:
            if salt_bytes is None or len(salt_bytes) != DIGEST:
                raise ValueError("root salting needs a 32-byte salt")
            return bytes(salt_bytes)
        raise ValueError("the radix form exists for unsalted and root-salted trees only")

    def insert(self, tokens, tok_offsets, principal, salt_list, mode) -> None:
        tok_offsets = np.asarray(tok_offsets, dtype=np.int64)
        for r in range(tok_offsets.shape[0] - 1):
            s = salt_list[int(principal[r])] if mode != NONE else None
            seq = np.array(tokens[int(tok_offsets[r]):int(tok_offsets[r + 1])], dtype=np.int64)
            self.trees.setdefault(self._tree(mode, s), []).append(seq)

    def match(self, tokens, tok_offsets, principal, salt_list, mode,
              requests: Optional[Iterable[int]] = None) -> np.ndarray:
        tok_offsets = np.asarray(tok_offsets, dtype=np.int64)
        rows = range(tok_offsets.shape[0] - 1) if requests is None else list(requests)
        out = []
        for r in rows:
            s = salt_list[int(principal[r])] if mode != NONE else None
            q = np.array(tokens[int(tok_offsets[r]):int(tok_offsets[r + 1])], dtype=np.int64)
            seqs = self.trees.get(self._tree(mode, s), [])
            out.append(max([lcp_tokens(q, x) for x in seqs] or [0]))
        return np.array(out, dtype=np.int32)
