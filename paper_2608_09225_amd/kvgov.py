"""Python binding of libkvgov (ctypes).

Argument marshalling only: every step of the hot path runs in the HIP
kernels behind the C ABI declared in include/kvgov.h.  torch supplies device
memory (tensor storage) and streams; nothing here computes a hash, a salt or
a lookup, and there is no CPU fallback: if the shared library is missing or
no GPU is present, the calls raise.

Calls mirror the C ABI one to one:

    kvgov_salts         -> salts(K, principal_ids)
    kvgov_block_offsets -> block_offsets(tok_offsets)
    kvgov_hash_chains   -> hash_chains(tokens, tok_offsets, principal, salts, mode, ...)
    kvgov_hash_chains_noalloc -> hash_chains_noalloc(..., blk_offsets, out, status)
    kvgov_time_next_chain_kernel -> time_next_chain_kernel(start_event, end_event)
    kvgov_hash_chains_resume -> hash_chains_resume(..., start_block, parents, ...)
    kvgov_resume_offsets -> resume_offsets(tok_offsets, start_block)
    kvgov_cache_*       -> Cache(log2_slots).insert / lookup / admit / set_recency / evict /
                           erase / clear / count / export
    kvgov_radix_*       -> Radix(log2_block_slots, log2_edge_slots).insert / match / clear / stats
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

NONE, ROOT, BOUNDARY = 0, 1, 2
BLOCK = 16

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvgov.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "kvgov.h")

_c_i32, _c_i64, _c_sz, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p

# argument types of every exported call, in header order
_SIGNATURES = {
    "kvgov_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "kvgov_version": (ctypes.c_int, []),
    "kvgov_salts": (ctypes.c_int, [_vp, _c_sz, _vp, _c_i32, _c_i32, _vp, _vp]),
    "kvgov_block_offsets": (ctypes.c_int, [_vp, _c_i32, _c_i32, _vp, _vp, _vp]),
    "kvgov_hash_chains": (ctypes.c_int, [_vp, _c_i64, _vp, _c_i32, _vp, _vp, _c_i32, _c_i32,
                                         _vp, _c_i32, _vp, _vp, _c_i64, _vp, _vp]),
    "kvgov_hash_chains_noalloc": (ctypes.c_int, [_vp, _c_i64, _vp, _c_i32, _vp, _vp, _c_i32,
                                                 _c_i32, _vp, _c_i32, _vp, _vp, _c_i64, _vp,
                                                 _vp]),
    "kvgov_time_next_chain_kernel": (ctypes.c_int, [_vp, _vp]),
    "kvgov_hash_chains_resume": (ctypes.c_int, [_vp, _c_i64, _vp, _c_i32, _vp, _vp, _c_i32,
                                                _c_i32, _vp, _c_i32, _vp, _vp, _vp, _vp,
                                                _c_i64, _vp, _vp]),
    "kvgov_resume_offsets": (ctypes.c_int, [_vp, _vp, _c_i32, _c_i32, _vp, _vp, _vp]),
    "kvgov_cache_create": (ctypes.c_int, [_c_i32, ctypes.POINTER(_vp)]),
    "kvgov_cache_destroy": (ctypes.c_int, [_vp]),
    "kvgov_cache_clear": (ctypes.c_int, [_vp, _vp]),
    "kvgov_cache_slots": (ctypes.c_int, [_vp, ctypes.POINTER(_c_i64)]),
    "kvgov_cache_insert": (ctypes.c_int, [_vp, _vp, _vp, _c_i32, _c_i64,
                                          ctypes.POINTER(_c_i64), _vp]),
    "kvgov_cache_lookup": (ctypes.c_int, [_vp, _vp, _vp, _c_i32, _c_i64, _vp, _vp]),
    "kvgov_cache_admit": (ctypes.c_int, [_vp, _vp, _vp, _c_i32, _c_i64, _vp, _vp,
                                         ctypes.POINTER(_c_i64), _vp]),
    "kvgov_radix_create": (ctypes.c_int, [_c_i32, _c_i32, ctypes.POINTER(_vp)]),
    "kvgov_radix_destroy": (ctypes.c_int, [_vp]),
    "kvgov_radix_clear": (ctypes.c_int, [_vp, _vp]),
    "kvgov_radix_insert": (ctypes.c_int, [_vp, _vp, _c_i64, _vp, _c_i32, _vp, _vp, _c_i32,
                                          _c_i32, _vp, _vp, _c_i64, _vp]),
    "kvgov_radix_match": (ctypes.c_int, [_vp, _vp, _c_i64, _vp, _c_i32, _vp, _vp, _c_i32,
                                         _c_i32, _vp, _vp, _c_i64, _vp, _vp]),
    "kvgov_radix_stats": (ctypes.c_int, [_vp, ctypes.POINTER(_c_i64), ctypes.POINTER(_c_i64),
                                         _vp]),
    "kvgov_cache_set_recency": (ctypes.c_int, [_vp, _c_i32]),
    "kvgov_cache_evict": (ctypes.c_int, [_vp, _c_i64, ctypes.POINTER(_c_i64), _vp]),
    "kvgov_cache_erase": (ctypes.c_int, [_vp, _vp, _c_i64, ctypes.POINTER(_c_i64), _vp]),
    "kvgov_cache_count": (ctypes.c_int, [_vp, ctypes.POINTER(_c_i64), _vp]),
    "kvgov_cache_export": (ctypes.c_int, [_vp, _vp, _c_i64, ctypes.POINTER(_c_i64), _vp]),
}

_LIB = None


class KvgovError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        self.code = code
        msg = strerror(code) if _LIB is not None else str(code)
        super().__init__(f"{what}: {msg} ({code})" if what else f"{msg} ({code})")


def header_constants() -> dict:
    """#define KVGOV_* integer constants of include/kvgov.h."""
    out = {}
    with open(HEADER_PATH) as f:
        for m in re.finditer(r"#define\s+(KVGOV_\w+)\s+\(?(-?\d+)\)?", f.read()):
            out[m.group(1)] = int(m.group(2))
    return out


def lib() -> ctypes.CDLL:
    """The loaded shared library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def strerror(code: int) -> str:
    return lib().kvgov_strerror(int(code)).decode()


def _check(rc: int, what: str):
    if rc != 0:
        raise KvgovError(rc, what)


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _dev(t: Optional[torch.Tensor], dtype, name: str, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def new_status(device=None) -> torch.Tensor:
    """A zeroed int32 status word for the hashing calls."""
    return torch.zeros(1, dtype=torch.int32, device=device or "cuda")


def check_status(status: torch.Tensor, what: str = "kernel"):
    """Waits for the status word's stream and raises the latched error, if any."""
    v = int(status.item())
    if v != 0:
        raise KvgovError(v, what)


# ---------------------------------------------------------------------------
# a1 salts
# ---------------------------------------------------------------------------

def salts(K: bytes, principal_ids: torch.Tensor, out: Optional[torch.Tensor] = None,
          stream=None) -> torch.Tensor:
    """salts[p] = HMAC-SHA256(K, principal_ids[p]); uint8 [P, 32] on the GPU."""
    ids = _dev(principal_ids, torch.uint8, "principal_ids")
    if ids.dim() != 2:
        raise ValueError("principal_ids must be [P, id_len]")
    P, L = ids.shape
    if out is None:
        out = torch.empty((P, 32), dtype=torch.uint8, device=ids.device)
    _dev(out, torch.uint8, "out")
    kb = (ctypes.c_uint8 * max(1, len(K))).from_buffer_copy(bytes(K) or b"\0")
    try:
        _check(lib().kvgov_salts(ctypes.cast(kb, _vp), len(K), _ptr(ids), L, P, _ptr(out),
                                 _stream(stream)), "kvgov_salts")
    finally:
        ctypes.memset(kb, 0, ctypes.sizeof(kb))
    return out


# ---------------------------------------------------------------------------
# a2/a3 chains
# ---------------------------------------------------------------------------

def block_offsets(tok_offsets: torch.Tensor, out: Optional[torch.Tensor] = None,
                  status: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    to = _dev(tok_offsets, torch.int64, "tok_offsets")
    n = to.numel() - 1
    if out is None:
        out = torch.empty(n + 1, dtype=torch.int64, device=to.device)
    own = status is None
    if own:
        status = new_status(to.device)
    _check(lib().kvgov_block_offsets(_ptr(to), n, BLOCK, _ptr(out), _ptr(status),
                                     _stream(stream)), "kvgov_block_offsets")
    if own:
        check_status(status, "kvgov_block_offsets")
    return out


def hash_chains(tokens: torch.Tensor, tok_offsets: torch.Tensor, principal: Optional[torch.Tensor],
                salt_table: Optional[torch.Tensor], mode: int,
                boundary_tok: Optional[torch.Tensor] = None,
                blk_offsets: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                status: Optional[torch.Tensor] = None, check: bool = True,
                stream=None) -> torch.Tensor:
    """Chained block hashes, uint8 [blk_offsets[-1], 32] on the GPU.

    With ``check`` the call waits and raises any error the kernels latched;
    pass ``check=False`` and a shared ``status`` to keep the stream running."""
    tk = _dev(tokens, torch.int32, "tokens")
    to = _dev(tok_offsets, torch.int64, "tok_offsets")
    n = to.numel() - 1
    pr = _dev(principal, torch.int32, "principal", allow_none=(mode == NONE))
    st = _dev(salt_table, torch.uint8, "salts", allow_none=(mode == NONE))
    bt = _dev(boundary_tok, torch.int32, "boundary_tok", allow_none=(mode != BOUNDARY))
    P = 0 if st is None else int(st.shape[0])
    if status is None:
        status = new_status(tk.device)
    if blk_offsets is None:
        blk_offsets = block_offsets(to, status=status, stream=stream)
    bo = _dev(blk_offsets, torch.int64, "blk_offsets")
    if out is None:
        out = torch.empty((int(bo[-1].item()), 32), dtype=torch.uint8, device=tk.device)
    _dev(out, torch.uint8, "out")
    _check(lib().kvgov_hash_chains(_ptr(tk), tk.numel(), _ptr(to), n, _ptr(pr), _ptr(st), P,
                                   int(mode), _ptr(bt), BLOCK, _ptr(bo), _ptr(out),
                                   out.shape[0] if out.dim() else 0, _ptr(status),
                                   _stream(stream)), "kvgov_hash_chains")
    if check:
        check_status(status, "kvgov_hash_chains")
    return out


def hash_chains_noalloc(tokens: torch.Tensor, tok_offsets: torch.Tensor,
                        principal: Optional[torch.Tensor], salt_table: Optional[torch.Tensor],
                        mode: int, boundary_tok: Optional[torch.Tensor],
                        blk_offsets: torch.Tensor, out: torch.Tensor, status: torch.Tensor,
                        stream=None) -> torch.Tensor:
    """kvgov_hash_chains_noalloc: as hash_chains, with every buffer given by
    the caller (block offsets, output rows, status word), so that neither
    the library nor this binding allocates device memory.  Does not wait:
    errors the kernels find stay latched in ``status``."""
    tk = _dev(tokens, torch.int32, "tokens")
    to = _dev(tok_offsets, torch.int64, "tok_offsets")
    n = to.numel() - 1
    pr = _dev(principal, torch.int32, "principal", allow_none=(mode == NONE))
    st = _dev(salt_table, torch.uint8, "salts", allow_none=(mode == NONE))
    bt = _dev(boundary_tok, torch.int32, "boundary_tok", allow_none=(mode != BOUNDARY))
    bo = _dev(blk_offsets, torch.int64, "blk_offsets")
    _dev(out, torch.uint8, "out")
    _dev(status, torch.int32, "status")
    P = 0 if st is None else int(st.shape[0])
    _check(lib().kvgov_hash_chains_noalloc(_ptr(tk), tk.numel(), _ptr(to), n, _ptr(pr),
                                           _ptr(st), P, int(mode), _ptr(bt), BLOCK, _ptr(bo),
                                           _ptr(out), out.shape[0] if out.dim() else 0,
                                           _ptr(status), _stream(stream)),
           "kvgov_hash_chains_noalloc")
    return out


def resume_offsets(tok_offsets: torch.Tensor, start_block: torch.Tensor,
                   out: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    to = _dev(tok_offsets, torch.int64, "tok_offsets")
    sb = _dev(start_block, torch.int32, "start_block")
    n = to.numel() - 1
    if sb.numel() != n:
        raise ValueError("start_block must hold one entry per request")
    if out is None:
        out = torch.empty(n + 1, dtype=torch.int64, device=to.device)
    own = status is None
    if own:
        status = new_status(to.device)
    _check(lib().kvgov_resume_offsets(_ptr(to), _ptr(sb), n, BLOCK, _ptr(out), _ptr(status),
                                      _stream(stream)), "kvgov_resume_offsets")
    if own:
        check_status(status, "kvgov_resume_offsets")
    return out


def time_next_chain_kernel(start: Optional[torch.cuda.Event],
                           end: Optional[torch.cuda.Event]) -> None:
    """kvgov_time_next_chain_kernel: the next chain call of this thread records
    `start` and `end` (timing events) around its chain kernel alone.  The
    events must exist on the device already (torch creates an event at its
    first record), so each is recorded once here if it has not been."""
    if start is None and end is None:
        _check(lib().kvgov_time_next_chain_kernel(None, None), "kvgov_time_next_chain_kernel")
        return
    for e in (start, end):
        if e is None:
            raise ValueError("time_next_chain_kernel: both events or neither")
        if not e.cuda_event:
            e.record()
    _check(lib().kvgov_time_next_chain_kernel(_vp(start.cuda_event), _vp(end.cuda_event)),
           "kvgov_time_next_chain_kernel")


def hash_chains_resume(tokens: torch.Tensor, tok_offsets: torch.Tensor,
                       principal: Optional[torch.Tensor], salt_table: Optional[torch.Tensor],
                       mode: int, start_block: torch.Tensor, parents: torch.Tensor,
                       boundary_tok: Optional[torch.Tensor] = None,
                       blk_offsets: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
                       check: bool = True, stream=None) -> torch.Tensor:
    """Blocks start_block[r] .. len_r // 16 - 1 of each chain, resumed from
    parents[r] = h_{start_block[r] - 1}; uint8 [blk_offsets[-1], 32]."""
    tk = _dev(tokens, torch.int32, "tokens")
    to = _dev(tok_offsets, torch.int64, "tok_offsets")
    n = to.numel() - 1
    pr = _dev(principal, torch.int32, "principal", allow_none=(mode == NONE))
    st = _dev(salt_table, torch.uint8, "salts", allow_none=(mode == NONE))
    bt = _dev(boundary_tok, torch.int32, "boundary_tok", allow_none=(mode != BOUNDARY))
    sb = _dev(start_block, torch.int32, "start_block")
    pa = _dev(parents, torch.uint8, "parents")
    if sb.numel() != n or pa.numel() != 32 * n:
        raise ValueError("start_block and parents must hold one entry per request")
    P = 0 if st is None else int(st.shape[0])
    if status is None:
        status = new_status(tk.device)
    if blk_offsets is None:
        blk_offsets = resume_offsets(to, sb, status=status, stream=stream)
    bo = _dev(blk_offsets, torch.int64, "blk_offsets")
    if out is None:
        out = torch.empty((int(bo[-1].item()), 32), dtype=torch.uint8, device=tk.device)
    _dev(out, torch.uint8, "out")
    _check(lib().kvgov_hash_chains_resume(_ptr(tk), tk.numel(), _ptr(to), n, _ptr(pr), _ptr(st),
                                          P, int(mode), _ptr(bt), BLOCK, _ptr(sb), _ptr(pa),
                                          _ptr(bo), _ptr(out), out.shape[0] if out.dim() else 0,
                                          _ptr(status), _stream(stream)),
           "kvgov_hash_chains_resume")
    if check:
        check_status(status, "kvgov_hash_chains_resume")
    return out


# ---------------------------------------------------------------------------
# a4/a5 cache
# ---------------------------------------------------------------------------

class Cache:
    """Device-resident prefix-cache table (kvgov_cache_*)."""

    def __init__(self, log2_slots: int):
        h = _vp()
        _check(lib().kvgov_cache_create(int(log2_slots), ctypes.byref(h)), "kvgov_cache_create")
        self._h = h
        self._pid = os.getpid()
        self.log2_slots = int(log2_slots)

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("cache is closed")
        return self._h

    def slots(self) -> int:
        v = _c_i64()
        _check(lib().kvgov_cache_slots(self.handle, ctypes.byref(v)), "kvgov_cache_slots")
        return int(v.value)

    def clear(self, stream=None):
        _check(lib().kvgov_cache_clear(self.handle, _stream(stream)), "kvgov_cache_clear")

    def insert(self, hashes: torch.Tensor, blk_offsets: torch.Tensor, sync: bool = True,
               stream=None) -> Optional[int]:
        """Insert every key of the batch; with ``sync`` returns how many were new."""
        hs = _dev(hashes, torch.uint8, "hashes")
        bo = _dev(blk_offsets, torch.int64, "blk_offsets")
        nn = _c_i64(-1)
        _check(lib().kvgov_cache_insert(self.handle, _ptr(hs), _ptr(bo), bo.numel() - 1,
                                        hs.shape[0] if hs.dim() else 0,
                                        ctypes.byref(nn) if sync else None, _stream(stream)),
               "kvgov_cache_insert")
        return int(nn.value) if sync else None

    def lookup(self, hashes: torch.Tensor, blk_offsets: torch.Tensor,
               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Per request, the number of leading blocks present (int32 [n])."""
        hs = _dev(hashes, torch.uint8, "hashes")
        bo = _dev(blk_offsets, torch.int64, "blk_offsets")
        n = bo.numel() - 1
        if out is None:
            out = torch.empty(n, dtype=torch.int32, device=bo.device)
        _dev(out, torch.int32, "out")
        _check(lib().kvgov_cache_lookup(self.handle, _ptr(hs), _ptr(bo), n,
                                        hs.shape[0] if hs.dim() else 0, _ptr(out),
                                        _stream(stream)), "kvgov_cache_lookup")
        return out

    def admit(self, hashes: torch.Tensor, blk_offsets: torch.Tensor, sync: bool = True,
              hits: Optional[torch.Tensor] = None, new: Optional[torch.Tensor] = None,
              stream=None):
        """Lookup-then-insert in request order: (hit_blocks, new_blocks, n_new);
        n_new is None unless ``sync``."""
        hs = _dev(hashes, torch.uint8, "hashes")
        bo = _dev(blk_offsets, torch.int64, "blk_offsets")
        n = bo.numel() - 1
        if hits is None:
            hits = torch.empty(n, dtype=torch.int32, device=bo.device)
        if new is None:
            new = torch.empty(n, dtype=torch.int32, device=bo.device)
        _dev(hits, torch.int32, "hits")
        _dev(new, torch.int32, "new")
        nn = _c_i64(-1)
        _check(lib().kvgov_cache_admit(self.handle, _ptr(hs), _ptr(bo), n,
                                       hs.shape[0] if hs.dim() else 0, _ptr(hits), _ptr(new),
                                       ctypes.byref(nn) if sync else None, _stream(stream)),
               "kvgov_cache_admit")
        return hits, new, (int(nn.value) if sync else None)

    def set_recency(self, on: bool = True):
        """Tracks recency (needed by evict) from the next insert on."""
        _check(lib().kvgov_cache_set_recency(self.handle, 1 if on else 0),
               "kvgov_cache_set_recency")

    def evict(self, max_keys: int, sync: bool = True, stream=None) -> Optional[int]:
        """Keeps the most recent rank classes that fit in max_keys; with
        ``sync`` returns the number of keys kept."""
        v = _c_i64(-1)
        _check(lib().kvgov_cache_evict(self.handle, int(max_keys),
                                       ctypes.byref(v) if sync else None, _stream(stream)),
               "kvgov_cache_evict")
        return int(v.value) if sync else None

    def erase(self, keys: torch.Tensor, sync: bool = True, stream=None) -> Optional[int]:
        """Removes the given keys (uint8 [n, 32]); with ``sync`` returns how
        many of them were present."""
        ks = _dev(keys, torch.uint8, "keys")
        v = _c_i64(-1)
        _check(lib().kvgov_cache_erase(self.handle, _ptr(ks), ks.shape[0] if ks.dim() else 0,
                                       ctypes.byref(v) if sync else None, _stream(stream)),
               "kvgov_cache_erase")
        return int(v.value) if sync else None

    def count(self, stream=None) -> int:
        v = _c_i64()
        _check(lib().kvgov_cache_count(self.handle, ctypes.byref(v), _stream(stream)),
               "kvgov_cache_count")
        return int(v.value)

    def export(self, cap: Optional[int] = None, stream=None) -> torch.Tensor:
        """Every key in the table, uint8 [count, 32], in no particular order."""
        if cap is None:
            cap = self.count(stream)
        buf = torch.empty((max(cap, 1), 32), dtype=torch.uint8, device="cuda")
        v = _c_i64()
        _check(lib().kvgov_cache_export(self.handle, _ptr(buf), int(cap), ctypes.byref(v),
                                        _stream(stream)), "kvgov_cache_export")
        return buf[:int(v.value)]

    def close(self):
        # a forked child (e.g. a worker pool) inherits the object but not the
        # GPU context: only the creating process frees the table
        if self._h is not None and self._pid == os.getpid():
            _check(lib().kvgov_cache_destroy(self._h), "kvgov_cache_destroy")
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


# ---------------------------------------------------------------------------
# radix index
# ---------------------------------------------------------------------------

class Radix:
    """A kvgov_radix index on the current GPU (token-granular prefix match,
    one tree per principal in root mode, one shared tree unsalted)."""

    def __init__(self, log2_block_slots: int, log2_edge_slots: int):
        h = _vp()
        _check(lib().kvgov_radix_create(int(log2_block_slots), int(log2_edge_slots),
                                        ctypes.byref(h)), "kvgov_radix_create")
        self._h = h
        self._pid = os.getpid()

    @property
    def handle(self):
        if self._h is None or not self._h.value:
            raise ValueError("radix index is closed")
        return self._h

    def clear(self, stream=None):
        _check(lib().kvgov_radix_clear(self.handle, _stream(stream)), "kvgov_radix_clear")

    def _args(self, tokens, tok_offsets, principal, salt_table, mode, hashes, blk_offsets):
        tk = _dev(tokens, torch.int32, "tokens")
        to = _dev(tok_offsets, torch.int64, "tok_offsets")
        pr = _dev(principal, torch.int32, "principal", allow_none=(mode == NONE))
        st = _dev(salt_table, torch.uint8, "salts", allow_none=(mode == NONE))
        hs = _dev(hashes, torch.uint8, "hashes")
        bo = _dev(blk_offsets, torch.int64, "blk_offsets")
        P = 0 if st is None else int(st.shape[0])
        return [_ptr(tk), tk.numel(), _ptr(to), to.numel() - 1, _ptr(pr), _ptr(st), P,
                int(mode), _ptr(hs), _ptr(bo), hs.shape[0] if hs.dim() else 0]

    def insert(self, tokens, tok_offsets, principal, salt_table, mode, hashes, blk_offsets,
               stream=None):
        """Adds each request's token sequence to its tree (asynchronous)."""
        a = self._args(tokens, tok_offsets, principal, salt_table, mode, hashes, blk_offsets)
        _check(lib().kvgov_radix_insert(self.handle, *a, _stream(stream)), "kvgov_radix_insert")

    def match(self, tokens, tok_offsets, principal, salt_table, mode, hashes, blk_offsets,
              out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Matched prefix length in tokens per request (int32 [n])."""
        a = self._args(tokens, tok_offsets, principal, salt_table, mode, hashes, blk_offsets)
        if out is None:
            out = torch.empty(a[3], dtype=torch.int32, device="cuda")
        _dev(out, torch.int32, "out")
        _check(lib().kvgov_radix_match(self.handle, *a, _ptr(out), _stream(stream)),
               "kvgov_radix_match")
        return out

    def stats(self, stream=None):
        """(block nodes, edges); waits and raises a latched error."""
        b, e = _c_i64(), _c_i64()
        _check(lib().kvgov_radix_stats(self.handle, ctypes.byref(b), ctypes.byref(e),
                                       _stream(stream)), "kvgov_radix_stats")
        return int(b.value), int(e.value)

    def close(self):
        # only the creating process frees the index (see Cache.close)
        if getattr(self, "_h", None) is not None and self._h.value and \
                self._pid == os.getpid():
            _check(lib().kvgov_radix_destroy(self._h), "kvgov_radix_destroy")
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
