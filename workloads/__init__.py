"""Seeded synthetic inputs for the KVGov hot path.

This module only draws random numbers and lays them out; it computes no hash,
no salt and no lookup.  Both the CPU oracle (in the tests) and the HIP path
consume exactly the arrays it returns, so the two sides see identical inputs.

Workload shapes follow the paper's setting:

* token ids are int32 drawn uniformly from [0, 152064), the vocabulary size of
  the Qwen2.5 model family the paper measures (Sec. 5.1, Sec. 5.6);
* block size B = 16 (Sec. 2.1, chained block hashes);
* the 2119-token shared system prefix is the prefix length of the paper's
  hardware TTFT measurement (Table "tab:ttft");
* per-principal request counts reach Gini ~ 0.63, the tenant heterogeneity of
  the adversarial-load experiment (Sec. 5.4, Table "tab:advload");
* template prompts interleave fixed segments with bounded fields, the
  structured-prompt setting of Sec. 3.4.

The paper's prompts and templates are not published; every array here is a
seeded stand-in with the stated shape.  Streams are independent: each named
stream ``<config>/<name>`` gets ``np.random.default_rng([seed, s])`` with the
master seed 2026 (the paper's seed, Sec. 5.1) and s the first 8 bytes,
little-endian, of the SHA-256 digest of the stream's name (the paper derives
each condition's stream from a SHA-256 digest of the condition's name, Sec. 7,
reproducibility paragraph).  That digest of a name is the only hashing here:
no token, block, salt or chain is hashed.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import hashlib

import numpy as np

VOCAB = 152064
SEED = 2026
BLOCK = 16

# salt-placement modes, numbered as in the C ABI (kvgov.h)
NONE, ROOT, BOUNDARY = 0, 1, 2
MODE_NAMES = {NONE: "none", ROOT: "root", BOUNDARY: "boundary"}


def stream_seed(name: str) -> int:
    """The per-stream half of a generator's seed: the first 8 bytes of
    SHA-256(name), read little-endian."""
    return int.from_bytes(hashlib.sha256(name.encode()).digest()[:8], "little")


def rng(name: str, seed: int = SEED) -> np.random.Generator:
    """Independent generator for the stream ``name``."""
    return np.random.default_rng([seed, stream_seed(name)])


@dataclass
class Batch:
    """A ragged batch of requests in the flat layout the C ABI takes.

    tokens       int32 [tok_offsets[-1]]   all prompts back to back
    tok_offsets  int64 [n + 1]             request r owns tokens[tok_offsets[r]:tok_offsets[r+1]]
    principal    int32 [n]                 index into the principal table
    boundary_tok int32 [n]                 token offset of the divergence boundary
                                           (used by boundary mode only)
    expect_hits  int32 [n] or None         hit-block count a lookup must return,
                                           known from how the batch was built
    """

    tokens: np.ndarray
    tok_offsets: np.ndarray
    principal: np.ndarray
    boundary_tok: np.ndarray
    expect_hits: Optional[Dict[int, np.ndarray]] = None

    @property
    def n(self) -> int:
        return int(self.tok_offsets.shape[0] - 1)

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.tok_offsets)

    def block_counts(self) -> np.ndarray:
        """Number of full 16-token blocks per request (layout of the output)."""
        return self.lengths // BLOCK

    def blk_offsets(self) -> np.ndarray:
        out = np.zeros(self.n + 1, dtype=np.int64)
        np.cumsum(self.block_counts(), out=out[1:])
        return out

    def row(self, r: int) -> np.ndarray:
        return self.tokens[self.tok_offsets[r]:self.tok_offsets[r + 1]]

    def subset(self, idx) -> "Batch":
        """Requests ``idx`` (in that order) as a new, compact batch."""
        idx = np.asarray(idx, dtype=np.int64)
        lens = self.lengths[idx]
        offs = np.zeros(idx.size + 1, dtype=np.int64)
        np.cumsum(lens, out=offs[1:])
        toks = np.empty(int(offs[-1]), dtype=np.int32)
        for i, r in enumerate(idx):
            toks[offs[i]:offs[i + 1]] = self.row(int(r))
        eh = None
        if self.expect_hits is not None:
            eh = {m: v[idx] for m, v in self.expect_hits.items()}
        return Batch(toks, offs, self.principal[idx].copy(),
                     self.boundary_tok[idx].copy(), eh)


@dataclass
class Workload:
    name: str
    K: bytes                        # server secret (host bytes)
    principal_ids: np.ndarray       # uint8 [P, 32]
    insert: Batch                   # batch whose chains are inserted
    lookup: Optional[Batch]         # batch probed after the insert
    modes: List[int]
    log2_slots: int
    notes: Dict[str, object] = field(default_factory=dict)

    @property
    def P(self) -> int:
        return int(self.principal_ids.shape[0])


def _flat(lengths: np.ndarray) -> np.ndarray:
    offs = np.zeros(lengths.size + 1, dtype=np.int64)
    np.cumsum(lengths, out=offs[1:])
    return offs


def _uniform_tokens(g: np.random.Generator, count: int) -> np.ndarray:
    return g.integers(0, VOCAB, size=int(count), dtype=np.int32)


def _secret_and_ids(cfg: str, P: int, seed: int):
    K = rng(f"{cfg}/secret", seed).integers(0, 256, size=32, dtype=np.uint8).tobytes()
    ids = rng(f"{cfg}/principal_ids", seed).integers(0, 256, size=(P, 32), dtype=np.uint8)
    return K, ids


def zipf_counts(total: int, P: int, s: float) -> np.ndarray:
    """Counts proportional to rank^-s, largest-remainder rounded, minimum 1."""
    w = np.arange(1, P + 1, dtype=np.float64) ** -s
    q = w / w.sum() * total
    c = np.maximum(np.floor(q).astype(np.int64), 1)
    frac_order = np.argsort(-(q - np.floor(q)), kind="stable")
    i = 0
    while c.sum() < total:
        c[frac_order[i % P]] += 1
        i += 1
    while c.sum() > total:  # only reachable if the minimum of 1 overshoots
        j = int(np.argmax(c))
        c[j] -= 1
    return c


def gini(counts: np.ndarray) -> float:
    x = np.sort(np.asarray(counts, dtype=np.float64))
    n = x.size
    cum = np.cumsum(x)
    return float((n + 1 - 2 * (cum / cum[-1]).sum()) / n)


# ---------------------------------------------------------------------------
# configurations
# ---------------------------------------------------------------------------

def tiny(seed: int = SEED) -> Workload:
    """64 requests x 256 tokens, 4 principals, root mode; insert the first 32,
    look up all 64 (hit 16 for the inserted half, 0 for the rest)."""
    n, L, P = 64, 256, 4
    K, ids = _secret_and_ids("tiny", P, seed)
    toks = _uniform_tokens(rng("tiny/tokens", seed), n * L)
    offs = _flat(np.full(n, L, dtype=np.int64))
    prin = rng("tiny/principal", seed).integers(0, P, size=n, dtype=np.int32)
    bt = np.zeros(n, dtype=np.int32)
    full = Batch(toks, offs, prin, bt)
    ins = full.subset(np.arange(32))
    exp = np.where(np.arange(n) < 32, L // BLOCK, 0).astype(np.int32)
    look = Batch(toks, offs, prin, bt, {ROOT: exp})
    return Workload("tiny", K, ids, ins, look, [ROOT], 12,
                    {"inserted_requests": 32})


def paper(seed: int = SEED, n: int = 4096, P: int = 64) -> Workload:
    """Paper-shaped shared prefix: one fixed 2119-token system prefix plus a
    private suffix of U{64..1024} tokens; per-principal counts Zipf-like with
    Gini ~ 0.63.  The lookup batch keeps the principals and the prefix and
    draws fresh suffixes, so every lookup must hit exactly 132 = 2119 // 16
    blocks in all three modes (boundary at token 2119)."""
    prefix_len = 2119
    K, ids = _secret_and_ids("paper", P, seed)
    prefix = _uniform_tokens(rng("paper/prefix", seed), prefix_len)
    counts = zipf_counts(n, P, 1.0627)
    prin = np.repeat(np.arange(P, dtype=np.int32), counts)
    rng("paper/assign", seed).shuffle(prin)

    def build(stream: str) -> Batch:
        g = rng(stream, seed)
        suf = g.integers(64, 1025, size=n).astype(np.int64)
        lens = prefix_len + suf
        offs = _flat(lens)
        toks = np.empty(int(offs[-1]), dtype=np.int32)
        body = _uniform_tokens(g, int(suf.sum()))
        pos = 0
        for r in range(n):
            a = int(offs[r])
            toks[a:a + prefix_len] = prefix
            toks[a + prefix_len:int(offs[r + 1])] = body[pos:pos + suf[r]]
            pos += int(suf[r])
        bt = np.full(n, prefix_len, dtype=np.int32)
        return Batch(toks, offs, prin.copy(), bt)

    ins = build("paper/suffix_insert")
    look = build("paper/suffix_lookup")
    hit = np.full(n, prefix_len // BLOCK, dtype=np.int32)
    look.expect_hits = {NONE: hit, ROOT: hit, BOUNDARY: hit}
    return Workload("paper", K, ids, ins, look, [ROOT, BOUNDARY], 20,
                    {"prefix_len": prefix_len, "gini": gini(counts),
                     "counts": counts})


def template(seed: int = SEED, n: int = 16384, P: int = 256) -> Workload:
    """Template-structured prompts: 12 fixed segments (32..128 tokens each)
    interleaved with 4 bounded fields (each one of 512 candidate strings of
    1..4 tokens), layout S0 S1 S2 F0 S3 S4 S5 F1 S6 S7 S8 F2 S9 S10 S11 F3.
    The boundary is the first field's offset.  Insert n draws, look up n fresh
    draws; no closed-form hit count."""
    K, ids = _secret_and_ids("template", P, seed)
    g = rng("template/segments", seed)
    seg_len = g.integers(32, 129, size=12)
    segs = [_uniform_tokens(g, int(l)) for l in seg_len]
    gf = rng("template/fields", seed)
    fields = []
    for _ in range(4):
        fl = gf.integers(1, 5, size=512)
        fields.append([_uniform_tokens(gf, int(l)) for l in fl])
    boundary = int(seg_len[0] + seg_len[1] + seg_len[2])

    def build(stream: str) -> Batch:
        gs = rng(stream, seed)
        choice = gs.integers(0, 512, size=(n, 4))
        prin = gs.integers(0, P, size=n, dtype=np.int32)
        rows = []
        for r in range(n):
            parts = []
            for f in range(4):
                parts.extend(segs[3 * f:3 * f + 3])
                parts.append(fields[f][choice[r, f]])
            rows.append(np.concatenate(parts))
        lens = np.array([x.size for x in rows], dtype=np.int64)
        offs = _flat(lens)
        toks = np.concatenate(rows).astype(np.int32)
        bt = np.full(n, boundary, dtype=np.int32)
        return Batch(toks, offs, prin, bt)

    return Workload("template", K, ids, build("template/insert"),
                    build("template/lookup"), [NONE, ROOT, BOUNDARY], 22,
                    {"boundary_tok": boundary, "segment_lengths": seg_len})


def probe(seed: int = SEED, n_res: int = 250_000, n_probe: int = 1_000_000,
          P: int = 1024) -> Workload:
    """Probe-heavy lookup: a resident set of n_res requests x 32 blocks (root
    mode, 8M keys at full size) in a 2^24-slot table, then n_probe probe
    requests of U{8..64} blocks.  70 % copy a resident request's first d
    blocks (d = U{1..min(L,32)}) under its own principal and then diverge
    (expected hit d); 30 % do the same under another principal (expected hit 0)."""
    K, ids = _secret_and_ids("probe", P, seed)
    L_res = 512
    res_toks = _uniform_tokens(rng("probe/resident_tokens", seed), n_res * L_res)
    res_offs = _flat(np.full(n_res, L_res, dtype=np.int64))
    res_prin = rng("probe/resident_principal", seed).integers(0, P, size=n_res, dtype=np.int32)
    resident = Batch(res_toks, res_offs, res_prin, np.zeros(n_res, dtype=np.int32))

    g = rng("probe/probes", seed)
    nblk = g.integers(8, 65, size=n_probe).astype(np.int64)
    src = g.integers(0, n_res, size=n_probe).astype(np.int64)
    own = g.random(n_probe) < 0.7
    d = (np.floor(g.random(n_probe) * np.minimum(nblk, 32)).astype(np.int64) + 1)
    lens = nblk * BLOCK
    offs = _flat(lens)
    toks = _uniform_tokens(g, int(offs[-1]))
    # copy the shared prefix: probe blocks [0, d) <- resident blocks [0, d)
    # (every probe starts on a block edge, so whole 16-token rows are copied)
    blk = toks.reshape(-1, BLOCK)
    res_blk = res_toks.reshape(-1, BLOCK)
    first = np.repeat(offs[:-1] // BLOCK - (np.cumsum(d) - d), d)
    within = np.arange(int(d.sum()), dtype=np.int64)
    src_first = np.repeat(src * (L_res // BLOCK) - (np.cumsum(d) - d), d)
    blk[first + within] = res_blk[src_first + within]
    # force divergence at token 16 d when the probe and the resident request
    # both have a block d
    div = (d < nblk) & (d < 32)
    pos_p = offs[:-1][div] + d[div] * BLOCK
    orig = res_toks[src[div] * L_res + d[div] * BLOCK].astype(np.int64)
    bump = g.integers(1, VOCAB, size=int(div.sum())).astype(np.int64)
    toks[pos_p] = ((orig + bump) % VOCAB).astype(np.int32)
    prin = res_prin[src].copy()
    other = g.integers(1, P, size=n_probe, dtype=np.int32)
    prin[~own] = (prin[~own] + other[~own]) % P
    hits = np.where(own, d, 0).astype(np.int32)
    probes = Batch(toks, offs, prin.astype(np.int32),
                   np.zeros(n_probe, dtype=np.int32), {ROOT: hits})
    return Workload("probe", K, ids, resident, probes, [ROOT], 24,
                    {"own_fraction": float(own.mean()), "source": src, "depth": d})


def large(seed: int = SEED, n: int = 65536, P: int = 4096,
          sigma: float = 1.0) -> Workload:
    """Large batch: lognormal lengths (median 2048, sigma 1.0, clipped to
    [1, 32768] tokens), 4096 principals, boundary uniform in [0, len].
    Chains plus insert; the lookup re-probes the same batch (hit = its block
    count)."""
    K, ids = _secret_and_ids("large", P, seed)
    g = rng("large/lengths", seed)
    lens = np.floor(np.exp(np.log(2048.0) + sigma * g.standard_normal(n)))
    lens = np.clip(lens, 1, 32768).astype(np.int64)
    offs = _flat(lens)
    toks = _uniform_tokens(rng("large/tokens", seed), int(offs[-1]))
    prin = rng("large/principal", seed).integers(0, P, size=n, dtype=np.int32)
    bt = np.floor(rng("large/boundary", seed).random(n) * (lens + 1)).astype(np.int32)
    b = Batch(toks, offs, prin, bt)
    full = (lens // BLOCK).astype(np.int32)
    look = Batch(toks, offs, prin, bt, {ROOT: full, BOUNDARY: full})
    return Workload("large", K, ids, b, look, [ROOT, BOUNDARY], 25,
                    {"sigma": sigma})


def session(seed: int = SEED, n: int = 4096, P: int = 64) -> Workload:
    """Multi-turn sessions (Sec. 5.7: turn n+1 extends turn n exactly).  Turn
    1 of each session is a request of the paper-shaped workload (2119-token
    shared prefix + U{64..1024} private suffix); turn 2 appends a follow-up of
    U{64..1024} tokens.  Turn 2 resumes each chain at turn 1's full-block
    count, from turn 1's last full-block digest, so only the blocks from there
    on are hashed (notes: ``turn1`` batch, ``start`` blocks).  Boundary at
    token 2119 in both turns.  The lookup re-probes the resumed rows (hit =
    the number of blocks hashed for the request)."""
    base = paper(seed=seed, n=n, P=P)
    t1 = base.insert
    g = rng("session/followup", seed)
    extra = g.integers(64, 1025, size=n).astype(np.int64)
    lens2 = t1.lengths + extra
    offs2 = _flat(lens2)
    toks2 = np.empty(int(offs2[-1]), dtype=np.int32)
    new = _uniform_tokens(g, int(extra.sum()))
    pos = 0
    for r in range(n):
        a, l1 = int(offs2[r]), int(t1.lengths[r])
        toks2[a:a + l1] = t1.row(r)
        toks2[a + l1:int(offs2[r + 1])] = new[pos:pos + extra[r]]
        pos += int(extra[r])
    t2 = Batch(toks2, offs2, t1.principal.copy(), t1.boundary_tok.copy())
    start = (t1.lengths // BLOCK).astype(np.int32)
    hashed = (lens2 // BLOCK - start).astype(np.int32)
    look = Batch(toks2, offs2, t2.principal, t2.boundary_tok,
                 {ROOT: hashed, BOUNDARY: hashed})
    return Workload("session", base.K, base.principal_ids, t2, look, [ROOT, BOUNDARY], 20,
                    {"turn1": t1, "start": start, "gini": base.notes["gini"],
                     "prefix_len": base.notes["prefix_len"]})


def admission(seed: int = SEED, n: int = 4096, P: int = 64) -> Workload:
    """The paper-shaped batches admitted in one call each mode: the insert
    batch then the re-lookup batch, 2n requests in order.  Hits are fixed by
    construction: a request sees the 132 prefix blocks once an earlier request
    of its salting domain (root: the same principal; boundary: any request,
    the prefix lies below the boundary) holds them, else nothing; the block
    after the prefix mixes prefix and private tokens and is never shared.
    notes["admit_hits"][mode] = int32 [2n]."""
    base = paper(seed=seed, n=n, P=P)
    pre = base.notes["prefix_len"] // BLOCK
    prin = np.concatenate([base.insert.principal, base.lookup.principal])
    first_of_principal = np.zeros(2 * n, dtype=bool)
    first_of_principal[np.unique(prin, return_index=True)[1]] = True
    root = np.where(first_of_principal, 0, pre).astype(np.int32)
    bnd = np.full(2 * n, pre, dtype=np.int32)
    bnd[0] = 0
    notes = dict(base.notes)
    notes["admit_hits"] = {ROOT: root, BOUNDARY: bnd}
    return Workload("admission", base.K, base.principal_ids, base.insert, base.lookup,
                    [ROOT, BOUNDARY], base.log2_slots, notes)


def radix(seed: int = SEED, n: int = 4096, P: int = 64) -> Workload:
    """The paper-shaped batches on the radix index: the insert batch's token
    sequences go into the index, the re-lookup batch is matched (token
    granular: every match is at least the 2119-token shared prefix, more
    where a fresh suffix happens to continue an inserted one).  Root salting
    (one tree per principal) and unsalted (one tree)."""
    base = paper(seed=seed, n=n, P=P)
    return Workload("radix", base.K, base.principal_ids, base.insert, base.lookup,
                    [ROOT, NONE], base.log2_slots, dict(base.notes))


def maintenance(seed: int = SEED, n: int = 4096, P: int = 64) -> Workload:
    """The paper-shaped batches on a table that tracks recency: the insert
    batch, then the re-lookup batch, in two insert calls; an eviction down
    to half of the keys present, an erase of the first tenth of the insert
    batch's rows, then a lookup of the re-lookup batch."""
    base = paper(seed=seed, n=n, P=P)
    notes = dict(base.notes)
    notes["evict_fraction"] = 0.5
    notes["erase_fraction"] = 0.1
    return Workload("maintenance", base.K, base.principal_ids, base.insert, base.lookup,
                    [ROOT, BOUNDARY], base.log2_slots, notes)


CONFIGS = {
    "tiny": tiny,
    "paper": paper,
    "template": template,
    "probe": probe,
    "large": large,
    "session": session,
    "admission": admission,
    "radix": radix,
    "maintenance": maintenance,
}


def make(name: str, seed: int = SEED, **kw) -> Workload:
    return CONFIGS[name](seed=seed, **kw)
