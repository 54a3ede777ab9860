"""Throughput of the KVGov hot path on one MI355X.

Default (the bench line): one step = one pass of the whole hot path over the
large-batch workload (65,536 requests with lognormal lengths, median 2048
tokens, clipped to 32,768; 4096 principals; ~13.7M full blocks):

    salts for the 4096 principals (HMAC-SHA256)
    for mode in (root, boundary at a uniform token of each request), each on
    its own stream:
        clear the table (concurrently with the salts)
        hash the batch in one call
        insert its keys, look the batch up again

Inputs are generated once and are resident in HBM before timing starts.
value = block tokens hashed per second over the whole step (16 tokens per
full block, both modes).  The roofline entry is for the chain kernel (the
dominant kernel), its fraction taken on 1672 integer ops per compression
(the FIPS 180-4 definition, one op per rotate, shift, xor, and, add or
3-input add; the gfx950 count with 3-input logic ops, 1384, is beside it).
The timed steps carry HIP events around the chain kernels only (the
library records them around the kernel itself, after the ordering kernels
of a large batch; a timing event costs its stream a few microseconds); the
per-phase launch times come from as many steps again, run after the timed
ones with events around every call.

After the line's own workload, the default run times the other
configurations, each with its own kind of step, and summarises each under
"configs" (tokens/s, lookups/s, the chain kernel's integer-VALU fraction,
the lookup's and insert's HBM fractions, gates):

    tiny      64 x 256 tokens, 4 principals, root; insert 32, look up 64
    paper     4096 requests x 2 batches, 2119-token shared prefix, root and
              boundary (token 2119): chains of both batches, insert, lookup
    template  16384 requests x 2 batches, 12 template segments + 4 fields;
              none, root, boundary
    probe     lookups alone: 1M probe requests against the 8M-key resident
              table (the resident chains, the probe chains and the insert
              are done before timing); its lookup roofline is the line's
              roofline_lookup and its lookups/s the line's lookups_per_s

Each step derives its salts during the previous step (two salt buffers; the
timed region holds one salts derivation per step).  --pipeline 2 keeps two
batches in flight.  Beside the line's own fields: per-phase rates for every
mode (median, mean and min launch times of salts, chains, clear, insert,
lookup), the insert kernel's HBM roofline, the critical-path ceiling (the
longest request hashed alone), the device's measured peaks (integer-VALU and
32-byte random-gather microbenchmarks, a 1 GiB copy) with the fractions of
those, and the CPU oracle on a bounded sample of the same workload, with the
host's core count, CPU model and SHA extension flag.  The oracle runs only in
that CPU-baseline leg (skipped with --no-cpu-baseline), where it is timed and
checks sampled outputs of each step bit for bit (gate G1).

--config NAME times one workload alone (also session, admission, radix,
maintenance: chains resumed from turn 1's digests; lookup-then-insert in
request order; the radix index; recency eviction and erase).  --mode runs a
single salt mode, --seed changes the master seed of the inputs (2026).

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--config NAME]
                       [--mode MODE] [--seed S] [--no-configs]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

# --- hardware figures (MI355X, published) ----------------------------------
CUS = 256
SIMDS_PER_CU = 4
LANES_PER_SIMD = 16
CLOCK_GHZ = 2.4
INT_PEAK_TOPS = CUS * SIMDS_PER_CU * LANES_PER_SIMD * CLOCK_GHZ * 1e9 / 1e12  # 39.32
HBM_PEAK_GBS = 8000.0

# --- algorithmic work --------------------------------------------------------
# One SHA-256 compression as the FIPS 180-4 definition writes it, one op per
# rotate, shift, xor, and, add or 3-input add: 64 rounds x 17 (two sigmas of
# 5, choose 1, majority 2, two 3-input adds for T1 and one each for e' and
# a') + 48 schedule words x 12 (two sigmas of 5, two adds) + 8 final adds =
# 1672.  The fractions are taken on this count.  gfx950 has 3-input xor,
# choose and majority in one op each (v_bitop3_b32): 64 x 14 + 48 x 10 + 8 =
# 1384, reported beside it.
OPS_PER_COMPRESSION = 1672
OPS_PER_COMPRESSION_GFX950 = 1384
# Lookup: per examined block a 32-byte query and a 32-byte slot key; per
# request two 8-byte offsets and a 4-byte result.
LOOKUP_BYTES_PER_BLOCK = 64
LOOKUP_BYTES_PER_REQUEST = 20
# Insert: a new key reads its 32-byte query and one slot, and writes the slot;
# a key already present reads the query and the slot holding it.
INSERT_BYTES_NEW = 96
INSERT_BYTES_PRESENT = 64
# Radix match: the block lookup's bytes, plus per request the 32-byte key of
# the last matched block (its node) and per token step one 8-byte edge key
# and the 4-byte token.  Radix insert: per record (full or partial block) its
# parent key (32 B) and per edge the 4-byte token and the 8-byte edge slot
# (read, and written when new).
RADIX_MATCH_BYTES_NODE = 32
RADIX_MATCH_BYTES_STEP = 12
RADIX_INSERT_BYTES_RECORD = 32
RADIX_INSERT_BYTES_EDGE = 12
RADIX_EDGE_SLOTS_LOG2 = 23
# Maintenance (evict, erase): per slot one scan of tag and recency word for
# the ranks, the compaction scan (tag + word) and the refill (key, tag, word
# written); per kept key its key read and 40 B written to scratch, then read
# back, a probe's tag read and its key, tag and word written again.  Erase
# marks: per listed key its 32 B, the slot key compared and the word swapped.
EVICT_BYTES_PER_SLOT = 16 + 16 + 48
ERASE_BYTES_PER_SLOT = 16 + 48
MAINT_BYTES_PER_KEPT = 32 + 40 + 40 + 8 + 48
ERASE_BYTES_PER_LISTED = 32 + 32 + 8
# Admission: the insert's bytes, plus per row a 4-byte code written and read
# back and an 8-byte tag read; per request two 8-byte offsets and two 4-byte
# outputs.
ADMIT_BYTES_PER_ROW = 16
ADMIT_BYTES_PER_REQUEST = 24

DESCRIPTIONS = {
    "paper": "paper-shaped shared prefix: 4096 requests x 2 batches (insert, re-lookup with "
             "fresh suffixes), 64 principals (Zipf, Gini {gini:.3f}), 2119-token shared prefix + "
             "U{{64..1024}} suffix, B=16, root and boundary (token 2119) modes",
    "tiny": "tiny: 64 requests x 256 tokens, 4 principals, root; insert 32, look up 64",
    "template": "template-structured: 16384 requests x 2 batches, 256 principals, 12 segments + "
                "4 fields of 512 candidates; none, root, boundary modes",
    "probe": "probe-heavy lookup: 8M resident keys (250k x 32 blocks, root, 2^24 slots), "
             "1M probes of U{{8..64}} blocks, 70% own-principal prefixes, 30% foreign",
    "large": "large batch: 65536 requests, lognormal lengths (median 2048, sigma 1, max "
             "32768 tokens), 4096 principals, root and boundary; chains + insert + re-lookup",
    "maintenance": "paper-shaped batches on a recency-tracking table: insert batch then "
                   "re-lookup batch (two insert calls), evict to half the keys, erase a tenth "
                   "of the insert batch's rows, look up the re-lookup batch; root and boundary",
    "radix": "paper-shaped batches on the radix index: 4096 insert-batch sequences inserted, "
             "4096 re-lookup-batch requests matched token by token, 64 principals, root "
             "(per-principal trees) and unsalted; chains + clear + insert + match",
    "admission": "paper-shaped batches admitted in order: 8192 requests (4096 insert-batch "
                 "then 4096 re-lookup-batch), 64 principals, root and boundary (token 2119); "
                 "chains + one lookup-then-insert call per mode",
    "session": "multi-turn sessions: 4096 turn-2 prompts (paper-shaped turn 1 + U{{64..1024}} "
               "follow-up tokens), 64 principals, root and boundary (token 2119); chains "
               "resumed at turn 1's last full block + insert + re-lookup of the new blocks",
}


# the workload of the bench line (the largest single-GPU configuration) and
# the configurations timed after it in the default run
HEADLINE = "large"
SECONDARY = ("tiny", "paper", "template", "probe")
# Batches in flight per workload (--pipeline 0).  Large batch: after the
# first ~1.2 ms of a chain launch only the CUs running the longest chains are
# busy, and the insert and re-lookup that follow are latency-bound; with a
# second batch in flight they overlap the next batch's chains.
PIPELINE = {"large": 2}
# Hardware queues per process.  Each batch in flight uses one stream per mode
# and one for the salts; streams that share a hardware queue run one after
# the other, which takes the overlap away (HIP's default is 4 queues).
HW_QUEUES = 8


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Kernel sources whose hash identifies the build a traffic record was taken on.
KERNEL_SOURCES = {
    "chains": ["chains.hip", "sha256_cdna4.h", "common.h"],
    "cache": ["cache.hip", "table.h", "common.h"],
    "radix": ["radix.hip", "table.h", "common.h"],
}
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "hbm_traffic.md")
TRAFFIC_FRAC_NOTE = ("HBM bytes the kernel actually moves per launch (traffic) over its mean "
                     "duration, against the same peak: how busy the memory is, where frac "
                     "counts algorithmic bytes only (a 32-byte slot probe fills a 128-byte "
                     "line)")


def sources_sha256(group: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[group]:
        with open(os.path.join(ROOT, "paper_2608_09225_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(kernel: str, workload: str, group: str):
    """HBM bytes per launch (fetch + write, scaled by a copy kernel) from the
    committed counter record, or None if the kernel's sources changed since."""
    try:
        with open(TRAFFIC_RECORD) as f:
            rows = [l for l in f if l.startswith("| `")]
    except OSError:
        return None
    want = sources_sha256(group)
    for row in rows:
        cells = [c.strip().strip("`") for c in row.strip().strip("|").split("|")]
        if len(cells) >= 5 and cells[0] == kernel and cells[1] == workload:
            if cells[2] != want:
                return None
            return {"fetch_bytes": int(cells[3]), "write_bytes": int(cells[4]),
                    "bytes": int(cells[3]) + int(cells[4])}
    return None


def start_blocks(wl: W.Workload, batch: W.Batch) -> np.ndarray:
    """Block each request's hashing starts at: turn 1's full-block count for
    the resumed sessions, else 0."""
    st = wl.notes.get("start") if wl.name == "session" else None
    return np.zeros(batch.n, np.int64) if st is None else np.asarray(st, np.int64)


def hashed_counts(wl: W.Workload, batch: W.Batch) -> np.ndarray:
    """Blocks hashed (and inserted / looked up) per request."""
    return batch.block_counts() - start_blocks(wl, batch)


def compressions(wl: W.Workload, batch: W.Batch, mode: int) -> int:
    """Compressions the definition needs: 2 per hashed block, plus one for
    the 128-byte boundary block (boundary mode, 0 < k < n_full, k at or
    after the start block)."""
    nf = batch.block_counts()
    j0 = start_blocks(wl, batch)
    c = 2 * int((nf - j0).sum())
    if mode == W.BOUNDARY:
        k = batch.boundary_tok.astype(np.int64) // W.BLOCK
        c += int(((k > 0) & (k < nf) & (k >= j0)).sum())
    return c


def radix_match_bytes(counts: np.ndarray, match: np.ndarray) -> int:
    """Algorithmic bytes of one radix match launch: the block lookup up to
    the first absent block, the node key of the last matched block, and the
    edge steps (the matched ones and the failing one)."""
    hits = np.minimum(match.astype(np.int64) // 16, counts)
    return (lookup_bytes(counts, hits) + RADIX_MATCH_BYTES_NODE * counts.size +
            RADIX_MATCH_BYTES_STEP * int((match.astype(np.int64) % 16 + 1).sum()))


def radix_insert_edges(batch: W.Batch) -> int:
    """Edges the insert walks: the first min(len, 15) tokens of every full or
    partial block."""
    L = batch.lengths.astype(np.int64)
    tail = L % 16
    return int(15 * (L // 16).sum() + tail.sum())


def admit_bytes(n_req: int, rows: int, n_new: int) -> int:
    """Algorithmic bytes of one admission call (both kernels)."""
    return (INSERT_BYTES_NEW * n_new + INSERT_BYTES_PRESENT * (rows - n_new) +
            ADMIT_BYTES_PER_ROW * rows + ADMIT_BYTES_PER_REQUEST * n_req)


def admit_group(n: int, rows: int) -> int:
    """Lanes per request of the admission scan, the plain insert and the radix
    edge walk (the library's rule)."""
    avg = rows // n if n else 0
    g = 4
    while g < 64 and g * 2 < avg:
        g <<= 1
    return g


def lookup_lanes(n: int, n_blocks: int) -> int:
    """Lanes per request of the lookup kernel (the library's rule)."""
    g = 1
    while g < 64 and n * g * 2 <= (1 << 18):
        g <<= 1
    avg = n_blocks // n if n else 0
    while g < 64 and g * 16 <= avg and n * g * 2 <= (1 << 21):
        g <<= 1
    if avg >= 128:
        while g < 64 and n * g * 2 <= (1 << 22):
            g <<= 1
    return g


def lookup_bytes(counts: np.ndarray, hits: np.ndarray) -> int:
    examined = np.minimum(hits.astype(np.int64) + 1, counts)
    return int(examined.sum()) * LOOKUP_BYTES_PER_BLOCK + counts.size * LOOKUP_BYTES_PER_REQUEST


def concat(A: W.Batch, B: W.Batch) -> W.Batch:
    return W.Batch(np.concatenate([A.tokens, B.tokens]),
                   np.concatenate([A.tok_offsets, B.tok_offsets[1:] + A.tok_offsets[-1]]),
                   np.concatenate([A.principal, B.principal]),
                   np.concatenate([A.boundary_tok, B.boundary_tok]))


def capped(b: W.Batch, max_blocks: int) -> W.Batch:
    """The first requests of ``b`` holding at most ``max_blocks`` blocks."""
    bo = b.blk_offsets()
    n = int(np.searchsorted(bo, max_blocks, side="right")) - 1
    return b if n >= b.n else b.subset(np.arange(max(n, 1)))


def host_cpu_info() -> dict:
    info = {"os_cpu_count": os.cpu_count(), "model": None, "sha_ni": None}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name") and info["model"] is None:
                    info["model"] = line.split(":", 1)[1].strip()
                if line.startswith("flags") and info["sha_ni"] is None:
                    info["sha_ni"] = "sha_ni" in line.split(":", 1)[1].split()
    except OSError:
        pass
    return info


def cpu_salt_cost(wl: W.Workload, min_seconds: float = 0.2) -> float:
    """Seconds per HMAC key derivation with the oracle (one process)."""
    import oracle as O
    n, t0 = 0, time.perf_counter()
    while True:
        O.salts(wl.K, wl.principal_ids)
        n += wl.P
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            return dt / n


def cpu_baseline(wl: W.Workload, processes: int, max_blocks: int):
    """The oracle, untouched, running the same step on the host cores (on the
    first requests of each batch when the workload is larger than
    ``max_blocks`` blocks per batch), each phase timed on its own; plus the
    chains of a few requests on one core and the per-key HMAC cost."""
    import oracle as O
    if wl.name == "probe":
        return cpu_baseline_probe(wl, processes)
    if wl.name == "session":
        return cpu_baseline_session(wl, processes)
    if wl.name == "admission":
        return cpu_baseline_admission(wl, processes)
    if wl.name == "radix":
        return cpu_baseline_radix(wl, processes)
    if wl.name == "maintenance":
        return cpu_baseline_maintenance(wl, processes)
    same = wl.name == "large"
    A = capped(wl.insert, max_blocks)
    B = A if same else capped(wl.lookup, max_blocks)
    clock = time.perf_counter
    t = {"salts": 0.0, "chains": 0.0, "insert": 0.0, "lookup": 0.0}
    t0 = clock()
    salts = O.salts(wl.K, wl.principal_ids)
    t["salts"] = clock() - t0
    tokens = keys = lookups = 0
    for mode in wl.modes:
        hashes = {}
        for name, b in (("insert", A), ("lookup", B)):
            if name == "lookup" and same:
                hashes[name] = hashes["insert"]
                continue
            t0 = clock()
            hashes[name] = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, salts,
                                                  mode, b.boundary_tok, processes=processes)
            t["chains"] += clock() - t0
            tokens += 16 * int(b.block_counts().sum())
        T = O.Table()
        t0 = clock()
        T.insert(hashes["insert"], A.blk_offsets())
        t["insert"] += clock() - t0
        keys += hashes["insert"].shape[0]
        t0 = clock()
        T.lookup(hashes["lookup"], B.blk_offsets())
        t["lookup"] += clock() - t0
        lookups += B.n
    dt = sum(t.values())
    # one core: the chains of the first requests of the insert batch
    one = capped(A, 20000)
    t0 = clock()
    O.hash_chains(one.tokens, one.tok_offsets, one.principal, salts, wl.modes[0],
                  one.boundary_tok)
    t1 = clock() - t0
    whole = A is wl.insert and (same or B is wl.lookup)
    what = "one full step of the same workload" if whole else \
        f"the step on the first {A.n} (insert) / {B.n} (lookup) requests"
    return {"value": tokens / dt, "unit": "tokens/s", "cores": processes, "kind": "oracle",
            "sample": (f"{what} ({tokens} block tokens hashed, {lookups} lookups, "
                       f"{len(wl.modes)} mode(s)) in {dt:.1f} s; chains over {processes} "
                       "worker processes, salts and table in one process"),
            "seconds": dt, "lookups_per_s": lookups / dt,
            "phases": {
                "salts_us_per_key": t["salts"] / wl.P * 1e6,
                "chains_tokens_per_s": tokens / t["chains"],
                "insert_keys_per_s": keys / t["insert"],
                "lookup_lookups_per_s": lookups / t["lookup"],
            },
            "single_core": {
                "chains_tokens_per_s": 16 * int(one.block_counts().sum()) / t1,
                "sample": f"chains of the first {one.n} insert requests, "
                          f"{W.MODE_NAMES[wl.modes[0]]} mode",
                "salts_us_per_key": cpu_salt_cost(wl) * 1e6,
            },
            "host": host_cpu_info()}


def cpu_baseline_maintenance(wl: W.Workload, processes: int):
    """The oracle's step on the same workload: chains of both batches (over
    worker processes), then in one process the two inserts, the eviction to
    half the keys, the erase of a tenth of the insert batch's rows and the
    lookup of the re-lookup batch."""
    import oracle as O
    A, B = wl.insert, wl.lookup
    X = concat(A, B)
    nA = int(A.block_counts().sum())
    clock = time.perf_counter
    t = {"salts": 0.0, "chains": 0.0, "insert": 0.0, "evict": 0.0, "erase": 0.0, "lookup": 0.0}
    t0 = clock()
    salts = O.salts(wl.K, wl.principal_ids)
    t["salts"] = clock() - t0
    tokens = 0
    for mode in wl.modes:
        t0 = clock()
        h = O.hash_chains_parallel(X.tokens, X.tok_offsets, X.principal, salts, mode,
                                   X.boundary_tok, processes=processes)
        t["chains"] += clock() - t0
        tokens += 16 * h.shape[0]
        T = O.Table()
        t0 = clock()
        T.insert(h[:nA], A.blk_offsets())
        T.insert(h[nA:], B.blk_offsets())
        t["insert"] += clock() - t0
        t0 = clock()
        T.evict(int(len(T.keys) * wl.notes["evict_fraction"]))
        t["evict"] += clock() - t0
        t0 = clock()
        T.erase(h[:int(nA * wl.notes["erase_fraction"])])
        t["erase"] += clock() - t0
        t0 = clock()
        T.lookup(h[nA:], B.blk_offsets())
        t["lookup"] += clock() - t0
    dt = sum(t.values())
    return {"value": tokens / dt, "unit": "tokens/s", "cores": processes, "kind": "oracle",
            "sample": (f"one full step of the same workload ({tokens} block tokens hashed, "
                       f"{len(wl.modes)} modes) in {dt:.1f} s; chains over {processes} worker "
                       "processes, the table steps in one process"),
            "seconds": dt,
            "phases": {k + "_s": v for k, v in t.items()},
            "host": host_cpu_info()}


def cpu_baseline_radix(wl: W.Workload, processes: int, sample: int = 128):
    """The oracle's chains of both batches (over worker processes), its radix
    insert of the insert batch and its match of the first ``sample`` requests
    of the re-lookup batch (one process; the match time is scaled to the
    whole batch, stated in ``sample``)."""
    import oracle as O
    A, B = wl.insert, wl.lookup
    X = concat(A, B)
    clock = time.perf_counter
    t = {"salts": 0.0, "chains": 0.0, "insert": 0.0, "match": 0.0}
    t0 = clock()
    salts = O.salts(wl.K, wl.principal_ids)
    t["salts"] = clock() - t0
    tokens = 0
    q = np.arange(min(sample, B.n))
    for mode in wl.modes:
        t0 = clock()
        h = O.hash_chains_parallel(X.tokens, X.tok_offsets, X.principal, salts, mode,
                                   X.boundary_tok, processes=processes)
        t["chains"] += clock() - t0
        tokens += 16 * h.shape[0]
        R = O.Radix()
        t0 = clock()
        R.insert(A.tokens, A.tok_offsets, A.principal, salts, mode)
        t["insert"] += clock() - t0
        t0 = clock()
        R.match(B.tokens, B.tok_offsets, B.principal, salts, mode, requests=q)
        t["match"] += (clock() - t0) * B.n / q.size
    dt = sum(t.values())
    return {"value": tokens / dt, "unit": "tokens/s", "cores": processes, "kind": "oracle",
            "sample": (f"chains of both batches ({tokens} block tokens) and the radix insert "
                       f"of the insert batch in full, the match of {q.size} of the {B.n} "
                       f"re-lookup requests scaled to the batch ({len(wl.modes)} modes); "
                       f"{dt:.1f} s with the scaling; chains over {processes} worker "
                       "processes, the rest in one process"),
            "seconds": dt, "matches_per_s": len(wl.modes) * B.n / dt,
            "phases": {
                "salts_us_per_key": t["salts"] / wl.P * 1e6,
                "chains_tokens_per_s": tokens / t["chains"],
                "radix_insert_sequences_per_s": len(wl.modes) * A.n / t["insert"],
                "radix_match_per_s": len(wl.modes) * B.n / t["match"],
            },
            "host": host_cpu_info()}


def cpu_baseline_admission(wl: W.Workload, processes: int):
    """The oracle's chains of both batches (over worker processes), then its
    admission (one process) of the 2n requests in order."""
    import oracle as O
    X = concat(wl.insert, wl.lookup)
    clock = time.perf_counter
    t = {"salts": 0.0, "chains": 0.0, "admit": 0.0}
    t0 = clock()
    salts = O.salts(wl.K, wl.principal_ids)
    t["salts"] = clock() - t0
    bo = X.blk_offsets()
    tokens = admitted = 0
    for mode in wl.modes:
        t0 = clock()
        h = O.hash_chains_parallel(X.tokens, X.tok_offsets, X.principal, salts, mode,
                                   X.boundary_tok, processes=processes)
        t["chains"] += clock() - t0
        tokens += 16 * h.shape[0]
        t0 = clock()
        O.Table().admit(h, bo)
        t["admit"] += clock() - t0
        admitted += X.n
    dt = sum(t.values())
    return {"value": tokens / dt, "unit": "tokens/s", "cores": processes, "kind": "oracle",
            "sample": (f"one full step of the same workload ({tokens} block tokens hashed, "
                       f"{admitted} requests admitted, {len(wl.modes)} modes) in {dt:.1f} s; "
                       f"chains over {processes} worker processes, salts and admission in one "
                       "process"),
            "seconds": dt, "requests_admitted_per_s": admitted / dt,
            "phases": {
                "salts_us_per_key": t["salts"] / wl.P * 1e6,
                "chains_tokens_per_s": tokens / t["chains"],
                "admit_requests_per_s": admitted / t["admit"],
                "admit_rows_per_s": tokens / 16 / t["admit"],
            },
            "host": host_cpu_info()}


def cpu_baseline_session(wl: W.Workload, processes: int):
    """The oracle's resumed chains (chain_from, one process) of every turn-2
    prompt, then the insert and re-lookup of the new blocks; turn 1's chains,
    which give the parents, are hashed before timing."""
    import oracle as O
    A = wl.insert
    T1 = wl.notes["turn1"]
    start = wl.notes["start"]
    clock = time.perf_counter
    t = {"salts": 0.0, "chains": 0.0, "insert": 0.0, "lookup": 0.0}
    t0 = clock()
    salts = O.salts(wl.K, wl.principal_ids)
    t["salts"] = clock() - t0
    cnt = hashed_counts(wl, A)
    bo = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    last = np.maximum(T1.blk_offsets()[1:] - 1, 0)
    tokens = lookups = 0
    for mode in wl.modes:
        h1 = O.hash_chains_parallel(T1.tokens, T1.tok_offsets, T1.principal, salts, mode,
                                    T1.boundary_tok, processes=processes)
        parents = h1[last]
        t0 = clock()
        h = O.hash_chains_resume(A.tokens, A.tok_offsets, A.principal, salts, mode, start,
                                 parents, A.boundary_tok)
        t["chains"] += clock() - t0
        tokens += 16 * int(cnt.sum())
        T = O.Table()
        t0 = clock()
        T.insert(h, bo)
        t["insert"] += clock() - t0
        t0 = clock()
        T.lookup(h, bo)
        t["lookup"] += clock() - t0
        lookups += A.n
    dt = sum(t.values())
    return {"value": tokens / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": (f"one full step of the same workload ({tokens} block tokens hashed "
                       f"from the start blocks, {lookups} lookups, {len(wl.modes)} modes) in "
                       f"{dt:.1f} s, one process; turn 1's chains (the parents) not timed"),
            "seconds": dt, "lookups_per_s": lookups / dt,
            "phases": {
                "salts_us_per_key": t["salts"] / wl.P * 1e6,
                "chains_tokens_per_s": tokens / t["chains"],
                "insert_keys_per_s": tokens / 16 / t["insert"],
                "lookup_lookups_per_s": lookups / t["lookup"],
            },
            "host": host_cpu_info()}


def cpu_baseline_probe(wl: W.Workload, processes: int, resident: int = 20000):
    """Oracle lookups of the probes copied from the first ``resident`` resident
    requests, against those requests' keys (the lookup phase is timed)."""
    import oracle as O
    salts = O.salts(wl.K, wl.principal_ids)
    R = wl.insert.subset(np.arange(resident))
    hr = O.hash_chains_parallel(R.tokens, R.tok_offsets, R.principal, salts, W.ROOT,
                                processes=processes)
    idx = np.nonzero(wl.notes["source"] < resident)[0]
    Pb = wl.lookup.subset(idx)
    hp = O.hash_chains_parallel(Pb.tokens, Pb.tok_offsets, Pb.principal, salts, W.ROOT,
                                processes=processes)
    T = O.Table()
    T.insert(hr)
    t0 = time.perf_counter()
    T.lookup(hp, Pb.blk_offsets())
    dt = time.perf_counter() - t0
    return {"value": Pb.n / dt, "unit": "lookups/s", "cores": 1, "kind": "oracle",
            "sample": (f"lookup of the {Pb.n} probes copied from the first {resident} resident "
                       f"requests, against their {hr.shape[0]} keys, in {dt:.1f} s "
                       "(one process; hashing not timed)"),
            "seconds": dt, "host": host_cpu_info()}


def measured_peaks(dev, slots: int = 1 << 24) -> dict:
    """What the device reaches on the microbenchmarks of libkvgov_peaks (the
    best of five launches each) and on a 1 GiB device-to-device copy."""
    import torch
    from paper_2608_09225_amd import peaks as P
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    s = torch.cuda.Stream(device=dev)
    out = torch.empty(cus * 32 * P.THREADS, dtype=torch.int32, device=dev)
    table = torch.zeros((slots, 32), dtype=torch.uint8, device=dev)
    src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)

    def best(launch):
        rates = []
        for i in range(6):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(s)
            work = launch()
            e1.record(s)
            e1.synchronize()
            if i:
                rates.append(work / (e0.elapsed_time(e1) * 1e-3))
        return max(rates)

    torch.cuda.synchronize()
    valu = best(lambda: P.valu(out, cus * 8, 4096, stream=s))
    gather = best(lambda: P.gather(table, out, cus * 32, 16, stream=s))

    def copy():
        with torch.cuda.stream(s):
            dst.copy_(src)
        return 2 * src.numel()
    cp = best(copy)
    torch.cuda.synchronize()
    del table, src, dst
    return {"int_valu_tops": valu / 1e12, "gather32_gbs": gather / 1e9,
            "gather32_table_bytes": slots * 32, "copy_gbs": cp / 1e9,
            "note": "best of 5 launches: independent rotate/add3/xor3 chains, 8 waves per "
                    "SIMD; 32-byte reads at random slots of a table; a 1 GiB copy (read + "
                    "write bytes)"}


def summarize(r: dict) -> dict:
    """The per-config entry of the bench line: rates, the fractions of the
    integer-VALU roofline (chain kernel) and of the HBM roofline (lookup,
    insert), and the gates."""
    s = {"workload": r["config"]["workload"], "value": r["value"], "unit": r["unit"],
         "ms_per_step": r["ms_per_step"], "steps": r["steps"]}
    for k in ("block_hashes_per_s", "lookups_per_s", "block_probes_per_s",
              "retention_boundary_vs_none", "retention_root_vs_none", "keys_in_table"):
        if k in r:
            s[k] = r[k]
    if r["unit"] == "tokens/s":
        s["tokens_per_s"] = r["value"]
    ro = r["roofline"]
    lk = r.get("roofline_lookup")
    if ro["bound"] == "alu":
        s["chains"] = {k: ro[k] for k in (
            "kernel", "achieved", "frac", "frac_gfx950_ops", "launch_ms", "traffic",
            "longest_chain_blocks", "parallelism_ceiling", "critical_path_ceiling",
            "us_per_block_on_critical_path") if k in ro}
    else:
        lk = ro
    if lk:
        s["lookup"] = {k: lk[k] for k in ("kernel", "achieved", "frac", "traffic", "launch_ms",
                                          "frac_of_measured_gather32") if k in lk}
    ins = r.get("roofline_insert")
    if ins:
        s["insert"] = {k: ins[k] for k in ("kernel", "achieved", "frac", "traffic") if k in ins}
    if "probe_hashing" in r:
        s["probe_hashing"] = r["probe_hashing"]
    s["gates"] = r["gates"]
    return s


def run_workload(name: str, args, dev, K, torch):
    """One workload's bench: set-up, warm-up, the timed steps, the per-phase
    steps, the gates, the rooflines (and, unless switched off, the extras and
    the CPU oracle baseline).  Returns (result, gates_ok)."""
    log(f"generating the {name} workload")
    wl = W.make(name, seed=args.seed)

    def to(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    ids = to(wl.principal_ids)
    A = wl.insert
    probe_only = wl.name == "probe"
    session = wl.name == "session"  # chains resumed from turn 1's digests
    # the lookup re-probes the inserted batch
    relookup_same = wl.name in ("large", "session")
    B = A if relookup_same else wl.lookup
    X = A if relookup_same else concat(A, B)  # what one hashing call covers
    cntX, cntB = hashed_counts(wl, X), hashed_counts(wl, B)
    nA = int(hashed_counts(wl, A).sum())
    nX = int(cntX.sum())
    boX = np.concatenate([[0], np.cumsum(cntX)]).astype(np.int64)
    x = dict(tokens=to(X.tokens), tok_offsets=to(X.tok_offsets), principal=to(X.principal),
             boundary_tok=to(X.boundary_tok), blk_offsets=to(boX))
    boA = boB = x["blk_offsets"]
    if not relookup_same:
        boA, boB = to(A.blk_offsets()), to(B.blk_offsets())
    modes = wl.modes if args.mode == "all" else \
        [m for m in wl.modes if W.MODE_NAMES[m] == args.mode]
    if not modes:
        raise SystemExit(f"the {name} workload has no {args.mode} mode "
                         f"(it runs {[W.MODE_NAMES[m] for m in wl.modes]})")
    status = K.new_status(dev)
    radix_cfg = wl.name == "radix"
    maint_cfg = wl.name == "maintenance"
    admission = wl.name == "admission"
    main_s = torch.cuda.current_stream()

    def buffer_set():
        """Everything one batch in flight writes: chain outputs, results,
        salts, tables, and a stream per mode plus one for the salts (all at
        the default priority)."""
        return dict(
            out={m: torch.empty((nX, 32), dtype=torch.uint8, device=dev) for m in modes},
            hits={m: torch.empty(B.n, dtype=torch.int32, device=dev) for m in modes},
            salts=torch.empty((wl.P, 32), dtype=torch.uint8, device=dev),
            caches={m: K.Cache(wl.log2_slots) for m in modes} if not radix_cfg else {},
            radixes={m: K.Radix(wl.log2_slots, RADIX_EDGE_SLOTS_LOG2) for m in modes}
            if radix_cfg else {},
            matched={m: torch.empty(B.n, dtype=torch.int32, device=dev) for m in modes},
            adm_hits={m: torch.empty(X.n, dtype=torch.int32, device=dev) for m in modes},
            adm_new={m: torch.empty(X.n, dtype=torch.int32, device=dev) for m in modes},
            streams={m: torch.cuda.Stream(device=dev) for m in modes},
            sstream=torch.cuda.Stream(device=dev),
            chains_done=[], step_done=[])

    depth = 1 if probe_only else (args.pipeline or PIPELINE.get(name, 1))
    sets = [buffer_set() for _ in range(depth)]

    def use_set(k):
        """Points the step's names at buffer set k."""
        nonlocal out, hits, salts, caches, radixes, matched, adm_hits, adm_new, streams
        st = sets[k]
        out, hits, salts, caches = st["out"], st["hits"], st["salts"], st["caches"]
        radixes, matched, adm_hits, adm_new = (st["radixes"], st["matched"], st["adm_hits"],
                                               st["adm_new"])
        streams = st["streams"]
        return st

    out = hits = salts = caches = radixes = matched = adm_hits = adm_new = streams = None
    use_set(0)
    ev_rins, ev_rmatch = [], []
    ev_chain, ev_look, ev_salts, ev_clear, ev_ins = [], [], [], [], []
    ev_adm = []

    def bview(m):
        return out[m][0:nA], (out[m][0:nA] if relookup_same else out[m][nA:])

    parents = {}
    if session:
        # untimed set-up: turn 1 hashed whole; each session's parent is the
        # digest of turn 1's last full block (rows of empty turns are unused)
        T1 = wl.notes["turn1"]
        x["start"] = to(wl.notes["start"])
        K.salts(wl.K, ids, out=salts)
        last = to(np.maximum(T1.blk_offsets()[1:] - 1, 0))
        for m in modes:
            h1 = K.hash_chains(to(T1.tokens), to(T1.tok_offsets), to(T1.principal), salts, m,
                               to(T1.boundary_tok))
            parents[m] = h1[last].contiguous()
            del h1
        torch.cuda.synchronize()

    def hash_call(m, s, xx=None, out_=None, par=None):
        xx = x if xx is None else xx
        if session:
            K.hash_chains_resume(xx["tokens"], xx["tok_offsets"], xx["principal"], salts, m,
                                 xx["start"], parents[m] if par is None else par,
                                 xx["boundary_tok"], blk_offsets=xx["blk_offsets"],
                                 out=out[m] if out_ is None else out_, status=status,
                                 check=False, stream=s)
        else:
            K.hash_chains(xx["tokens"], xx["tok_offsets"], xx["principal"], salts, m,
                          xx["boundary_tok"], blk_offsets=xx["blk_offsets"],
                          out=out[m] if out_ is None else out_, status=status, check=False,
                          stream=s)

    ev_ins_b, ev_evict, ev_erase = [], [], []
    max_keys, n_erase, new_a = {}, 0, {}
    if maint_cfg:
        # untimed set-up: the keys both inserts leave in the table fix the
        # eviction target (half of them); the erase list is the first tenth
        # of the insert batch's rows
        K.salts(wl.K, ids, out=salts)
        n_erase = int(nA * wl.notes["erase_fraction"])
        for st in sets:
            for c in st["caches"].values():
                c.set_recency(True)
        for m in modes:
            hash_call(m, main_s)
            new_a[m] = caches[m].insert(out[m][0:nA], boA)
            caches[m].insert(out[m][nA:], boB)
            max_keys[m] = int(caches[m].count() * wl.notes["evict_fraction"])
            caches[m].clear()
        torch.cuda.synchronize()

    probe_hash_ms = None
    if probe_only:
        # untimed set-up: resident chains + insert, probe chains
        m = W.ROOT
        K.salts(wl.K, ids, out=salts)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        K.hash_chains(x["tokens"], x["tok_offsets"], x["principal"], salts, m,
                      x["boundary_tok"], blk_offsets=x["blk_offsets"], out=out[m],
                      status=status, check=False)
        e1.record()
        n_new = caches[m].insert(bview(m)[0], boA)
        torch.cuda.synchronize()
        probe_hash_ms = e0.elapsed_time(e1)
        log(f"set-up: {nX} blocks hashed in {probe_hash_ms:.2f} ms, {n_new} keys resident")

    def timed(evs, key, s):
        """Records a start event now on ``s``; returns a closure recording the end."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s)

        def end():
            e1.record(s)
            evs.append((key, e0, e1))
        return end

    # One batch in flight: the salts of step i + 1 are derived while step i
    # runs (two salt buffers), so that a step's chains start without waiting
    # for its salts kernel (a single wave, slow on an otherwise idle GPU);
    # each step still derives one set of salts.
    early = depth == 1 and not probe_only and not args.salts_in_step
    salt_bufs = [sets[0]["salts"], torch.empty_like(sets[0]["salts"])]
    salted_evs = [None, None]
    readers = [[], []]  # chains that read each salt buffer last

    def enqueue_salts(k: int, record: bool):
        sst = sets[0]["sstream"]
        for ev in readers[k % 2]:
            sst.wait_event(ev)
        end = timed(ev_salts, None, sst) if record else None
        K.salts(wl.K, ids, out=salt_bufs[k % 2], stream=sst)
        if end:
            end()
        ev = torch.cuda.Event()
        ev.record(sst)
        salted_evs[k % 2] = ev

    def step(i: int, chains_ev: bool, phase_ev: bool):
        """Step i.  chains_ev: timing events around the dominant launches
        (the chains; the probe workload's lookups); phase_ev: timing events
        around every other call.  Each timing event costs the stream a few
        microseconds, so the timed steps carry only the first kind."""
        nonlocal salts
        st = use_set(i % depth)
        sst = st["sstream"]
        if early:
            salts = salt_bufs[i % 2]
            if salted_evs[i % 2] is None:
                enqueue_salts(i, False)
            salted = salted_evs[i % 2]
        else:
            # the salts of this set are rewritten once the set's previous
            # chains have read them (one batch in flight: once its step is done)
            for ev in st["chains_done"] + (st["step_done"] if depth == 1 else []):
                sst.wait_event(ev)
            if not probe_only:
                end = timed(ev_salts, None, sst) if phase_ev else None
                K.salts(wl.K, ids, out=salts, stream=sst)
                if end:
                    end()
            salted = torch.cuda.Event()
            salted.record(sst)
        st["chains_done"] = []
        done = []
        for m in modes:
            s = streams[m]
            hA, hB = bview(m)
            if not probe_only:
                # the table clear needs no salts: it overlaps the salts kernel
                end = timed(ev_clear, m, s) if phase_ev else None
                (radixes if radix_cfg else caches)[m].clear(stream=s)
                if end:
                    end()
            s.wait_event(salted)
            if not probe_only:
                if chains_ev:
                    # the library records this pair around the chain kernel
                    # itself (not the ordering kernels before it)
                    e0, e1 = chain_events.pop()
                    K.time_next_chain_kernel(e0, e1)
                hash_call(m, s)
                # the chains' end (the salts buffer they read may be
                # rewritten after it); the timing event serves when there is one
                if chains_ev:
                    ev_chain.append((m, e0, e1))
                    cd = e1
                else:
                    cd = torch.cuda.Event()
                    cd.record(s)
                st["chains_done"].append(cd)
                if radix_cfg:
                    # insert batch A's sequences, match batch B's (views of
                    # the concatenated arrays: A's requests come first)
                    pr = x["principal"] if m != W.NONE else None
                    sd = salts if m != W.NONE else None
                    end = timed(ev_rins, m, s) if phase_ev else None
                    radixes[m].insert(x["tokens"], x["tok_offsets"][:A.n + 1],
                                      None if pr is None else pr[:A.n], sd, m, out[m],
                                      x["blk_offsets"][:A.n + 1], stream=s)
                    if end:
                        end()
                    end = timed(ev_rmatch, m, s) if phase_ev else None
                    radixes[m].match(x["tokens"], x["tok_offsets"][A.n:],
                                     None if pr is None else pr[A.n:], sd, m, out[m],
                                     x["blk_offsets"][A.n:], out=matched[m], stream=s)
                    if end:
                        end()
                elif admission:
                    end = timed(ev_adm, m, s) if phase_ev else None
                    caches[m].admit(out[m], x["blk_offsets"], sync=False, hits=adm_hits[m],
                                    new=adm_new[m], stream=s)
                    if end:
                        end()
                else:
                    end = timed(ev_ins, m, s) if phase_ev else None
                    caches[m].insert(hA, boA, sync=False, stream=s)
                    if end:
                        end()
                if maint_cfg:
                    # the second insert call, then the maintenance calls
                    end = timed(ev_ins_b, m, s) if phase_ev else None
                    caches[m].insert(hB, boB, sync=False, stream=s)
                    if end:
                        end()
                    end = timed(ev_evict, m, s) if phase_ev else None
                    caches[m].evict(max_keys[m], sync=False, stream=s)
                    if end:
                        end()
                    end = timed(ev_erase, m, s) if phase_ev else None
                    caches[m].erase(hA[:n_erase], sync=False, stream=s)
                    if end:
                        end()
            if not admission and not radix_cfg:
                rec_look = chains_ev if probe_only else phase_ev
                if rec_look:
                    l0 = torch.cuda.Event(enable_timing=True)
                    l1 = torch.cuda.Event(enable_timing=True)
                    l0.record(s)
                caches[m].lookup(hB, boB, out=hits[m], stream=s)
                if rec_look:
                    l1.record(s)
                    ev_look.append((m, l0, l1))
            if not early or depth > 1:
                # waited on by the next step's salts (derived in the step)
                ev = torch.cuda.Event()
                ev.record(s)
                done.append(ev)
        st["step_done"] = done
        if early:
            readers[i % 2] = list(st["chains_done"])
            salted_evs[i % 2] = None
            enqueue_salts(i + 1, phase_ev)

    log(f"warmup {args.warmup} steps ({depth} batch(es) in flight)")
    for i in range(args.warmup):
        step(i, False, False)
    torch.cuda.synchronize()
    # timing events of the chain kernels, created (by a first record) before
    # the timed region, which then holds only the library's records of them
    chain_events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for _ in range(args.steps * len(modes))]
    for e0, e1 in chain_events:
        e0.record()
        e1.record()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, True, False)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    t_step = elapsed / args.steps
    last = args.warmup + args.steps - 1
    if not probe_only:
        # the per-phase launch times: as many steps again, after the timed
        # ones, with events around every call
        log(f"{args.steps} more steps with per-phase events")
        for i in range(args.steps):
            step(args.warmup + args.steps + i, False, True)
        torch.cuda.synchronize()
        last += args.steps
    # the results below are those of the last step's buffer set
    use_set(last % depth)

    # ---- gates: latched errors, bit-exactness on a sample, by-construction hits
    K.check_status(status, "bench step")
    if radix_cfg:
        rstats = {W.MODE_NAMES[m]: radixes[m].stats() for m in modes}
        n_keys = {k: v[0] for k, v in rstats.items()}
    else:
        n_keys = {W.MODE_NAMES[m]: caches[m].count() for m in modes}
    gates = {}
    got_hits = {m: hits[m].cpu().numpy() for m in modes}
    # a re-lookup of the inserted batch takes its expected hits from the
    # lookup batch the workload built for it
    exp = (wl.lookup if relookup_same else B).expect_hits
    if admission:
        # hits fixed by construction; each request's new blocks are the rest
        # of its chain (chains share only a leading run of blocks)
        exp = wl.notes["admit_hits"]
        got_hits = {m: adm_hits[m].cpu().numpy() for m in modes}
        got_new = {m: adm_new[m].cpu().numpy() for m in modes}
        gates["G4_new_blocks_by_construction"] = all(
            bool(np.array_equal(got_new[m], X.block_counts() - exp[m])) for m in modes)
    # The oracle is touched only in the CPU-baseline leg (skipped with
    # --no-cpu-baseline): there it is timed, and it checks sampled outputs of
    # the step bit for bit (G1) and, for maintenance, the whole table (G4).
    oracle_leg = not args.no_cpu_baseline
    if maint_cfg:
        exp = None
    if maint_cfg and oracle_leg:
        # the table after the last step, replayed by the oracle: both inserts,
        # the eviction, the erase; then the re-lookup batch and the count
        import oracle as O
        osl = O.salts(wl.K, wl.principal_ids)
        okm = True
        for m in modes:
            ho = O.hash_chains_parallel(X.tokens, X.tok_offsets, X.principal, osl, m,
                                        X.boundary_tok,
                                        processes=min(16, len(os.sched_getaffinity(0))))
            T = O.Table()
            T.insert(ho[:nA], A.blk_offsets())
            T.insert(ho[nA:], B.blk_offsets())
            T.evict(max_keys[m])
            T.erase(ho[:n_erase])
            okm &= n_keys[W.MODE_NAMES[m]] == len(T.keys)
            okm &= bool(np.array_equal(got_hits[m], T.lookup(ho[nA:], B.blk_offsets())))
        gates["G4_maintained_state_matches_oracle"] = bool(okm)
    if radix_cfg:
        exp = None
        got_match = {m: matched[m].cpu().numpy() for m in modes}
        # every request of the matched batch shares the 2119-token prefix with
        # inserted requests of its principal (root) or of any principal
        gates["G4_match_covers_shared_prefix"] = all(
            bool((got_match[m] >= wl.notes["prefix_len"]).all()) for m in modes)
    if exp is not None:
        gates["G4_hits_by_construction"] = all(
            bool(np.array_equal(got_hits[m], exp[m])) for m in modes)
    bo = boX
    if oracle_leg:
        import oracle as O
        osalts = O.salts(wl.K, wl.principal_ids)
        gs = np.random.default_rng(7)
        ok = bytes(salts.cpu().numpy().tobytes()) == b"".join(osalts)
        j0X = start_blocks(wl, X)
        sample = np.sort(gs.choice(X.n, min(96, X.n), replace=False))
        for m in modes:
            got = out[m].cpu().numpy()
            for r in sample:
                # the whole chain by definition; a resumed request keeps its
                # rows from the start block on
                want = O.hash_chains(X.tokens, X.tok_offsets, X.principal, osalts, m,
                                     X.boundary_tok, requests=[int(r)])[j0X[r]:]
                ok &= bool(np.array_equal(got[bo[r]:bo[r + 1]], want))
        if radix_cfg:
            # sampled match lengths against the oracle's index of the insert batch
            qs = np.sort(gs.choice(B.n, min(96, B.n), replace=False))
            for m in modes:
                R = O.Radix()
                R.insert(A.tokens, A.tok_offsets, A.principal, osalts, m)
                want = R.match(B.tokens, B.tok_offsets, B.principal, osalts, m, requests=qs)
                ok &= bool(np.array_equal(got_match[m][qs], want))
        gates["G1_bitexact_sampled"] = bool(ok)

    def per(evs):
        d = {}
        for m, e0, e1 in evs:
            d.setdefault(m, []).append(e0.elapsed_time(e1) * 1e-3)
        return d

    result = {
        "metric": "salted block hashes/sec (tokens/sec) + prefix lookups/sec, 1 MI355X",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": DESCRIPTIONS[wl.name].format(gini=wl.notes.get("gini", 0.0)),
            "requests_per_batch": A.n,
            "principals": wl.P,
            "modes": [W.MODE_NAMES[m] for m in modes],
            "table_slots": 1 << wl.log2_slots,
            "batches_in_flight": depth,
        },
    }
    if admission:
        # the admission call stands where the lookup stands in the other
        # configs: its two kernels together, HBM-bound
        look_t = per(ev_adm)
        look_bytes = {m: admit_bytes(X.n, nX, n_keys[W.MODE_NAMES[m]]) for m in modes}
    elif radix_cfg:
        look_t = per(ev_rmatch)
        look_bytes = {m: radix_match_bytes(B.block_counts(), got_match[m]) for m in modes}
    else:
        look_t = per(ev_look)
        look_bytes = {m: lookup_bytes(cntB, got_hits[m]) for m in modes}
    look_mean = {m: float(np.mean(ts)) for m, ts in look_t.items()}
    look_gbs = float(np.mean([look_bytes[m] / look_mean[m] for m in modes])) / 1e9
    g_look = lookup_lanes(B.n, int(cntB.sum()))
    ltr = recorded_traffic(f"k_lookup<{g_look}>", wl.name, "cache")
    roof_lookup = {
        "bound": "hbm", "kernel": "k_lookup (first-miss prefix lookup)",
        "achieved": look_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": look_gbs / HBM_PEAK_GBS, "traffic": None if ltr is None else ltr["bytes"],
        "traffic_frac": None if ltr is None else
        ltr["bytes"] / float(np.mean(list(look_mean.values()))) / 1e9 / HBM_PEAK_GBS,
        "traffic_frac_note": TRAFFIC_FRAC_NOTE,
        "bytes_per_launch": {W.MODE_NAMES[m]: b for m, b in look_bytes.items()},
        "launch_ms": {W.MODE_NAMES[m]: t * 1e3 for m, t in look_mean.items()},
        "examined_blocks_per_launch": {
            W.MODE_NAMES[m]: (look_bytes[m] - B.n * LOOKUP_BYTES_PER_REQUEST) //
            LOOKUP_BYTES_PER_BLOCK for m in modes},
    }
    if admission:
        atr = [recorded_traffic(k, wl.name, "cache")
               for k in ("k_chunk_insert<true>", f"k_admit_scan<{admit_group(X.n, nX)}>")]
        roof_lookup = {
            "bound": "hbm", "kernel": "k_chunk_insert<true> + k_admit_scan (kvgov_cache_admit)",
            "achieved": look_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": look_gbs / HBM_PEAK_GBS,
            "traffic": None if None in atr else sum(t["bytes"] for t in atr),
            "bytes_per_launch": {W.MODE_NAMES[m]: b for m, b in look_bytes.items()},
            "launch_ms": {W.MODE_NAMES[m]: t * 1e3 for m, t in look_mean.items()},
            "bytes_note": f"{INSERT_BYTES_NEW} B per new key, {INSERT_BYTES_PRESENT} B per "
                          f"present key, {ADMIT_BYTES_PER_ROW} B per row (code write and "
                          f"read, tag read), {ADMIT_BYTES_PER_REQUEST} B per request "
                          "(offsets, two outputs); both kernels of the call",
            "requests": X.n, "rows": nX,
        }
    if radix_cfg:
        g_r = 64 if admit_group(B.n, int(B.block_counts().sum())) > 16 else 16
        rtr = recorded_traffic(f"k_radix_match<{g_r}>", wl.name, "radix")
        roof_lookup = {
            "bound": "hbm", "kernel": f"k_radix_match<{g_r}> (token-granular match)",
            "achieved": look_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": look_gbs / HBM_PEAK_GBS, "traffic": None if rtr is None else rtr["bytes"],
            "bytes_per_launch": {W.MODE_NAMES[m]: b for m, b in look_bytes.items()},
            "launch_ms": {W.MODE_NAMES[m]: t * 1e3 for m, t in look_mean.items()},
            "bytes_note": f"block lookup up to the first absent block "
                          f"({LOOKUP_BYTES_PER_BLOCK} B per examined block, "
                          f"{LOOKUP_BYTES_PER_REQUEST} B per request), "
                          f"{RADIX_MATCH_BYTES_NODE} B node key per request, "
                          f"{RADIX_MATCH_BYTES_STEP} B per edge step",
            "mean_match_tokens": {W.MODE_NAMES[m]: float(got_match[m].mean()) for m in modes},
        }
    if probe_only:
        result["value"] = len(modes) * B.n / t_step
        result["unit"] = "lookups/s"
        result["block_probes_per_s"] = \
            sum(roof_lookup["examined_blocks_per_launch"].values()) / t_step
        ph_ops = OPS_PER_COMPRESSION * compressions(wl, X, W.ROOT)
        ph_tops = ph_ops / (probe_hash_ms * 1e-3) / 1e12
        result["probe_hashing"] = {"blocks": nX, "requests": X.n, "ms": probe_hash_ms,
                                   "tokens_per_s": 16 * nX / (probe_hash_ms * 1e-3),
                                   "kernel": "k_chains_mixed<1> (one set-up launch)",
                                   "int_valu_achieved_tops": ph_tops,
                                   "int_valu_frac": ph_tops / INT_PEAK_TOPS}
        result["roofline"] = roof_lookup
        per_step = [sum(look_t[m][i] for m in modes) for i in range(args.steps)]
    else:
        blocks = len(modes) * nX
        result["value"] = 16 * blocks / t_step
        result["unit"] = "tokens/s"
        result["block_hashes_per_s"] = blocks / t_step
        if admission:
            result["requests_admitted_per_s"] = len(modes) * X.n / t_step
        elif radix_cfg:
            result["matches_per_s"] = len(modes) * B.n / t_step
        else:
            result["lookups_per_s"] = len(modes) * B.n / t_step
            result["step_lookups_per_s"] = result["lookups_per_s"]
        chain_t = per(ev_chain)
        ops = {m: OPS_PER_COMPRESSION * compressions(wl, X, m) for m in modes}
        mean_t = {m: float(np.mean(ts)) for m, ts in chain_t.items()}
        achieved = float(np.mean([ops[m] / mean_t[m] for m in modes])) / 1e12
        spans = []
        for i in range(0, len(ev_chain), len(modes)):
            grp = ev_chain[i:i + len(modes)]
            ref = grp[0][1]
            starts = [ref.elapsed_time(e0) for _, e0, _ in grp]
            ends = [ref.elapsed_time(e1) for _, _, e1 in grp]
            spans.append((max(ends) - min(starts)) * 1e-3)
        concurrent = sum(ops.values()) / float(np.mean(spans)) / 1e12
        waves = int(np.ceil(X.n / 64))  # one lane per request
        cus = torch.cuda.get_device_properties(dev).multi_processor_count
        # the library's launch policy: the lane-pair kernel while the batch
        # fits in two 64-request workgroups per CU, else the mixed kernel
        # (longest requests on lane-pair workgroups, the rest one lane each)
        kname = "k_chains_lp" if X.n <= 2 * 64 * cus else "k_chains_mixed"
        # the lane-pair kernel's second template argument: a fourth wave
        # sharing the schedule (one workgroup per CU) or not (two per CU)
        pair = "" if kname == "k_chains_mixed" else (",true" if X.n <= 64 * cus else ",false")
        tr = {m: recorded_traffic(f"{kname}<{m}{pair}>", wl.name, "chains") for m in modes}
        traffic = None
        if all(t is not None for t in tr.values()):
            traffic = float(np.mean([t["bytes"] for t in tr.values()]))
        result["roofline"] = {
            "bound": "alu", "kernel": f"{kname} (chained block hashing)",
            "achieved": achieved, "peak": INT_PEAK_TOPS,
            "unit": "Tops/s (32-bit integer vector ops)", "frac": achieved / INT_PEAK_TOPS,
            "traffic": traffic,
            "traffic_note": "HBM bytes per launch, FETCH_SIZE + WRITE_SIZE scaled by a 1 GiB "
                            "copy kernel (profiles/hbm_traffic.md); null if the kernel "
                            "sources changed since",
            "algorithmic_bytes_per_launch": 64 * nX + 32 * nX,
            "ops_per_compression": OPS_PER_COMPRESSION,
            "ops_per_compression_gfx950": OPS_PER_COMPRESSION_GFX950,
            "frac_gfx950_ops": achieved * OPS_PER_COMPRESSION_GFX950 / OPS_PER_COMPRESSION /
            INT_PEAK_TOPS,
            "ops_per_launch": {W.MODE_NAMES[m]: o for m, o in ops.items()},
            "mean_launch_ms": float(np.mean(list(mean_t.values()))) * 1e3,
            "launch_ms": {W.MODE_NAMES[m]: t * 1e3 for m, t in mean_t.items()},
            "launch_requests": X.n,
            "longest_chain_blocks": int(cntX.max()),
            "parallelism_ceiling": min(1.0, waves / (CUS * SIMDS_PER_CU)),
            "parallelism_ceiling_note": "ceil(requests / 64) / 1024 SIMDs: waves at one lane "
                                        "per request (the lane-pair kernel runs three waves "
                                        "per 64 requests)",
            "concurrent_modes_achieved": concurrent,
            "concurrent_modes_frac": concurrent / INT_PEAK_TOPS,
        }
        result["roofline_admit" if admission else
               "roofline_radix_match" if radix_cfg else "roofline_lookup"] = roof_lookup
        # per step: the interval between consecutive steps' last chain ends
        # (the steady-state step time; the modes' launches overlap and how
        # they share the chip shifts between steps, so their durations are
        # the noisier figure)
        # (with several batches in flight the steps' chains may end out of
        # order, so the interval is taken between steps `depth` apart)
        nm = len(modes)
        ref = ev_chain[0][1]
        ends = [max(ref.elapsed_time(e1) for _, _, e1 in ev_chain[i * nm:(i + 1) * nm]) * 1e-3
                for i in range(args.steps)]
        per_step = [(ends[i + depth] - ends[i]) / depth for i in range(len(ends) - depth)]
        if wl.name == "template":
            s = {W.MODE_NAMES[m]: int(got_hits[m].sum()) for m in modes}
            result["hit_blocks"] = s
            result["retention_boundary_vs_none"] = s["boundary"] / max(1, s["none"])
            result["retention_root_vs_none"] = s["root"] / max(1, s["none"])
    result["keys_in_table"] = n_keys

    # ---- per-phase rates (HIP events on each call's own stream) ----------
    def stats(ts):
        a = np.asarray(ts) * 1e3
        return {"ms_mean": float(a.mean()), "ms_median": float(np.median(a)),
                "ms_min": float(a.min())}

    phases = {}
    if ev_salts:
        st = stats(per(ev_salts)[None])
        phases["salts"] = {**st, "salts_per_s": wl.P / (st["ms_median"] * 1e-3)}
    clear_t, ins_t = per(ev_clear), per(ev_ins)
    for m in modes:
        ph = {}
        if not probe_only:
            st = stats(chain_t[m])
            sec = st["ms_median"] * 1e-3
            ph["chains"] = {**st, "blocks": nX, "tokens_per_s": 16 * nX / sec,
                            "block_hashes_per_s": nX / sec,
                            "compressions_per_s": compressions(wl, X, m) / sec}
            ph["clear"] = stats(clear_t[m])
        if admission:
            st = stats(look_t[m])
            sec = st["ms_median"] * 1e-3
            b = look_bytes[m]
            ph["admit"] = {**st, "requests": X.n, "rows": nX,
                           "new_keys": n_keys[W.MODE_NAMES[m]],
                           "requests_per_s": X.n / sec, "rows_per_s": nX / sec,
                           "algorithmic_bytes": b, "gbs": b / sec / 1e9}
            phases[W.MODE_NAMES[m]] = ph
            continue
        if radix_cfg:
            nb, ne = rstats[W.MODE_NAMES[m]]
            st = stats(per(ev_rins)[m])
            sec = st["ms_median"] * 1e-3
            edges = radix_insert_edges(A)
            recs = int(((A.lengths + 15) // 16).sum())
            b = (INSERT_BYTES_NEW * nb + INSERT_BYTES_PRESENT * max(nA - nb, 0) +
                 RADIX_INSERT_BYTES_RECORD * recs + RADIX_INSERT_BYTES_EDGE * edges)
            ph["radix_insert"] = {**st, "sequences": A.n, "tokens": int(A.lengths.sum()),
                                  "block_nodes": nb, "edges_walked": edges,
                                  "edges_in_index": ne, "sequences_per_s": A.n / sec,
                                  "algorithmic_bytes": b, "gbs": b / sec / 1e9}
            st = stats(look_t[m])
            sec = st["ms_median"] * 1e-3
            ph["radix_match"] = {**st, "matches_per_s": B.n / sec,
                                 "algorithmic_bytes": look_bytes[m],
                                 "gbs": look_bytes[m] / sec / 1e9}
            phases[W.MODE_NAMES[m]] = ph
            continue
        if maint_cfg:
            slots = 1 << wl.log2_slots
            kept = max_keys[m]  # an upper bound of the keys the eviction keeps
            st = stats(per(ev_ins_b)[m])
            ph["insert_b"] = {**st, "keys": nX - nA,
                              "keys_per_s": (nX - nA) / (st["ms_median"] * 1e-3)}
            st = stats(per(ev_evict)[m])
            b = EVICT_BYTES_PER_SLOT * slots + MAINT_BYTES_PER_KEPT * kept
            ph["evict"] = {**st, "slots": slots, "max_keys": kept, "algorithmic_bytes": b,
                           "gbs": b / (st["ms_median"] * 1e-3) / 1e9}
            st = stats(per(ev_erase)[m])
            b = (ERASE_BYTES_PER_SLOT * slots + MAINT_BYTES_PER_KEPT * n_keys[W.MODE_NAMES[m]] +
                 ERASE_BYTES_PER_LISTED * n_erase)
            ph["erase"] = {**st, "listed_keys": n_erase, "algorithmic_bytes": b,
                           "gbs": b / (st["ms_median"] * 1e-3) / 1e9}
        if not probe_only:
            st = stats(ins_t[m])
            sec = st["ms_median"] * 1e-3
            n_new = n_keys[W.MODE_NAMES[m]]
            if maint_cfg:
                n_new = new_a[m]  # the insert batch's new keys, from the set-up run
            ibytes = INSERT_BYTES_NEW * n_new + INSERT_BYTES_PRESENT * (nA - n_new)
            ph["insert"] = {**st, "keys": nA, "new_keys": n_new, "keys_per_s": nA / sec,
                            "algorithmic_bytes": ibytes, "gbs": ibytes / sec / 1e9}
        st = stats(look_t[m])
        sec = st["ms_median"] * 1e-3
        ex = roof_lookup["examined_blocks_per_launch"][W.MODE_NAMES[m]]
        ph["lookup"] = {**st, "lookups_per_s": B.n / sec, "block_probes_per_s": ex / sec}
        phases[W.MODE_NAMES[m]] = ph
    result["phases"] = phases

    if radix_cfg:
        ins_gbs = float(np.mean([phases[W.MODE_NAMES[m]]["radix_insert"]["gbs"]
                                 for m in modes]))
        g_i = admit_group(A.n, nA)
        itr = [recorded_traffic(k, wl.name, t) for k, t in
               (("k_radix_roots", "radix"), (f"k_insert_req<{g_i}>", "cache"),
                (f"k_radix_edges<{g_i}>", "radix"))]
        result["roofline_radix_insert"] = {
            "bound": "hbm", "kernel": f"k_radix_roots + k_insert_req<{g_i}> + k_radix_edges<{g_i}> "
                                      "(kvgov_radix_insert)",
            "achieved": ins_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": ins_gbs / HBM_PEAK_GBS,
            "traffic": None if None in itr else sum(t["bytes"] for t in itr),
            "bytes_note": f"the block insert's {INSERT_BYTES_NEW}/{INSERT_BYTES_PRESENT} B per "
                          f"new/present key, {RADIX_INSERT_BYTES_RECORD} B per record (parent "
                          f"key), {RADIX_INSERT_BYTES_EDGE} B per edge walked",
        }
    if maint_cfg:
        eg = float(np.mean([phases[W.MODE_NAMES[m]]["evict"]["gbs"] for m in modes]))
        result["roofline_evict"] = {
            "bound": "hbm", "kernel": "k_rank_hist/k_rank_select x 8 + k_compact + "
                                      "k_rebuild_fill + k_reinsert (kvgov_cache_evict)",
            "achieved": eg, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": eg / HBM_PEAK_GBS,
            "traffic": None,
            "bytes_note": f"{EVICT_BYTES_PER_SLOT} B per slot, {MAINT_BYTES_PER_KEPT} B per kept "
                          "key (max_keys used as the kept count)",
            "launch_ms": {W.MODE_NAMES[m]: phases[W.MODE_NAMES[m]]["evict"]["ms_median"]
                          for m in modes},
        }
    if not probe_only and not admission and not radix_cfg:
        ins_gbs = float(np.mean([phases[W.MODE_NAMES[m]]["insert"]["gbs"] for m in modes]))
        g_ins = admit_group(A.n, nA)
        itr = recorded_traffic(f"k_insert_req<{g_ins}>", wl.name, "cache")
        ins_s = float(np.mean([phases[W.MODE_NAMES[m]]["insert"]["ms_median"]
                               for m in modes])) / 1e3
        result["roofline_insert"] = {
            "bound": "hbm", "kernel": f"k_insert_req<{g_ins}> (set-union insert)",
            "achieved": ins_gbs,
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ins_gbs / HBM_PEAK_GBS,
            "traffic": None if itr is None else itr["bytes"],
            "traffic_frac": None if itr is None else itr["bytes"] / ins_s / 1e9 / HBM_PEAK_GBS,
            "traffic_frac_note": TRAFFIC_FRAC_NOTE,
            "bytes_note": f"{INSERT_BYTES_NEW} B per new key (query read, slot read, slot "
                          f"write), {INSERT_BYTES_PRESENT} B per present key",
        }
    if not probe_only and not args.no_extras:
        # Critical path: the per-block latency of the lane-pair kernel under a
        # realistic load (the longest request replicated into one 64-request
        # workgroup per CU; a single workgroup on an otherwise idle GPU runs
        # at a lower clock), times the longest chain.
        r = int(np.argmax(cntX))
        nb = int(cntX[r])
        one = X.subset(np.array([r]))
        nrep = 64 * cus
        L1 = int(one.tok_offsets[-1])
        rep = W.Batch(np.tile(one.tokens, nrep), np.arange(nrep + 1, dtype=np.int64) * L1,
                      np.repeat(one.principal, nrep), np.repeat(one.boundary_tok, nrep))
        o = dict(tokens=to(rep.tokens), tok_offsets=to(rep.tok_offsets),
                 principal=to(rep.principal), boundary_tok=to(rep.boundary_tok),
                 blk_offsets=to(np.arange(nrep + 1, dtype=np.int64) * nb))
        m0 = modes[0]
        par = None
        if session:
            o["start"] = to(np.full(nrep, start_blocks(wl, X)[r], np.int32))
            par = parents[m0][r:r + 1].repeat(nrep, 1).contiguous()
        oh = torch.empty((nrep * nb, 32), dtype=torch.uint8, device=dev)
        ts = []
        for i in range(4):
            end = timed(ts, None, main_s)
            hash_call(m0, main_s, xx=o, out_=oh, par=par)
            end()
        torch.cuda.synchronize()
        K.check_status(status, "critical-path launch")
        ok_rep = bool(np.array_equal(oh[:nb].cpu().numpy(),
                                     out[m0][int(bo[r]):int(bo[r + 1])].cpu().numpy()))
        gates["G1b_replicas_agree"] = ok_rep
        t_crit = min(e0.elapsed_time(e1) for _, e0, e1 in ts[1:]) * 1e-3
        ideal = ops[m0] / (INT_PEAK_TOPS * 1e12)
        roof = result["roofline"]
        roof["critical_path_ms"] = t_crit * 1e3
        roof["us_per_block_on_critical_path"] = t_crit / nb * 1e6
        roof["critical_path_ceiling"] = min(1.0, ideal / t_crit)
        roof["critical_path_note"] = (f"the longest request ({nb} blocks hashed) "
                                      f"replicated {nrep} times, one launch; ceiling = "
                                      "(launch ops at peak) / its duration")
        del o, oh, par
        if session:
            # the same turn-2 chains rehashed from block 0 (what a stack without
            # chain extension hashes each turn), for comparison
            xf = dict(x, blk_offsets=to(X.blk_offsets()))
            of = torch.empty((int(X.block_counts().sum()), 32), dtype=torch.uint8, device=dev)
            full = {}
            for m in modes:
                ts = []
                for i in range(4):
                    end = timed(ts, None, main_s)
                    K.hash_chains(xf["tokens"], xf["tok_offsets"], xf["principal"], salts, m,
                                  xf["boundary_tok"], blk_offsets=xf["blk_offsets"], out=of,
                                  status=status, check=False, stream=main_s)
                    end()
                torch.cuda.synchronize()
                full[W.MODE_NAMES[m]] = min(e0.elapsed_time(e1) for _, e0, e1 in ts[1:])
                rows = of.cpu().numpy()[np.concatenate(
                    [np.arange(X.blk_offsets()[q] + start_blocks(wl, X)[q],
                               X.blk_offsets()[q + 1]) for q in range(X.n)])]
                gates["G1b_replicas_agree"] = bool(
                    gates.get("G1b_replicas_agree", True) and
                    np.array_equal(rows, out[m].cpu().numpy()))
            K.check_status(status, "full rehash")
            res_ms = {W.MODE_NAMES[m]: float(np.min(chain_t[m])) * 1e3 for m in modes}
            result["session"] = {
                "blocks_hashed": nX, "blocks_in_prompts": int(X.block_counts().sum()),
                "resume_chain_ms_min": res_ms, "full_rehash_chain_ms_min": full,
                "speedup": {k: full[k] / res_ms[k] for k in full},
                "prompt_tokens_per_s": 16 * len(modes) * int(X.block_counts().sum()) / t_step,
                "note": "min launch times; full rehash = kvgov_hash_chains over the whole "
                        "turn-2 prompts (its rows from the start block equal the resumed ones)",
            }
            del of

    if not args.no_extras:
        log("measuring device peaks (microbenchmarks)")
        mp = measured_peaks(dev)
        result["measured_peaks"] = mp
        roof = result["roofline"]
        if roof["bound"] == "alu":
            roof["frac_of_measured_peak"] = roof["achieved"] / mp["int_valu_tops"]
        for key in ("roofline_lookup", "roofline_insert", "roofline_admit",
                    "roofline_radix_match", "roofline_radix_insert", "roofline_evict",
                    "roofline"):
            rr = result.get(key)
            if rr and rr["bound"] == "hbm":
                rr["frac_of_measured_gather32"] = rr["achieved"] / mp["gather32_gbs"]

    # medians, so that one disturbed step does not decide the gate
    h = len(per_step) // 2
    if h:
        a1, a2 = np.median(per_step[:h]), np.median(per_step[h:])
        gates["G3_two_halves_within_5pct"] = bool(abs(a1 - a2) / max(a1, a2) < 0.05)
    result["gate_steps_ms"] = [round(float(v) * 1e3, 4) for v in per_step]
    gates["G2_below_peak"] = bool(result["roofline"]["frac"] <= 1.0 and roof_lookup["frac"] <= 1.0)
    result["gates"] = gates
    if not args.no_cpu_baseline and getattr(args, "cpu_timing", True):
        procs = min(16, len(os.sched_getaffinity(0)))
        log(f"timing the CPU oracle on {procs} processes")
        result["cpu_baseline"] = cpu_baseline(wl, procs, max_blocks=3_000_000)
    for st in sets:
        for c in list(st["caches"].values()) + list(st["radixes"].values()):
            c.close()
    ok = all(gates.get(g, True) for g in ("G1_bitexact_sampled", "G1b_replicas_agree",
                                          "G4_hits_by_construction",
                                          "G4_new_blocks_by_construction",
                                          "G4_maintained_state_matches_oracle",
                                          "G4_match_covers_shared_prefix"))
    if not ok:
        log(f"{name}: correctness gate failure: {gates}")
    return result, ok


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default=HEADLINE, choices=sorted(DESCRIPTIONS),
                    help=f"workload of the bench line (default {HEADLINE}; with the default, "
                         f"the other configs {', '.join(SECONDARY)} are timed after it and "
                         "summarised under \"configs\")")
    ap.add_argument("--mode", default="all", choices=["all", "none", "root", "boundary"],
                    help="run only this salt mode of the workload (default: all of its modes)")
    ap.add_argument("--seed", type=int, default=W.SEED,
                    help=f"master seed of the synthetic inputs (default {W.SEED})")
    ap.add_argument("--no-configs", action="store_true",
                    help="time the bench line's workload only, not the other configs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the critical-path launch and the measured-peak "
                         "microbenchmarks (counter runs: only the step's own launches)")
    ap.add_argument("--pipeline", type=int, default=0, choices=(0, 1, 2, 3),
                    help="batches in flight: 1 runs the steps one after another; 2 runs "
                         "batch i+1's salts and chains while batch i's insert and lookup "
                         "finish (a set of tables, buffers and streams per batch); 0 (the "
                         "default) takes each workload's own setting: 2 for the large batch, "
                         "whose longest chains leave most CUs idle for most of the chain "
                         "launch, 1 for the others")
    ap.add_argument("--salts-in-step", action="store_true",
                    help="derive each step's salts at its start, before its chains (default: "
                         "during the previous step)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before the bench, run one device-to-device copy of this many MiB "
                         "(a kernel of known traffic, to scale HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the bench runs on one GPU only; --gpus must be 1 "
                                   "(sharding over several GPUs is not implemented)"}))
        sys.exit(2)

    # before the HIP runtime starts (it reads the setting once)
    if int(os.environ.get("GPU_MAX_HW_QUEUES", "0") or 0) < HW_QUEUES:
        os.environ["GPU_MAX_HW_QUEUES"] = str(HW_QUEUES)
    import torch
    from paper_2608_09225_amd import kvgov as K

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    K.lib()  # fails loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"copy probe: {n} bytes read and written by one copy kernel")

    result, ok = run_workload(args.config, args, dev, K, torch)
    if args.config == HEADLINE and not args.no_configs:
        # the other configs, each a bench of its own kind after the headline
        # (at most 30 timed steps, no extras, no CPU timing; the oracle's
        # sampled bit-exact gate still runs unless --no-cpu-baseline)
        configs = {args.config: summarize(result)}
        for name in SECONDARY:
            sub = argparse.Namespace(**vars(args))
            sub.steps, sub.warmup = min(args.steps, 30), min(args.warmup, 5)
            sub.no_extras, sub.cpu_timing, sub.mode = True, False, "all"
            r, ok_r = run_workload(name, sub, dev, K, torch)
            ok &= ok_r
            configs[name] = summarize(r)
            if name == "probe":
                # the lookup roofline of the line: the lookup-only workload
                result["lookups_per_s"] = r["value"]
                result["lookups_note"] = ("probe-heavy workload: 1M probe requests of 8..64 "
                                          "blocks against 8M resident keys, lookup only")
                result["roofline_relookup"] = result.get("roofline_lookup")
                result["roofline_lookup"] = r["roofline"]
            torch.cuda.empty_cache()
        result["configs"] = configs
    print(json.dumps(result), flush=True)
    if not ok:
        sys.exit(1)




if __name__ == "__main__":
    main()
