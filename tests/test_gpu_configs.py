"""GPU parity on the six workloads at full size, in the launch shapes bench.py
uses (one hashing call per batch and mode, the table sizes of the configs).

* tiny, paper, template: every digest, every hit count and n_new against the
  oracle.
* probe (8M resident keys, 1M probes): every digest of both batches against
  the oracle, every hit count against the oracle's lookup of its own probe
  digests in its own resident set, and against the value fixed by
  construction (d for a probe copying d blocks under its own principal, 0
  under another principal).
* large (65,536 requests, 13.7M blocks per mode): every digest of both modes
  against the oracle; n_new and every hit count of the re-lookup against the
  oracle's (all keys distinct, so a lookup of the inserted batch hits every
  block).
* session (4096 two-turn sessions): turn 2's chains resumed from turn 1's
  last digests, every digest, n_new and hit count against the oracle's own
  resumed chains.
* admission, radix, maintenance (the paper-shaped batches on the three
  later stages, one call shape each as bench.py times them): every admitted
  request's hits and new blocks against the oracle's sequential admission;
  every token-granular match against the oracle's index (root: per-principal
  trees; unsalted: 256 sampled requests, since each is compared with all 4096
  sequences) and every match against the shared prefix; the maintained table
  (two tracked inserts, an eviction to half, an erase, a re-lookup) replayed
  by the oracle.

The probe and large workloads are compared in request ranges on forked worker
processes: each worker hashes its range with the oracle and compares it with
the same rows of the GPU output (copied to host memory before the fork), so
no process holds a whole batch's oracle digests at once.
"""
import hashlib
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

K = pytest.importorskip("paper_2608_09225_amd.kvgov")
PROCS = min(16, len(os.sched_getaffinity(0)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def gpu_chains(b, salts_dev, mode):
    return K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), salts_dev, mode,
                         dev(b.boundary_tok))


def oracle_chains(b, salts, mode, requests=None):
    if requests is None:
        return O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, salts, mode,
                                      b.boundary_tok, processes=PROCS)
    return O.hash_chains(b.tokens, b.tok_offsets, b.principal, salts, mode, b.boundary_tok,
                         requests=requests)


_BO = {}


def rows_of(b, hashes_np, r):
    if id(b) not in _BO:
        _BO[id(b)] = (b, b.blk_offsets())
    bo = _BO[id(b)][1]
    return hashes_np[bo[r]:bo[r + 1]]


# ---------------------------------------------------------------------------
# whole-batch comparisons on worker processes
# ---------------------------------------------------------------------------

_SHARED = {}


def _ranges(n, procs, per_proc=8):
    step = max(1, -(-n // (procs * per_proc)))
    return [(a, min(a + step, n)) for a in range(0, n, step)]


def _cmp_range(rng_):
    """Oracle digests of requests [a, b) against the GPU rows of the same
    requests; with a resident key set, also the oracle's lookup of those
    digests against the GPU hit counts.  Returns (a, b, bad request or -1,
    bad hit request or -1)."""
    a, b = rng_
    sh = _SHARED
    bt, bo = sh["batch"], sh["bo"]
    want = O.hash_chains(bt.tokens, bt.tok_offsets, bt.principal, sh["salts"], sh["mode"],
                         bt.boundary_tok, requests=range(a, b))
    got = sh["gpu"][bo[a]:bo[b]]
    bad = -1
    if not np.array_equal(got, want):
        for r in range(a, b):
            if not np.array_equal(got[bo[r]:bo[r + 1]], want[bo[r] - bo[a]:bo[r + 1] - bo[a]]):
                bad = r
                break
    bad_hit = -1
    if sh.get("keys") is not None:
        local = bo[a:b + 1] - bo[a]
        hits = O.lookup_hits(sh["keys"], want, local)
        diff = np.nonzero(hits != sh["hits"][a:b])[0]
        bad_hit = int(a + diff[0]) if diff.size else -1
    return a, b, bad, bad_hit


def key_set(rows):
    """The rows of a uint8 [n, 32] array as a set of 32-byte keys."""
    raw = np.ascontiguousarray(rows).tobytes()
    return {raw[i:i + 32] for i in range(0, len(raw), 32)}


def compare_all(b, osalts, mode, gpu_rows, keys=None, gpu_hits=None):
    """Every request of ``b``: the oracle's chains against ``gpu_rows`` (host
    uint8 [rows, 32]) and, given a key set, the oracle's lookup hits against
    ``gpu_hits``."""
    import multiprocessing as mp
    bo = b.blk_offsets()
    assert gpu_rows.shape == (int(bo[-1]), 32)
    _SHARED.update(batch=b, bo=bo, salts=osalts, mode=mode, gpu=gpu_rows, keys=keys,
                   hits=gpu_hits)
    try:
        with mp.get_context("fork").Pool(PROCS) as pool:
            res = pool.map(_cmp_range, _ranges(b.n, PROCS))
    finally:
        _SHARED.clear()
    bad = [r for _, _, r, _ in res if r >= 0]
    assert not bad, f"digests of request {bad[0]} differ from the oracle"
    bad_hit = [r for _, _, _, r in res if r >= 0]
    assert not bad_hit, f"hit count of request {bad_hit[0]} differs from the oracle"
    assert sum(y - x for x, y, _, _ in res) == b.n


def full_pipeline(wl, mode):
    """GPU: chains of both batches, insert, lookup.  Oracle: the same."""
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    assert sd.cpu().numpy().tobytes() == b"".join(osalts)
    hi = gpu_chains(wl.insert, sd, mode)
    hl = gpu_chains(wl.lookup, sd, mode)
    with K.Cache(wl.log2_slots) as c:
        n_new = c.insert(hi, dev(wl.insert.blk_offsets()))
        hits = c.lookup(hl, dev(wl.lookup.blk_offsets())).cpu().numpy()
        count = c.count()
    wi = oracle_chains(wl.insert, osalts, mode)
    wlk = oracle_chains(wl.lookup, osalts, mode)
    assert np.array_equal(hi.cpu().numpy(), wi)
    assert np.array_equal(hl.cpu().numpy(), wlk)
    T = O.Table()
    assert n_new == T.insert(wi) == count
    want_hits = T.lookup(wlk, wl.lookup.blk_offsets())
    assert np.array_equal(hits, want_hits)
    return hits


def test_tiny_config():
    wl = W.make("tiny")
    hits = full_pipeline(wl, W.ROOT)
    assert np.array_equal(hits, wl.lookup.expect_hits[W.ROOT])


@pytest.fixture(scope="module")
def paper_wl():
    return W.make("paper")


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY, W.NONE])
def test_paper_config(paper_wl, mode):
    wl = paper_wl
    hits = full_pipeline(wl, mode)
    assert np.array_equal(hits, wl.lookup.expect_hits[mode])  # 132 for every request


def test_template_config():
    """All three modes; the hit-block retention of boundary salting relative to
    no salting is the same number on both sides (it is computed from hits that
    are compared exactly)."""
    wl = W.make("template")
    hits = {m: full_pipeline(wl, m) for m in (W.NONE, W.ROOT, W.BOUNDARY)}
    k = wl.notes["boundary_tok"] // 16
    # by construction: every request shares the first k template blocks
    assert np.all(hits[W.BOUNDARY] >= k) and np.all(hits[W.NONE] >= hits[W.BOUNDARY])
    assert np.all(hits[W.ROOT] <= hits[W.NONE])
    retention = hits[W.BOUNDARY].sum() / hits[W.NONE].sum()
    assert 0 < retention <= 1


@pytest.fixture(scope="module")
def probe_wl():
    return W.make("probe")


def test_probe_config(probe_wl):
    """Every resident and probe digest against the oracle, n_new, and every
    probe's hit count against the oracle's first-miss lookup in the oracle's
    resident key set (and the value fixed by construction)."""
    wl = probe_wl
    res, pr = wl.insert, wl.lookup
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    h_res = gpu_chains(res, sd, W.ROOT)
    h_pr = gpu_chains(pr, sd, W.ROOT)
    with K.Cache(wl.log2_slots) as c:
        assert c.slots() == 1 << 24
        n_new = c.insert(h_res, dev(res.blk_offsets()))
        hits = c.lookup(h_pr, dev(pr.blk_offsets())).cpu().numpy()
    assert np.array_equal(hits, pr.expect_hits[W.ROOT])
    hr = h_res.cpu().numpy()
    del h_res
    # resident chains: every digest; the oracle's key set is built from its
    # own digests, which equal the GPU's once the comparison has passed
    compare_all(res, osalts, W.ROOT, hr)
    keys = key_set(hr)
    assert n_new == len(keys) == res.n * 32  # random 512-token prompts: all distinct
    del hr
    hp = h_pr.cpu().numpy()
    del h_pr
    compare_all(pr, osalts, W.ROOT, hp, keys=keys, gpu_hits=hits)


def test_probe_sources_checked_by_oracle(probe_wl):
    """For sampled own-principal probes, the oracle hashes the probe and the
    resident request it was copied from and counts leading common keys."""
    wl = probe_wl
    res, pr = wl.insert, wl.lookup
    osalts = O.salts(wl.K, wl.principal_ids)
    L = 512
    first_block = {res.tokens[L * r:L * r + 16].tobytes(): r for r in range(res.n)}
    g = np.random.default_rng(6)
    checked = 0
    for p in g.choice(pr.n, 400, replace=False):
        d = int(pr.expect_hits[W.ROOT][p])
        if d == 0:
            continue
        # the source is the resident request whose first block equals the probe's
        r = first_block[pr.row(int(p))[:16].tobytes()]
        keys = set(bytes(x) for x in oracle_chains(res, osalts, W.ROOT, [r]))
        ph = oracle_chains(pr, osalts, W.ROOT, [int(p)])
        j = 0
        while j < len(ph) and bytes(ph[j]) in keys:
            j += 1
        assert j == d
        checked += 1
    assert checked > 200


@pytest.fixture(scope="module")
def large_wl():
    return W.make("large")


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY])
def test_large_config(large_wl, mode):
    """Every digest of the 65,536-request batch against the oracle; the
    insert's n_new and every hit of the re-lookup against the oracle's."""
    wl = large_wl
    b = wl.insert
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    h = gpu_chains(b, sd, mode)
    nb = int(b.block_counts().sum())
    with K.Cache(wl.log2_slots) as c:
        n_new = c.insert(h, dev(b.blk_offsets()))
        hits = c.lookup(h, dev(b.blk_offsets())).cpu().numpy()
    hn = h.cpu().numpy()
    del h
    # the key set is built from the GPU rows before the workers fork; the
    # workers first compare those rows with the oracle's, so once the call
    # returns it is the oracle's set
    keys = key_set(hn)
    compare_all(b, osalts, mode, hn, keys=keys, gpu_hits=hits)
    assert n_new == len(keys) == nb  # all keys distinct
    assert np.array_equal(hits, b.block_counts())


def test_many_requests_longest_first_ordering():
    """A batch above the longest-first threshold (40,000 short requests)."""
    g = np.random.default_rng(8)
    lens = g.integers(0, 200, 40000).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)])
    toks = g.integers(0, W.VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 50, lens.size).astype(np.int32)
    bt = np.floor(g.random(lens.size) * (lens + 1)).astype(np.int32)
    b = W.Batch(toks, offs, prin, bt)
    Kb = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, (50, 32), dtype=np.uint8)
    sd = K.salts(Kb, dev(ids))
    osalts = O.salts(Kb, ids)
    for mode in (W.NONE, W.ROOT, W.BOUNDARY):
        got = gpu_chains(b, sd, mode).cpu().numpy()
        assert np.array_equal(got, oracle_chains(b, osalts, mode))


@pytest.fixture(scope="module")
def session_wl():
    return W.make("session")


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY])
def test_session_config(session_wl, mode):
    """Multi-turn sessions at full size: turn 1 hashed whole on the GPU, turn 2
    resumed from its last full-block digests, then insert and re-lookup of
    the new blocks.  The oracle hashes turn 1 and resumes turn 2 on its own
    (chain_from); every digest, n_new and every hit count are compared."""
    wl = session_wl
    T1, T2, start = wl.notes["turn1"], wl.insert, wl.notes["start"]
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    last = np.maximum(T1.blk_offsets()[1:] - 1, 0)
    h1 = gpu_chains(T1, sd, mode)
    parents = h1[dev(last)].contiguous()
    h2 = K.hash_chains_resume(dev(T2.tokens), dev(T2.tok_offsets), dev(T2.principal), sd, mode,
                              dev(start), parents, dev(T2.boundary_tok))
    cnt = T2.block_counts() - start
    bo = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    with K.Cache(wl.log2_slots) as c:
        n_new = c.insert(h2, dev(bo))
        hits = c.lookup(h2, dev(bo)).cpu().numpy()
    o1 = oracle_chains(T1, osalts, mode)
    want = O.hash_chains_resume(T2.tokens, T2.tok_offsets, T2.principal, osalts, mode, start,
                                o1[last], T2.boundary_tok)
    assert np.array_equal(h2.cpu().numpy(), want)
    assert n_new == O.Table().insert(want) == int(cnt.sum())
    assert np.array_equal(hits, cnt)
    assert np.array_equal(hits, wl.lookup.expect_hits[mode])


# ---------------------------------------------------------------------------
# the later stages on the paper-shaped batches
# ---------------------------------------------------------------------------

_CHAINS = {}


def oracle_chains_cached(b, salts, mode):
    """The oracle's digests of a whole batch, computed once per content (the
    three workloads below share the paper-shaped batches)."""
    h = hashlib.sha256()
    for a in (b.tokens, b.tok_offsets, b.principal, b.boundary_tok):
        h.update(np.ascontiguousarray(a).tobytes())
    h.update(b"".join(salts))
    key = (h.hexdigest(), mode)
    if key not in _CHAINS:
        _CHAINS[key] = oracle_chains(b, salts, mode)
    return _CHAINS[key]


def concat(A, B):
    return W.Batch(np.concatenate([A.tokens, B.tokens]),
                   np.concatenate([A.tok_offsets, B.tok_offsets[1:] + A.tok_offsets[-1]]),
                   np.concatenate([A.principal, B.principal]),
                   np.concatenate([A.boundary_tok, B.boundary_tok]))


@pytest.fixture(scope="module")
def admission_wl():
    return W.make("admission")


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY])
def test_admission_config(admission_wl, mode):
    """Both batches (8192 requests) admitted in one call, as bench.py does:
    every request's hit blocks and new blocks against the oracle's requests
    taken in order, and the hits fixed by construction."""
    wl = admission_wl
    A, B = wl.insert, wl.lookup
    X = concat(A, B)
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    h = gpu_chains(X, sd, mode)
    with K.Cache(wl.log2_slots) as c:
        hits, new, n_new = c.admit(h, dev(X.blk_offsets()))
        count = c.count()
    want_h = np.concatenate([oracle_chains_cached(A, osalts, mode),
                             oracle_chains_cached(B, osalts, mode)])
    assert np.array_equal(h.cpu().numpy(), want_h)
    T = O.Table()
    wh, wn = T.admit(want_h, X.blk_offsets())
    assert np.array_equal(hits.cpu().numpy(), wh)
    assert np.array_equal(new.cpu().numpy(), wn)
    assert n_new == int(wn.sum()) == len(T.keys) == count
    assert np.array_equal(wh, wl.notes["admit_hits"][mode])


@pytest.fixture(scope="module")
def radix_wl():
    return W.make("radix")


@pytest.mark.parametrize("mode", [W.ROOT, W.NONE])
def test_radix_config(radix_wl, mode):
    """The insert batch's sequences into the radix index (2^23 edge slots, as
    bench.py), the re-lookup batch matched: every match covers the shared
    2119-token prefix and equals the oracle's, and the index holds one block
    node per distinct digest plus its roots."""
    wl = radix_wl
    A, B = wl.insert, wl.lookup
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    salted = mode != W.NONE

    def args(b):
        h = gpu_chains(b, sd, mode) if salted else \
            K.hash_chains(dev(b.tokens), dev(b.tok_offsets), None, None, W.NONE)
        return (dev(b.tokens), dev(b.tok_offsets), dev(b.principal) if salted else None,
                sd if salted else None, mode, h, dev(b.blk_offsets()))

    with K.Radix(wl.log2_slots, 23) as x:
        x.insert(*args(A))
        got = x.match(*args(B)).cpu().numpy()
        blocks, edges = x.stats()
    assert (got >= wl.notes["prefix_len"]).all()
    ha = oracle_chains_cached(A, osalts, mode)
    roots = wl.P if salted else 1  # a root per salt of the table, or the zero root
    assert blocks == roots + len({ha[i].tobytes() for i in range(ha.shape[0])})
    R = O.Radix()
    R.insert(A.tokens, A.tok_offsets, A.principal, osalts, mode)
    # every request: with root salting compared with its principal's
    # sequences, unsalted with all 4096 inserted sequences (~35 ms each on
    # one core, spread over the worker processes)
    qs = np.arange(B.n)
    want = radix_match_parallel(R, B, osalts, mode, qs)
    assert np.array_equal(got[qs], want)


def _radix_range(rng_):
    a, b = rng_
    sh = _SHARED
    return sh["R"].match(sh["B"].tokens, sh["B"].tok_offsets, sh["B"].principal, sh["salts"],
                         sh["mode"], requests=sh["qs"][a:b])


def radix_match_parallel(R, B, osalts, mode, qs):
    """The oracle index's matches of requests ``qs``, split over workers."""
    import multiprocessing as mp
    _SHARED.update(R=R, B=B, salts=osalts, mode=mode, qs=qs)
    try:
        with mp.get_context("fork").Pool(PROCS) as pool:
            parts = pool.map(_radix_range, _ranges(len(qs), PROCS))
    finally:
        _SHARED.clear()
    return np.concatenate(parts)


@pytest.fixture(scope="module")
def maintenance_wl():
    return W.make("maintenance")


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY])
def test_maintenance_config(maintenance_wl, mode):
    """A recency-tracking table: the insert batch and the re-lookup batch in
    two insert calls, an eviction to half of the keys present, an erase of
    the first tenth of the insert batch's rows, a lookup of the re-lookup
    batch; every count, the kept key set and every hit against the oracle."""
    wl = maintenance_wl
    A, B = wl.insert, wl.lookup
    sd = K.salts(wl.K, dev(wl.principal_ids))
    osalts = O.salts(wl.K, wl.principal_ids)
    hA, hB = gpu_chains(A, sd, mode), gpu_chains(B, sd, mode)
    oA, oB = oracle_chains_cached(A, osalts, mode), oracle_chains_cached(B, osalts, mode)
    n_erase = int(A.block_counts().sum() * wl.notes["erase_fraction"])
    T = O.Table()
    with K.Cache(wl.log2_slots) as c:
        c.set_recency(True)
        assert c.insert(hA, dev(A.blk_offsets())) == T.insert(oA, A.blk_offsets())
        assert c.insert(hB, dev(B.blk_offsets())) == T.insert(oB, B.blk_offsets())
        max_keys = int(c.count() * wl.notes["evict_fraction"])
        assert c.evict(max_keys) == T.evict(max_keys)
        assert c.erase(hA[:n_erase]) == T.erase(oA[:n_erase])
        hits = c.lookup(hB, dev(B.blk_offsets())).cpu().numpy()
        assert c.count() == len(T.keys)
        kept = c.export().cpu().numpy()
    assert {kept[i].tobytes() for i in range(kept.shape[0])} == T.keys
    assert np.array_equal(hits, T.lookup(oB, B.blk_offsets()))
