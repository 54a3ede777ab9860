"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every comparison is bit-exact (digests, hit counts, key sets, n_new): the
path computes integers only.  Slot placement inside the table is not part of
the contract and is never compared; the exported key *set* is.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import Batch, VOCAB

pytestmark = pytest.mark.gpu

K = pytest.importorskip("paper_2608_09225_amd.kvgov")


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


def ragged(seed, lens, P=4, bt_mode="random"):
    g = np.random.default_rng(seed)
    lens = np.asarray(lens, dtype=np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(-2 ** 31, 2 ** 31 - 1, int(offs[-1]), dtype=np.int64).astype(np.int32) \
        if bt_mode == "wide" else g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, P, lens.size).astype(np.int32)
    bt = np.floor(g.random(lens.size) * (lens + 1)).astype(np.int32)
    return Batch(toks, offs, prin, bt)


def secret(seed, P, klen=32, idlen=32):
    g = np.random.default_rng(1000 + seed)
    Kb = g.integers(0, 256, klen, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, (P, idlen), dtype=np.uint8)
    return Kb, ids


def gpu_chains(b: Batch, salts_dev, mode, status=None, check=True):
    return K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), salts_dev, mode,
                         dev(b.boundary_tok), status=status, check=check)


# ---------------------------------------------------------------------------
# a1 salts
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("klen", [1, 31, 32, 55, 64])
@pytest.mark.parametrize("idlen", [0, 1, 32, 55, 56, 64, 119, 120, 300])
def test_salts(klen, idlen):
    for P in (1, 65):
        Kb, ids = secret(klen * 7 + idlen, P, klen, idlen)
        got = K.salts(Kb, dev(ids)).cpu().numpy()
        want = O.salts(Kb, ids)
        for p in range(P):
            assert bytes(got[p]) == want[p], (klen, idlen, P, p)


def test_salts_many_principals():
    Kb, ids = secret(3, 4096)
    got = K.salts(Kb, dev(ids)).cpu().numpy()
    want = O.salts(Kb, ids)
    assert all(bytes(got[p]) == want[p] for p in range(4096))


# ---------------------------------------------------------------------------
# output layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [0, 1, 1023, 1024, 1025, 5000, 70000])
def test_block_offsets(n):
    g = np.random.default_rng(n)
    lens = g.integers(0, 100, n).astype(np.int64)
    if n:
        lens[:min(n, 8)] = [0, 15, 16, 17, 31, 32, 33, 99][:min(n, 8)]
    b = Batch(np.zeros(int(lens.sum()), np.int32), np.concatenate([[0], np.cumsum(lens)]),
              np.zeros(n, np.int32), np.zeros(n, np.int32))
    got = K.block_offsets(dev(b.tok_offsets)).cpu().numpy()
    assert np.array_equal(got, b.blk_offsets())


def test_block_offsets_negative_length_latched():
    offs = np.array([0, 40, 30, 50], dtype=np.int64)
    with pytest.raises(K.KvgovError) as e:
        K.block_offsets(dev(offs))
    assert e.value.code == K.header_constants()["KVGOV_E_OFFSETS"]


# ---------------------------------------------------------------------------
# a2/a3 chains
# ---------------------------------------------------------------------------

EDGE_LENS = [0, 1, 15, 16, 17, 31, 32, 33, 47, 48, 63, 64, 65, 160, 161, 500, 1023, 1024]


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_chains_edge_lengths(mode):
    """Ragged lengths around block edges; boundary at 0, inside, on a block
    edge, at and past the last full block."""
    lens = EDGE_LENS * 6
    b = ragged(11 + mode, lens)
    L = b.lengths
    bt = b.boundary_tok
    for i in range(len(lens)):
        kind = i // len(EDGE_LENS)
        bt[i] = [0, min(15, L[i]), min(16, L[i]), L[i] // 2, L[i], (L[i] // 16) * 16][kind]
    Kb, ids = secret(5, 4)
    sd = K.salts(Kb, dev(ids))
    got = gpu_chains(b, sd, mode).cpu().numpy()
    want = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode, bt)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_chains_full_int32_range(mode):
    b = ragged(21, [16, 48, 100, 33], bt_mode="wide")
    Kb, ids = secret(6, 4)
    got = gpu_chains(b, K.salts(Kb, dev(ids)), mode).cpu().numpy()
    want = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                         b.boundary_tok)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_chains_many_waves_and_ordering(mode):
    """9000 requests (above the longest-first ordering threshold), lengths
    0..400 tokens, so waves mix lengths and boundaries."""
    g = np.random.default_rng(31)
    lens = g.integers(0, 400, 9000)
    b = ragged(33 + mode, lens, P=37)
    Kb, ids = secret(7, 37)
    got = gpu_chains(b, K.salts(Kb, dev(ids)), mode).cpu().numpy()
    want = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                                  b.boundary_tok)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", [W.ROOT, W.BOUNDARY])
def test_chains_long_with_scattered_boundaries(mode):
    """Long chains (94..200 blocks) whose boundaries fall on different blocks
    across each 64-request workgroup, some on the first or last block or
    past it: the lane-pair kernel switches between the first compression's
    precomputed schedule terms and the plain schedule at every iteration
    where some request of the workgroup has its boundary block."""
    g = np.random.default_rng(41)
    lens = g.integers(1500, 3200, 256)
    b = ragged(43 + mode, lens, P=9)
    bt = b.boundary_tok
    L = b.lengths
    for i in range(0, 256, 16):
        bt[i] = 0
        bt[i + 1] = (L[i + 1] // 16) * 16 - 16  # the last full block
        bt[i + 2] = L[i + 2]
    Kb, ids = secret(8, 9)
    got = gpu_chains(b, K.salts(Kb, dev(ids)), mode).cpu().numpy()
    want = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                                  bt)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("n_req", [3000, 40000])
def test_chains_permutation_invariance(n_req):
    """A request's digests depend only on its own tokens, principal and
    boundary, not on where it sits in the batch: the same batch permuted
    (lane-pair launch at 3000 requests, longest-first ordered mixed launch at
    40,000, where a request's rank decides its workgroup kind) gives every
    request the same rows, and a request repeated at the other end of the
    batch gets identical digests."""
    g = np.random.default_rng(51 + n_req)
    lens = g.integers(0, 500, n_req)
    lens[g.integers(0, n_req, 20)] = g.integers(3000, 6000, 20)  # a few long chains
    b = ragged(53 + n_req, lens, P=11)
    perm = g.permutation(n_req)
    perm[-1] = perm[0]  # request perm[0] twice: first and last
    bp = b.subset(perm)
    Kb, ids = secret(12, 11)
    sd = K.salts(Kb, dev(ids))
    bo, bop = b.blk_offsets(), bp.blk_offsets()
    rows = np.concatenate([np.arange(bo[r], bo[r + 1]) for r in perm])
    for mode in (W.ROOT, W.BOUNDARY):
        h = gpu_chains(b, sd, mode).cpu().numpy()
        hp = gpu_chains(bp, sd, mode).cpu().numpy()
        assert np.array_equal(h[rows], hp)
        assert np.array_equal(hp[bop[0]:bop[1]], hp[bop[-2]:bop[-1]])


def test_chains_unaligned_token_offsets():
    """Requests starting at any token offset (tokens not 16-byte aligned)."""
    b = ragged(41, [1, 35, 2, 70, 3, 17, 5, 64])
    Kb, ids = secret(8, 4)
    sd = K.salts(Kb, dev(ids))
    for mode in (W.NONE, W.ROOT, W.BOUNDARY):
        got = gpu_chains(b, sd, mode).cpu().numpy()
        want = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                             b.boundary_tok)
        assert np.array_equal(got, want)


def test_chains_rejects_bad_requests_and_keeps_the_rest():
    c = K.header_constants()
    b = ragged(51, [64, 64, 64, 64, 64])
    Kb, ids = secret(9, 4)
    sd = K.salts(Kb, dev(ids))
    want = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), W.BOUNDARY,
                         b.boundary_tok)
    for field, val, code in (("principal", 4, "KVGOV_E_PRINCIPAL"),
                             ("principal", -1, "KVGOV_E_PRINCIPAL"),
                             ("boundary_tok", 65, "KVGOV_E_BOUNDARY"),
                             ("boundary_tok", -1, "KVGOV_E_BOUNDARY")):
        bb = Batch(b.tokens, b.tok_offsets, b.principal.copy(), b.boundary_tok.copy())
        getattr(bb, field)[2] = val
        status = K.new_status()
        out = torch.full((20, 32), 7, dtype=torch.uint8, device="cuda")
        K.hash_chains(dev(bb.tokens), dev(bb.tok_offsets), dev(bb.principal), sd, W.BOUNDARY,
                      dev(bb.boundary_tok), blk_offsets=dev(b.blk_offsets()), out=out,
                      status=status, check=False)
        assert int(status.item()) == c[code], (field, val)
        o = out.cpu().numpy()
        assert np.array_equal(o[:8], want[:8]) and np.array_equal(o[12:], want[12:])
        assert np.all(o[8:12] == 7)  # the rejected request wrote nothing
    # blk_offsets that do not match len // 16, and a hashes buffer too small
    status = K.new_status()
    bo = b.blk_offsets().copy()
    bo[3] += 1
    out = torch.zeros((21, 32), dtype=torch.uint8, device="cuda")
    K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), sd, W.ROOT,
                  blk_offsets=dev(bo), out=out, status=status, check=False)
    assert int(status.item()) == c["KVGOV_E_OFFSETS"]
    status = K.new_status()
    out = torch.zeros((19, 32), dtype=torch.uint8, device="cuda")
    K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), sd, W.ROOT,
                  blk_offsets=dev(b.blk_offsets()), out=out, status=status, check=False)
    assert int(status.item()) == c["KVGOV_E_OFFSETS"]


def test_chains_invariants_on_gpu():
    """Root salting equals boundary salting at k = 0; boundary past the last
    block equals no salting; blocks below k are shared across principals."""
    b = ragged(61, [300] * 64)
    Kb, ids = secret(10, 4)
    sd = K.salts(Kb, dev(ids))
    none = gpu_chains(b, sd, W.NONE).cpu().numpy()
    root = gpu_chains(b, sd, W.ROOT).cpu().numpy()
    b0 = Batch(b.tokens, b.tok_offsets, b.principal, np.zeros(64, np.int32))
    assert np.array_equal(gpu_chains(b0, sd, W.BOUNDARY).cpu().numpy(), root)
    bL = Batch(b.tokens, b.tok_offsets, b.principal, np.full(64, 300, np.int32))
    assert np.array_equal(gpu_chains(bL, sd, W.BOUNDARY).cpu().numpy(), none)
    bk = Batch(b.tokens, b.tok_offsets, b.principal, np.full(64, 100, np.int32))
    bnd = gpu_chains(bk, sd, W.BOUNDARY).cpu().numpy().reshape(64, 18, 32)
    assert np.array_equal(bnd[:, :6], none.reshape(64, 18, 32)[:, :6])


def test_chains_principals_disjoint_on_gpu():
    """The same token sequences under four principals: root salting gives
    four disjoint key sets (no block of one principal's chains equals any
    block of another's), boundary salting gives identical blocks below k
    and disjoint ones from k on, and the unsalted chains coincide."""
    g = np.random.default_rng(71)
    base = ragged(73, g.integers(16, 900, 50))
    n = base.n
    idx = np.tile(np.arange(n), 4)
    b = base.subset(idx)
    b.principal[:] = np.repeat(np.arange(4, dtype=np.int32), n)
    b.boundary_tok[:] = np.tile(base.boundary_tok, 4)
    Kb, ids = secret(13, 4)
    sd = K.salts(Kb, dev(ids))
    bo = b.blk_offsets()
    per = int(bo[n])  # rows of one principal's copy of the batch
    none = gpu_chains(b, sd, W.NONE).cpu().numpy()
    for p_ in range(1, 4):
        assert np.array_equal(none[p_ * per:(p_ + 1) * per], none[:per])
    root = gpu_chains(b, sd, W.ROOT).cpu().numpy()
    sets = [key_set(root[p_ * per:(p_ + 1) * per]) for p_ in range(4)]
    for p_ in range(4):
        for q in range(p_ + 1, 4):
            assert not (sets[p_] & sets[q])
    bnd = gpu_chains(b, sd, W.BOUNDARY).cpu().numpy()
    k = base.boundary_tok // 16
    below = np.concatenate([np.arange(bo[r], bo[r] + min(int(k[r]), bo[r + 1] - bo[r]))
                            for r in range(n)]).astype(np.int64)
    above = np.setdiff1d(np.arange(per), below)
    for p_ in range(1, 4):
        assert np.array_equal(bnd[p_ * per + below], bnd[below])
        assert np.array_equal(bnd[p_ * per + below], none[below])
    upper = [key_set(bnd[p_ * per + above]) for p_ in range(4)]
    for p_ in range(4):
        for q in range(p_ + 1, 4):
            assert not (upper[p_] & upper[q])


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _gpu_cross_hit(pa, pb, mode, boundary, Kb, ids):
    """Principal 0 caches prompt pa; principal 1 looks up pb: the hit blocks
    of pb, through salts, chains, insert and lookup on the GPU."""
    lens = np.array([pa.size, pb.size], np.int64)
    b = Batch(np.concatenate([pa, pb]).astype(np.int32),
              np.concatenate([[0], np.cumsum(lens)]).astype(np.int64),
              np.array([0, 1], np.int32), np.array([boundary, boundary], np.int32))
    hs = gpu_chains(b, K.salts(Kb, dev(ids)), mode)
    bo = b.blk_offsets()
    with K.Cache(12) as c:
        c.insert(hs, dev(bo[:2]))
        return int(c.lookup(hs, dev(bo[1:])).cpu().numpy()[0])


def test_worked_examples_end_to_end():
    """The paper's worked examples through the whole GPU path, against the
    hit counts the paper prints or fixes (fixtures in tests/golden): a
    prompt diverging from a cached 2119-token preamble at token 1990 keeps
    124 blocks and at token 5 none (Sec. 5.6); another principal with the
    same 2000- or 1500-token preamble hits 125 or 93 blocks unsalted and
    with the salt at the boundary, and none with root salting (Sec. 4.2)."""
    Kb, ids = secret(14, 2)
    g = np.random.default_rng(81)
    w1 = _golden("W1_divergence_position.json")
    pre = g.integers(0, VOCAB, w1["preamble_tokens"], dtype=np.int32)
    for mode in (W.NONE, W.ROOT):
        for case in w1["cases"]:
            probe = pre.copy()
            i = case["diverge_at_token"]
            probe[i] = (probe[i] + 1) % VOCAB
            # both requests under principal 0 here: W1 is about one namespace
            lens = np.array([pre.size, probe.size], np.int64)
            b = Batch(np.concatenate([pre, probe]),
                      np.concatenate([[0], np.cumsum(lens)]).astype(np.int64),
                      np.zeros(2, np.int32), np.zeros(2, np.int32))
            hs = gpu_chains(b, K.salts(Kb, dev(ids)), mode)
            bo = b.blk_offsets()
            with K.Cache(12) as c:
                c.insert(hs, dev(bo[:2]))
                hit = int(c.lookup(hs, dev(bo[1:])).cpu().numpy()[0])
            assert hit == case["hit_blocks"], (mode, case)
    for name in ("W2_boundary_preamble.json", "W3_short_preamble.json"):
        w = _golden(name)
        shared = g.integers(0, VOCAB, w["preamble_tokens"], dtype=np.int32)
        pa = np.concatenate([shared, g.integers(0, VOCAB, w["tail_tokens"], dtype=np.int32)])
        pb = np.concatenate([shared, g.integers(0, VOCAB, w["tail_tokens"], dtype=np.int32)])
        for mname, mode in (("none", W.NONE), ("root", W.ROOT), ("boundary", W.BOUNDARY)):
            hit = _gpu_cross_hit(pa, pb, mode, w["preamble_tokens"], Kb, ids)
            assert hit == w["cross_principal_hit_blocks"][mname], (name, mname)


# ---------------------------------------------------------------------------
# a4/a5 cache
# ---------------------------------------------------------------------------

def key_set(arr):
    raw = np.ascontiguousarray(arr).tobytes()
    return {raw[i:i + 32] for i in range(0, len(raw), 32)}


def test_cache_insert_lookup_small():
    b = ragged(71, W_LENS := [0, 15, 16, 17, 100, 256, 300, 32] * 8, P=3)
    Kb, ids = secret(11, 3)
    sd = K.salts(Kb, dev(ids))
    hs = gpu_chains(b, sd, W.ROOT)
    bo = dev(b.blk_offsets())
    want_h = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), W.ROOT)
    with K.Cache(10) as c:
        assert c.slots() == 1024
        assert c.lookup(hs, bo).cpu().numpy().tolist() == [0] * len(W_LENS)
        half = dev(b.blk_offsets()[:33])
        T = O.Table()
        assert c.insert(hs, half) == T.insert(want_h, b.blk_offsets()[:33])
        assert np.array_equal(c.lookup(hs, bo).cpu().numpy(), T.lookup(want_h, b.blk_offsets()))
        assert c.insert(hs, half) == 0
        assert c.insert(hs, bo) == T.insert(want_h, b.blk_offsets())
        got = c.lookup(hs, bo).cpu().numpy()
        assert np.array_equal(got, T.lookup(want_h, b.blk_offsets()))
        assert np.array_equal(got, b.lengths // 16)
        assert c.count() == len(T.keys)
        assert key_set(c.export().cpu().numpy()) == T.keys


def test_cache_duplicates_and_special_keys():
    """Duplicate keys in one batch count once; the all-zero and all-0xFF keys
    (the latter is the empty-slot pattern) are ordinary keys."""
    g = np.random.default_rng(81)
    base = g.integers(0, 256, (300, 32), dtype=np.uint8)
    base[0] = 0
    base[1] = 255
    base[2, :31] = 255  # one byte away from the empty pattern
    keys = np.concatenate([base, base[::-1], base[:50]])
    g.shuffle(keys)
    bo = np.array([0, keys.shape[0]], dtype=np.int64)
    with K.Cache(12) as c:
        assert c.insert(dev(keys), dev(bo)) == 300
        assert c.insert(dev(keys), dev(bo)) == 0
        assert c.count() == 300
        assert key_set(c.export().cpu().numpy()) == key_set(base)
        # each special key alone as a one-block request
        q = np.stack([base[0], base[1], base[2], g.integers(0, 256, 32, dtype=np.uint8)])
        hits = c.lookup(dev(q), dev(np.arange(5, dtype=np.int64))).cpu().numpy()
        assert hits.tolist() == [1, 1, 1, 0]
    with K.Cache(6) as c:  # 64 slots
        q = np.stack([np.full(32, 255, np.uint8)])
        assert c.lookup(dev(q), dev(np.array([0, 1], np.int64))).cpu().numpy().tolist() == [0]
        assert c.insert(dev(q), dev(np.array([0, 1], np.int64))) == 1
        assert c.lookup(dev(q), dev(np.array([0, 1], np.int64))).cpu().numpy().tolist() == [1]


def test_cache_heavy_duplicates_repeatable():
    """Many lanes insert the same few keys at once; results and key sets are
    identical run after run."""
    g = np.random.default_rng(91)
    uniq = g.integers(0, 256, (37, 32), dtype=np.uint8)
    keys = uniq[g.integers(0, 37, 200000)]
    bo = np.array([0, keys.shape[0]], dtype=np.int64)
    for _ in range(3):
        with K.Cache(8) as c:
            assert c.insert(dev(keys), dev(bo)) == 37
            assert key_set(c.export().cpu().numpy()) == key_set(uniq)


def test_cache_full_is_latched():
    c_ = K.header_constants()
    g = np.random.default_rng(101)
    keys = g.integers(0, 256, (40, 32), dtype=np.uint8)
    with K.Cache(4) as c:  # 16 slots
        with pytest.raises(K.KvgovError) as e:
            c.insert(dev(keys), dev(np.array([0, 40], np.int64)))
        assert e.value.code == c_["KVGOV_E_FULL"]
        got = key_set(c.export(cap=64).cpu().numpy()) if c.slots() else set()
        assert len(got) == 16 and got <= key_set(keys)
        c.clear()
        assert c.count() == 0
        assert c.insert(dev(keys[:10]), dev(np.array([0, 10], np.int64))) == 10


def test_cache_bad_offsets_latched():
    c_ = K.header_constants()
    keys = np.zeros((4, 32), np.uint8)
    with K.Cache(6) as c:
        with pytest.raises(K.KvgovError) as e:
            c.insert(dev(keys), dev(np.array([0, 5], np.int64)))
        assert e.value.code == c_["KVGOV_E_OFFSETS"]
        c.clear()
        hits = c.lookup(dev(keys), dev(np.array([0, 2, 1, 9], np.int64)))
        assert hits.cpu().numpy().tolist()[1:] == [0, 0]
        with pytest.raises(K.KvgovError):
            c.count()


def test_cache_insert_shared_prefixes():
    """Requests sharing prefixes with their neighbours (the insert skips keys
    equal to the previous request's key at the same position), runs of empty
    and one-block requests, and duplicates far apart: the table receives
    exactly the batch's key set."""
    g = np.random.default_rng(111)
    fam = g.integers(0, 256, (12, 300, 32), dtype=np.uint8)
    lens, rows = [], []
    for r in range(4000):
        kind = r % 10
        if kind == 0:
            L = 0
        elif kind in (1, 2):
            L = 1
        else:
            L = int(g.integers(1, 250))
        f = (r // 7) % 12 if kind < 8 else int(g.integers(0, 12))  # runs, then random
        s = int(g.integers(0, L + 1))
        k = g.integers(0, 256, (L, 32), dtype=np.uint8)
        k[:s] = fam[f, :s]
        lens.append(L)
        rows.append(k)
    # a long run of one-block requests with identical keys (window overflow)
    for r in range(300):
        lens.append(1)
        rows.append(fam[0, :1].copy())
    keys = np.concatenate(rows)
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    want = key_set(keys)
    with K.Cache(20) as c:
        assert c.insert(dev(keys), dev(bo)) == len(want)
        assert c.count() == len(want)
        assert key_set(c.export().cpu().numpy()) == want
        assert c.insert(dev(keys), dev(bo)) == 0
        hits = c.lookup(dev(keys), dev(bo)).cpu().numpy()
    assert np.array_equal(hits, np.asarray(lens))


def test_cache_insert_interleaved_shared_heads():
    """Requests of many prefix families interleaved at random, as the requests
    of root-salted principals are (the insert compares a row with the row at
    the same depth of the earliest request that starts with the same block):
    shared heads with tails that diverge at once, requests shorter and longer
    than their family's earliest one, a family's keys at shifted depths, the
    head key repeated deeper, and the same batch with recency tracking on."""
    g = np.random.default_rng(131)
    fam = g.integers(0, 256, (30, 300, 32), dtype=np.uint8)
    lens, rows = [], []
    for r in range(6000):
        f = int(g.integers(0, 30))
        L = int(g.integers(1, 250))
        kind = r % 8
        k = g.integers(0, 256, (L, 32), dtype=np.uint8)
        if kind <= 3:  # a shared prefix of random depth
            s = int(g.integers(1, L + 1))
            k[:s] = fam[f, :s]
        elif kind == 4:  # the head only, then another family's rows at the same depths
            k[:] = fam[(f + 1) % 30, :L]
            k[0] = fam[f, 0]
        elif kind == 5:  # the head, then the family's rows shifted by three
            k[0] = fam[f, 0]
            k[1:] = fam[f, 4:L + 3]
        elif kind == 6:  # the whole family prefix, the head key again at depth 7
            k[:] = fam[f, :L]
            if L > 7:
                k[7] = fam[f, 0]
        lens.append(L)
        rows.append(k)
    keys = np.concatenate(rows)
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    want = key_set(keys)
    for track in (False, False, True):
        with K.Cache(21) as c:
            if track:
                c.set_recency(True)
            assert c.insert(dev(keys), dev(bo)) == len(want)
            assert c.count() == len(want)
            assert key_set(c.export().cpu().numpy()) == want
            assert c.insert(dev(keys), dev(bo)) == 0
            hits = c.lookup(dev(keys), dev(bo)).cpu().numpy()
        assert np.array_equal(hits, np.asarray(lens))


@pytest.mark.parametrize("max_len", [3, 20, 40])
def test_cache_insert_shared_heads_short_requests(max_len):
    """Short requests (few lanes per request: 4, 8, 16) of interleaved
    families whose first keys repeat, with the all-zero and all-0xFF keys as
    first keys of some families, empty requests between them, and rows
    that equal an earlier family member's at the same depth only sometimes."""
    g = np.random.default_rng(141 + max_len)
    fam = g.integers(0, 256, (12, max_len, 32), dtype=np.uint8)
    fam[0, 0] = 0
    fam[1, 0] = 255
    lens, rows = [], []
    for r in range(20000):
        L = int(g.integers(0, max_len + 1))
        f = int(g.integers(0, 12))
        k = g.integers(0, 256, (L, 32), dtype=np.uint8)
        if L:
            s_ = int(g.integers(1, L + 1))
            k[:s_] = fam[f, :s_]
        lens.append(L)
        rows.append(k)
    keys = np.concatenate(rows)
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    want = key_set(keys)
    with K.Cache(20) as c:
        assert c.insert(dev(keys), dev(bo)) == len(want)
        assert c.count() == len(want)
        assert key_set(c.export().cpu().numpy()) == want
        hits = c.lookup(dev(keys), dev(bo)).cpu().numpy()
    assert np.array_equal(hits, np.asarray(lens))


@pytest.mark.parametrize("scale", [1, 10])
def test_cache_insert_ignores_interior_offsets(scale):
    """Insert adds the flat range [blk_offsets[0], blk_offsets[n]); interior
    offsets that are not monotone change nothing.  At scale 10 the requests
    average over 4096 rows, which the insert walks in chunks of rows instead
    of a group of lanes per request."""
    g = np.random.default_rng(121)
    uniq = g.integers(0, 256, (500 * scale, 32), dtype=np.uint8)
    keys = uniq[g.integers(0, 500 * scale, 9000 * scale)]
    keys[4000 * scale:4500 * scale] = keys[3000 * scale:3500 * scale]  # a repeated stretch
    bo = np.array([0, 5000, 100, 7000, 20, 8999, 3, 9000], np.int64) * scale
    with K.Cache(12 + scale // 5) as c:
        assert c.insert(dev(keys), dev(bo)) == len(key_set(keys))
        assert key_set(c.export().cpu().numpy()) == key_set(keys)


def test_cache_insert_few_long_requests_with_shared_prefixes():
    """Requests of tens of thousands of rows (the chunked walk), sharing
    prefixes with their neighbours, then the same batch as short requests
    (a group of lanes per request): the same key set either way."""
    g = np.random.default_rng(151)
    base = g.integers(0, 256, (30000, 32), dtype=np.uint8)
    rows, lens = [], []
    for r in range(6):
        s_ = int(g.integers(0, 30000))
        k = g.integers(0, 256, (30000, 32), dtype=np.uint8)
        k[:s_] = base[:s_]
        rows.append(k)
        lens.append(30000)
    keys = np.concatenate(rows)
    want = key_set(keys)
    for bo in (np.concatenate([[0], np.cumsum(lens)]).astype(np.int64),
               np.arange(0, keys.shape[0] + 1, 100, dtype=np.int64)):
        with K.Cache(20) as c:
            assert c.insert(dev(keys), dev(bo)) == len(want)
            assert key_set(c.export().cpu().numpy()) == want
            hits = c.lookup(dev(keys), dev(bo)).cpu().numpy()
        assert np.array_equal(hits, np.diff(bo))


@pytest.mark.parametrize("n_req", [1, 7, 64, 3000, 5000, 20000, 300000])
def test_cache_lookup_group_sizes(n_req):
    """Lookups at batch sizes that select every lanes-per-request width
    (3000 long requests: many rounds per request, first misses at chosen
    positions)."""
    g = np.random.default_rng(n_req)
    # long requests at 20000 and 3000 (lanes per request from the average length)
    hi = {20000: 400, 3000: 900}.get(n_req, 70)
    nb = g.integers(0, hi, n_req).astype(np.int64)
    edge = [0, 1, 255, 256, 257, 511, 512, 513, 767, 768, 799, 800, 800, 100]
    if n_req == 3000:
        nb[:len(edge)] = 800  # first misses at the rounds' edges, and none
    bo = np.concatenate([[0], np.cumsum(nb)])
    keys = g.integers(0, 256, (int(bo[-1]), 32), dtype=np.uint8)
    # insert a random prefix of each request's keys
    pre = np.floor(g.random(n_req) * (nb + 1)).astype(np.int64)
    if n_req == 3000:
        pre[:len(edge)] = edge
    ins = np.concatenate([keys[bo[r]:bo[r] + pre[r]] for r in range(n_req)] +
                         [np.zeros((0, 32), np.uint8)])
    with K.Cache(max(6, int(np.ceil(np.log2(max(ins.shape[0], 1) * 2 + 1))))) as c:
        if ins.shape[0]:
            c.insert(dev(ins), dev(np.array([0, ins.shape[0]], np.int64)))
        hits = c.lookup(dev(keys), dev(bo)).cpu().numpy()
    assert np.array_equal(hits, pre)


# ---------------------------------------------------------------------------
# the small workload end to end
# ---------------------------------------------------------------------------

def test_tiny_workload_end_to_end():
    wl = W.make("tiny")
    sd = K.salts(wl.K, dev(wl.principal_ids))
    want_s = O.salts(wl.K, wl.principal_ids)
    hi = gpu_chains(wl.insert, sd, W.ROOT)
    hl = gpu_chains(wl.lookup, sd, W.ROOT)
    T = O.Table()
    wi = O.hash_chains(wl.insert.tokens, wl.insert.tok_offsets, wl.insert.principal, want_s, W.ROOT)
    wlk = O.hash_chains(wl.lookup.tokens, wl.lookup.tok_offsets, wl.lookup.principal, want_s,
                        W.ROOT)
    assert np.array_equal(hi.cpu().numpy(), wi) and np.array_equal(hl.cpu().numpy(), wlk)
    with K.Cache(wl.log2_slots) as c:
        assert c.insert(hi, dev(wl.insert.blk_offsets())) == T.insert(wi)
        hits = c.lookup(hl, dev(wl.lookup.blk_offsets())).cpu().numpy()
    assert np.array_equal(hits, T.lookup(wlk, wl.lookup.blk_offsets()))
    assert np.array_equal(hits, wl.lookup.expect_hits[W.ROOT])


@pytest.mark.parametrize("n_req", [20000, 30000])
def test_chains_between_one_and_two_pairs_per_cu(n_req):
    """Batch sizes where the wave-pair kernel runs two pairs per CU
    (between 64 and 128 requests per CU on a 256-CU device)."""
    g = np.random.default_rng(n_req)
    lens = g.integers(0, 300, n_req)
    b = ragged(n_req, lens, P=11)
    Kb, ids = secret(12, 11)
    sd = K.salts(Kb, dev(ids))
    osalts = O.salts(Kb, ids)
    for mode in (W.NONE, W.ROOT, W.BOUNDARY):
        got = gpu_chains(b, sd, mode).cpu().numpy()
        want = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, osalts, mode,
                                      b.boundary_tok)
        assert np.array_equal(got, want), mode


def test_chains_concurrent_streams_and_scratch_growth():
    """Ordered batches (above 128 requests per CU) hashed on three streams at
    once, twice, the second time with larger batches (each stream's scratch
    grows between the rounds): every digest equals the oracle's and no
    kernel latches an error."""
    Kb, ids = secret(21, 29)
    sd = K.salts(Kb, dev(ids))
    osalts = O.salts(Kb, ids)
    streams = [torch.cuda.Stream() for _ in range(3)]
    main = torch.cuda.current_stream()
    for rnd, base in enumerate((34000, 52000)):
        jobs = []
        for k, s in enumerate(streams):
            n = base + 3001 * k
            g = np.random.default_rng(700 + 10 * rnd + k)
            b = ragged(800 + 10 * rnd + k, g.integers(0, 120, n), P=29)
            mode = (W.NONE, W.ROOT, W.BOUNDARY)[(k + rnd) % 3]
            args = [dev(b.tokens), dev(b.tok_offsets), dev(b.principal), dev(b.boundary_tok)]
            bo = K.block_offsets(args[1])
            jobs.append((b, mode, args, bo))
        torch.cuda.synchronize()
        outs = []
        for (b, mode, args, bo), s in zip(jobs, streams):
            s.wait_stream(main)
            with torch.cuda.stream(s):
                st = K.new_status()
                out = torch.empty((int(bo[-1].item()), 32), dtype=torch.uint8, device="cuda")
                K.hash_chains(args[0], args[1], args[2], sd, mode, args[3], blk_offsets=bo,
                              out=out, status=st, check=False, stream=s)
            outs.append((out, st))
        torch.cuda.synchronize()
        for (b, mode, _, _), (out, st) in zip(jobs, outs):
            assert int(st.item()) == 0, (rnd, mode)
            want = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, osalts, mode,
                                          b.boundary_tok)
            assert np.array_equal(out.cpu().numpy(), want), (rnd, mode)
