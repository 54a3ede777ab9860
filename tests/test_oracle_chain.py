"""Pins for the oracle's chained block hashes and cache (CPU only).

What pins what:

* the chain formulas (Sec. 2.1 / 4.1 / 4.2 displays): each digest recomputed
  from its definition with the FIPS code and an independently built byte
  string, its parent taken from the oracle's own output;
* the paper's invariants: same principal and prefix give the same hashes
  (Sec. 4.1, "Cache efficiency"), root salting gives disjoint key sets across
  principals (Sec. 4.1, "Why this works"), boundary salting keeps blocks below
  k shared and makes the rest disjoint (Sec. 4.2), root salting is the k = 0
  case of boundary salting (Sec. 4.2, "Deployment");
* the paper's worked examples (tests/golden/W*.json);
* lookup: brute-force longest common prefix over token blocks, which uses no
  hashing at all, on small batches built to contain shared prefixes, repeated
  blocks at other positions and cross-principal copies;
* planted mistakes: each plausible slip in the oracle (see ``MUTANTS``) makes
  at least one of the pins above fail.
"""
import hashlib
import json
import os
import struct

import numpy as np
import pytest

import oracle
from oracle import fips_sha256 as F
from oracle import kvgov as O
from workloads import Batch, rng, VOCAB

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
B = 16


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _salt_pair(seed=3):
    g = np.random.default_rng(seed)
    K = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, (2, 32), dtype=np.uint8)
    return O.salts(K, ids)


def _tokens(seed, n):
    return np.random.default_rng(seed).integers(0, VOCAB, n, dtype=np.int32)


# ---------------------------------------------------------------------------
# pin functions, parameterised by the chain implementation so that the
# planted-mistake tests can run them against a broken copy
# ---------------------------------------------------------------------------

def pin_closed_form(chain_fn):
    """Each h_j equals SHA-256 of its defining message (FIPS code, bytes built
    with numpy rather than struct)."""
    s0, _ = _salt_pair()
    toks = _tokens(1, 16 * 6 + 5)  # 6 full blocks + ragged tail

    def T(j):
        return toks[B * j:B * (j + 1)].astype("<i4").tobytes()

    h = chain_fn(toks, O.NONE, None, None)
    assert len(h) == 6
    assert h[0] == F.sha256(T(0))
    for j in range(1, 6):
        assert h[j] == F.sha256(h[j - 1] + T(j))
    h = chain_fn(toks, O.ROOT, s0, None)
    assert h[0] == F.sha256(s0 + T(0))
    for j in range(1, 6):
        assert h[j] == F.sha256(h[j - 1] + T(j))
    for bt, k in ((16 * 3 + 7, 3), (0, 0), (15, 0)):
        h = chain_fn(toks, O.BOUNDARY, s0, bt)
        for j in range(6):
            if j < k:
                want = F.sha256((h[j - 1] if j else b"") + T(j))
            elif j == k:
                want = F.sha256(s0 + (h[j - 1] if j else b"") + T(j))
            else:
                want = F.sha256(h[j - 1] + T(j))
            assert h[j] == want, (bt, j)


def pin_prefix_property(chain_fn):
    """h_0..h_{m-1} depend only on the first 16 m tokens: appending tokens or a
    partial block never changes them (Sec. 2.1, truncation to a block)."""
    s0, _ = _salt_pair()
    toks = _tokens(2, 16 * 8)
    for mode, salt, bt in ((O.NONE, None, None), (O.ROOT, s0, None), (O.BOUNDARY, s0, 40)):
        full = chain_fn(toks, mode, salt, bt)
        for m in (3, 5, 8):
            for extra in (0, 1, 15):
                part = chain_fn(toks[:16 * m + extra], mode, salt,
                                bt if bt is None else min(bt, 16 * m + extra))
                assert part == full[:m]
    assert chain_fn(toks[:15], O.NONE, None, None) == []
    one = chain_fn(toks[:16], O.NONE, None, None)
    for L in range(16, 32):
        assert chain_fn(toks[:L], O.NONE, None, None) == one


def pin_invariants(chain_fn):
    s0, s1 = _salt_pair()
    n = 10
    longer = _tokens(4, 16 * n + 9)
    toks = longer[:16 * n]
    plain = chain_fn(toks, O.NONE, None, None)
    r0 = chain_fn(toks, O.ROOT, s0, None)
    r1 = chain_fn(toks, O.ROOT, s1, None)
    # determinism: the same principal and tokens give the same chain
    assert chain_fn(toks.copy(), O.ROOT, s0, None) == r0
    # root disjointness
    assert not set(r0) & set(r1)
    assert not set(r0) & set(plain)
    for k in (1, 4, 9):
        b0 = chain_fn(toks, O.BOUNDARY, s0, 16 * k + 3)
        b1 = chain_fn(toks, O.BOUNDARY, s1, 16 * k + 3)
        assert b0[:k] == plain[:k] == b1[:k]       # shared below k
        assert not set(b0[k:]) & set(b1[k:])       # disjoint from k on
        assert not set(b0[k:]) & set(plain)
    # special cases: k = 0 is root salting, k >= n_full salts nothing
    assert chain_fn(toks, O.BOUNDARY, s0, 0) == r0
    assert chain_fn(toks, O.BOUNDARY, s0, 15) == r0
    assert chain_fn(toks, O.BOUNDARY, s0, 16 * n) == plain
    assert chain_fn(longer, O.BOUNDARY, s0, 16 * n + 9) == plain
    # all digests within a chain are distinct
    assert len(set(r0)) == n


def pin_worked_examples(chain_fn):
    """W1-W3: hit counts printed in (or derived from) the paper."""
    w1 = _golden("W1_divergence_position.json")
    pre = _tokens(10, w1["preamble_tokens"])
    for mode in (O.NONE, O.ROOT):
        s0, _ = _salt_pair()
        salt = s0 if mode == O.ROOT else None
        keys = set(chain_fn(pre, mode, salt, None))
        for case in w1["cases"]:
            probe = pre.copy()
            i = case["diverge_at_token"]
            probe[i] = (probe[i] + 1) % VOCAB
            h = chain_fn(probe, mode, salt, None)
            hit = 0
            while hit < len(h) and h[hit] in keys:
                hit += 1
            assert hit == case["hit_blocks"], (mode, case)
    for name in ("W2_boundary_preamble.json", "W3_short_preamble.json"):
        w = _golden(name)
        s0, s1 = _salt_pair()
        pre = _tokens(20, w["preamble_tokens"])
        tail_a = _tokens(21, w["tail_tokens"])
        tail_b = _tokens(22, w["tail_tokens"])
        pa = np.concatenate([pre, tail_a])
        pb = np.concatenate([pre, tail_b])
        if "blocks_total_including_partial" in w:
            assert -(-pa.size // B) == w["blocks_total_including_partial"]
        for mname, mode in (("none", O.NONE), ("root", O.ROOT), ("boundary", O.BOUNDARY)):
            bt = w["preamble_tokens"] if mode == O.BOUNDARY else None
            keys = set(chain_fn(pa, mode, s0, bt))
            h = chain_fn(pb, mode, s1, bt)
            hit = 0
            while hit < len(h) and h[hit] in keys:
                hit += 1
            assert hit == w["cross_principal_hit_blocks"][mname], (name, mname)
            if mode == O.BOUNDARY and "blocks_to_prefill_boundary" in w:
                assert w["blocks_total_including_partial"] - hit == w["blocks_to_prefill_boundary"]


def _oracle_chain(toks, mode, salt, bt):
    return O.chain(toks, mode, salt, bt)


def test_closed_form():
    pin_closed_form(_oracle_chain)


def test_prefix_property():
    pin_prefix_property(_oracle_chain)


def test_invariants():
    pin_invariants(_oracle_chain)


def test_worked_examples():
    pin_worked_examples(_oracle_chain)


def test_block_bytes_encoding():
    """Tokens are 4-byte little-endian two's complement, back to back."""
    toks = [0, 1, -1, 0x01020304, 152063, -2 ** 31, 2 ** 31 - 1] + list(range(9))
    b = O.block_bytes(toks, 0)
    assert len(b) == 64
    assert b[:4] == b"\x00\x00\x00\x00" and b[4:8] == b"\x01\x00\x00\x00"
    assert b[8:12] == b"\xff\xff\xff\xff" and b[12:16] == b"\x04\x03\x02\x01"
    assert b == np.asarray(toks, dtype="<i4").tobytes()


def test_boundary_out_of_range_rejected():
    s0, _ = _salt_pair()
    toks = _tokens(5, 40)
    with pytest.raises(ValueError):
        O.chain(toks, O.BOUNDARY, s0, 41)
    with pytest.raises(ValueError):
        O.chain(toks, O.BOUNDARY, s0, -1)
    assert len(O.chain(toks, O.BOUNDARY, s0, 40)) == 2


def test_batch_layout_and_permutation():
    """hash_chains lays requests out back to back; permuting the batch permutes
    the rows and changes no digest."""
    salts_ = _salt_pair()
    g = np.random.default_rng(9)
    lens = np.array([0, 5, 16, 17, 33, 64, 100, 15, 48], dtype=np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)])
    toks = g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 2, lens.size).astype(np.int32)
    bt = (lens // 2).astype(np.int32)
    b = Batch(toks, offs, prin, bt)
    for mode in (O.NONE, O.ROOT, O.BOUNDARY):
        out = O.hash_chains(toks, offs, prin, salts_, mode, bt)
        bo = b.blk_offsets()
        assert out.shape == (bo[-1], 32)
        for r in range(lens.size):
            s = salts_[prin[r]] if mode != O.NONE else None
            rowh = O.chain(b.row(r), mode, s, int(bt[r]) if mode == O.BOUNDARY else None)
            assert [bytes(x) for x in out[bo[r]:bo[r + 1]]] == rowh
        perm = g.permutation(lens.size)
        pb = b.subset(perm)
        outp = O.hash_chains(pb.tokens, pb.tok_offsets, pb.principal, salts_, mode, pb.boundary_tok)
        pbo = pb.blk_offsets()
        for i, r in enumerate(perm):
            assert np.array_equal(outp[pbo[i]:pbo[i + 1]], out[bo[r]:bo[r + 1]])


def test_parallel_matches_serial():
    salts_ = _salt_pair()
    g = np.random.default_rng(12)
    lens = g.integers(0, 200, 37).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)])
    toks = g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 2, 37).astype(np.int32)
    bt = (lens // 3).astype(np.int32)
    a = O.hash_chains(toks, offs, prin, salts_, O.BOUNDARY, bt)
    b = O.hash_chains_parallel(toks, offs, prin, salts_, O.BOUNDARY, bt, processes=3)
    assert np.array_equal(a, b)
    c = O.hash_chains_parallel(toks, offs, prin, salts_, O.BOUNDARY, bt, processes=2,
                               requests=range(5, 20))
    bo = np.concatenate([[0], np.cumsum(lens // 16)])
    assert np.array_equal(c, a[bo[5]:bo[20]])


# ---------------------------------------------------------------------------
# lookup: brute force over token blocks, no hashing
# ---------------------------------------------------------------------------

def brute_force_hits(queries, residents, mode):
    """hit(q) = max over resident r of the number m of leading blocks such that
    for every j < m the token blocks are equal and the salt regime agrees:
    both below their boundary (unsalted, shared), or both at or past it with
    the same boundary block and the same principal (salted)."""
    INF = 1 << 30
    out = []
    for qt, qp, qb in queries:
        nq = len(qt) // B
        kq = INF if mode == O.NONE else (0 if mode == O.ROOT else qb // B)
        best = 0
        for rt, rp, rb in residents:
            nr = len(rt) // B
            kr = INF if mode == O.NONE else (0 if mode == O.ROOT else rb // B)
            m = 0
            while m < min(nq, nr):
                same = np.array_equal(qt[B * m:B * (m + 1)], rt[B * m:B * (m + 1)])
                regime = (m < kq and m < kr) or (m >= kq and m >= kr and kq == kr and qp == rp)
                if not (same and regime):
                    break
                m += 1
            best = max(best, m)
        out.append(best)
    return np.array(out, dtype=np.int32)


def _lcp_batches(seed):
    """Small batches with shared prefixes, blocks repeated at shifted
    positions, cross-principal copies and ragged lengths."""
    g = np.random.default_rng(seed)
    base = g.integers(0, 50, 16 * 12, dtype=np.int32)  # small alphabet: repeats
    res, qry = [], []
    for i in range(12):
        L = int(g.integers(0, 16 * 12))
        t = base[:L].copy()
        if i % 3 == 1 and L > 40:
            t[int(g.integers(0, L))] += 1000
        res.append((t, int(g.integers(0, 3)), int(g.integers(0, L + 1))))
    for i in range(24):
        L = int(g.integers(0, 16 * 12))
        kind = i % 4
        if kind == 0:
            t = base[:L].copy()
        elif kind == 1:  # shifted by one block: same blocks, wrong positions
            t = np.concatenate([base[16:16 + L], base[:max(0, L - (base.size - 16))]])[:L].copy()
        elif kind == 2:
            t = base[:L].copy()
            if L:
                t[int(g.integers(0, L))] += 7
        else:
            t = g.integers(0, 50, L, dtype=np.int32)
        qry.append((t, int(g.integers(0, 3)), int(g.integers(0, L + 1))))
    # a resident made of the base blocks in reverse order: every block exists
    # somewhere in the table, but not as a chain prefix
    rev = np.concatenate([base[16 * j:16 * (j + 1)] for j in range(11, -1, -1)])
    res.append((rev, 0, 0))
    return res, qry


def oracle_hits(chain_fn, queries, residents, mode, salts_):
    keys = set()
    for t, p, b in residents:
        keys |= set(chain_fn(t, mode, salts_[p] if mode != O.NONE else None,
                             b if mode == O.BOUNDARY else None))
    out = []
    for t, p, b in queries:
        h = chain_fn(t, mode, salts_[p] if mode != O.NONE else None,
                     b if mode == O.BOUNDARY else None)
        m = 0
        while m < len(h) and h[m] in keys:
            m += 1
        out.append(m)
    return np.array(out, dtype=np.int32)


def pin_brute_force(chain_fn):
    g = np.random.default_rng(77)
    K = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
    salts_ = O.salts(K, g.integers(0, 256, (3, 32), dtype=np.uint8))
    for seed in (1, 2, 3):
        res, qry = _lcp_batches(seed)
        for mode in (O.NONE, O.ROOT, O.BOUNDARY):
            want = brute_force_hits(qry, res, mode)
            got = oracle_hits(chain_fn, qry, res, mode, salts_)
            assert np.array_equal(want, got), (seed, mode, want, got)
            assert want.max() > 0  # the batches do exercise hits


def test_lookup_matches_brute_force():
    pin_brute_force(_oracle_chain)


def test_table_lookup_is_first_miss():
    """Lookup reports leading blocks matched (first miss), not how many of the
    request's keys are present (Table "tab:taxonomy", block prefix cache)."""
    ks = [bytes([i]) * 32 for i in range(4)]
    T = O.Table()
    assert T.insert(np.frombuffer(ks[0] + ks[2] + ks[3], np.uint8).reshape(-1, 32)) == 3
    q = np.frombuffer(b"".join(ks), np.uint8).reshape(-1, 32)
    assert T.lookup(q, [0, 4]).tolist() == [1]
    assert T.lookup(q, [0, 0, 1, 4]).tolist() == [0, 1, 0]
    assert T.lookup(q, [0, 2, 4]).tolist() == [1, 2]


def test_table_laws():
    """Empty table hits 0; inserting a batch makes it hit fully; a second insert
    adds nothing; hits only grow as the table grows; duplicates count once."""
    salts_ = _salt_pair()
    g = np.random.default_rng(31)
    lens = g.integers(0, 150, 20).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)])
    toks = g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 2, 20).astype(np.int32)
    h = O.hash_chains(toks, offs, prin, salts_, O.ROOT)
    bo = np.concatenate([[0], np.cumsum(lens // 16)])
    T = O.Table()
    assert T.lookup(h, bo).tolist() == [0] * 20
    half = bo[:11]
    n1 = T.insert(h, half)
    assert n1 == len(set(bytes(x) for x in h[:bo[10]]))
    hits_half = T.lookup(h, bo)
    assert np.array_equal(hits_half[:10], lens[:10] // 16)
    assert T.insert(h, half) == 0
    T.insert(h, bo)
    full = T.lookup(h, bo)
    assert np.array_equal(full, lens // 16)
    assert np.all(full >= hits_half)
    dup = np.concatenate([h, h])
    T2 = O.Table()
    assert T2.insert(dup) == len(set(bytes(x) for x in h))


# ---------------------------------------------------------------------------
# planted mistakes: each must trip at least one pin
# ---------------------------------------------------------------------------

def _mut_chain(variant):
    def chain(tokens, mode, salt, bt):
        n_full = len(tokens) // B if variant != "partial_block" else -(-len(tokens) // B)
        k = None
        if mode == O.BOUNDARY:
            k = bt // B if variant != "boundary_ceil" else -(-bt // B)
        out, prev = [], b""
        for j in range(n_full):
            blk = tokens[B * j:B * (j + 1)]
            if variant == "big_endian":
                T = struct.pack(">%di" % len(blk), *[int(x) for x in blk])
            else:
                T = struct.pack("<%di" % len(blk), *[int(x) for x in blk])
            salted = (mode == O.ROOT and j == 0) or (mode == O.BOUNDARY and j == k)
            if variant == "no_parent":
                prev = b""
            if variant == "salt_after" and salted:
                msg = prev + T + salt
            elif variant == "boundary_salt_after_parent" and salted:
                msg = prev + salt + T
            elif variant == "salt_every_block" and mode != O.NONE:
                msg = salt + prev + T
            elif variant == "root_salts_boundary_too" and mode == O.BOUNDARY and j == 0:
                msg = salt + prev + T
            else:
                msg = (salt if salted else b"") + prev + T
            if variant == "parent_hex":
                msg = msg.replace(prev, prev.hex().encode()) if prev else msg
            prev = hashlib.sha256(msg).digest()
            out.append(prev)
        return out
    return chain


MUTANTS = ["partial_block", "boundary_ceil", "big_endian", "no_parent", "salt_after",
           "boundary_salt_after_parent", "salt_every_block", "root_salts_boundary_too",
           "parent_hex"]


@pytest.mark.parametrize("variant", MUTANTS)
def test_planted_mistake_is_caught(variant):
    fn = _mut_chain(variant)
    caught = []
    for pin in (pin_closed_form, pin_prefix_property, pin_invariants, pin_worked_examples,
                pin_brute_force):
        try:
            pin(fn)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {variant!r}"


def test_unmutated_copy_passes_all_pins():
    fn = _mut_chain("none")
    for pin in (pin_closed_form, pin_prefix_property, pin_invariants, pin_worked_examples,
                pin_brute_force):
        pin(fn)
