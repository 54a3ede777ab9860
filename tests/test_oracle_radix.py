"""Pins for the oracle's radix index (token-granular longest prefix match).

``Radix.match`` is the definition: the longest token prefix a request shares
with any sequence of its tree (one tree per principal under root salting,
one shared tree unsalted).  What pins it:

* the block cache, computed independently (chained SHA-256 digests in a key
  set, first-miss lookup): for every request, floor(match / 16) equals the
  block cache's hit count on the same sequences (a block of the request is
  cached exactly when some sequence shares its first 16 (j + 1) tokens);
* hand-built sequences with the expected lengths written out: divergence at
  every position of a block, partial blocks inserted and queried, empty
  sequences, queries longer and shorter than what is stored;
* laws: an inserted sequence matches in full; inserting never lowers a
  match; root salting separates principals and unsalted trees share;
* planted mistakes (``MUTANTS``) each trip at least one pin.
"""
import numpy as np
import pytest

from oracle import kvgov as O
from tests.test_oracle_chain import _lcp_batches, B


def _flat(seqs):
    lens = [len(s) for s in seqs]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = np.concatenate([np.asarray(s, dtype=np.int32) for s in seqs]) if seqs \
        else np.zeros(0, np.int32)
    return toks, offs


# fn(inserted: [(tokens, principal)], queries: [(tokens, principal)], mode, salts)
#    -> match lengths of the queries

def pin_block_cache_agrees(fn):
    g = np.random.default_rng(3)
    salts_ = O.salts(bytes(range(32)), g.integers(0, 256, (3, 32), dtype=np.uint8))
    for seed in (1, 2, 3):
        res, qry = _lcp_batches(seed)
        ins = [(t, p) for t, p, _ in res]
        qs = [(t, p) for t, p, _ in qry] + [(t[:len(t) - 3], p) for t, p, _ in res[:5]]
        for mode in (O.NONE, O.ROOT):
            got = fn(ins, qs, mode, salts_)
            T = O.Table()
            for t, p in ins:
                T.keys |= set(O.chain(t, mode, salts_[p] if mode else None))
            hits = []
            for t, p in qs:
                h = O.chain(t, mode, salts_[p] if mode else None)
                m = 0
                while m < len(h) and h[m] in T.keys:
                    m += 1
                hits.append(m)
            assert np.array_equal(np.asarray(got) // B, hits), (seed, mode)
            assert (np.asarray(got) % B).any()  # the finer signal is exercised


def pin_hand_built(fn):
    base = np.arange(100, 180, dtype=np.int32)  # 80 tokens = 5 blocks
    ins = [(base[:40], 0),                      # 2 full blocks + 8 tokens
           (np.r_[base[:20], 7, 7, 7], 0),      # diverges at token 20
           (base[:5], 1),                       # partial first block only
           (np.zeros(0, np.int32), 0)]          # empty
    cases = [  # (query, principal, expected in the shared tree, expected per principal)
        (base[:40], 0, 40, 40),
        (base[:80], 0, 40, 40),
        (base[:33], 0, 33, 33),
        (base[:16], 0, 16, 16),
        (np.r_[base[:15], 1], 0, 15, 15),
        (np.r_[base[:16], 1], 0, 16, 16),
        (np.r_[base[:17], 1], 0, 17, 17),
        (np.r_[base[:20], 7, 7, 7, 7], 0, 23, 23),
        (np.r_[base[:20], 7, 8], 0, 21, 21),
        (np.r_[1, base[1:40]], 0, 0, 0),
        (base[:40], 1, 40, 5),                  # principal 1 holds only base[:5]
        (base[:3], 1, 3, 3),
        (np.zeros(0, np.int32), 0, 0, 0),
        (base[:40], 2, 40, 0),                  # principal 2 has an empty tree
    ]
    salts_ = O.salts(b"k", np.arange(3 * 8, dtype=np.uint8).reshape(3, 8))
    qs = [(q, p) for q, p, _, _ in cases]
    assert list(fn(ins, qs, O.NONE, salts_)) == [c[2] for c in cases]
    assert list(fn(ins, qs, O.ROOT, salts_)) == [c[3] for c in cases]


def pin_laws(fn):
    g = np.random.default_rng(4)
    salts_ = O.salts(b"key", g.integers(0, 256, (4, 16), dtype=np.uint8))
    pre = g.integers(0, 9, 70).astype(np.int32)
    seqs = []
    for i in range(24):
        L = int(g.integers(0, 120))
        t = np.r_[pre[:min(L, int(g.integers(0, 71)))], g.integers(0, 9, L)][:L].astype(np.int32)
        seqs.append((t, int(g.integers(0, 4))))
    queries = [(np.r_[t, 5, 5].astype(np.int32), p) for t, p in seqs]
    for mode in (O.NONE, O.ROOT):
        full = fn(seqs, [(t, p) for t, p in seqs], mode, salts_)
        assert list(full) == [len(t) for t, _ in seqs]
        prev = np.zeros(len(queries), np.int64)
        for k in (0, 6, 12, 24):
            cur = np.asarray(fn(seqs[:k], queries, mode, salts_))
            assert (cur >= prev).all()
            prev = cur
    # principals: the same sequence under another principal
    t = pre[:50]
    assert list(fn([(t, 0)], [(t, 1)], O.ROOT, salts_)) == [0]
    assert list(fn([(t, 0)], [(t, 1)], O.NONE, salts_)) == [50]


PINS = (pin_block_cache_agrees, pin_hand_built, pin_laws)


def _oracle(ins, qs, mode, salts_):
    R = O.Radix()
    if ins:
        toks, offs = _flat([t for t, _ in ins])
        R.insert(toks, offs, [p for _, p in ins], salts_, mode)
    toks, offs = _flat([t for t, _ in qs])
    return R.match(toks, offs, [p for _, p in qs], salts_, mode)


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_radix(pin):
    pin(_oracle)


def test_boundary_mode_has_no_radix_form():
    R = O.Radix()
    with pytest.raises(ValueError):
        R.insert(np.arange(16), [0, 16], [0], [bytes(32)], O.BOUNDARY)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def _mut(variant):
    def fn(ins, qs, mode, salts_):
        trees = {}
        for t, p in ins:
            key = p if (mode == O.ROOT and variant != "ignore_principal") else -1
            trees.setdefault(key, []).append(np.asarray(t))
            if variant == "latest_only":
                trees[key] = trees[key][-1:]
        out = []
        for q, p in qs:
            key = p if (mode == O.ROOT and variant != "ignore_principal") else -1
            best = 0
            for s in trees.get(key, []):
                n = min(len(q), len(s))
                k = 0
                while k < n and q[k] == s[k]:
                    k += 1
                if variant == "count_first_mismatch" and k < n:
                    k += 1
                best = max(best, k)
            if variant == "block_quantised":
                best = best // B * B
            out.append(best)
        return out
    return fn


MUTANTS = ["ignore_principal", "latest_only", "count_first_mismatch", "block_quantised"]


@pytest.mark.parametrize("variant", MUTANTS)
def test_planted_mistake_is_caught(variant):
    fn = _mut(variant)
    caught = []
    for pin in PINS:
        try:
            pin(fn)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {variant!r}"


def test_unmutated_copy_passes_all_pins():
    fn = _mut("none")
    for pin in PINS:
        pin(fn)
