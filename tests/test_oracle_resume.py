"""Pins for the oracle's chain extension (CPU only).

``chain_from`` enters the chain recurrence of Sec. 2.1 at block j0 with the
parent digest h_{j0-1} (Sec. 5.7: turn n+1 of a session extends turn n
exactly).  What pins it:

* the definition: every digest recomputed with the FIPS code from a byte
  string built here (parent first, salt in front on the salted block only);
* the whole-chain oracle ``chain`` (pinned on its own in
  test_oracle_chain.py): for every start block, every mode and boundaries
  below, at and above the start, the resumed chain equals the suffix of the
  whole chain;
* composition: resuming twice equals resuming once;
* the two-turn session: turn 2's chain resumed from turn 1's last full block
  equals turn 2's whole chain from there, including a turn 1 that ends in a
  partial block;
* planted mistakes (``MUTANTS``) each trip at least one of these pins.
"""
import hashlib
import struct

import numpy as np
import pytest

from oracle import fips_sha256 as F
from oracle import kvgov as O
from workloads import VOCAB

B = 16


def _salt_pair(seed=5):
    g = np.random.default_rng(seed)
    K = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, (2, 24), dtype=np.uint8)
    return O.salts(K, ids)


def _tokens(seed, n):
    return np.random.default_rng(seed).integers(0, VOCAB, n, dtype=np.int32)


def _T(toks, j):
    return toks[B * j:B * (j + 1)].astype("<i4").tobytes()


# ---------------------------------------------------------------------------
# pins, parameterised by the implementation under test
# ---------------------------------------------------------------------------

def pin_definition(fn):
    """h_{j0} = SHA256([sigma] || parent || T_{j0}), then chained."""
    s0, _ = _salt_pair()
    toks = _tokens(31, 16 * 7 + 9)  # 7 full blocks + ragged tail
    parent = hashlib.sha256(b"some earlier digest").digest()
    for j0 in (1, 3, 6):
        # unsalted and root: no salt anywhere from j0 on
        for mode, salt in ((O.NONE, None), (O.ROOT, s0)):
            h = fn(toks, j0, parent, mode, salt, None)
            assert len(h) == 7 - j0
            prev = parent
            for i, j in enumerate(range(j0, 7)):
                assert h[i] == F.sha256(prev + _T(toks, j)), (mode, j0, j)
                prev = h[i]
        # boundary at, above and below the start block
        for k in (j0, j0 + 1, j0 - 1):
            h = fn(toks, j0, parent, O.BOUNDARY, s0, 16 * k + 5)
            prev = parent
            for i, j in enumerate(range(j0, 7)):
                sig = s0 if j == k else b""
                assert h[i] == F.sha256(sig + prev + _T(toks, j)), (k, j0, j)
                prev = h[i]
    # j0 = 0 reads no parent: the chain's usual root
    h = fn(toks, 0, None, O.ROOT, s0, None)
    assert h[0] == F.sha256(s0 + _T(toks, 0))
    h = fn(toks, 0, None, O.NONE, None, None)
    assert h[0] == F.sha256(_T(toks, 0))


def pin_suffix_of_whole_chain(fn):
    s0, s1 = _salt_pair()
    toks = _tokens(32, 16 * 9 + 3)
    cases = [(O.NONE, None, None), (O.ROOT, s0, None)]
    cases += [(O.BOUNDARY, s1, bt) for bt in (0, 7, 16, 16 * 3 + 2, 16 * 5, 16 * 9, 16 * 9 + 3)]
    for mode, salt, bt in cases:
        whole = O.chain(toks, mode, salt, bt)
        for j0 in range(0, 10):
            parent = whole[j0 - 1] if j0 else None
            assert fn(toks, j0, parent, mode, salt, bt) == whole[j0:], (mode, bt, j0)


def pin_composition(fn):
    s0, _ = _salt_pair()
    toks = _tokens(33, 16 * 8)
    parent = hashlib.sha256(b"p").digest()
    for mode, salt, bt in ((O.NONE, None, None), (O.ROOT, s0, None), (O.BOUNDARY, s0, 16 * 4)):
        for j0 in (1, 2):
            once = fn(toks, j0, parent, mode, salt, bt)
            for j1 in range(j0 + 1, 9):
                again = fn(toks, j1, once[j1 - j0 - 1], mode, salt, bt)
                assert again == once[j1 - j0:], (mode, j0, j1)


def pin_two_turn_session(fn):
    """Turn 2 = turn 1 + new tokens; resume at turn 1's full-block count from
    its last full block's digest."""
    s0, _ = _salt_pair()
    turn2 = _tokens(34, 16 * 11 + 4)
    for t1_len in (16 * 4, 16 * 4 + 9, 16 * 7 + 15):
        turn1 = turn2[:t1_len]
        for mode, salt, bt in ((O.NONE, None, None), (O.ROOT, s0, None),
                               (O.BOUNDARY, s0, 16 * 2 + 1), (O.BOUNDARY, s0, t1_len)):
            # a boundary at or past turn 1's last full block leaves turn 1
            # unsalted; turn 2 salts block bt // 16 >= j0 after resuming
            h1 = O.chain(turn1, mode, salt, min(bt, t1_len) if bt is not None else None)
            j0 = t1_len // B
            h2 = fn(turn2, j0, h1[-1], mode, salt, bt)
            assert h2 == O.chain(turn2, mode, salt, bt)[j0:], (t1_len, mode, bt)


def pin_edges(fn):
    toks = _tokens(35, 16 * 3 + 1)
    parent = hashlib.sha256(b"q").digest()
    assert fn(toks, 3, parent, O.NONE, None, None) == []
    assert fn(toks[:15], 0, None, O.NONE, None, None) == []


PINS = (pin_definition, pin_suffix_of_whole_chain, pin_composition, pin_two_turn_session,
        pin_edges)


def _oracle(toks, j0, parent, mode, salt, bt):
    return O.chain_from(toks, j0, parent, mode, salt, bt)


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_chain_from(pin):
    pin(_oracle)


def test_chain_from_rejects_bad_arguments():
    toks = _tokens(36, 16 * 3)
    p = bytes(32)
    with pytest.raises(ValueError):
        O.chain_from(toks, 4, p, O.NONE)
    with pytest.raises(ValueError):
        O.chain_from(toks, -1, p, O.NONE)
    with pytest.raises(ValueError):
        O.chain_from(toks, 1, None, O.NONE)
    with pytest.raises(ValueError):
        O.chain_from(toks, 1, b"short", O.NONE)
    with pytest.raises(ValueError):
        O.chain_from(toks, 1, p, O.ROOT)  # no salt


def test_batch_layout_matches_whole_chains():
    """hash_chains_resume's rows are the whole chains' rows from each start."""
    s0, s1 = _salt_pair()
    g = np.random.default_rng(37)
    lens = np.array([0, 15, 16, 40, 16 * 6, 16 * 9 + 7, 33], dtype=np.int64)
    tok_offsets = np.concatenate([[0], np.cumsum(lens)])
    tokens = g.integers(0, VOCAB, int(tok_offsets[-1]), dtype=np.int32)
    principal = g.integers(0, 2, lens.size).astype(np.int32)
    bt = np.minimum(g.integers(0, 200, lens.size), lens).astype(np.int32)
    for mode in (O.NONE, O.ROOT, O.BOUNDARY):
        whole = [O.chain(tokens[tok_offsets[r]:tok_offsets[r + 1]], mode,
                         (s0, s1)[principal[r]] if mode else None,
                         int(bt[r]) if mode == O.BOUNDARY else None) for r in range(lens.size)]
        start = np.array([g.integers(0, len(w) + 1) for w in whole], dtype=np.int32)
        parents = np.zeros((lens.size, 32), dtype=np.uint8)
        for r, w in enumerate(whole):
            if start[r]:
                parents[r] = np.frombuffer(w[start[r] - 1], dtype=np.uint8)
        got = O.hash_chains_resume(tokens, tok_offsets, principal, [s0, s1], mode, start,
                                   parents, bt if mode == O.BOUNDARY else None)
        want = b"".join(b"".join(w[start[r]:]) for r, w in enumerate(whole))
        assert got.tobytes() == want


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def _mut(variant):
    def fn(tokens, j0, parent, mode, salt, bt):
        n_full = len(tokens) // B
        k = 0 if mode == O.ROOT else (bt // B if mode == O.BOUNDARY else None)
        h = bytes(parent) if j0 > 0 else b""
        if variant == "ignore_parent":
            h = b""
        out = []
        first = j0 - 1 if variant == "start_one_early" and j0 > 0 else j0
        for j in range(first, n_full):
            blk = tokens[B * j:B * (j + 1)]
            T = struct.pack("<%di" % len(blk), *[int(x) for x in blk])
            if variant == "boundary_relative":
                salted = k is not None and (j - j0) == k
            elif variant == "salt_at_start":
                salted = (k is not None and j == k) or (mode != O.NONE and j == j0)
            else:
                salted = k is not None and j == k
            if variant == "skip_parent_on_salted" and salted:
                msg = salt + T
            else:
                msg = (salt if salted else b"") + h + T
            h = hashlib.sha256(msg).digest()
            out.append(h)
        return out
    return fn


MUTANTS = ["ignore_parent", "start_one_early", "boundary_relative", "salt_at_start",
           "skip_parent_on_salted"]


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
