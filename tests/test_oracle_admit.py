"""Pins for the oracle's admission (lookup-then-insert in request order).

``Table.admit`` takes the requests of a batch one after another: request r
is looked up against the table holding everything inserted before the call
and every key of requests 0..r-1, then its keys join the table.  What pins
it:

* brute force without hashing: for chains, the keys of request r present
  when it comes are exactly its first m blocks, m = the longest run of
  leading token blocks (with matching salt regime) shared with any earlier
  request or any request inserted before; so hits = m and new = n_r - m;
* a one-request batch is a lookup followed by an insert;
* the final key set and the total of new keys equal a plain insert's, for
  any request order;
* hand-built batches of arbitrary keys (repeats inside a request, a miss
  followed by present keys, the all-0xFF key) with their values written out;
* planted mistakes (``MUTANTS``) each trip at least one of these pins.
"""
import numpy as np
import pytest

from oracle import kvgov as O
from tests.test_oracle_chain import _lcp_batches, B

# ---------------------------------------------------------------------------
# brute force
# ---------------------------------------------------------------------------

INF = 1 << 30


def _lcp(a, b, mode):
    """Leading blocks shared by requests a and b = (tokens, principal,
    boundary_tok), salt regimes included (as in the lookup brute force)."""
    (at, ap, ab), (bt, bp, bb) = a, b
    ka = INF if mode == O.NONE else (0 if mode == O.ROOT else ab // B)
    kb = INF if mode == O.NONE else (0 if mode == O.ROOT else bb // B)
    m = 0
    while m < min(len(at), len(bt)) // B:
        same = np.array_equal(at[B * m:B * (m + 1)], bt[B * m:B * (m + 1)])
        regime = (m < ka and m < kb) or (m >= ka and m >= kb and ka == kb and ap == bp)
        if not (same and regime):
            break
        m += 1
    return m


def brute_force_admit(batch, resident, mode):
    hits, new = [], []
    for i, q in enumerate(batch):
        best = max([_lcp(q, r, mode) for r in list(resident) + list(batch[:i])] or [0])
        hits.append(best)
        new.append(len(q[0]) // B - best)
    return np.array(hits, np.int32), np.array(new, np.int32)


def _hashes(reqs, mode, salts_):
    rows, lens = [], []
    for t, p, b in reqs:
        h = O.chain(t, mode, salts_[p] if mode != O.NONE else None,
                    b if mode == O.BOUNDARY else None)
        rows.extend(h)
        lens.append(len(h))
    arr = np.frombuffer(b"".join(rows), dtype=np.uint8).reshape(-1, 32) if rows \
        else np.zeros((0, 32), np.uint8)
    return arr, np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


# ---------------------------------------------------------------------------
# pins, parameterised by the admission under test:
#   fn(keys_before: set, hashes, blk_offsets) -> (hits, new, keys_after)
# ---------------------------------------------------------------------------

def pin_brute_force(fn):
    g = np.random.default_rng(5)
    salts_ = O.salts(bytes(range(32)), g.integers(0, 256, (3, 32), dtype=np.uint8))
    for seed in (1, 2, 3):
        res, qry = _lcp_batches(seed)
        batch = qry + res[:4]  # also copies of residents, and repeats in the batch
        for mode in (O.NONE, O.ROOT, O.BOUNDARY):
            rh, rbo = _hashes(res[4:], mode, salts_)
            keys = O.Table()
            keys.insert(rh, rbo)
            qh, qbo = _hashes(batch, mode, salts_)
            hits, new, _ = fn(set(keys.keys), qh, qbo)
            wh, wn = brute_force_admit(batch, res[4:], mode)
            assert np.array_equal(hits, wh), (seed, mode)
            assert np.array_equal(new, wn), (seed, mode)
            assert (wh > 0).any() and (wn > 0).any()


def pin_single_request_is_lookup_then_insert(fn):
    g = np.random.default_rng(6)
    pre = g.integers(0, 256, (40, 32), dtype=np.uint8)
    T = O.Table()
    T.insert(pre)
    for trial in range(6):
        n = int(g.integers(0, 12))
        rows = [pre[int(i)] for i in g.integers(0, 40, n)]
        rows += [g.integers(0, 256, 32, dtype=np.uint8) for _ in range(int(g.integers(0, 4)))]
        order = g.permutation(len(rows))
        h = np.array([rows[i] for i in order], np.uint8).reshape(-1, 32)
        bo = np.array([0, h.shape[0]], np.int64)
        T2 = O.Table()
        T2.keys = set(T.keys)
        want_hits = T2.lookup(h, bo)
        want_new = T2.insert(h, bo)
        hits, new, after = fn(set(T.keys), h, bo)
        assert hits.tolist() == want_hits.tolist(), trial
        assert new.tolist() == [want_new], trial
        assert after == T2.keys


def pin_total_matches_insert(fn):
    g = np.random.default_rng(7)
    pool = g.integers(0, 256, (30, 32), dtype=np.uint8)
    for trial in range(5):
        lens = g.integers(0, 8, 9)
        bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        h = pool[g.integers(0, 30, int(bo[-1]))]
        pre = set(O._keys(pool[:5]))
        T = O.Table()
        T.keys = set(pre)
        n_ins = T.insert(h, bo)
        for perm in (np.arange(9), g.permutation(9)):
            hp = np.concatenate([h[bo[r]:bo[r + 1]] for r in perm]) if bo[-1] else h
            bp = np.concatenate([[0], np.cumsum(lens[perm])]).astype(np.int64)
            hits, new, after = fn(set(pre), hp, bp)
            assert int(new.sum()) == n_ins and after == T.keys, trial


def pin_hand_built(fn):
    A, Bk, C, X, Y = (bytes([v]) * 32 for v in (1, 2, 3, 4, 5))
    F = b"\xff" * 32

    def arr(keys):
        return np.frombuffer(b"".join(keys), np.uint8).reshape(-1, 32)
    # request 0: A B A C   (A repeated inside the request)
    # request 1: A X       (A from request 0, X new)
    # request 2: Y A B     (Y new: miss at 0, then A, B present)
    # request 3: (empty)
    # request 4: F F Y     (the all-0xFF key twice, Y from request 2)
    # request 5: C F X A   (all present)
    reqs = [[A, Bk, A, C], [A, X], [Y, A, Bk], [], [F, F, Y], [C, F, X, A]]
    bo = np.concatenate([[0], np.cumsum([len(q) for q in reqs])]).astype(np.int64)
    h = arr([k for q in reqs for k in q])
    hits, new, after = fn(set(), h, bo)
    assert hits.tolist() == [0, 1, 0, 0, 0, 4]
    assert new.tolist() == [3, 1, 1, 0, 1, 0]
    assert after == {A, Bk, C, X, Y, F}
    # with B and F present before the call: request 4 now hits F, F and Y
    hits, new, after = fn({Bk, F}, h, bo)
    assert hits.tolist() == [0, 1, 0, 0, 3, 4]
    assert new.tolist() == [2, 1, 1, 0, 0, 0]


PINS = (pin_brute_force, pin_single_request_is_lookup_then_insert, pin_total_matches_insert,
        pin_hand_built)


def _oracle(keys, h, bo):
    T = O.Table()
    T.keys = set(keys)
    hits, new = T.admit(h, bo)
    return hits, new, T.keys


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_admit(pin):
    pin(_oracle)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def _mut(variant):
    def fn(keys, h, bo):
        T = set(keys)
        n = bo.shape[0] - 1
        hits = np.zeros(n, np.int32)
        new = np.zeros(n, np.int32)
        if variant == "pre_batch_visibility":
            snapshot = set(T)
        for r in range(n):
            ks = [h[i].tobytes() for i in range(int(bo[r]), int(bo[r + 1]))]
            if variant == "insert_before_lookup":
                T |= set(ks)
            seen = snapshot if variant == "pre_batch_visibility" else T
            j = 0
            while j < len(ks) and ks[j] in seen:
                j += 1
            hits[r] = j
            if variant == "new_counts_repeats":
                new[r] = sum(1 for k in ks if k not in T)
            elif variant == "new_is_rows_after_first_miss":
                new[r] = len(ks) - j
            else:
                new[r] = len(set(ks) - T)
            T |= set(ks)
        return hits, new, T
    return fn


MUTANTS = ["pre_batch_visibility", "insert_before_lookup", "new_counts_repeats",
           "new_is_rows_after_first_miss"]


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
