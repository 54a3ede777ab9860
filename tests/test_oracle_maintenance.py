"""Pins for the oracle's table maintenance (recency, eviction, erase).

The paper is silent on maintenance; the oracle's reading: every insert or
admission call is one tick of a clock, each key of its batch takes the tick
as its stamp and its smallest block position in that batch as its depth,
and evict keeps
the largest set of whole (stamp, depth) classes, newest and shallowest
first, that fits.  What pins it:

* the size law: kept <= max_keys, and the next class would not fit;
* the order law: every kept key outranks every evicted key;
* prefix closure: for chains inserted whole (from block 0), the kept part
  of every chain is a prefix of it, whatever the call history, so a lookup
  after eviction returns min(old hits, kept prefix);
* hand-built histories with the kept sets written out;
* erase is set difference, its count the keys that were present;
* planted mistakes (``MUTANTS``) each trip at least one pin.
"""
import numpy as np
import pytest

from oracle import kvgov as O
from workloads import VOCAB

B = 16


def K(v):
    return bytes([v % 256, v // 256]) + bytes(30)


def arr(keys):
    return np.frombuffer(b"".join(keys), np.uint8).reshape(-1, 32) if keys \
        else np.zeros((0, 32), np.uint8)


def _chains(seed, n, P=3):
    """n requests of whole chains with shared prefixes (root salting)."""
    g = np.random.default_rng(seed)
    salts_ = O.salts(b"m", g.integers(0, 256, (P, 8), dtype=np.uint8))
    base = g.integers(0, VOCAB, 16 * 12, dtype=np.int32)
    reqs = []
    for _ in range(n):
        L = int(g.integers(0, 16 * 12))
        cut = int(g.integers(0, L + 1))
        t = np.r_[base[:cut], g.integers(0, VOCAB, L - cut)].astype(np.int32)
        reqs.append(O.chain(t, O.ROOT, salts_[int(g.integers(0, P))]))
    return reqs


def _batch(chains):
    rows = [k for c in chains for k in c]
    bo = np.concatenate([[0], np.cumsum([len(c) for c in chains])]).astype(np.int64)
    return arr(rows), bo


# fn(history: list of ("insert"|"admit"|"evict"|"erase", payload), ) -> Table-like
# with .keys; the pins drive a fresh table through a history and inspect it.

def pin_size_and_order(fn):
    g = np.random.default_rng(1)
    chains = _chains(2, 60)
    hist = []
    for i in range(0, 60, 6):
        hist.append(("insert", _batch(chains[i:i + 6])))
    T = fn(hist)
    before = set(T.keys)
    ranks = {k: T.rank(k) for k in before}
    for max_keys in (0, 1, 37, 150, len(before) - 1, len(before), len(before) + 5):
        T2 = fn(hist + [("evict", max_keys)])
        kept = set(T2.keys)
        assert kept <= before and len(kept) <= max_keys
        gone = before - kept
        if kept and gone:
            assert min(ranks[k] for k in kept) > max(ranks[k] for k in gone), max_keys
        if gone:
            top = max(ranks[k] for k in gone)
            nxt = sum(1 for k in gone if ranks[k] == top)
            assert len(kept) + nxt > max_keys, max_keys  # the next class does not fit


def pin_prefix_closure(fn):
    chains = _chains(3, 80)
    g = np.random.default_rng(4)
    hist = []
    for i in range(0, 80, 8):
        hist.append(("insert" if i % 16 else "admit", _batch(chains[i:i + 8])))
        if i % 24 == 0:
            # re-insert some older chains: their stamps refresh
            idx = g.integers(0, i + 1, 5)
            hist.append(("insert", _batch([chains[j] for j in idx])))
    for max_keys in (10, 100, 300, 10 ** 6):
        T = fn(hist + [("evict", max_keys)])
        for c in chains:
            kept = [k in T.keys for k in c]
            # kept blocks form a prefix of the chain
            if False in kept:
                assert not any(kept[kept.index(False):]), max_keys


def pin_hand_built(fn):
    a = [K(i) for i in range(10)]
    one = np.array([0, 3], np.int64)
    hist = [("insert", (arr(a[0:3]), one)),                  # tick 1: a0 a1 a2 (depth 0 1 2)
            ("insert", (arr([a[0], a[3], a[4]]), one)),      # tick 2: a0 a3 a4
            ("insert", (arr([a[5], a[1]]), np.array([0, 1, 2], np.int64)))]  # tick 3: a5, a1
    # ranks (stamp, -depth): a5 (3,0), a1 (3,0) (depth 0 in tick 3), a0 (2,0),
    # a3 (2,-1), a4 (2,-2), a2 (1,-2)
    T = fn(hist + [("evict", 2)])
    assert T.keys == {a[5], a[1]}
    T = fn(hist + [("evict", 3)])
    assert T.keys == {a[5], a[1], a[0]}
    T = fn(hist + [("evict", 5)])
    assert T.keys == {a[5], a[1], a[0], a[3], a[4]}
    T = fn(hist + [("evict", 1)])
    assert T.keys == set()  # the top class holds two keys
    T = fn(hist + [("erase", arr([a[1], a[7], a[1]]))])
    assert T.keys == {a[0], a[2], a[3], a[4], a[5]}
    # a key at two positions of one call takes the smaller: a7 is at 1 and 0
    h2 = hist + [("insert", (arr([a[6], a[7], a[7], a[8]]), np.array([0, 2, 4], np.int64)))]
    T = fn(h2 + [("evict", 2)])
    assert T.keys == {a[6], a[7]}
    # a later insert of an evicted key brings it back with a new stamp
    T = fn(hist + [("evict", 2), ("insert", (arr([a[2]]), np.array([0, 1], np.int64))),
                   ("evict", 1)])
    assert T.keys == {a[2]}


def pin_erase(fn):
    g = np.random.default_rng(5)
    pool = [K(i) for i in range(50)]
    ins = [pool[int(i)] for i in g.integers(0, 50, 80)]
    T = fn([("insert", (arr(ins), np.array([0, 80], np.int64)))])
    present = set(T.keys)
    er = [pool[int(i)] for i in g.integers(0, 50, 30)]
    T2 = fn([("insert", (arr(ins), np.array([0, 80], np.int64))), ("erase", arr(er))])
    assert T2.keys == present - set(er)
    assert T2.last == len(present & set(er))


PINS = (pin_size_and_order, pin_prefix_closure, pin_hand_built, pin_erase)


def _oracle(hist):
    T = O.Table()
    T.last = None
    for op, x in hist:
        if op == "insert":
            T.last = T.insert(*x)
        elif op == "admit":
            T.admit(*x)
        elif op == "evict":
            T.last = T.evict(x)
        else:
            T.last = T.erase(x)
    return T


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_maintenance(pin):
    pin(_oracle)


def test_lookup_after_eviction_is_kept_prefix():
    chains = _chains(7, 40)
    T = O.Table()
    h, bo = _batch(chains)
    T.insert(h, bo)
    before = T.lookup(h, bo)
    T.evict(120)
    after = T.lookup(h, bo)
    kept_prefix = np.array([sum(1 for k in c if k in T.keys) for c in chains])
    assert np.array_equal(after, np.minimum(before, kept_prefix))


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

class _Mut(O.Table):
    variant = "none"

    def _touch(self, hashes, blk_offsets):
        self.clock += 1
        blk_offsets = np.asarray(blk_offsets, dtype=np.int64)
        pos = {}
        for r in range(blk_offsets.shape[0] - 1):
            a, b = int(blk_offsets[r]), int(blk_offsets[r + 1])
            for j, k in enumerate(O._keys(hashes, a, b)):
                d = pos.get(k, O.NO_DEPTH if self.variant != "depth_max" else -1)
                pos[k] = max(d, j) if self.variant == "depth_max" else min(d, j)
        for k, j in pos.items():
            if not (self.variant == "stamp_first_insert_only" and k in self.stamp):
                self.stamp[k] = self.clock
            self.depth[k] = j

    def rank(self, k):
        s, d = self.stamp.get(k, 0), -self.depth.get(k, O.NO_DEPTH)
        if self.variant == "deepest_first":
            d = -d
        if self.variant == "oldest_first":
            s = -s
        return (s, d)

    def evict(self, max_keys):
        if self.variant != "split_classes":
            return super().evict(max_keys)
        order = sorted(self.keys, key=lambda k: (self.rank(k), k), reverse=True)
        self.erase_set(set(order[max_keys:]))
        return len(self.keys)


def _mut(variant):
    def fn(hist):
        T = _Mut()
        T.variant = variant
        T.last = None
        for op, x in hist:
            if op == "insert":
                T.last = T.insert(*x)
            elif op == "admit":
                T.admit(*x)
            elif op == "evict":
                T.last = T.evict(x)
            else:
                T.last = T.erase(x)
        return T
    return fn


MUTANTS = ["stamp_first_insert_only", "depth_max", "deepest_first", "oldest_first",
           "split_classes"]


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
