"""GPU parity of table maintenance (kvgov_cache_evict / kvgov_cache_erase)
against the oracle's Table: after every step of a history of inserts,
admissions, evictions and erasures, the exported key set, the counts and
later lookups are compared exactly."""
import numpy as np
import pytest
import torch

import oracle as O
from tests.test_oracle_maintenance import K as key_of, arr, _chains, _batch

pytestmark = pytest.mark.gpu

KV = pytest.importorskip("paper_2608_09225_amd.kvgov")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    KV.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def dev(x):
    return torch.from_numpy(np.require(x, requirements=["C", "W"])).cuda()


def key_set(t):
    a = t.cpu().numpy()
    return {a[i].tobytes() for i in range(a.shape[0])}


def replay(hist, log2_slots=16, probes=None):
    """Runs `hist` on a GPU table and on the oracle, checking after each step."""
    T = O.Table()
    with KV.Cache(log2_slots) as c:
        c.set_recency(True)
        for op, x in hist:
            if op == "insert":
                h, bo = x
                assert c.insert(dev(h), dev(bo)) == T.insert(h, bo)
            elif op == "admit":
                h, bo = x
                hits, new, n_new = c.admit(dev(h), dev(bo))
                wh, wn = T.admit(h, bo)
                assert np.array_equal(hits.cpu().numpy(), wh)
                assert np.array_equal(new.cpu().numpy(), wn)
            elif op == "evict":
                assert c.evict(x) == T.evict(x), ("evict", x)
            else:
                assert c.erase(dev(x)) == T.erase(x), "erase"
            assert key_set(c.export()) == T.keys, op
            assert c.count() == len(T.keys)
        if probes is not None:
            h, bo = probes
            assert np.array_equal(c.lookup(dev(h), dev(bo)).cpu().numpy(), T.lookup(h, bo))
    return T


def test_hand_built_history():
    a = [key_of(i) for i in range(10)]
    one = np.array([0, 3], np.int64)
    base = [("insert", (arr(a[0:3]), one)),
            ("insert", (arr([a[0], a[3], a[4]]), one)),
            ("insert", (arr([a[5], a[1]]), np.array([0, 1, 2], np.int64)))]
    for max_keys in (0, 1, 2, 3, 4, 5, 6, 100):
        replay(base + [("evict", max_keys)])
    replay(base + [("erase", arr([a[1], a[7], a[1]]))])
    T = replay(base + [("evict", 2), ("insert", (arr([a[2]]), np.array([0, 1], np.int64))),
                       ("evict", 1)])
    assert T.keys == {a[2]}


def test_chain_history_with_admissions():
    chains = _chains(3, 160)
    g = np.random.default_rng(4)
    hist = []
    for i in range(0, 160, 16):
        hist.append(("insert" if i % 32 else "admit", _batch(chains[i:i + 16])))
        if i % 48 == 0:
            idx = g.integers(0, i + 1, 9)
            hist.append(("insert", _batch([chains[j] for j in idx])))
        if i % 64 == 32:
            hist.append(("evict", int(g.integers(50, 600))))
    hist.append(("evict", 250))
    hist.append(("insert", _batch(chains[:20])))
    hist.append(("erase", arr([k for c in chains[20:40] for k in c[:2]])))
    hist.append(("admit", _batch(chains[40:80])))
    T = replay(hist, probes=_batch(chains))
    # prefix closure of what the last eviction kept, among chains inserted whole
    assert len(T.keys) > 0


def test_arbitrary_keys_repeats_and_all_ff():
    g = np.random.default_rng(5)
    pool = [key_of(i) for i in range(300)] + [b"\xff" * 32]
    hist = []
    for step in range(8):
        lens = g.integers(0, 9, 40)
        bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        rows = [pool[int(i)] for i in g.integers(0, len(pool), int(bo[-1]))]
        hist.append(("insert" if step % 2 else "admit", (arr(rows), bo)))
        if step % 3 == 2:
            hist.append(("evict", int(g.integers(20, 200))))
    hist.append(("erase", arr([pool[-1], pool[0], pool[0], key_of(999)])))
    hist.append(("evict", 0))
    replay(hist, log2_slots=12)


def test_eviction_at_scale():
    """~200k keys over 6 insert calls of whole chains; evictions to several
    sizes, then the table keeps working (insert, lookup)."""
    g = np.random.default_rng(6)
    n = 6000
    lens = g.integers(1, 60, n)
    keys = g.integers(0, 256, (int(lens.sum()), 32), dtype=np.uint8)
    keys[:, 0] = 7  # never the all-0xFF key
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    hist = []
    for k in range(6):
        sel = np.arange(k * 1000, (k + 1) * 1000)
        rows = np.concatenate([keys[bo[r]:bo[r + 1]] for r in sel])
        sb = np.concatenate([[0], np.cumsum(lens[sel])]).astype(np.int64)
        hist.append(("insert", (rows, sb)))
    hist += [("evict", 150000), ("evict", 90000), ("evict", 90000), ("evict", 12345)]
    hist.append(("insert", (keys[:bo[500]], bo[:501])))
    replay(hist, log2_slots=19, probes=(keys, bo))


def test_evict_and_erase_async_then_count():
    g = np.random.default_rng(7)
    h = g.integers(0, 256, (500, 32), dtype=np.uint8)
    with KV.Cache(12) as c:
        c.set_recency(True)
        c.insert(dev(h), dev(np.array([0, 500], np.int64)))
        assert c.evict(100, sync=False) is None
        assert c.erase(dev(h[:10]), sync=False) is None
        n = c.count()
    T = O.Table()
    T.insert(h, np.array([0, 500], np.int64))
    T.evict(100)
    T.erase(h[:10])
    assert n == len(T.keys)


def test_untracked_table_erases_but_does_not_evict():
    c_ = KV.header_constants()
    g = np.random.default_rng(8)
    h = g.integers(0, 256, (300, 32), dtype=np.uint8)
    bo = np.array([0, 300], np.int64)
    with KV.Cache(12) as c:
        c.insert(dev(h), dev(bo))
        with pytest.raises(KV.KvgovError) as e:
            c.evict(10)
        assert e.value.code == c_["KVGOV_E_UNSUPPORTED"]
        assert c.erase(dev(h[:40])) == 40
        assert key_set(c.export()) == {h[i].tobytes() for i in range(40, 300)}
        # switched on later: the tracked keys rank above the untracked ones
        c.set_recency(True)
        c.insert(dev(h[100:150]), dev(np.array([0, 50], np.int64)))
        assert c.evict(50) == 50
        assert key_set(c.export()) == {h[i].tobytes() for i in range(100, 150)}


@pytest.mark.parametrize("op", ["insert", "admit"])
@pytest.mark.parametrize("empties", [False, True])
def test_depth_when_a_stretch_spans_many_requests(empties, op):
    """Every key of a batch of one-block requests (with an empty request
    before each, or not) sits at depth 0, so the batch is one rank class:
    64 consecutive rows then span more requests than a window of 64 request
    starts reaches, and a wrong depth would split the class and change what
    an eviction keeps."""
    n = 1000
    keys = arr([key_of(i) for i in range(n)])
    bo = np.repeat(np.arange(n + 1), 2)[:2 * n + 1] if empties else np.arange(n + 1)
    bo = bo.astype(np.int64)
    replay([(op, (keys, bo)), ("evict", n - 1), (op, (keys, bo)), ("evict", n)],
           log2_slots=12)


@pytest.mark.parametrize("keep", ["all", "all_but_one", "tracked_only"])
def test_untracked_keys_in_a_sparse_table(keep):
    """Keys inserted while tracking is off (recency word 0) form the lowest
    rank class.  In a sparse table most waves of the rank gather hold only
    untracked keys or only tracked ones, and the untracked class must still
    enter the select: evict(count) keeps every key, evict(count - 1) drops
    exactly the untracked class (it no longer fits whole)."""
    untracked = arr([key_of(1000 + i) for i in range(3)])
    tracked = arr([key_of(2000 + i) for i in range(5)])
    bo = np.array([0, 5], np.int64)
    T = O.Table()
    T.keys |= {untracked[i].tobytes() for i in range(3)}  # no recency recorded
    T.insert(tracked, bo)
    max_keys = {"all": 8, "all_but_one": 7, "tracked_only": 5}[keep]
    with KV.Cache(16) as c:
        c.insert(dev(untracked), dev(np.array([0, 3], np.int64)))
        c.set_recency(True)
        c.insert(dev(tracked), dev(bo))
        assert c.count() == 8
        assert c.evict(max_keys) == T.evict(max_keys)
        assert key_set(c.export()) == T.keys
    assert len(T.keys) == (8 if keep == "all" else 5)


def test_clear_resets_recency_of_a_tracked_table():
    """A clear skips the recency words unless a call since the last clear may
    have written them.  Keys ranked by tracked inserts (stamps up to 5), a
    clear, the same keys again untracked and other keys tracked (stamps 1
    and 2): the untracked keys must rank lowest, as if the table were new."""
    a = arr([key_of(3000 + i) for i in range(3)])
    b = arr([key_of(4000 + i) for i in range(5)])
    bo_a = np.array([0, 3], np.int64)
    bo_b = np.array([0, 5], np.int64)
    T = O.Table()
    T.keys |= {a[i].tobytes() for i in range(3)}  # untracked after the clear
    T.insert(b, bo_b)
    with KV.Cache(16) as c:
        c.set_recency(True)
        for _ in range(5):
            c.insert(dev(a), dev(bo_a))
        c.clear()
        c.set_recency(False)
        c.insert(dev(a), dev(bo_a))
        c.set_recency(True)
        c.insert(dev(b), dev(bo_b))
        assert c.evict(5) == T.evict(5)
        assert key_set(c.export()) == T.keys == {b[i].tobytes() for i in range(5)}
        # a table that never tracked: clears skip the words, erasure still exact
    with KV.Cache(12) as c:
        for _ in range(2):
            c.insert(dev(a), dev(bo_a))
            assert c.erase(dev(a[:1])) == 1
            assert key_set(c.export()) == {a[i].tobytes() for i in (1, 2)}
            c.clear()
            assert c.count() == 0


def test_concurrent_maintenance_on_two_streams():
    """Two tables, each on a stream of its own, run their inserts, eviction
    and erase at the same time (every call asynchronous), three times over
    with a clear before each round, as the two modes of the maintenance
    bench step do; then each table holds what the oracle's does and answers
    lookups the same way."""
    g = np.random.default_rng(11)
    jobs = []
    for t in range(2):
        lens = g.integers(1, 80, 3000)
        keys = g.integers(0, 256, (int(lens.sum()), 32), dtype=np.uint8)
        keys[:, 0] = 9 + t  # distinct per table, never the all-0xFF key
        keys[:, 1] = 0
        bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        half = int(bo[1500])
        a = (keys[:half], bo[:1501])
        b = (keys[half:], bo[1500:] - half)
        T = O.Table()
        T.insert(*a)
        T.insert(*b)
        max_keys = len(T.keys) // 2
        T.evict(max_keys)
        erase = keys[:half // 10]
        T.erase(erase)
        jobs.append(dict(a=a, b=b, max_keys=max_keys, erase=erase, T=T, keys=keys, bo=bo))
    streams = [torch.cuda.Stream() for _ in jobs]
    caches = [KV.Cache(18) for _ in jobs]
    try:
        dj = []
        for j in jobs:
            dj.append(dict(a=(dev(j["a"][0]), dev(j["a"][1])), b=(dev(j["b"][0]), dev(j["b"][1])),
                           erase=dev(j["erase"]), keys=dev(j["keys"]), bo=dev(j["bo"])))
        for c in caches:
            c.set_recency(True)
        torch.cuda.synchronize()
        for _ in range(3):
            for j, d, c, s in zip(jobs, dj, caches, streams):
                c.clear(stream=s)
                c.insert(*d["a"], sync=False, stream=s)
                c.insert(*d["b"], sync=False, stream=s)
                c.evict(j["max_keys"], sync=False, stream=s)
                c.erase(d["erase"], sync=False, stream=s)
        torch.cuda.synchronize()
        for j, d, c in zip(jobs, dj, caches):
            assert c.count() == len(j["T"].keys)
            assert key_set(c.export()) == j["T"].keys
            hits = c.lookup(d["keys"], d["bo"]).cpu().numpy()
            assert np.array_equal(hits, j["T"].lookup(j["keys"], j["bo"]))
    finally:
        for c in caches:
            c.close()
