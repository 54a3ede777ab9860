"""GPU parity of the admission call (lookup-then-insert in request order)
against the oracle's ``Table.admit``; hit counts, new-block counts, n_new and
the exported key set are compared exactly."""
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
    return torch.from_numpy(np.require(x, requirements=["C", "W"])).cuda()


def key_set(arr):
    a = np.ascontiguousarray(arr, dtype=np.uint8)
    return {a[i].tobytes() for i in range(a.shape[0])}


def check_admit(h, bo, pre=None, log2_slots=16, pre_bo=None):
    """Admit (h, bo) on the GPU into a table holding `pre`, and compare with
    the oracle; returns (hits, new)."""
    T = O.Table()
    with K.Cache(log2_slots) as c:
        if pre is not None and pre.shape[0]:
            pb = pre_bo if pre_bo is not None else np.array([0, pre.shape[0]], np.int64)
            c.insert(dev(pre), dev(pb))
            T.insert(pre, pb)
        hits, new, n_new = c.admit(dev(h), dev(bo))
        hits, new = hits.cpu().numpy(), new.cpu().numpy()
        got_keys = key_set(c.export().cpu().numpy())
        count = c.count()
    before = len(T.keys)
    wh, wn = T.admit(h, bo)
    assert np.array_equal(hits, wh)
    assert np.array_equal(new, wn)
    assert n_new == int(wn.sum()) == len(T.keys) - before
    assert got_keys == T.keys and count == len(T.keys)
    return hits, new


def test_admit_hand_built():
    A, Bk, C, X, Y = (np.full(32, v, np.uint8) for v in (1, 2, 3, 4, 5))
    F = np.full(32, 0xFF, np.uint8)
    reqs = [[A, Bk, A, C], [A, X], [Y, A, Bk], [], [F, F, Y], [C, F, X, A]]
    bo = np.concatenate([[0], np.cumsum([len(q) for q in reqs])]).astype(np.int64)
    h = np.stack([k for q in reqs for k in q])
    hits, new = check_admit(h, bo)
    assert hits.tolist() == [0, 1, 0, 0, 0, 4] and new.tolist() == [3, 1, 1, 0, 1, 0]
    hits, new = check_admit(h, bo, pre=np.stack([Bk, F]))
    assert hits.tolist() == [0, 1, 0, 0, 3, 4] and new.tolist() == [2, 1, 1, 0, 0, 0]


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_admit_key_pool_with_repeats(seed):
    """Arbitrary keys from a small pool (heavy repeats inside and across
    requests, the all-0xFF key among them), some present before the call."""
    g = np.random.default_rng(seed)
    pool = g.integers(0, 256, (60, 32), dtype=np.uint8)
    pool[7] = 0xFF
    lens = g.integers(0, 24, 3000)
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    h = pool[g.integers(0, 60, int(bo[-1]))]
    check_admit(h, bo, pre=pool[g.integers(0, 60, 12)])


def _batch(seed, n, P, prefix, suffix_hi):
    g = np.random.default_rng(seed)
    pre = g.integers(0, VOCAB, prefix, dtype=np.int32)
    suf = g.integers(0, suffix_hi, n)
    lens = prefix + suf
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    for r in range(n):
        toks[offs[r]:offs[r] + prefix] = pre
    prin = g.integers(0, P, n).astype(np.int32)
    bt = np.full(n, prefix, np.int32)
    return Batch(toks, offs, prin, bt)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_admit_shared_prefix_chains(mode):
    """Chains of 3000 requests sharing a 500-token prefix over 7 principals:
    every key of the prefix is claimed by many requests at once."""
    b = _batch(10 + mode, 3000, 7, 500, 400)
    g = np.random.default_rng(11)
    Kb = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
    ids = g.integers(0, 256, (7, 32), dtype=np.uint8)
    sd = K.salts(Kb, dev(ids))
    h = K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), sd, mode,
                      dev(b.boundary_tok)).cpu().numpy()
    want = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                                  b.boundary_tok)
    assert np.array_equal(h, want)
    hits, new = check_admit(want, b.blk_offsets(), log2_slots=20)
    # the first request of each salting domain computes the prefix
    assert (hits >= 500 // 16).sum() >= 3000 - 7


def test_admit_many_short_requests_and_empty():
    g = np.random.default_rng(21)
    pool = g.integers(0, 256, (5000, 32), dtype=np.uint8)
    lens = g.integers(0, 5, 200000)
    bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    h = pool[g.integers(0, 5000, int(bo[-1]))]
    check_admit(h, bo, pre=pool[:100], log2_slots=14)


def test_admit_twice_and_with_lookup():
    """Keys admitted by one call are visible to the next as keys present
    before it; a lookup after admission sees the union."""
    g = np.random.default_rng(31)
    pool = g.integers(0, 256, (300, 32), dtype=np.uint8)
    lens1, lens2 = g.integers(0, 10, 400), g.integers(0, 10, 400)
    bo1 = np.concatenate([[0], np.cumsum(lens1)]).astype(np.int64)
    bo2 = np.concatenate([[0], np.cumsum(lens2)]).astype(np.int64)
    h1 = pool[g.integers(0, 200, int(bo1[-1]))]
    h2 = pool[g.integers(100, 300, int(bo2[-1]))]
    T = O.Table()
    with K.Cache(12) as c:
        for h, bo in ((h1, bo1), (h2, bo2)):
            hits, new, n_new = c.admit(dev(h), dev(bo))
            wh, wn = T.admit(h, bo)
            assert np.array_equal(hits.cpu().numpy(), wh)
            assert np.array_equal(new.cpu().numpy(), wn) and n_new == int(wn.sum())
        got = c.lookup(dev(h1), dev(bo1)).cpu().numpy()
        assert np.array_equal(got, T.lookup(h1, bo1))
        assert np.array_equal(got, np.diff(bo1))


def test_admit_no_requests_and_async():
    with K.Cache(8) as c:
        h = torch.zeros((0, 32), dtype=torch.uint8, device="cuda")
        hits, new, n_new = c.admit(h, dev(np.zeros(1, np.int64)))
        assert n_new == 0 and hits.numel() == 0
        g = np.random.default_rng(41)
        hk = g.integers(0, 256, (50, 32), dtype=np.uint8)
        bo = np.array([0, 20, 20, 50], np.int64)
        hits, new, n_new = c.admit(dev(hk), dev(bo), sync=False)
        assert n_new is None
        assert c.count() == 50
        assert hits.cpu().tolist() == [0, 0, 0] and new.cpu().tolist() == [20, 0, 30]


def test_admit_bad_offsets_latched():
    c_ = K.header_constants()
    g = np.random.default_rng(51)
    hk = dev(g.integers(0, 256, (30, 32), dtype=np.uint8))
    for bo in ([0, 20, 10, 30], [0, 10, 40], [-1, 10, 30]):
        with K.Cache(8) as c:
            hits, new, _ = c.admit(hk, dev(np.array(bo, np.int64)), sync=False)
            with pytest.raises(K.KvgovError) as e:
                c.count()
            assert e.value.code == c_["KVGOV_E_OFFSETS"], bo


def test_admit_table_full_latched():
    c_ = K.header_constants()
    g = np.random.default_rng(61)
    hk = dev(g.integers(0, 256, (40, 32), dtype=np.uint8))
    with K.Cache(4) as c:
        with pytest.raises(K.KvgovError) as e:
            c.admit(hk, dev(np.array([0, 25, 40], np.int64)))
        assert e.value.code == c_["KVGOV_E_FULL"]


def test_concurrent_admission_on_two_streams():
    """Two tables, each on a stream of its own, admit different batches at
    the same time (the per-row codes live in each stream's scratch), three
    rounds with a clear before each, every call asynchronous; each round's
    hits and new blocks equal the oracle's."""
    g = np.random.default_rng(23)
    jobs = []
    for t in range(2):
        fam = g.integers(0, 256, (40, 120, 32), dtype=np.uint8)
        fam[:, :, 0] = 3 + t
        rows, lens = [], []
        for r in range(2500):
            L = int(g.integers(0, 120))
            k = g.integers(0, 256, (L, 32), dtype=np.uint8)
            s_ = int(g.integers(0, L + 1))
            k[:s_] = fam[int(g.integers(0, 40)), :s_]
            rows.append(k)
            lens.append(L)
        h = np.concatenate(rows)
        bo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        wh, wn = O.Table().admit(h, bo)
        jobs.append(dict(h=h, bo=bo, wh=wh, wn=wn))
    streams = [torch.cuda.Stream() for _ in jobs]
    caches = [K.Cache(18) for _ in jobs]
    try:
        dj = [dict(h=dev(j["h"]), bo=dev(j["bo"]),
                   hits=[torch.empty(j["bo"].size - 1, dtype=torch.int32, device="cuda")
                         for _ in range(3)],
                   new=[torch.empty(j["bo"].size - 1, dtype=torch.int32, device="cuda")
                        for _ in range(3)]) for j in jobs]
        torch.cuda.synchronize()
        for rnd in range(3):
            for d, c, s in zip(dj, caches, streams):
                c.clear(stream=s)
                c.admit(d["h"], d["bo"], sync=False, hits=d["hits"][rnd], new=d["new"][rnd],
                        stream=s)
        torch.cuda.synchronize()
        for j, d, c in zip(jobs, dj, caches):
            for rnd in range(3):
                assert np.array_equal(d["hits"][rnd].cpu().numpy(), j["wh"])
                assert np.array_equal(d["new"][rnd].cpu().numpy(), j["wn"])
            assert c.count() == int(j["wn"].sum())
    finally:
        for c in caches:
            c.close()
