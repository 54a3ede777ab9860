"""GPU parity of the radix index (kvgov_radix_*) against the oracle's
``Radix``: every match length is compared exactly."""
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


def flat(seqs, prin):
    lens = [len(s) for s in seqs]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = np.concatenate([np.asarray(s, np.int32) for s in seqs]) if seqs \
        else np.zeros(0, np.int32)
    return Batch(toks, offs, np.asarray(prin, np.int32), np.zeros(len(seqs), np.int32))


class Run:
    """Both sides of one test: a GPU index and the oracle, same salts.  Use
    as a context manager: the index is freed on exit."""

    def __init__(self, mode, P=5, log2_blocks=16, log2_edges=18, seed=0):
        g = np.random.default_rng(500 + seed)
        self.Kb = g.integers(0, 256, 32, dtype=np.uint8).tobytes()
        self.ids = g.integers(0, 256, (P, 32), dtype=np.uint8)
        self.sd = K.salts(self.Kb, dev(self.ids))
        self.osalts = O.salts(self.Kb, self.ids)
        self.mode = mode
        self.x = K.Radix(log2_blocks, log2_edges)
        self.R = O.Radix()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.x.close()

    def _gpu_args(self, b):
        h = K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), self.sd,
                          self.mode) if self.mode != W.NONE else \
            K.hash_chains(dev(b.tokens), dev(b.tok_offsets), None, None, W.NONE)
        pr = dev(b.principal) if self.mode != W.NONE else None
        sd = self.sd if self.mode != W.NONE else None
        return (dev(b.tokens), dev(b.tok_offsets), pr, sd, self.mode, h,
                dev(b.blk_offsets()))

    def insert(self, b):
        self.x.insert(*self._gpu_args(b))
        self.R.insert(b.tokens, b.tok_offsets, b.principal, self.osalts, self.mode)

    def check(self, b):
        got = self.x.match(*self._gpu_args(b)).cpu().numpy()
        want = self.R.match(b.tokens, b.tok_offsets, b.principal, self.osalts, self.mode)
        assert np.array_equal(got, want), (np.nonzero(got != want)[0][:10],)
        return got


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT])
def test_radix_hand_built(mode):
    base = np.arange(100, 180, dtype=np.int32)
    ins = flat([base[:40], np.r_[base[:20], 7, 7, 7], base[:5], []], [0, 0, 1, 0])
    queries = [base[:40], base[:80], base[:33], base[:16], np.r_[base[:15], 1],
               np.r_[base[:16], 1], np.r_[base[:17], 1], np.r_[base[:20], 7, 7, 7, 7],
               np.r_[base[:20], 7, 8], np.r_[1, base[1:40]], base[:40], base[:3], [],
               base[:40]]
    prin = [0] * 10 + [1, 1, 0, 2]
    with Run(mode) as r:
        r.insert(ins)
        got = r.check(flat(queries, prin))
        want = [40, 40, 33, 16, 15, 16, 17, 23, 21, 0] + ([40, 3, 0, 40] if mode == W.NONE
                                                          else [5, 3, 0, 0])
        assert got.tolist() == want


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT])
def test_radix_divergence_at_every_position(mode):
    """Queries copy an inserted sequence up to token d and then differ, for
    every d across four blocks, under their own and other principals."""
    g = np.random.default_rng(7)
    seqs = [g.integers(0, 50, int(L)).astype(np.int32) for L in g.integers(0, 70, 40)]
    prin = g.integers(0, 5, 40)
    with Run(mode, seed=1) as r:
        r.insert(flat(seqs, prin))
        qs, qp = [], []
        for i, s in enumerate(seqs):
            for d in range(0, len(s) + 2, 3):
                q = np.r_[s[:d], 999, g.integers(0, 50, int(g.integers(0, 20)))].astype(np.int32)
                qs.append(q)
                qp.append(prin[i] if i % 4 else (prin[i] + 1) % 5)
        r.check(flat(qs, qp))


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT])
def test_radix_shared_prefix_batch(mode):
    """3000 requests sharing a 500-token prefix over 7 principals (token
    nodes shared by many sequences are created concurrently), inserted in two
    calls; queries with fresh suffixes and copies of inserted requests cut
    at random points."""
    g = np.random.default_rng(11 + mode)
    pre = g.integers(0, VOCAB, 500, dtype=np.int32)

    def batch(n, seed):
        gg = np.random.default_rng(seed)
        seqs = [np.r_[pre[:int(gg.integers(0, 501))], gg.integers(0, 20, int(gg.integers(0, 300)))]
                .astype(np.int32) for _ in range(n)]
        return seqs, gg.integers(0, 7, n)

    with Run(mode, P=7, log2_blocks=18, log2_edges=21, seed=2) as r:
        s1, p1 = batch(1500, 1)
        s2, p2 = batch(1500, 2)
        r.insert(flat(s1, p1))
        r.insert(flat(s2, p2))
        qs, qp = batch(2000, 3)
        cut = [s[:int(g.integers(0, len(s) + 1))] for s in s1[:500]]
        got = r.check(flat(qs + cut, list(qp) + list(p1[:500])))
        assert (got % 16).any() and (got >= 16).any()


def test_radix_clear_and_stats():
    with Run(W.ROOT, seed=3) as r:
        g = np.random.default_rng(21)
        seqs = [g.integers(0, VOCAB, 37).astype(np.int32) for _ in range(10)]
        b = flat(seqs, [0] * 10)
        r.insert(b)
        blocks, edges = r.x.stats()
        # 5 roots + 2 full blocks per sequence; edges: 15 + 15 + 5 per sequence
        assert blocks == 5 + 20 and edges == 10 * 35
        r.x.clear()
        assert r.x.stats() == (0, 0)
        got = r.x.match(*r._gpu_args(b)).cpu().numpy()
        assert (got == 0).all()


def test_radix_full_table_latched():
    c = K.header_constants()
    with Run(W.NONE, log2_blocks=16, log2_edges=4, seed=4) as r:
        g = np.random.default_rng(31)
        seqs = [g.integers(0, VOCAB, 30).astype(np.int32) for _ in range(4)]
        r.x.insert(*r._gpu_args(flat(seqs, [0] * 4)))
        with pytest.raises(K.KvgovError) as e:
            r.x.stats()
        assert e.value.code == c["KVGOV_E_FULL"]


def test_radix_rejects_boundary_mode_and_bad_offsets():
    c = K.header_constants()
    with Run(W.ROOT, seed=5) as r:
        b = flat([np.arange(40, dtype=np.int32)], [0])
        toks, offs, pr, sd, _, h, bo = r._gpu_args(b)
        with pytest.raises(K.KvgovError) as e:
            r.x.insert(toks, offs, pr, sd, W.BOUNDARY, h, bo)
        assert e.value.code == c["KVGOV_E_UNSUPPORTED"]
        bad = dev(np.array([0, 3], np.int64))  # 2 full blocks given as 3
        r.x.insert(toks, offs, pr, sd, W.ROOT, h, bad)
        with pytest.raises(K.KvgovError) as e:
            r.x.stats()
        assert e.value.code == c["KVGOV_E_OFFSETS"]
