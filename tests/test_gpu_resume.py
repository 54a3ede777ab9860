"""GPU parity of chain extension (resume from a parent digest and a start
block) against the oracle's ``chain_from``; bit-exact.

Parents are either arbitrary 32-byte strings (the resumed chain is then
defined by the recurrence alone) or the oracle's own digests of the whole
chain, so that the resumed rows must equal the whole chain's suffix.
"""
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


def ragged(seed, lens, P=4):
    g = np.random.default_rng(seed)
    lens = np.asarray(lens, dtype=np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(0, VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, P, lens.size).astype(np.int32)
    bt = np.floor(g.random(lens.size) * (lens + 1)).astype(np.int32)
    return Batch(toks, offs, prin, bt)


def secret(seed, P):
    g = np.random.default_rng(2000 + seed)
    return g.integers(0, 256, 32, dtype=np.uint8).tobytes(), \
        g.integers(0, 256, (P, 32), dtype=np.uint8)


def resume_offsets_np(lens, start):
    return np.concatenate([[0], np.cumsum(lens // 16 - start)]).astype(np.int64)


def gpu_resume(b, sd, mode, start, parents, **kw):
    return K.hash_chains_resume(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), sd, mode,
                                dev(start), dev(parents), dev(b.boundary_tok), **kw)


def oracle_resume(b, osalts, mode, start, parents):
    return O.hash_chains_resume(b.tokens, b.tok_offsets, b.principal, osalts, mode, start,
                                parents, b.boundary_tok)


def test_resume_offsets():
    g = np.random.default_rng(3)
    for n in (0, 1, 1023, 1025, 70000):
        lens = g.integers(0, 300, n).astype(np.int64)
        start = np.floor(g.random(n) * (lens // 16 + 1)).astype(np.int32)
        offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        got = K.resume_offsets(dev(offs), dev(start)).cpu().numpy()
        assert np.array_equal(got, resume_offsets_np(lens, start)), n


def test_resume_offsets_bad_start_latched():
    offs = np.array([0, 40, 80, 100], dtype=np.int64)
    for bad in (3, -1):
        start = np.array([0, bad, 1], dtype=np.int32)
        with pytest.raises(K.KvgovError) as e:
            K.resume_offsets(dev(offs), dev(start))
        assert e.value.code == K.header_constants()["KVGOV_E_OFFSETS"]


EDGE_LENS = [0, 15, 16, 17, 32, 33, 64, 65, 160, 161, 500, 1024]


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_resume_edge_starts(mode):
    """Start blocks 0, 1, k - 1, k, k + 1, the last block and n_full (nothing
    to hash), with boundaries at 0, inside, on a block edge and past the end;
    arbitrary parents."""
    lens = EDGE_LENS * 7 * 5
    b = ragged(71 + mode, lens)
    L = b.lengths
    nf = L // 16
    n = len(lens)
    start = np.zeros(n, np.int32)
    for i in range(n):
        bk = (i // len(EDGE_LENS)) % 5
        b.boundary_tok[i] = [0, min(15, L[i]), min(16, L[i]), L[i] // 2, L[i]][bk]
        k = b.boundary_tok[i] // 16
        sk = i // (len(EDGE_LENS) * 5)
        start[i] = int(np.clip([0, 1, k - 1, k, k + 1, nf[i] - 1, nf[i]][sk], 0, nf[i]))
    parents = np.random.default_rng(5).integers(0, 256, (n, 32), dtype=np.uint8)
    Kb, ids = secret(1, 4)
    got = gpu_resume(b, K.salts(Kb, dev(ids)), mode, start, parents).cpu().numpy()
    want = oracle_resume(b, O.salts(Kb, ids), mode, start, parents)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_resume_equals_whole_chain_suffix(mode):
    """Parents taken from the oracle's whole chains: the resumed rows are the
    whole chains' rows from each start block."""
    g = np.random.default_rng(81)
    lens = g.integers(0, 700, 3000)
    b = ragged(82 + mode, lens, P=9)
    Kb, ids = secret(2, 9)
    osalts = O.salts(Kb, ids)
    whole = O.hash_chains_parallel(b.tokens, b.tok_offsets, b.principal, osalts, mode,
                                   b.boundary_tok)
    nf = b.lengths // 16
    start = np.floor(g.random(lens.size) * (nf + 1)).astype(np.int32)
    wo = np.concatenate([[0], np.cumsum(nf)])
    parents = np.zeros((lens.size, 32), np.uint8)
    keep = np.zeros(whole.shape[0], bool)
    for r in range(lens.size):
        if start[r]:
            parents[r] = whole[wo[r] + start[r] - 1]
        keep[wo[r] + start[r]:wo[r + 1]] = True
    got = gpu_resume(b, K.salts(Kb, dev(ids)), mode, start, parents).cpu().numpy()
    assert np.array_equal(got, whole[keep])


def test_resume_large_ordered_batch():
    """40000 requests: above the size at which the batch is ordered by the
    blocks left to hash and run on the mixed kernel; starts spread so that the
    order differs from the order by length."""
    g = np.random.default_rng(91)
    n = 40000
    lens = g.integers(0, 400, n)
    b = ragged(92, lens, P=13)
    nf = b.lengths // 16
    start = np.floor(g.random(n) ** 0.5 * (nf + 1)).astype(np.int32)
    start = np.minimum(start, nf).astype(np.int32)
    parents = g.integers(0, 256, (n, 32), dtype=np.uint8)
    Kb, ids = secret(3, 13)
    sd = K.salts(Kb, dev(ids))
    osalts = O.salts(Kb, ids)
    for mode in (W.ROOT, W.BOUNDARY):
        got = gpu_resume(b, sd, mode, start, parents).cpu().numpy()
        want = oracle_resume(b, osalts, mode, start, parents)
        assert np.array_equal(got, want), mode


def test_two_turn_session():
    """Turn 2 extends turn 1; turn 1's chains are hashed on the GPU, turn 2
    resumes from its last full block.  Expected: the oracle's whole chain of
    turn 2 from that block on."""
    g = np.random.default_rng(101)
    n = 257
    l1 = g.integers(0, 600, n)
    l2 = l1 + g.integers(0, 300, n)
    t2 = ragged(102, l2, P=5)
    t1_tokens = np.concatenate([t2.tokens[t2.tok_offsets[r]:t2.tok_offsets[r] + l1[r]]
                                for r in range(n)])
    t1 = Batch(t1_tokens, np.concatenate([[0], np.cumsum(l1)]).astype(np.int64),
               t2.principal, np.minimum(t2.boundary_tok, l1).astype(np.int32))
    Kb, ids = secret(4, 5)
    sd = K.salts(Kb, dev(ids))
    osalts = O.salts(Kb, ids)
    for mode in (W.NONE, W.ROOT, W.BOUNDARY):
        # the boundary of turn 2 must not fall in turn 1's full blocks unless
        # turn 1 used the same one; keep turn 2's where turn 1 salted a block
        bt2 = t2.boundary_tok.copy()
        past = bt2 // 16 >= l1 // 16
        t1.boundary_tok[:] = np.where(past, l1, bt2)
        b2 = Batch(t2.tokens, t2.tok_offsets, t2.principal, bt2)
        h1 = K.hash_chains(dev(t1.tokens), dev(t1.tok_offsets), dev(t1.principal), sd, mode,
                           dev(t1.boundary_tok)).cpu().numpy()
        nf1 = l1 // 16
        o1 = np.concatenate([[0], np.cumsum(nf1)])
        parents = np.zeros((n, 32), np.uint8)
        for r in range(n):
            if nf1[r]:
                parents[r] = h1[o1[r + 1] - 1]
        start = nf1.astype(np.int32)
        got = gpu_resume(b2, sd, mode, start, parents).cpu().numpy()
        want = b"".join(b"".join(O.chain(t2.tokens[t2.tok_offsets[r]:t2.tok_offsets[r + 1]],
                                         mode, osalts[t2.principal[r]] if mode else None,
                                         int(bt2[r]) if mode == W.BOUNDARY else None)[nf1[r]:])
                        for r in range(n))
        assert got.tobytes() == want, mode


def test_resume_bad_start_skips_the_request():
    c = K.header_constants()
    b = ragged(111, [64, 64, 64, 64])
    Kb, ids = secret(5, 4)
    sd = K.salts(Kb, dev(ids))
    start = np.array([1, 2, 0, 3], np.int32)
    parents = np.random.default_rng(6).integers(0, 256, (4, 32), dtype=np.uint8)
    want = oracle_resume(b, O.salts(Kb, ids), W.ROOT, start, parents)
    bo = resume_offsets_np(b.lengths, start)
    for bad in (5, -1):
        s2 = start.copy()
        s2[2] = bad
        status = K.new_status()
        out = torch.full((int(bo[-1]), 32), 7, dtype=torch.uint8, device="cuda")
        gpu_resume(b, sd, W.ROOT, s2, parents, blk_offsets=dev(bo), out=out, status=status,
                   check=False)
        assert int(status.item()) == c["KVGOV_E_OFFSETS"], bad
        o = out.cpu().numpy()
        assert np.array_equal(o[:5], want[:5]) and np.array_equal(o[9:], want[9:])
        assert np.all(o[5:9] == 7)


def test_resume_from_zero_ignores_parents():
    b = ragged(121, [0, 16, 100, 333, 64])
    Kb, ids = secret(6, 4)
    sd = K.salts(Kb, dev(ids))
    start = np.zeros(5, np.int32)
    parents = np.full((5, 32), 0xAB, np.uint8)
    for mode in (W.NONE, W.ROOT, W.BOUNDARY):
        got = gpu_resume(b, sd, mode, start, parents).cpu().numpy()
        full = K.hash_chains(dev(b.tokens), dev(b.tok_offsets), dev(b.principal), sd, mode,
                             dev(b.boundary_tok)).cpu().numpy()
        want = O.hash_chains(b.tokens, b.tok_offsets, b.principal, O.salts(Kb, ids), mode,
                             b.boundary_tok)
        assert np.array_equal(got, want) and np.array_equal(full, want)
