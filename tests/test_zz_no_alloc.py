"""The allocation-free hashing entry point (kvgov_hash_chains_noalloc)
against kvgov_hash_chains, through the C ABI: two calls in a row on batches
large enough to be ordered longest first (so the library's fixed scratch
array holds the order), the second smaller than the first, then a batch on
the lane-pair path, in every salt mode.  Outputs must be byte-identical."""
import numpy as np
import pytest
import torch

import workloads as W

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


def batch(n, seed):
    g = np.random.default_rng(seed)
    lens = g.integers(0, 400, n).astype(np.int64)
    lens[g.integers(0, n, 8)] = g.integers(2000, 5000, 8)  # a few long chains
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(0, W.VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 37, n).astype(np.int32)
    bt = np.floor(g.random(n) * (lens + 1)).astype(np.int32)
    return W.Batch(toks, offs, prin, bt)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_noalloc_matches_hash_chains(mode):
    g = np.random.default_rng(3)
    ids = dev(g.integers(0, 256, (37, 32), dtype=np.uint8))
    salts = K.salts(g.integers(0, 256, 32, dtype=np.uint8).tobytes(), ids)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ordered = 128 * cus  # above this many requests the batch is ordered
    for n, seed in ((ordered + 17000, 1), (ordered + 7000, 2), (1000, 3)):
        b = batch(n, seed)
        x = [dev(b.tokens), dev(b.tok_offsets), dev(b.principal), salts, mode,
             dev(b.boundary_tok)]
        bo = dev(b.blk_offsets())
        want = K.hash_chains(*x, blk_offsets=bo)
        out = torch.full_like(want, 0xAB)  # stale bytes must all be overwritten
        status = K.new_status()
        K.hash_chains_noalloc(*x, blk_offsets=bo, out=out, status=status)
        K.check_status(status, "kvgov_hash_chains_noalloc")
        assert torch.equal(out, want), (n, mode)


def test_noalloc_rejects_batches_above_the_limit():
    c = K.header_constants()
    n = c["KVGOV_NOALLOC_MAX_REQUESTS"] + 1
    offs = torch.zeros(n + 1, dtype=torch.int64, device="cuda")
    toks = torch.zeros(16, dtype=torch.int32, device="cuda")
    out = torch.empty((0, 32), dtype=torch.uint8, device="cuda")
    with pytest.raises(K.KvgovError) as e:
        K.hash_chains_noalloc(toks, offs, None, None, W.NONE, None, blk_offsets=offs, out=out,
                              status=K.new_status())
    assert e.value.code == c["KVGOV_E_TOO_LARGE"]
