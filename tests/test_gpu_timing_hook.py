"""kvgov_time_next_chain_kernel on the GPU: the events it hands to the next
chain call bracket the chain kernel alone (inside the call's own span), on
the lane-pair path and on the ordered mixed path, and timing a call changes
none of its output bytes; the pair is used once."""
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
    K.time_next_chain_kernel(None, None)
    torch.cuda.synchronize()


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def batch(n, seed):
    g = np.random.default_rng(seed)
    lens = g.integers(0, 600, n).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(0, W.VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 11, n).astype(np.int32)
    bt = np.floor(g.random(n) * (lens + 1)).astype(np.int32)
    return W.Batch(toks, offs, prin, bt)


def ev():
    return torch.cuda.Event(enable_timing=True)


@pytest.mark.parametrize("ordered", [False, True])
def test_events_bracket_the_chain_kernel(ordered):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 128 * cus + 5000 if ordered else 3000
    b = batch(n, 7 + int(ordered))
    g = np.random.default_rng(1)
    salts = K.salts(g.integers(0, 256, 32, dtype=np.uint8).tobytes(),
                    dev(g.integers(0, 256, (11, 16), dtype=np.uint8)))
    x = [dev(b.tokens), dev(b.tok_offsets), dev(b.principal), salts, W.BOUNDARY,
         dev(b.boundary_tok)]
    bo = dev(b.blk_offsets())
    want = K.hash_chains(*x, blk_offsets=bo)
    c0, c1, k0, k1 = ev(), ev(), ev(), ev()
    K.time_next_chain_kernel(k0, k1)
    c0.record()
    got = K.hash_chains(*x, blk_offsets=bo)
    c1.record()
    torch.cuda.synchronize()
    assert torch.equal(got, want)
    kernel, call = k0.elapsed_time(k1), c0.elapsed_time(c1)
    assert 0 < kernel <= call, (kernel, call)
    assert c0.elapsed_time(k0) >= 0 and k1.elapsed_time(c1) >= 0
    # used once: the next call records nothing, so the pair keeps its times
    again = K.hash_chains(*x, blk_offsets=bo)
    torch.cuda.synchronize()
    assert torch.equal(again, want)
    assert k0.elapsed_time(k1) == kernel
