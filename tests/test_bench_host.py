"""Host-side arithmetic of bench.py (no GPU): the algorithmic work and bytes
the rooflines divide by, the traffic records they read, and the one-GPU
guard.  Each figure is recomputed here from its definition (by brute force
over small seeded batches where it depends on the inputs), not by calling
the formula it checks."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _sha256_blocks(msg_len: int) -> int:
    """Compressions SHA-256 runs on a message of msg_len bytes (FIPS 180-4
    padding: a 0x80 byte and the 8-byte length, then zeros to a multiple of
    64 bytes)."""
    return (msg_len + 1 + 8 + 63) // 64


def _brute_compressions(batch: W.Batch, mode: int, start=None) -> int:
    """The definition walked block by block: a block's message is its 64
    token bytes, after the parent digest (32 B) when it has one, after the
    salt (32 B) when it is salted."""
    total = 0
    for r in range(batch.n):
        n_full = int(batch.lengths[r]) // 16
        k = int(batch.boundary_tok[r]) // 16
        j0 = 0 if start is None else int(start[r])
        for j in range(j0, n_full):
            salted = (mode == W.ROOT and j == 0) or (mode == W.BOUNDARY and j == k)
            msg = 64 + (32 if j > 0 else 0) + (32 if salted else 0)
            total += _sha256_blocks(msg)
    return total


def _ragged(seed, n, max_len):
    g = np.random.default_rng(seed)
    lens = g.integers(0, max_len, n).astype(np.int64)
    lens[:4] = [0, 15, 16, 33]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = g.integers(0, W.VOCAB, int(offs[-1]), dtype=np.int32)
    prin = g.integers(0, 3, n).astype(np.int32)
    bt = np.floor(g.random(n) * (lens + 1)).astype(np.int32)
    bt[4:8] = 0  # k = 0: the first block is the salted one
    return W.Batch(toks, offs, prin, bt)


@pytest.mark.parametrize("mode", [W.NONE, W.ROOT, W.BOUNDARY])
def test_compressions_match_the_definition(mode):
    b = _ragged(1, 300, 700)
    wl = W.Workload("paper", b"", np.zeros((3, 32), np.uint8), b, None, [mode], 10, {})
    assert bench.compressions(wl, b, mode) == _brute_compressions(b, mode)


def test_compressions_of_resumed_chains():
    """A resumed request hashes its blocks from the start block on; its
    boundary block costs the extra compression only at or after it."""
    b = _ragged(2, 200, 600)
    g = np.random.default_rng(3)
    start = np.minimum(g.integers(0, 20, b.n), b.lengths // 16).astype(np.int64)
    wl = W.Workload("session", b"", np.zeros((3, 32), np.uint8), b, None, [W.BOUNDARY], 10,
                    {"start": start})
    for mode in (W.ROOT, W.BOUNDARY):
        assert bench.compressions(wl, b, mode) == _brute_compressions(b, mode, start)


def test_compression_op_counts():
    """The per-compression op counts the fractions use, from the operation
    counts of the FIPS 180-4 round and schedule: a big sigma is two xors of
    three rotates, a small sigma two xors of two rotates and a shift."""
    big_sigma, small_sigma = 3 + 2, 3 + 2
    choose, majority = 1, 2      # one bit-select; and-xor with the shared term
    t1, e_new, a_new = 2, 1, 1   # two 3-input adds; d + T1; T1 + T2 as one 3-input add
    per_round = 2 * big_sigma + choose + majority + t1 + e_new + a_new
    per_word = 2 * small_sigma + 2  # two 3-input adds
    assert 64 * per_round + 48 * per_word + 8 == bench.OPS_PER_COMPRESSION
    # gfx950: xor3 makes each sigma 3 rotates + 1 op, bitop3 makes the
    # majority one op
    per_round_3 = 2 * (3 + 1) + 1 + 1 + t1 + e_new + a_new
    per_word_3 = 2 * (3 + 1) + 2
    assert 64 * per_round_3 + 48 * per_word_3 + 8 == bench.OPS_PER_COMPRESSION_GFX950


def test_lookup_bytes_by_brute_force():
    """Per request: every block up to and including the first absent one
    (none past the last), 64 bytes each, plus 20 bytes of offsets and
    result."""
    g = np.random.default_rng(4)
    counts = g.integers(0, 50, 500)
    hits = np.array([int(g.integers(0, c + 1)) for c in counts])
    want = 0
    for c, h in zip(counts, hits):
        examined = 0
        for j in range(c):
            examined += 1
            if j == h:  # the first absent block
                break
        want += 64 * examined + 20
    assert bench.lookup_bytes(counts, hits) == want


def test_recorded_traffic_follows_the_sources(monkeypatch):
    """A record is used only while the kernel sources hash to the value it
    was taken with."""
    with open(bench.TRAFFIC_RECORD) as f:
        rows = [l for l in f if l.startswith("| `")]
    current = {bench.sources_sha256(gname): gname for gname in bench.KERNEL_SOURCES}
    for row in rows:
        cells = [c.strip().strip("`") for c in row.strip().strip("|").split("|")]
        if cells[2] in current:
            break
    else:
        pytest.skip("no record was taken on the present sources")
    kernel, workload, sha, fetch, write = cells[:5]
    group = current[sha]
    # the group hash is SHA-256 over the group's files in order
    h = hashlib.sha256()
    for fname in bench.KERNEL_SOURCES[group]:
        with open(os.path.join(ROOT, "paper_2608_09225_amd", "csrc", fname), "rb") as fh:
            h.update(fh.read())
    assert h.hexdigest() == sha
    got = bench.recorded_traffic(kernel, workload, group)
    assert got == {"fetch_bytes": int(fetch), "write_bytes": int(write),
                   "bytes": int(fetch) + int(write)}
    monkeypatch.setattr(bench, "sources_sha256", lambda g: "0" * 64)
    assert bench.recorded_traffic(kernel, workload, group) is None
    assert bench.recorded_traffic("no_such_kernel", workload, group) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]
