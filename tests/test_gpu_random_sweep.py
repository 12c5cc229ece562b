"""GPU parity over a seeded random sweep of shapes: row widths from 1 to 700 words, cluster
sizes from 1 to past the row count, every value structure of the test generators, both
schemes, every payload placement, ranges and gathers with duplicates, unsorted ids and
ragged tails, and the compressed cache on zero-copy handles. Each case decodes the oracle's
stream on the GPU and compares every row, bit for bit, with the oracle's bit-serial decode
(and the original rows)."""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import structured_rows

pytestmark = pytest.mark.gpu

KINDS = ["random", "identical", "zeros", "ones", "onebit", "alternating", "floats", "specials", "sparse",
         "smallint"]
PLACEMENTS = [ibp.IBP_OPEN_PAYLOAD_DEVICE, ibp.IBP_OPEN_PAYLOAD_HOST, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
              ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED]
N_CASES = 600


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def draw_case(k):
    """Case k of the sweep: shape, structure, scheme and placement from one seeded stream."""
    rng = np.random.default_rng(10_000 + k)
    W = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 65, 100, 127, 128, 129, 200, 256, 257, 400, 512, 513, 700]))
    n = int(rng.integers(1, 400))
    G = int(rng.choice([1, 2, 5, 16, 32, 33, 64, 100, n, n + 7]))
    kind = str(rng.choice(KINDS))
    part = bool(rng.random() < 0.35)
    chunk = 0
    threshold = (1, 1)
    if part:
        divisors = [4 * d for d in range(1, W + 1) if W % d == 0 and d <= 8]
        chunk = int(rng.choice(divisors))
        threshold = [(1, 1), (4, 5), (3, 5), (9, 10)][int(rng.integers(0, 4))]
    flags = int(rng.choice(PLACEMENTS))
    if part and flags == ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED:
        flags = ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY
    return rng, W, n, G, kind, part, chunk, threshold, flags


@pytest.mark.parametrize("k", range(N_CASES))
def test_random_case(torch, k):
    rng, W, n, G, kind, part, chunk, threshold, flags = draw_case(k)
    L = 4 * W
    rows = structured_rows(kind, n, L, seed=k)
    stream = (oracle.compress(rows, G, chunk_bytes=chunk, threshold=threshold) if part
              else oracle.compress(rows, G))
    first = int(rng.integers(0, n))
    count = int(rng.integers(1, n - first + 1))
    ids = rng.integers(0, n, size=int(rng.integers(1, 3 * n + 2))).astype(np.int64)
    if rng.random() < 0.5:
        ids = np.sort(ids)
    say(f"[sweep {k}] W={W} n={n} G={G} kind={kind} part={part} chunk={chunk} T={threshold} flags={flags} "
        f"range=({first},{count}) ids={ids.size}")
    want_range = oracle.decode_rows(stream, np.arange(first, first + count, dtype=np.int64), L)
    want_ids = oracle.decode_rows(stream, ids, L)
    assert np.array_equal(want_range, rows[first:first + count])
    assert np.array_equal(want_ids, rows[ids])
    with ibp.ibp_open(stream, 0, flags) as h:
        out = torch.full((max(count, ids.size) * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")
        ibp.ibp_decompress(h, first, count, out)
        torch.cuda.synchronize()
        got = out[:count * L].cpu().numpy().reshape(count, L)
        assert (out[count * L:].cpu().numpy() == 0xA5).all(), "decompress wrote past its rows"
        assert np.array_equal(got, want_range)
        out.fill_(0xA5)
        if flags != ibp.IBP_OPEN_PAYLOAD_HOST and rng.random() < 0.5:
            ibp.ibp_gather_decompress_device(h, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
        else:
            ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        got = out[:ids.size * L].cpu().numpy().reshape(ids.size, L)
        assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "gather wrote past its rows"
        assert np.array_equal(got, want_ids)
        if flags == ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY and not part and W <= 512:
            # the compressed cache over the same handle: a random third of the rows cached
            cached = np.flatnonzero(rng.random(n) < 1 / 3)
            out.fill_(0xA5)
            with ibp.ibp_cache_create(h, cached) as c:
                ibp.ibp_cache_gather(c, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
                torch.cuda.synchronize()
                st = ibp.ibp_cache_get_stats(c)
            got = out[:ids.size * L].cpu().numpy().reshape(ids.size, L)
            assert np.array_equal(got, want_ids)
            hits = int(np.isin(ids, cached).sum())
            assert st["hits"] == hits and st["misses"] == ids.size - hits
        assert ibp.ibp_device_errors(h) == 0
