"""The allocation-free host-id gather (ibp_gather_decompress_noalloc) against the
allocating one (ibp_gather_decompress), through the C ABI: bit-exact on two calls in a
row, the second with fewer ids, on every placement whose kernels read the payload in
place; plus its size limit and argument checks, which fire before anything is enqueued.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import structured_rows

pytestmark = pytest.mark.gpu

MAX_IDS = 4 << 20
PLACEMENTS = {"device": ibp.IBP_OPEN_PAYLOAD_DEVICE, "zero_copy": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
              "zero_copy_aligned": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def _out(torch, n, L):
    return torch.full((n * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")


CASES = [("floats", 3000, 400, 32, "clustered"), ("sparse", 2000, 512, 64, "clustered"),
         ("floats", 1500, 2400, 16, "clustered"), ("floats", 2500, 256, 2500, "participation")]


@pytest.mark.parametrize("placement", list(PLACEMENTS))
@pytest.mark.parametrize("kind,n,L,G,scheme", CASES, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}-{c[4]}" for c in CASES])
def test_noalloc_matches_allocating_gather(torch, kind, n, L, G, scheme, placement):
    rows = structured_rows(kind, n, L, seed=n + L)
    if scheme == "participation":
        stream = oracle.compress(rows, G, chunk_bytes=8, threshold=(4, 5))
        if placement == "zero_copy_aligned":   # aligned rows hold clustered-scheme streams only
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_open(stream, 0, PLACEMENTS[placement])
            assert e.value.status == ibp.IBP_EINVAL
            return
    else:
        stream = oracle.compress(rows, G)
    rng = np.random.default_rng(n * 7 + L)
    first = rng.integers(0, n, size=5 * n).astype(np.int64)            # unsorted, duplicates
    second = np.sort(rng.choice(n, size=n // 3, replace=False)).astype(np.int64)
    say(f"[noalloc] {kind} n={n} L={L} G={G} {scheme} {placement}: {first.size} then {second.size} ids")
    with ibp.ibp_open(stream, 0, PLACEMENTS[placement]) as h:
        for ids in (first, second):
            want = _out(torch, ids.size, L)
            got = _out(torch, ids.size, L)
            ibp.ibp_gather_decompress(h, ids, want, out_cap=ids.size * L)
            ibp.ibp_gather_decompress_noalloc(h, ids, got, out_cap=ids.size * L)
            torch.cuda.synchronize()
            assert torch.equal(got, want)                   # canary bytes past the end too
            g = got[:ids.size * L].cpu().numpy().reshape(-1, L)
            assert np.array_equal(g, rows[ids])
            assert np.array_equal(g[:200], oracle.decode_rows(stream, ids[:200], L))
            assert (got[ids.size * L:].cpu().numpy() == 0xA5).all()
        assert ibp.ibp_device_errors(h) == 0


def test_noalloc_reads_pageable_ids_before_returning(torch):
    """Ids in pageable host memory may be overwritten as soon as the call returns."""
    rows = structured_rows("floats", 4000, 400, seed=5)
    stream = oracle.compress(rows, 32)
    rng = np.random.default_rng(3)
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        ids = rng.integers(0, 4000, size=200_000).astype(np.int64)
        keep = ids.copy()
        out = _out(torch, ids.size, 400)
        ibp.ibp_gather_decompress_noalloc(h, ids, out, out_cap=ids.size * 400)
        ids[:] = (ids + 1) % 4000                # still in range: a stale read decodes other rows
        torch.cuda.synchronize()
        assert np.array_equal(out[:ids.size * 400].cpu().numpy().reshape(-1, 400), rows[keep])


def test_noalloc_limits_and_arguments(torch):
    rows = structured_rows("floats", 100, 64, seed=4)
    stream = oracle.compress(rows, 16)
    out = _out(torch, 4, 64)
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        too_many = np.zeros(MAX_IDS + 1, np.int64)
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_gather_decompress_noalloc(h, too_many, out, out_cap=10 ** 12)
        assert e.value.status == ibp.IBP_EINVAL and "scratch" in str(e.value)
        for bad in ([1, 100, 2], [-1], [5, 2 ** 40]):
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_gather_decompress_noalloc(h, np.array(bad, np.int64), out, out_cap=3 * 64)
            assert e.value.status == ibp.IBP_ERANGE
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_gather_decompress_noalloc(h, np.arange(4, dtype=np.int64), out, out_cap=3 * 64)
        assert e.value.status == ibp.IBP_ENOMEM
        ibp.ibp_gather_decompress_noalloc(h, np.zeros(0, np.int64), out)    # empty call
        torch.cuda.synchronize()
        assert (out.cpu().numpy() == 0xA5).all()
        # the largest call the scratch holds
        ids = np.arange(MAX_IDS, dtype=np.int64) % 100
        big = torch.empty(MAX_IDS * 64, dtype=torch.uint8, device="cuda")
        ibp.ibp_gather_decompress_noalloc(h, ids, big)
        torch.cuda.synchronize()
        sample = np.random.default_rng(1).integers(0, MAX_IDS, 5000)
        got = big.view(-1, 64)[torch.from_numpy(sample).cuda()].cpu().numpy()
        assert np.array_equal(got, rows[ids[sample]])
        assert ibp.ibp_device_errors(h) == 0
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST) as h:
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_gather_decompress_noalloc(h, np.arange(4, dtype=np.int64), out, out_cap=4 * 64)
        assert e.value.status == ibp.IBP_EINVAL
