"""GPU parity of the compressed device cache: hits decoded from the slab in HBM and misses
from the pinned host payload, element by element against the CPU oracle, plus the hit /
miss accounting and the error cases."""
import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import structured_rows

pytestmark = pytest.mark.gpu

ZC = ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY
CASES = [("floats", 3000, 400, 32), ("sparse", 1000, 512, 64), ("random", 500, 12, 5),
         ("specials", 700, 16, 7), ("floats", 2000, 256, 1), ("alternating", 900, 2048, 16),
         ("smallint", 640, 4, 32)]


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _gather(torch, c, ids, L):
    d_ids = torch.from_numpy(np.ascontiguousarray(ids, np.int64)).cuda()
    out = torch.full((ids.size * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")
    ibp.ibp_cache_gather(c, d_ids, out, out_cap=ids.size * L)
    torch.cuda.synchronize()
    assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
    return out[:ids.size * L].cpu().numpy().reshape(ids.size, L)


@pytest.mark.parametrize("kind,n,L,G", CASES, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}" for c in CASES])
def test_cache_gather_matches_oracle(torch, kind, n, L, G):
    rows = structured_rows(kind, n, L, seed=n + L)
    s = oracle.compress(rows, G)
    rng = np.random.default_rng(n)
    cached = rng.choice(n, size=n // 3, replace=False)
    ids = np.concatenate([rng.integers(0, n, size=2 * n), cached[:50], [0, n - 1]]).astype(np.int64)
    want = oracle.decode_rows(s, ids, L)
    say(f"[cache] {kind} n={n} L={L} G={G} cached={cached.size} n_ids={ids.size}")
    with ibp.ibp_open(s, 0, ZC) as h:
        with ibp.ibp_cache_create(h, np.concatenate([cached, cached[:10]])) as c:
            got = _gather(torch, c, ids, L)
            assert np.array_equal(got, want)
            st = ibp.ibp_cache_get_stats(c)
            hits = int(np.isin(ids, cached).sum())
            assert st["rows"] == cached.size
            assert st["hits"] == hits and st["misses"] == ids.size - hits
            assert st["slab_bytes"] == sum(oracle.packed_row_bytes(
                oracle.group_masks(rows[(r // G) * G:(r // G + 1) * G])[0]) for r in np.unique(cached))
            ibp.ibp_cache_reset_stats(c)
            assert ibp.ibp_cache_get_stats(c)["hits"] == 0
        assert ibp.ibp_device_errors(h) == 0


def test_cache_all_hits_all_misses_and_bad_ids(torch):
    rows = structured_rows("floats", 400, 64, seed=1)
    s = oracle.compress(rows, 16)
    say("[cache edge] all hits, all misses, empty cache, bad ids")
    with ibp.ibp_open(s, 0, ZC) as h:
        with ibp.ibp_cache_create(h, np.arange(400)) as c:
            ids = np.random.default_rng(2).integers(0, 400, size=999)
            assert np.array_equal(_gather(torch, c, ids, 64), rows[ids])
            assert ibp.ibp_cache_get_stats(c)["misses"] == 0
        with ibp.ibp_cache_create(h, np.zeros(0, np.int64)) as c:
            ids = np.arange(400)[::-1].copy()
            assert np.array_equal(_gather(torch, c, ids, 64), rows[ids])
            st = ibp.ibp_cache_get_stats(c)
            assert st["hits"] == 0 and st["misses"] == 400 and st["rows"] == 0
        with ibp.ibp_cache_create(h, np.arange(0, 400, 3)) as c:
            ids = np.array([5, 400, -1, 9, 2 ** 40, 399], np.int64)
            got = _gather(torch, c, ids, 64)
            assert ibp.ibp_device_errors(h) == 3
            assert np.array_equal(got[[0, 3, 5]], rows[[5, 9, 399]])
            assert not got[[1, 2, 4]].any()
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_close(h)
            assert e.value.status == ibp.IBP_ESTATE and h.ptr   # still open, closed on exit
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_cache_create(h, np.array([400], np.int64))
        assert e.value.status == ibp.IBP_ERANGE


def test_cache_rejects_other_placements_and_schemes(torch):
    rows = structured_rows("floats", 100, 64, seed=3)
    for flags in (ibp.IBP_OPEN_PAYLOAD_DEVICE, ibp.IBP_OPEN_PAYLOAD_HOST):
        with ibp.ibp_open(oracle.compress(rows, 16), 0, flags) as h:
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_cache_create(h, np.arange(10))
            assert e.value.status == ibp.IBP_EINVAL
    ps = oracle.compress(rows, 100, chunk_bytes=8, threshold=(4, 5))
    with ibp.ibp_open(ps, 0, ZC) as h:
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_cache_create(h, np.arange(10))
        assert e.value.status == ibp.IBP_EINVAL
    wide = structured_rows("floats", 10, 4096, seed=4)
    with ibp.ibp_open(oracle.compress(wide, 8), 0, ZC) as h:
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_cache_create(h, np.arange(3))
        assert e.value.status == ibp.IBP_EINVAL
