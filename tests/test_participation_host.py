"""Host half of the thresholded scheme with participation bits (no GPU needed):
the library's streams against the oracle's, parameter checks, and validation."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import CONFIGS, gen_rows, structured_rows

# (kind, n_rows, row_bytes, group_rows, chunk_bytes, threshold, sample_every)
PCASES = [("floats", 300, 400, 32, 4, (4, 5), 1), ("floats", 300, 400, 1000, 8, (4, 5), 1),
          ("sparse", 129, 256, 32, 8, (3, 4), 2), ("random", 97, 12, 5, 4, (9, 10), 1),
          ("specials", 70, 16, 7, 8, (7, 10), 3), ("smallint", 33, 4, 32, 4, (1, 1), 1),
          ("onebit", 50, 36, 10, 12, (5, 6), 1), ("alternating", 80, 24, 8, 4, (2, 3), 1),
          ("identical", 66, 20, 16, 4, (4, 5), 1), ("floats", 600, 2400, 700, 8, (4, 5), 4),
          ("random", 40, 64, 40, 4, (11, 20), 1), ("floats", 1, 8, 4, 8, (4, 5), 1),
          ("sparse", 200, 512, 1, 16, (4, 5), 1)]
IDS = [f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}-C{c[4]}-T{c[5][0]}of{c[5][1]}-s{c[6]}" for c in PCASES]


@pytest.mark.parametrize("kind,n,L,G,cs,thr,every", PCASES, ids=IDS)
@pytest.mark.parametrize("threads", [1, 5, 16])
def test_participation_stream_matches_oracle(kind, n, L, G, cs, thr, every, threads):
    rows = structured_rows(kind, n, L, seed=n + L)
    want = oracle.compress(rows, G, chunk_bytes=cs, threshold=thr, sample_every=every)
    got = ibp.ibp_compress_ex(rows, G, cs, thr, every, n_threads=threads)
    assert np.array_equal(got, want)
    d = ibp.ibp_describe(got)
    assert d["flags"] == ibp.IBP_STREAM_PARTICIPATION and d["chunk_bytes"] == cs
    assert d["stream_bytes"] == want.size and d["n_rows"] == n


def test_clustered_parameters_give_the_clustered_stream():
    rows = structured_rows("floats", 200, 64, seed=2)
    assert np.array_equal(ibp.ibp_compress_ex(rows, 32), ibp.ibp_compress(rows, 32))
    assert np.array_equal(ibp.ibp_compress_ex(rows, 32), oracle.compress(rows, 32))


def test_global_mask_on_gnn_features():
    """One Mask for 20,000 GNN feature rows at T = 0.8 n (the paper's default), counted
    over all rows and over every 10th row (a sampled Mask)."""
    cfg = CONFIGS["gnn_gather"]
    rows = gen_rows(cfg, 0, 20000)
    for every in (1, 10):
        s = ibp.ibp_compress_ex(rows, 20000, 8, (4, 5), every)
        assert np.array_equal(s, oracle.compress(rows, 20000, chunk_bytes=8, threshold=(4, 5), sample_every=every))
        ids = np.random.default_rng(every).integers(0, 20000, size=300)
        assert np.array_equal(oracle.decode_rows(s, ids, cfg.row_bytes), rows[ids])


@pytest.mark.parametrize("G,cs,thr,every", [(32, 6, (4, 5), 1), (32, 12, (4, 5), 1), (32, 0, (4, 5), 1),
                                             (32, 0, (1, 1), 2), (32, 4, (1, 2), 1), (32, 4, (6, 5), 1),
                                             (32, 4, (4, 0), 1), (32, 4, (4, 5), 0), (0, 4, (4, 5), 1)])
def test_compress_ex_rejects_bad_parameters(G, cs, thr, every):
    rows = structured_rows("floats", 10, 16, seed=1)
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_compress_ex(rows, G, cs, thr, every)
    assert e.value.status == ibp.IBP_EINVAL


def test_compress_ex_reports_size_and_writes_nothing_when_small():
    rows = structured_rows("floats", 50, 64, seed=3)
    want = oracle.compress(rows, 16, chunk_bytes=8, threshold=(4, 5))
    p = ibp.ibp_params(16, 8, 4, 5, 1)
    got = ctypes.c_uint64(0)
    buf = np.full(want.size - 1, 0xAB, np.uint8)
    st = ibp.lib().ibp_compress_ex(rows.ctypes.data, 50, 64, ctypes.byref(p), 0, buf.ctypes.data, buf.size,
                                   ctypes.byref(got))
    assert st == ibp.IBP_ENOMEM and got.value == want.size
    assert (buf == 0xAB).all()


@pytest.fixture(scope="module")
def part_stream():
    rows = structured_rows("floats", 120, 64, seed=9)
    s = ibp.ibp_compress_ex(rows, 40, 4, (4, 5), 1)
    return rows, s


def _u64(s, off):
    return int(s[off:off + 8].view(np.uint64)[0])


def _set_u64(s, off, v):
    s[off:off + 8] = np.frombuffer(np.uint64(v).tobytes(), np.uint8)


def _first_compressed_row(s):
    L, n = 64, 120
    index_off, payload_off = _u64(s, 48), _u64(s, 56)
    for r in range(n):
        if _u64(s, index_off + 8 * (r + 1)) - _u64(s, index_off + 8 * r) < L:
            return r, payload_off + _u64(s, index_off + 8 * r)
    raise AssertionError("no compressed row")


def _flip_part_bit(s):
    r, pos = _first_compressed_row(s)
    s[pos] ^= np.uint8(1)


def _index_decreases(s):
    index_off = _u64(s, 48)
    _set_u64(s, index_off + 8 * 5, _u64(s, index_off + 8 * 6) + 1)


PCORRUPT = {
    "participation bit flipped": _flip_part_bit,
    "index decreases": _index_decreases,
    "chunk_bytes 6": lambda s: s.__setitem__(slice(36, 40), np.frombuffer(np.uint32(6).tobytes(), np.uint8)),
    "chunk_bytes 0": lambda s: s.__setitem__(slice(36, 40), 0),
    "flags 2": lambda s: s.__setitem__(32, 2),
    "flags 0 with chunk bytes": lambda s: s.__setitem__(32, 0),
    "last offset past the end": lambda s: _set_u64(s, _u64(s, 48) + 8 * 120, _u64(s, _u64(s, 48) + 8 * 120) + 50),
    "bitval outside mask": lambda s: _bitval_outside_mask(s),
}


def _bitval_outside_mask(s):
    """Set a Bitval bit of group 0 where its Mask bit is 0."""
    L = 64
    for k in range(L):
        m = int(s[64 + k])
        if m != 0xFF:
            s[64 + L + k] |= np.uint8((~m & 0xFF) & -(~m & 0xFF))
            return
    raise AssertionError("group 0 has no variant bit")


@pytest.mark.parametrize("name", sorted(PCORRUPT))
def test_describe_rejects_participation_corruption(part_stream, name):
    rows, s = part_stream
    bad = s.copy()
    PCORRUPT[name](bad)
    if np.array_equal(bad, s):
        pytest.skip("corruption did not change this stream")
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_describe(bad)
    assert e.value.status == ibp.IBP_ECORRUPT, str(e.value)


def test_participation_truncation(part_stream):
    rows, s = part_stream
    for cut in (63, 100, _u64(s, 56), s.size - 1):
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_describe(s[:cut])
        assert e.value.status == ibp.IBP_ECORRUPT
