"""Byte identity of a library stream of the clustered scheme with the oracle's, at sizes
where one single-threaded oracle call over the whole tensor would take minutes.

Clusters are independent in this scheme (a cluster's Mask, Bitval and packed rows depend
on its own rows only), so the oracle compresses runs of consecutive clusters, one
single-threaded call per run on several threads, and each run's sections are compared
with the library stream's: the Mask/Bitval bytes, the index steps and the packed bytes.
For a whole stream the runs tile every cluster and the header is compared too: the
oracle's header of the first run with its four size fields (row count, cluster count,
index and payload offsets) replaced by the sums over the runs' own headers.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle


def _u64(b, off):
    return int(np.frombuffer(b[off:off + 8].tobytes(), np.uint64)[0])


def _sections(s):
    """(meta, index as int64, payload) of a stream, plus its header fields."""
    hdr = {"n_rows": _u64(s, 16), "n_groups": _u64(s, 24), "index_off": _u64(s, 48), "payload_off": _u64(s, 56)}
    idx = s[hdr["index_off"]:hdr["payload_off"]].view(np.uint64).astype(np.int64)
    return s[64:hdr["index_off"]], idx, s[hdr["payload_off"]:], hdr


def check_runs(stream, rows, G, runs, threads=16):
    """Every run [g0, g1) of clusters: the library stream's sections equal the oracle's
    compression of rows [g0*G, min(g1*G, n)). Returns the oracle's header fields of every
    run, in run order."""
    n, L = rows.shape
    meta_all, idx_all, pay_all, hdr = _sections(stream)
    assert hdr["n_rows"] == n and hdr["n_groups"] == (n + G - 1) // G

    def one(run):
        g0, g1 = run
        o = oracle.compress(rows[g0 * G:min(g1 * G, n)], G)
        meta, idx, pay, h = _sections(o)
        if not np.array_equal(meta_all[g0 * 2 * L:g1 * 2 * L], meta):
            return f"metadata of clusters [{g0}, {g1})", h
        if not np.array_equal(idx_all[g0:g1 + 1] - idx_all[g0], idx):
            return f"index of clusters [{g0}, {g1})", h
        if not np.array_equal(pay_all[idx_all[g0]:idx_all[g1]], pay):
            return f"payload of clusters [{g0}, {g1})", h
        return None, (h, o[:64].copy())

    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(one, runs))
    bad = [r for r, _ in res if r]
    assert not bad, bad[:5]
    return [h for _, h in res]


def check_whole(stream, rows, G, pieces=64, threads=16):
    """The whole stream, byte for byte: every cluster through check_runs, then the header
    against the oracle's first run header with its size fields summed over the runs (each
    run's index has its own closing entry; the whole stream has one)."""
    n, L = rows.shape
    ng = (n + G - 1) // G
    cuts = np.linspace(0, ng, min(pieces, max(ng, 1)) + 1).astype(np.int64)
    runs = [(int(a), int(b)) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
    heads = check_runs(stream, rows, G, runs, threads)
    fields = [h for h, _ in heads]
    n_rows = sum(h["n_rows"] for h in fields)
    n_groups = sum(h["n_groups"] for h in fields)
    meta = sum(h["index_off"] - 64 for h in fields)
    index = sum(h["payload_off"] - h["index_off"] for h in fields) - 8 * (len(runs) - 1)
    want = heads[0][1]
    for off, v in ((16, n_rows), (24, n_groups), (48, 64 + meta), (56, 64 + meta + index)):
        want[off:off + 8] = np.frombuffer(np.uint64(v).tobytes(), np.uint8)
    assert n_rows == n and n_groups == ng
    assert np.array_equal(stream[:64], want)
    _, idx, _, _ = _sections(stream)
    assert stream.size == 64 + meta + index + int(idx[-1])
    return ng


def sampled_runs(n_groups, fraction, run_len, seed, must=()):
    """Runs of run_len clusters covering about `fraction` of n_groups clusters (seeded
    starts), plus the first and last cluster and every cluster in `must` (single runs)."""
    rng = np.random.default_rng(seed)
    k = max(1, int(round(n_groups * fraction / run_len)))
    starts = np.unique(rng.integers(0, max(1, n_groups - run_len), size=k))
    runs = {(int(a), int(min(a + run_len, n_groups))) for a in starts}
    runs.add((0, 1))
    runs.add((n_groups - 1, n_groups))
    for g in np.unique(np.asarray(must, dtype=np.int64)):
        runs.add((int(g), int(g) + 1))
    return sorted(runs)
