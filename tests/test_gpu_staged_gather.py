"""Row gathers through the staged PCIe placement (IBP_OPEN_PAYLOAD_HOST) whose requests
span several 128 MiB staging buffers: the host packs each chunk of requests into pinned
staging, the copy stream moves it and the kernel decodes it into d_out at the chunk's
first request, while the buffers rotate with host waits on their previous copies (the
paper's one-call lookup + transfer + decompress, Sec. 4.4 and Sec. 6.3).

Ids are unsorted with duplicates, so chunk boundaries fall inside clusters; every row is
compared with the oracle's bit-serial decode of the same stream and with the original
rows, and the bytes past the output are checked untouched.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import structured_rows

pytestmark = pytest.mark.gpu

STAGE_BYTES = 128 << 20


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def par_decode(stream, ids, L, parts=16):
    """The oracle's decode of every requested row, in parts on several threads (each part
    one single-threaded oracle call)."""
    from concurrent.futures import ThreadPoolExecutor
    cuts = np.linspace(0, ids.size, parts + 1).astype(np.int64)
    with ThreadPoolExecutor(parts) as ex:
        pieces = list(ex.map(lambda k: oracle.decode_rows(stream, ids[cuts[k]:cuts[k + 1]], L), range(parts)))
    return np.concatenate(pieces)


def max_packed_row(stream):
    """Largest packed row of a stream (what sizes a staged chunk): per cluster from the
    index for the clustered scheme; a raw row for the participation scheme."""
    d = ibp.ibp_describe(stream)
    if d["flags"] == ibp.IBP_STREAM_PARTICIPATION:
        return d["row_bytes"]
    ng, G = d["n_groups"], d["group_rows"]
    idx = stream[d["index_off"]:d["index_off"] + 8 * (ng + 1)].view(np.uint64).astype(np.int64)
    per = np.full(ng, G, np.int64)
    per[-1] = d["n_rows"] - G * (ng - 1)
    return int((np.diff(idx) // per).max())


def rows_per_stage(stream):
    # one staged chunk: 8 B of tables (cluster, offset) + the largest packed row per request,
    # in whole packing blocks of 256 requests
    return (STAGE_BYTES - 64) // (8 + max_packed_row(stream)) // 256 * 256


CASES = [("floats", 600_000, 400, 32, "clustered"), ("sparse", 300_000, 512, 64, "clustered"),
         ("floats", 400_000, 400, 400_000, "participation"), ("random", 200_000, 256, 32, "participation")]


@pytest.mark.parametrize("kind,n,L,G,scheme", CASES, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}-{c[4]}" for c in CASES])
def test_staged_gather_spans_several_stages(torch, kind, n, L, G, scheme):
    rows = structured_rows(kind, n, L, seed=n + L + 17)
    if scheme == "participation":
        stream = ibp.ibp_compress_ex(rows, G, chunk_bytes=8, threshold=(4, 5))
    else:
        stream = ibp.ibp_compress(rows, G)
    per_stage = rows_per_stage(stream)
    n_ids = int(3.3 * per_stage) + 77                      # a ragged last chunk
    rng = np.random.default_rng(n * 3 + L)
    ids = rng.integers(0, n, size=n_ids).astype(np.int64)
    ids[:1000] = ids[0]                                    # a run of one id
    ids[-5:] = [n - 1, 0, n - 1, 1, n - 2]
    chunks = (n_ids + per_stage - 1) // per_stage
    say(f"[staged gather] {kind} n={n} L={L} G={G} {scheme}: {n_ids} ids, {per_stage} per stage -> {chunks} chunks")
    assert chunks >= 4
    want = par_decode(stream, ids, L)
    assert np.array_equal(want, rows[ids])
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST) as h:
        out = torch.full((n_ids * L + 4096,), 0xA5, dtype=torch.uint8, device="cuda")
        for rep in range(2):            # the second call reuses buffers the first left busy
            ibp.ibp_gather_decompress(h, ids, out, out_cap=n_ids * L)
            torch.cuda.synchronize()
            got = out[:n_ids * L].cpu().numpy().reshape(n_ids, L)
            assert np.array_equal(got, want), rep
            assert (out[n_ids * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
        st = ibp.ibp_get_stats(h)
        assert st["calls"] == 2 and st["rows_out"] == 2 * n_ids
        # the packed rows crossed PCIe once per request, plus 8 B of tables per request and
        # 4 B per chunk
        d = ibp.ibp_describe(stream)
        idx_n = d["n_rows"] + 1 if d["flags"] else d["n_groups"] + 1
        idx = stream[d["index_off"]:d["index_off"] + 8 * idx_n].view(np.uint64).astype(np.int64)
        if d["flags"]:
            sizes = np.diff(idx)[ids]
        else:
            per = np.full(d["n_groups"], G, np.int64)
            per[-1] = n - G * (d["n_groups"] - 1)
            sizes = (np.diff(idx) // per)[ids // G]
        assert st["h2d_payload_bytes"] == 2 * int(sizes.sum())
        assert st["h2d_bytes"] == 2 * (int(sizes.sum()) + 8 * n_ids + 4 * chunks)
        assert ibp.ibp_device_errors(h) == 0
