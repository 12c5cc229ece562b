"""GPU parity of the thresholded scheme with participation bits: every decode path of
the library (device-resident payload, pinned host payload through staging, zero-copy;
ranges and gathers with host or device ids) against the CPU oracle, element by element."""
import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import CONFIGS, gen_all_rows, gnn_batch_ids, structured_rows

pytestmark = pytest.mark.gpu

FLAGS = {"device": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host": ibp.IBP_OPEN_PAYLOAD_HOST,
         "zero_copy": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY}

# (kind, n_rows, row_bytes, group_rows, chunk_bytes, threshold, sample_every): chunk sizes
# of 1-4 words, thresholds from 0.55 to 1, global and per-cluster masks, sampled masks,
# rows needing several tiles (W > 512) under one global and per-cluster masks, rows stored
# raw, clusters of one row
PCASES = [("floats", 300, 400, 32, 4, (4, 5), 1), ("floats", 300, 400, 1000, 8, (4, 5), 1),
          ("sparse", 129, 256, 32, 8, (3, 4), 2), ("random", 97, 12, 5, 4, (9, 10), 1),
          ("specials", 70, 16, 7, 8, (7, 10), 3), ("onebit", 50, 36, 10, 12, (5, 6), 1),
          ("alternating", 80, 24, 8, 4, (2, 3), 1), ("floats", 150, 2400, 700, 8, (4, 5), 4),
          ("random", 40, 64, 40, 4, (11, 20), 1), ("floats", 70, 4096, 100, 16, (4, 5), 1),
          ("sparse", 200, 512, 1, 16, (4, 5), 1), ("floats", 333, 256, 64, 4, (1, 1), 1),
          ("smallint", 65, 128, 1000, 4, (3, 5), 1), ("floats", 90, 2400, 16, 8, (4, 5), 1),
          ("specials", 60, 3000, 1000, 12, (7, 10), 1)]
IDS = [f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}-C{c[4]}-T{c[5][0]}of{c[5][1]}-s{c[6]}" for c in PCASES]


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _stream(kind, n, L, G, cs, thr, every):
    rows = structured_rows(kind, n, L, seed=n + 5 * L)
    s = oracle.compress(rows, G, chunk_bytes=cs, threshold=thr, sample_every=every)
    return rows, s


def _out(torch, n, L):
    return torch.full((n * L + 256,), 0xA5, dtype=torch.uint8, device="cuda")


def _rows(out, n, L):
    return out[:n * L].cpu().numpy().reshape(n, L)


@pytest.mark.parametrize("flags", ["device", "host", "zero_copy"])
@pytest.mark.parametrize("kind,n,L,G,cs,thr,every", PCASES, ids=IDS)
def test_participation_decompress(torch, kind, n, L, G, cs, thr, every, flags):
    rows, s = _stream(kind, n, L, G, cs, thr, every)
    want = oracle.decompress(s, n, L)
    assert np.array_equal(want, rows)
    say(f"[part decompress] {kind} n={n} L={L} G={G} C={cs} T={thr} every={every} flags={flags}")
    a, b = min(n - 1, 3), max(min(n, n - 2), min(n - 1, 3) + 1)
    with ibp.ibp_open(s, 0, FLAGS[flags]) as h:
        for first, cnt in ((0, n), (a, b - a)):
            out = _out(torch, cnt, L)
            ibp.ibp_decompress(h, first, cnt, out)
            torch.cuda.synchronize()
            assert np.array_equal(_rows(out, cnt, L), want[first:first + cnt]), (first, cnt)
            assert (out[cnt * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"


@pytest.mark.parametrize("mode", ["device_payload_host_ids", "device_payload_device_ids", "host_payload",
                                  "zero_copy_host_ids", "zero_copy_device_ids"])
@pytest.mark.parametrize("kind,n,L,G,cs,thr,every", PCASES, ids=IDS)
def test_participation_gather(torch, kind, n, L, G, cs, thr, every, mode):
    rows, s = _stream(kind, n, L, G, cs, thr, every)
    rng = np.random.default_rng(n * L + cs)
    ids = np.concatenate([rng.integers(0, n, size=3 * n), np.sort(rng.choice(n, size=n // 2, replace=False)),
                          [0, n - 1, n - 1]]).astype(np.int64)
    want = oracle.decode_rows(s, ids, L)
    say(f"[part gather] {kind} n={n} L={L} G={G} C={cs} mode={mode} n_ids={ids.size}")
    flags = (ibp.IBP_OPEN_PAYLOAD_HOST if mode == "host_payload" else
             ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY if mode.startswith("zero_copy") else ibp.IBP_OPEN_PAYLOAD_DEVICE)
    with ibp.ibp_open(s, 0, flags) as h:
        out = _out(torch, ids.size, L)
        if mode.endswith("device_ids"):
            ibp.ibp_gather_decompress_device(h, torch.from_numpy(ids).cuda(), out, out_cap=ids.size * L)
        else:
            ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * L)
        torch.cuda.synchronize()
        assert np.array_equal(_rows(out, ids.size, L), want)
        assert (out[ids.size * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
        assert ibp.ibp_device_errors(h) == 0


def test_participation_device_id_errors(torch):
    rows, s = _stream("floats", 100, 64, 100, 8, (4, 5), 1)
    say("[part edge] device ids out of range")
    d_ids = torch.tensor([3, 100, -7, 50, 2 ** 40], dtype=torch.int64, device="cuda")
    for flags in (ibp.IBP_OPEN_PAYLOAD_DEVICE, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY):
        with ibp.ibp_open(s, 0, flags) as h:
            out = _out(torch, 5, 64)
            ibp.ibp_gather_decompress_device(h, d_ids, out, out_cap=5 * 64)
            assert ibp.ibp_device_errors(h) == 3
            got = _rows(out, 5, 64)
            assert np.array_equal(got[0], rows[3]) and np.array_equal(got[3], rows[50])
            assert not got[1].any() and not got[2].any() and not got[4].any()


def test_participation_library_stream(torch):
    """The library's own compressor output decodes on the GPU to the original rows."""
    rows = structured_rows("floats", 5000, 400, seed=12)
    s = ibp.ibp_compress_ex(rows, 5000, 8, (4, 5), 1)
    assert np.array_equal(s, oracle.compress(rows, 5000, chunk_bytes=8, threshold=(4, 5)))
    say("[part library stream] 5000x400 global mask C=8 T=0.8")
    with ibp.ibp_open(s, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        out = _out(torch, 5000, 400)
        ibp.ibp_decompress(h, 0, 5000, out)
        torch.cuda.synchronize()
        assert np.array_equal(_rows(out, 5000, 400), rows)


DEFERRED = [(256, 270_000, 32, 4), (256, 270_000, 32, 8), (256, 270_000, 0, 8), (1024, 70_000, 0, 8),
            (1024, 70_000, 32, 16), (2048, 40_000, 0, 8), (2048, 40_000, 32, 8)]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("L,n,G,cs", DEFERRED, ids=[f"{c[0]}B-G{c[2] or 'all'}-C{c[3]}" for c in DEFERRED])
def test_participation_deferred_batches(torch, L, n, G, cs):
    """Launches large enough for two batches per wave (deferred stores) at one, four and
    eight words per lane: per-cluster Masks, where batches straddle clusters and decode row
    by row, and one global Mask; 32 to 256 chunks per row (participation dwords fetched with
    the lookup or loaded per batch). Range decode from an unaligned first row with a ragged
    count, gathers of random and of sorted ids; every row checked against the original rows,
    a sample of the stream against the oracle."""
    rows = structured_rows("floats", n, L, seed=77)
    s = ibp.ibp_compress_ex(rows, G or n, cs, (4, 5), 1)
    sample = np.random.default_rng(5).choice(n, 500, replace=False)
    assert np.array_equal(oracle.decode_rows(s, sample, L), rows[sample])
    with ibp.ibp_open(s, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        first, count = 5, n - 11
        say(f"[part deferred] G={G or n} chunk={cs} range ({first}, {count})")
        out = _out(torch, count, L)
        ibp.ibp_decompress(h, first, count, out)
        torch.cuda.synchronize()
        assert np.array_equal(_rows(out, count, L), rows[first:first + count])
        assert (out[count * L:].cpu().numpy() == 0xA5).all()
        rng = np.random.default_rng(6)
        for order, ids in (("random", rng.integers(0, n, size=n)), ("sorted", np.sort(rng.integers(0, n, size=n)))):
            say(f"[part deferred] G={G or n} chunk={cs} gather {order} ids={ids.size}")
            out = _out(torch, ids.size, L)
            ibp.ibp_gather_decompress_device(h, torch.from_numpy(ids.astype(np.int64)).cuda(), out,
                                             out_cap=ids.size * L)
            torch.cuda.synchronize()
            assert np.array_equal(_rows(out, ids.size, L), rows[ids])
        assert ibp.ibp_device_errors(h) == 0


@pytest.mark.timeout(600)
def test_participation_gnn_gather_full(torch):
    """The 2.4M x 100 fp32 GNN features under one global Mask at T = 0.8 n (8-byte
    chunks): a full minibatch gather on every path, checked against the original rows
    and, on a sample, against the oracle."""
    cfg = CONFIGS["gnn_gather"]
    rows = gen_all_rows(cfg)
    s = ibp.ibp_compress_ex(rows, cfg.n_rows, 8, (4, 5), 1)
    d = ibp.ibp_describe(s)
    say(f"[part gnn full] payload {d['payload_bytes'] / 1e6:.1f} MB (CR {rows.nbytes / d['payload_bytes']:.3f})")
    ids = gnn_batch_ids(cfg.n_rows, cfg.extra["seeds"], cfg.extra["fanouts"], batch_index=0)
    want = rows[ids]
    sample = np.random.default_rng(3).choice(ids.size, 1500, replace=False)
    assert np.array_equal(oracle.decode_rows(s, ids[sample], cfg.row_bytes), want[sample])
    for mode, flags in (("device", ibp.IBP_OPEN_PAYLOAD_DEVICE), ("host", ibp.IBP_OPEN_PAYLOAD_HOST),
                        ("zero_copy", ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)):
        say(f"[part gnn full] mode={mode} n_ids={ids.size}")
        with ibp.ibp_open(s, 0, flags) as h:
            out = _out(torch, ids.size, cfg.row_bytes)
            ibp.ibp_gather_decompress(h, ids, out, out_cap=ids.size * cfg.row_bytes)
            torch.cuda.synchronize()
            assert np.array_equal(_rows(out, ids.size, cfg.row_bytes), want)



@pytest.mark.timeout(600)
def test_participation_kv_full(torch):
    """All 32 layers of the bf16 KV workload (4 GiB raw) under one global Mask at T = 0.8n
    with 8-byte chunks, streamed layer by layer through every placement; layers checked
    against the original rows, sampled rows against the oracle."""
    import gc
    cfg = CONFIGS["kv_bf16"]
    rows = gen_all_rows(cfg)
    s = ibp.ibp_compress_ex(rows, cfg.n_rows, 8, (4, 5), 1)
    n = cfg.extra["rows_per_layer"]
    sample = np.random.default_rng(4).choice(cfg.n_rows, 1500, replace=False)
    assert np.array_equal(oracle.decode_rows(s, sample, cfg.row_bytes), rows[sample])
    for flags in (ibp.IBP_OPEN_PAYLOAD_DEVICE, ibp.IBP_OPEN_PAYLOAD_HOST, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY):
        say(f"[part kv full] flags={flags}")
        with ibp.ibp_open(s, 0, flags) as h:
            out = torch.empty(n * cfg.row_bytes, dtype=torch.uint8, device="cuda")
            for layer in range(cfg.extra["layers"]):
                ibp.ibp_decompress(h, layer * n, n, out)
                torch.cuda.synchronize()
                got = out.cpu().numpy().reshape(n, cfg.row_bytes)
                assert np.array_equal(got, rows[layer * n:(layer + 1) * n]), (flags, layer)
    del rows, s
    gc.collect()
