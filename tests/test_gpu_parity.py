"""GPU parity: the HIP decompression path against the CPU oracle, element by element.

Every expected value comes from the oracle (its bit-serial decode) or from the original
rows drawn by the seeded generators; the GPU decodes the oracle's own stream, and the
library's stream is compared with the oracle's separately. Decompressed rows must be
bit-exact.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import CONFIGS, gen_all_rows, gen_rows, gnn_batch_ids, structured_rows

pytestmark = pytest.mark.gpu

FLAGS = {"device": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host": ibp.IBP_OPEN_PAYLOAD_HOST,
         "zero_copy": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
         "zero_copy_aligned": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    ibp.lib()
    return t


def _out(torch, n, L, fill=0xA5):
    return torch.full((n * L + 256,), fill, dtype=torch.uint8, device="cuda")


def _rows(out, n, L):
    return out[:n * L].cpu().numpy().reshape(n, L)


def gpu_decompress(torch, stream, first, n, L, flags):
    with ibp.ibp_open(stream, 0, flags) as h:
        out = _out(torch, n, L)
        ibp.ibp_decompress(h, first, n, out)
        torch.cuda.synchronize()
        got = _rows(out, n, L)
        assert (out[n * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
    return got


def gpu_gather(torch, stream, ids, L, flags, device_ids=False):
    with ibp.ibp_open(stream, 0, flags) as h:
        n = len(ids)
        out = _out(torch, n, L)
        if device_ids:
            d_ids = torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int64)).cuda()
            ibp.ibp_gather_decompress_device(h, d_ids, out, out_cap=n * L)
        else:
            ibp.ibp_gather_decompress(h, ids, out, out_cap=n * L)
        torch.cuda.synchronize()
        got = _rows(out, n, L)
        assert (out[n * L:].cpu().numpy() == 0xA5).all(), "wrote past the output"
        errs = ibp.ibp_device_errors(h)
    return got, errs


SMALL = [("floats", 300, 400, 32), ("random", 97, 12, 5), ("specials", 70, 16, 7),
         ("sparse", 129, 256, 32), ("alternating", 80, 24, 8), ("identical", 66, 20, 16),
         ("smallint", 33, 4, 32), ("onebit", 50, 36, 1), ("floats", 200, 516, 100),
         ("sparse", 90, 1024, 32), ("floats", 70, 2400, 16), ("floats", 61, 260, 64),
         ("alternating", 45, 520, 9), ("floats", 40, 4096, 32), ("random", 19, 4096, 8),
         ("floats", 300, 400, 300), ("sparse", 90, 256, 1000)]


@pytest.mark.parametrize("flags", ["device", "host", "zero_copy", "zero_copy_aligned"])
@pytest.mark.parametrize("kind,n,L,G", SMALL, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}" for c in SMALL])
def test_decompress_small(torch, kind, n, L, G, flags):
    rows = structured_rows(kind, n, L, seed=n + 3 * L)
    stream = oracle.compress(rows, G)
    want = oracle.decompress(stream, n, L)
    assert np.array_equal(want, rows)
    say(f"[decompress] {kind} n={n} L={L} G={G} flags={flags}")
    got = gpu_decompress(torch, stream, 0, n, L, FLAGS[flags])
    assert np.array_equal(got, want)
    # a range starting and ending inside clusters
    a, b = min(n - 1, G // 2 + 1), max(min(n, n - G // 3), min(n - 1, G // 2 + 1) + 1)
    got = gpu_decompress(torch, stream, a, b - a, L, FLAGS[flags])
    assert np.array_equal(got, want[a:b])


@pytest.mark.parametrize("mode", ["device_payload_host_ids", "device_payload_device_ids", "host_payload",
                                  "zero_copy_host_ids", "zero_copy_device_ids", "zero_copy_aligned_host_ids",
                                  "zero_copy_aligned_device_ids"])
@pytest.mark.parametrize("kind,n,L,G", SMALL, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}" for c in SMALL])
def test_gather_small(torch, kind, n, L, G, mode):
    rows = structured_rows(kind, n, L, seed=n + 3 * L)
    stream = oracle.compress(rows, G)
    rng = np.random.default_rng(n * L)
    ids = np.concatenate([rng.integers(0, n, size=3 * n), np.sort(rng.choice(n, size=n // 2, replace=False)),
                          [0, n - 1, n - 1]]).astype(np.int64)
    want = oracle.decode_rows(stream, ids, L)
    say(f"[gather] {kind} n={n} L={L} G={G} mode={mode} n_ids={ids.size}")
    flags = (ibp.IBP_OPEN_PAYLOAD_HOST if mode == "host_payload" else
             ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED if mode.startswith("zero_copy_aligned") else
             ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY if mode.startswith("zero_copy") else ibp.IBP_OPEN_PAYLOAD_DEVICE)
    got, errs = gpu_gather(torch, stream, ids, L, flags, device_ids=mode.endswith("device_ids"))
    assert errs == 0
    assert np.array_equal(got, want)


def test_library_stream_decodes_identically(torch):
    rows = structured_rows("floats", 500, 400, seed=11)
    lib_stream = ibp.ibp_compress(rows, 32)
    assert np.array_equal(lib_stream, oracle.compress(rows, 32))
    say("[library stream] 500x400 G=32")
    got = gpu_decompress(torch, lib_stream, 0, 500, 400, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    assert np.array_equal(got, rows)


def test_edge_cases(torch):
    rows = structured_rows("floats", 100, 64, seed=4)
    stream = oracle.compress(rows, 16)
    say("[edge] empty calls, one row, the last row")
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        out = _out(torch, 1, 64)
        ibp.ibp_decompress(h, 100, 0, out)                       # empty range at the end
        ibp.ibp_gather_decompress(h, np.zeros(0, np.int64), out)  # no ids
        ibp.ibp_decompress(h, 99, 1, out)
        torch.cuda.synchronize()
        assert np.array_equal(_rows(out, 1, 64)[0], rows[99])
        for first, n in [(100, 1), (101, 0), (0, 101)]:
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_decompress(h, first, n, out, out_cap=10 ** 9)
            assert e.value.status == ibp.IBP_ERANGE
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_decompress(h, 0, 2, out, out_cap=64)
        assert e.value.status == ibp.IBP_ENOMEM
        # host ids out of range: IBP_ERANGE and nothing written
        out2 = _out(torch, 3, 64)
        for bad in ([1, 100, 2], [-1], [5, 2 ** 40]):
            with pytest.raises(ibp.IbpError) as e:
                ibp.ibp_gather_decompress(h, np.array(bad, np.int64), out2, out_cap=3 * 64)
            assert e.value.status == ibp.IBP_ERANGE
        torch.cuda.synchronize()
        assert (out2.cpu().numpy() == 0xA5).all()
        # device ids out of range: zero rows and a device error count
        d_ids = torch.tensor([3, 100, -7, 50, 2 ** 40], dtype=torch.int64, device="cuda")
        out3 = _out(torch, 5, 64)
        ibp.ibp_gather_decompress_device(h, d_ids, out3, out_cap=5 * 64)
        assert ibp.ibp_device_errors(h) == 3
        got = _rows(out3, 5, 64)
        assert np.array_equal(got[0], rows[3]) and np.array_equal(got[3], rows[50])
        assert not got[1].any() and not got[2].any() and not got[4].any()
        assert ibp.ibp_device_errors(h) == 0
        st = ibp.ibp_get_stats(h)
        assert st["calls"] == 2   # the two calls that enqueued work; empty calls do not count
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST) as h:
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_gather_decompress_device(h, d_ids, out3, out_cap=5 * 64)
        assert e.value.status == ibp.IBP_EINVAL
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY) as h:
        out4 = _out(torch, 5, 64)
        ibp.ibp_gather_decompress_device(h, d_ids, out4, out_cap=5 * 64)
        assert ibp.ibp_device_errors(h) == 3
        assert np.array_equal(_rows(out4, 5, 64), got)


def test_open_rejects_corrupt_stream(torch):
    rows = structured_rows("floats", 40, 64, seed=4)
    stream = oracle.compress(rows, 16).copy()
    stream[0] = ord("Z")
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    assert e.value.status == ibp.IBP_ECORRUPT
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_open(oracle.compress(rows, 16), 0, 7)
    assert e.value.status == ibp.IBP_EINVAL


def test_tiny_gnn_full(torch):
    """The 4,096 x 128 fp32 workload: whole tensor, both payload placements."""
    cfg = CONFIGS["tiny_gnn"]
    rows = gen_rows(cfg, 0, cfg.n_rows)
    stream = oracle.compress(rows, cfg.group_rows)
    assert np.array_equal(ibp.ibp_compress(rows, cfg.group_rows), stream)
    want = oracle.decompress(stream, cfg.n_rows, cfg.row_bytes)
    for flags in FLAGS.values():
        say(f"[tiny_gnn] flags={flags}")
        got = gpu_decompress(torch, stream, 0, cfg.n_rows, cfg.row_bytes, flags)
        assert np.array_equal(got, want)
        assert np.array_equal(got, rows)


def _sampled_groups_match_oracle(stream, rows, G, L, n_groups, n_sample, seed):
    """Library stream sections of sampled groups equal the oracle's compression of them."""
    d = ibp.ibp_describe(stream)
    rng = np.random.default_rng(seed)
    groups = np.unique(np.concatenate([[0, n_groups - 1], rng.integers(0, n_groups, n_sample)]))
    index = stream[d["index_off"]:d["index_off"] + 8 * (n_groups + 1)].view(np.uint64)
    for g in groups:
        g = int(g)
        grp = rows[g * G:(g + 1) * G]
        o = oracle.compress(grp, G)
        od = 64 + 2 * L + 16
        meta = stream[64 + g * 2 * L:64 + (g + 1) * 2 * L]
        assert np.array_equal(meta, o[64:64 + 2 * L]), g
        pay = stream[d["payload_off"] + int(index[g]):d["payload_off"] + int(index[g + 1])]
        assert np.array_equal(pay, o[od:]), g


# packed bytes of 2.5-3 staging buffers of 128 MiB: ~4,096, ~199 and ~464 B per packed row
@pytest.mark.parametrize("kind,n,L,G", [("random", 84000, 4096, 32), ("floats", 1700000, 400, 32),
                                         ("sparse", 730000, 512, 64)])
def test_staged_multi_chunk(torch, kind, n, L, G):
    """Ranges whose packed bytes span several staging buffers on the pinned-host path, cut
    at arbitrary rows (chunk ends fall inside clusters), starting and ending mid-cluster."""
    rows = structured_rows(kind, n, L, seed=n + L)
    stream = ibp.ibp_compress(rows, G)
    a, b = G // 2 + 1, n - G // 3 - 1
    say(f"[staged multi-chunk] {kind} n={n} L={L} G={G} rows [{a}, {b})")
    got = gpu_decompress(torch, stream, a, b - a, L, ibp.IBP_OPEN_PAYLOAD_HOST)
    assert np.array_equal(got, rows[a:b])
    # the same range through the device-resident path as a cross-check of the range logic
    got = gpu_decompress(torch, stream, a, b - a, L, ibp.IBP_OPEN_PAYLOAD_DEVICE)
    assert np.array_equal(got, rows[a:b])


def test_kv_layer(torch):
    """One layer of the bf16 KV workload (524,288 rows of 256 B), device and PCIe paths."""
    cfg = CONFIGS["kv_bf16"]
    n = cfg.extra["rows_per_layer"]
    layer = 3
    rows = gen_rows(cfg, layer * n, (layer + 1) * n)
    stream = ibp.ibp_compress(rows, cfg.group_rows)
    _sampled_groups_match_oracle(stream, rows, cfg.group_rows, cfg.row_bytes, n // cfg.group_rows, 64, 1)
    for flags in FLAGS.values():
        say(f"[kv layer] flags={flags}")
        got = gpu_decompress(torch, stream, 0, n, cfg.row_bytes, flags)
        assert np.array_equal(got, rows)
    sample = np.random.default_rng(2).integers(0, n, 2000)
    assert np.array_equal(oracle.decode_rows(stream, sample, cfg.row_bytes), got[sample])


def test_gnn_gather_full(torch):
    """The 2.4M x 100 fp32 workload at full size: a whole minibatch gathered three ways."""
    cfg = CONFIGS["gnn_gather"]
    rows = gen_all_rows(cfg)
    stream = ibp.ibp_compress(rows, cfg.group_rows)
    _sampled_groups_match_oracle(stream, rows, cfg.group_rows, cfg.row_bytes, 75_000, 64, 3)
    ids = gnn_batch_ids(cfg.n_rows, cfg.extra["seeds"], cfg.extra["fanouts"], batch_index=0)
    sample = np.random.default_rng(5).choice(ids.size, 3000, replace=False)
    want_sample = oracle.decode_rows(stream, ids[sample], cfg.row_bytes)
    for mode in ("device_ids", "host_ids", "host_payload", "zero_copy_device_ids", "zero_copy_aligned_device_ids"):
        say(f"[gnn gather] mode={mode} n_ids={ids.size}")
        flags = (ibp.IBP_OPEN_PAYLOAD_HOST if mode == "host_payload" else
                 ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED if mode.startswith("zero_copy_aligned") else
                 ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY if mode.startswith("zero_copy") else ibp.IBP_OPEN_PAYLOAD_DEVICE)
        got, errs = gpu_gather(torch, stream, ids, cfg.row_bytes, flags, device_ids=mode.endswith("device_ids"))
        assert errs == 0
        assert np.array_equal(got, rows[ids])
        assert np.array_equal(got[sample], want_sample)


# ---------------------------------------------------------------- full-size workloads
# These hold tens of GB of host memory (the raw tables) and take a minute or two each,
# mostly drawing the synthetic rows.

def _full_stream(cfg):
    import time
    t = time.time()
    rows = gen_all_rows(cfg)
    say(f"[{cfg.key}] drew {rows.shape[0]} x {rows.shape[1]} B in {time.time() - t:.0f}s")
    t = time.time()
    stream = ibp.ibp_compress(rows, cfg.group_rows)
    d = ibp.ibp_describe(stream)
    say(f"[{cfg.key}] compressed in {time.time() - t:.0f}s: payload {d['payload_bytes'] / 1e9:.2f} GB "
        f"(CR {rows.nbytes / d['payload_bytes']:.2f}), stream {d['stream_bytes'] / 1e9:.2f} GB")
    return rows, stream, d


MODE_FLAGS = {"device_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host_ids": ibp.IBP_OPEN_PAYLOAD_DEVICE,
              "host_payload": ibp.IBP_OPEN_PAYLOAD_HOST,
              "zero_copy_device_ids": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
              "zero_copy_host_ids": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY,
              "zero_copy_aligned_device_ids": ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED}


def _full_gathers(torch, key, stream, ids, want, L, modes):
    """One batch through every mode; each output must equal the original rows."""
    for mode in modes:
        say(f"[{key}] gather mode={mode} n_ids={ids.size}")
        got, errs = gpu_gather(torch, stream, ids, L, MODE_FLAGS[mode], device_ids=mode.endswith("device_ids"))
        assert errs == 0
        assert np.array_equal(got, want), mode
        del got


def _full_participation(torch, key, rows, ids, want, L):
    """The thresholded scheme at full size (one global Mask sampled from every row,
    T = 4/5, 8-byte chunks): the same batch through every placement it supports, and a
    sample of rows decoded by the oracle from the library's stream."""
    import gc
    import time
    t = time.time()
    ps = ibp.ibp_compress_ex(rows, rows.shape[0], chunk_bytes=8, threshold=(4, 5))
    d = ibp.ibp_describe(ps)
    say(f"[{key}] thresholded stream in {time.time() - t:.0f}s: payload {d['payload_bytes'] / 1e9:.2f} GB")
    sample = np.random.default_rng(13).choice(ids.size, 2000, replace=False)
    assert np.array_equal(oracle.decode_rows(ps, ids[sample], L), want[sample])
    _full_gathers(torch, key + " thresholded", ps, ids, want, L,
                  ("device_ids", "host_ids", "host_payload", "zero_copy_device_ids"))
    del ps
    gc.collect()


@pytest.mark.timeout(1200)
def test_dlrm_full(torch):
    """26 tables x 4M rows x 128 fp32 (53 GB raw), one batch of 2,048 x 26 Zipf lookups."""
    import gc
    import stream_check
    from workloads import dlrm_batch_ids
    cfg = CONFIGS["dlrm"]
    G, L = cfg.group_rows, cfg.row_bytes
    rows, stream, d = _full_stream(cfg)
    x = cfg.extra
    ids = dlrm_batch_ids(x["tables"], x["rows_per_table"], x["batch"], x["zipf_s"], batch_index=0)
    # stream identity: runs covering 1% of the clusters, plus every cluster the batch touches
    runs = stream_check.sampled_runs(d["n_groups"], 0.01, 50, seed=7, must=ids // G)
    heads = stream_check.check_runs(stream, rows, G, runs)
    say(f"[dlrm] {sum(b - a for a, b in runs)} of {d['n_groups']} clusters identical to the oracle's "
        f"({len(heads)} runs)")
    want = rows[ids]
    sample = np.random.default_rng(9).choice(ids.size, 2000, replace=False)
    assert np.array_equal(oracle.decode_rows(stream, ids[sample], L), want[sample])
    _full_gathers(torch, "dlrm", stream, ids, want, L,
                  ("device_ids", "host_ids", "host_payload", "zero_copy_device_ids", "zero_copy_host_ids",
                   "zero_copy_aligned_device_ids"))
    # the compressed device cache over the full tables: the 2M most popular rows cached,
    # hits decoded from HBM and misses from pinned host memory in one kernel
    from workloads import dlrm_hot_order
    hot = dlrm_hot_order(x["tables"], x["rows_per_table"], n=2_000_000)
    say(f"[dlrm] cache of {hot.size} rows, n_ids={ids.size}")
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY) as h:
        with ibp.ibp_cache_create(h, hot) as c:
            d_ids = torch.from_numpy(ids).cuda()
            out = torch.empty(ids.size * L, dtype=torch.uint8, device="cuda")
            ibp.ibp_cache_gather(c, d_ids, out)
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy().reshape(-1, L), want)
            st = ibp.ibp_cache_get_stats(c)
            hits = int(np.isin(ids, hot).sum())
            assert st["hits"] == hits and st["misses"] == ids.size - hits and hits > ids.size // 2
        assert ibp.ibp_device_errors(h) == 0
    del stream
    gc.collect()
    _full_participation(torch, "dlrm", rows, ids, want, L)
    del rows
    gc.collect()


@pytest.mark.timeout(1200)
def test_big_gnn_full(torch):
    """111M rows x 128 fp32 (57 GB raw), G = 64, a 3-hop (15,10,5) minibatch of ~3.69M
    rows: every placement, including the staged one, whose ~0.94 GB of packed rows cross
    PCIe in about eight 128 MiB stages."""
    import gc
    import stream_check
    cfg = CONFIGS["big_gnn"]
    G, L = cfg.group_rows, cfg.row_bytes
    rows, stream, d = _full_stream(cfg)
    runs = stream_check.sampled_runs(d["n_groups"], 0.01, 50, seed=8)
    stream_check.check_runs(stream, rows, G, runs)
    say(f"[big_gnn] {sum(b - a for a, b in runs)} of {d['n_groups']} clusters identical to the oracle's")
    ids = gnn_batch_ids(cfg.n_rows, cfg.extra["seeds"], cfg.extra["fanouts"], batch_index=0)
    want = rows[ids]
    sample = np.random.default_rng(10).choice(ids.size, 2000, replace=False)
    assert np.array_equal(oracle.decode_rows(stream, ids[sample], L), want[sample])
    _full_gathers(torch, "big_gnn", stream, ids, want, L,
                  ("device_ids", "host_ids", "host_payload", "zero_copy_device_ids", "zero_copy_host_ids",
                   "zero_copy_aligned_device_ids"))
    del stream
    gc.collect()
    _full_participation(torch, "big_gnn", rows, ids, want, L)
    del rows, want
    gc.collect()


@pytest.mark.timeout(900)
def test_kv_full(torch):
    """All 32 layers of the bf16 KV workload (4 GiB raw), streamed layer by layer."""
    import gc
    cfg = CONFIGS["kv_bf16"]
    rows, stream, d = _full_stream(cfg)
    _sampled_groups_match_oracle(stream, rows, cfg.group_rows, cfg.row_bytes, d["n_groups"], 48, 11)
    n = cfg.extra["rows_per_layer"]
    for flags in (ibp.IBP_OPEN_PAYLOAD_DEVICE, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY, ibp.IBP_OPEN_PAYLOAD_HOST):
        say(f"[kv full] flags={flags}")
        with ibp.ibp_open(stream, 0, flags) as h:
            out = torch.empty(n * cfg.row_bytes, dtype=torch.uint8, device="cuda")
            for layer in range(cfg.extra["layers"]):
                ibp.ibp_decompress(h, layer * n, n, out)
                got = out.cpu().numpy().reshape(n, cfg.row_bytes)
                assert np.array_equal(got, rows[layer * n:(layer + 1) * n]), layer
    sample = np.random.default_rng(12).integers(0, cfg.n_rows, 2000)
    assert np.array_equal(oracle.decode_rows(stream, sample, cfg.row_bytes), rows[sample])
    del rows, stream
    gc.collect()


def test_independent_handles_on_threads(torch):
    """Distinct handles are independent: four host threads, each with its own handle
    (every placement) and its own HIP stream, gather and decompress concurrently; every
    result equals the oracle's."""
    import threading
    rows = structured_rows("floats", 4000, 256, seed=77)
    stream = oracle.compress(rows, 32)
    rng = np.random.default_rng(5)
    jobs = [(flags, rng.integers(0, 4000, size=3000).astype(np.int64))
            for flags in (FLAGS["device"], FLAGS["host"], FLAGS["zero_copy"], FLAGS["zero_copy_aligned"])]
    wants = [oracle.decode_rows(stream, ids, 256) for _, ids in jobs]
    results, errors = [None] * len(jobs), []
    say("[threads] 4 handles on 4 threads")

    def work(k, flags, ids):
        try:
            s = torch.cuda.Stream()
            with ibp.ibp_open(stream, 0, flags) as h:
                out = torch.empty(ids.size * 256, dtype=torch.uint8, device="cuda")
                whole = torch.empty(4000 * 256, dtype=torch.uint8, device="cuda")
                for _ in range(5):
                    ibp.ibp_gather_decompress(h, ids, out, stream=s)
                    ibp.ibp_decompress(h, 0, 4000, whole, stream=s)
                s.synchronize()
                results[k] = (out.cpu().numpy().reshape(-1, 256), whole.cpu().numpy().reshape(-1, 256))
        except Exception as e:      # reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=(k, f, ids)) for k, (f, ids) in enumerate(jobs)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for k in range(len(jobs)):
        assert np.array_equal(results[k][0], wants[k])
        assert np.array_equal(results[k][1], rows)



def test_aligned_zero_copy_rejects_participation_streams(torch):
    rows = structured_rows("floats", 100, 64, seed=8)
    ps = oracle.compress(rows, 100, chunk_bytes=8, threshold=(4, 5))
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_open(ps, 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED)
    assert e.value.status == ibp.IBP_EINVAL
    with ibp.ibp_open(oracle.compress(rows, 16), 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED) as h:
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_cache_create(h, np.arange(10))
        assert e.value.status == ibp.IBP_EINVAL



def test_host_placement_rejects_rows_larger_than_a_stage(torch):
    """A row that cannot fit one 128 MiB staging buffer is refused at open for the staged
    placement (and accepted by the others)."""
    L = 128 << 20
    rows = np.zeros((1, L), np.uint8)
    rows[0, ::4097] = 7
    stream = ibp.ibp_compress(rows, 1)
    say("[edge] 128 MiB row on the staged placement")
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST)
    assert e.value.status == ibp.IBP_EINVAL
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_DEVICE) as h:
        out = torch.empty(L, dtype=torch.uint8, device="cuda")
        ibp.ibp_decompress(h, 0, 1, out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), rows[0])
