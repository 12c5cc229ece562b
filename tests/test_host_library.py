"""The library's host half (no GPU needed): its compressed stream must be byte-identical
to the oracle's, its validation must reject corrupted streams, and the C ABI must export
every entry point that include/ibp.h declares."""
import os
import re
import sys

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import CONFIGS, gen_rows, structured_rows

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ibp.h")


def declared_entry_points():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:ibp_status|const char \*)\s*(ibp_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_entry_points()
    assert len(names) >= 14
    L = ibp.lib()
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/ibp.h but not exported"
    assert sorted(names) == sorted(ibp.EXPORTS), "binding and header disagree"
    assert "stream format 1" in ibp.ibp_version()


CASES = [("random", 37, 12, 5), ("floats", 100, 64, 32), ("specials", 70, 16, 7),
         ("sparse", 65, 400, 32), ("smallint", 33, 8, 32), ("alternating", 40, 24, 8),
         ("onebit", 50, 36, 10), ("zeros", 3, 4, 2), ("floats", 1, 4, 32), ("identical", 64, 20, 16),
         ("floats", 64, 4, 64), ("random", 9, 4, 3), ("random", 130, 1028, 1), ("sparse", 200, 2052, 33),
         ("floats", 257, 1024, 64), ("specials", 31, 260, 31)]


@pytest.mark.parametrize("kind,n,L,G", CASES, ids=[f"{c[0]}-{c[1]}x{c[2]}-G{c[3]}" for c in CASES])
@pytest.mark.parametrize("threads", [1, 4])
def test_stream_matches_oracle(kind, n, L, G, threads):
    rows = structured_rows(kind, n, L, seed=n * 7 + L)
    want = oracle.compress(rows, G)
    got = ibp.ibp_compress(rows, G, n_threads=threads)
    assert got.size == want.size
    assert np.array_equal(got, want)
    d = ibp.ibp_describe(got)
    assert d["n_rows"] == n and d["row_bytes"] == L and d["group_rows"] == G
    assert d["stream_bytes"] == got.size
    assert ibp.ibp_compress_bound(n, L, G) >= got.size


def test_empty_input():
    rows = np.zeros((0, 16), np.uint8)
    s = ibp.ibp_compress(rows, 4)
    assert s.size == 64 + 8
    assert np.array_equal(s, oracle.compress(rows, 4))
    d = ibp.ibp_describe(s)
    assert d["n_rows"] == 0 and d["n_groups"] == 0 and d["payload_bytes"] == 0


@pytest.mark.parametrize("key", ["tiny_gnn", "gnn_gather", "kv_bf16", "dlrm", "big_gnn"])
def test_workload_slices_match_oracle(key):
    """A slice of each workload (several clusters and a ragged tail), byte for byte."""
    cfg = CONFIGS[key]
    n = 4096 if key == "tiny_gnn" else 32 * cfg.group_rows + 5
    rows = gen_rows(cfg, 0, n)
    want = oracle.compress(rows, cfg.group_rows)
    got = ibp.ibp_compress(rows, cfg.group_rows)
    assert np.array_equal(got, want)


def test_tiny_gnn_closed_form_size():
    cfg = CONFIGS["tiny_gnn"]
    rows = gen_rows(cfg, 0, cfg.n_rows)
    s = ibp.ibp_compress(rows, cfg.group_rows)
    d = ibp.ibp_describe(s)
    # every cluster keeps sign, bit 30 and mantissa bits 15..0 invariant: <= 224 B per row
    assert d["payload_bytes"] <= cfg.n_rows * 224
    assert d["n_groups"] == 128 and d["payload_off"] == 64 + 128 * 1024 + 8 * 129


@pytest.mark.parametrize("args,status", [
    ((np.zeros((4, 3), np.uint8), 2), ibp.IBP_EINVAL),     # row_bytes not a multiple of 4
    ((np.zeros((4, 4), np.uint8), 0), ibp.IBP_EINVAL),     # group_rows == 0
])
def test_compress_rejects_bad_arguments(args, status):
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_compress(*args)
    assert e.value.status == status


def test_compress_reports_size_when_capacity_is_small():
    import ctypes
    rows = structured_rows("floats", 40, 64, seed=2)
    want = oracle.compress(rows, 8)
    got = ctypes.c_uint64(0)
    buf = np.full(want.size - 1, 0xAB, np.uint8)
    st = ibp.lib().ibp_compress(rows.ctypes.data, 40, 64, 8, 0, buf.ctypes.data, buf.size, ctypes.byref(got))
    assert st == ibp.IBP_ENOMEM and got.value == want.size
    assert (buf == 0xAB).all(), "nothing may be written on failure"


def _corrupt(s, fn):
    s = s.copy()
    fn(s)
    return s


def _set_u64(s, off, v):
    s[off:off + 8] = np.frombuffer(np.uint64(v).tobytes(), np.uint8)


@pytest.fixture(scope="module")
def good_stream():
    rows = structured_rows("floats", 100, 64, seed=5)
    return ibp.ibp_compress(rows, 16)


CORRUPTIONS = {
    "bad magic": lambda s: s.__setitem__(0, ord("X")),
    "bad version": lambda s: s.__setitem__(4, 2),
    "row_bytes 6": lambda s: s.__setitem__(8, 6),
    "group_rows 0": lambda s: s.__setitem__(slice(12, 16), 0),
    "n_groups wrong": lambda s: _set_u64(s, 24, 3),
    "flags set": lambda s: s.__setitem__(32, 1),
    "index_off wrong": lambda s: _set_u64(s, 48, 999),
    "index not from 0": lambda s: _set_u64(s, 64 + 7 * 128, 1),
    "index step wrong": lambda s: _set_u64(s, 64 + 7 * 128 + 8 * 3, int(s[64 + 7 * 128 + 24:64 + 7 * 128 + 32].view(np.uint64)[0]) + 1),
    "bitval outside mask": lambda s: _bitval_outside_mask(s),
}


def _bitval_outside_mask(s):
    """Set a Bitval bit of group 0 where its Mask bit is 0 (the index stays consistent)."""
    L = 64
    for k in range(L):
        m = int(s[64 + k])
        if m != 0xFF:
            zero_bit = (~m & 0xFF) & -(~m & 0xFF)
            s[64 + L + k] |= np.uint8(zero_bit)
            return
    raise AssertionError("group 0 has no variant bit")


@pytest.mark.parametrize("name", sorted(CORRUPTIONS))
def test_describe_rejects_corruption(good_stream, name):
    bad = _corrupt(good_stream, CORRUPTIONS[name])
    with pytest.raises(ibp.IbpError) as e:
        ibp.ibp_describe(bad)
    assert e.value.status == ibp.IBP_ECORRUPT, str(e.value)


def test_describe_rejects_truncation(good_stream):
    for cut in (10, 63, 64 + 100, good_stream.size - 1):
        with pytest.raises(ibp.IbpError) as e:
            ibp.ibp_describe(good_stream[:cut])
        assert e.value.status == ibp.IBP_ECORRUPT


def test_last_error_is_set():
    with pytest.raises(ibp.IbpError):
        ibp.ibp_describe(np.zeros(8, np.uint8))
    assert ibp.ibp_last_error() != ""


def test_big_row_tiled_streams_match():
    """Rows wider than one wave tile (more than 512 words) still match the oracle."""
    rows = structured_rows("sparse", 70, 4 * 1500, seed=9)
    assert np.array_equal(ibp.ibp_compress(rows, 32), oracle.compress(rows, 32))


def test_identity_stream_is_valid_and_raw():
    """The uncompressed baseline stream of bench.py (every Mask 0) validates and decodes,
    bit by bit through the oracle, to exactly the raw rows."""
    import bench
    rows = structured_rows("floats", 70, 64, seed=21)
    s = bench.identity_stream(rows, 16)
    d = ibp.ibp_describe(s)
    assert d["payload_bytes"] == rows.nbytes and d["n_groups"] == 5
    assert np.array_equal(oracle.decompress(s, 70, 64), rows)


def test_kernel_code_hash_ignores_comments_only():
    """The hash that decides whether the stored counter traffic still describes the kernels:
    comment and blank-line edits keep it, any code edit changes it."""
    import bench
    src = "// header\n__global__ void k(int *p) {\n    p[0] = 1;   // store\n}\n"
    same = "/* a block\n   comment */\n__global__ void k(int *p) {\n\n    p[0] = 1;\n}\n// trailer\n"
    other = "__global__ void k(int *p) {\n    p[0] = 2;\n}\n"
    assert bench.code_sha256([src]) == bench.code_sha256([same])
    assert bench.code_sha256([src]) != bench.code_sha256([other])
    assert len(bench.kernel_sources_sha256()) == 64


def test_traffic_gate_reads_the_profile_only_while_the_code_matches(monkeypatch):
    """bench.py reports a kernel's measured HBM traffic from its committed rocprofv3 summary
    only while the hashed sources match the hash recorded there; any other hash, or a
    profile without the two lines, gives None (the line then carries traffic null)."""
    import bench
    text = open(os.path.join(bench.ROOT, "profiles", "k_gather_rows_big_gnn.md")).read()
    want = int(re.search(r"traffic_bytes_per_launch:\s*(\d+)", text).group(1))
    recorded = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text).group(1)
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: recorded)
    assert bench.measured_traffic("big_gnn") == want
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: "0" * 64)
    assert bench.measured_traffic("big_gnn") is None
    assert bench.measured_traffic("no_such_workload") is None


@pytest.mark.skipif(__import__("shutil").which("gcc") is None, reason="needs gcc")
def test_header_is_plain_c():
    """include/ibp.h is a C ABI: it compiles as pedantic C99 (and as C++), with no torch or
    HIP types in it."""
    import subprocess
    for cmd in (["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                ["g++", "-std=c++11", "-Wall", "-Werror", "-fsyntax-only", "-x", "c++", HEADER]):
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, r.stderr
    text = open(HEADER).read()
    assert "torch" not in text.lower().replace("pytorch", "") and "hip_runtime" not in text


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus 2 exits with status 2 and says why, before any
    device work."""
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def test_binding_rejects_host_buffers_for_device_arguments():
    """Device arguments are checked in the binding before any address reaches the library:
    CPU tensors, numpy arrays, int32 ids and strided views are refused with TypeError."""
    import torch
    h = ibp.Handle(None)
    ids64 = torch.arange(4, dtype=torch.int64)
    out = torch.empty(4 * 64, dtype=torch.uint8)
    for call in (lambda: ibp.ibp_gather_decompress_device(h, ids64, out),
                 lambda: ibp.ibp_decompress(h, 0, 4, out),
                 lambda: ibp.ibp_decompress(h, 0, 4, np.zeros(256, np.uint8)),
                 lambda: ibp.ibp_gather_decompress(h, np.arange(4), out),
                 lambda: ibp.ibp_gather_decompress_noalloc(h, np.arange(4), out),
                 lambda: ibp.ibp_cache_gather(ibp.Cache(None, h), ids64, out),
                 lambda: ibp.ibp_gather_decompress_device(h, ids64.to(torch.int32), out),
                 lambda: ibp.ibp_gather_decompress_device(h, torch.arange(8, dtype=torch.int64)[::2], out)):
        with pytest.raises(TypeError):
            call()


@pytest.mark.parametrize("scheme", ["clustered", "participation"])
def test_compress_allocation_failure_writes_nothing(scheme, monkeypatch):
    """IBP_TEST_FAIL_ALLOC=n fails the n-th allocation of one compress call: IBP_ENOMEM and
    an untouched output, for every n up to the call's allocation count; beyond it the
    stream equals the oracle's."""
    import ctypes
    rows = structured_rows("floats", 300, 64, seed=9)
    if scheme == "participation":
        want = oracle.compress(rows, 300, chunk_bytes=8, threshold=(4, 5))
        p = ibp.ibp_params(300, 8, 4, 5, 1)
        call = lambda buf, got: ibp.lib().ibp_compress_ex(rows.ctypes.data, 300, 64, ctypes.byref(p), 1,
                                                          buf.ctypes.data, buf.size, ctypes.byref(got))
    else:
        want = oracle.compress(rows, 16)
        call = lambda buf, got: ibp.lib().ibp_compress(rows.ctypes.data, 300, 64, 16, 1, buf.ctypes.data,
                                                       buf.size, ctypes.byref(got))
    failures = 0
    for n in range(1, 10):
        monkeypatch.setenv("IBP_TEST_FAIL_ALLOC", str(n))
        buf = np.full(want.size, 0xAB, np.uint8)
        got = ctypes.c_uint64(0)
        st = call(buf, got)
        if st == ibp.IBP_OK:
            assert np.array_equal(buf, want)
            break
        assert st == ibp.IBP_ENOMEM, st
        assert (buf == 0xAB).all(), n
        failures += 1
    else:
        raise AssertionError("the call never succeeded")
    assert failures >= 2
    monkeypatch.delenv("IBP_TEST_FAIL_ALLOC")
    assert np.array_equal(ibp.ibp_compress_ex(rows, 300, 8, (4, 5)) if scheme == "participation"
                          else ibp.ibp_compress(rows, 16), want)


def test_memory_usage_without_handles():
    dev, pin = ibp.ibp_memory_usage()
    assert dev == 0 and pin == 0


@pytest.mark.slow
@pytest.mark.parametrize("key", ["gnn_gather", "kv_bf16"])
def test_whole_workload_stream_matches_oracle(key):
    """The whole 2.4M x 400 B GNN table and the whole 4 GiB bf16 KV cache: the library's
    stream equals the oracle's byte for byte (every cluster's metadata, index and packed
    rows, and the header), the oracle running on cluster runs in parallel threads."""
    import time
    import stream_check
    from workloads import gen_all_rows
    cfg = CONFIGS[key]
    rows = gen_all_rows(cfg)
    stream = ibp.ibp_compress(rows, cfg.group_rows)
    t = time.time()
    ng = stream_check.check_whole(stream, rows, cfg.group_rows, pieces=256, threads=min(16, os.cpu_count() or 1))
    assert ng == (cfg.n_rows + cfg.group_rows - 1) // cfg.group_rows
    print(f"{key}: {ng} clusters identical to the oracle's in {time.time() - t:.1f}s")
