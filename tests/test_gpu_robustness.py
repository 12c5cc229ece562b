"""Documented failure statuses of the C ABI on a GPU: closed handles and destroyed caches,
two threads on one handle, and allocation failures forced from the host (the test hook
IBP_TEST_FAIL_ALLOC), each with no writes to the outputs and no memory left held.
"""
import ctypes
import sys
import threading

import numpy as np
import pytest

import oracle
import paper_2605_30728_amd as ibp
from workloads import structured_rows

pytestmark = pytest.mark.gpu

PLACEMENTS = {"device": ibp.IBP_OPEN_PAYLOAD_DEVICE, "host": ibp.IBP_OPEN_PAYLOAD_HOST,
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


def _raw_open(stream, flags):
    h = ctypes.c_void_p(0)
    st = ibp.lib().ibp_open(stream.ctypes.data, stream.nbytes, 0, flags, ctypes.byref(h))
    return st, h.value


def test_closed_handle_and_destroyed_cache(torch):
    """A second ibp_close, and every call on a closed handle, returns IBP_ESTATE; so does a
    second ibp_cache_destroy and every call on a destroyed cache."""
    L = ibp.lib()
    base = ibp.ibp_memory_usage()
    rows = structured_rows("floats", 200, 64, seed=3)
    stream = oracle.compress(rows, 16)
    st, hp = _raw_open(stream, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY)
    assert st == ibp.IBP_OK
    c = ctypes.c_void_p(0)
    ids = np.arange(50, dtype=np.int64)
    assert L.ibp_cache_create(hp, ids.ctypes.data, ids.size, ctypes.byref(c)) == ibp.IBP_OK
    assert L.ibp_close(hp) == ibp.IBP_ESTATE                 # a cache still lives on it
    d_ids = torch.arange(10, dtype=torch.int64, device="cuda")
    out = torch.full((10 * 64 + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert L.ibp_cache_gather(c.value, d_ids.data_ptr(), 10, out.data_ptr(), 10 * 64, s) == ibp.IBP_OK
    torch.cuda.synchronize()
    assert np.array_equal(out[:640].cpu().numpy().reshape(10, 64), rows[:10])
    assert L.ibp_cache_destroy(c.value) == ibp.IBP_OK
    out.fill_(0xA5)
    assert L.ibp_cache_destroy(c.value) == ibp.IBP_ESTATE
    assert L.ibp_cache_gather(c.value, d_ids.data_ptr(), 10, out.data_ptr(), 10 * 64, s) == ibp.IBP_ESTATE
    st_buf = ibp.ibp_cache_stats()
    assert L.ibp_cache_get_stats(c.value, ctypes.byref(st_buf)) == ibp.IBP_ESTATE
    assert L.ibp_cache_reset_stats(c.value) == ibp.IBP_ESTATE
    assert L.ibp_close(hp) == ibp.IBP_OK
    assert L.ibp_close(hp) == ibp.IBP_ESTATE
    assert "closed" in ibp.ibp_last_error()
    assert L.ibp_decompress(hp, 0, 10, out.data_ptr(), out.numel(), s) == ibp.IBP_ESTATE
    assert L.ibp_gather_decompress(hp, ids.ctypes.data, 10, out.data_ptr(), out.numel(), s) == ibp.IBP_ESTATE
    assert L.ibp_gather_decompress_device(hp, d_ids.data_ptr(), 10, out.data_ptr(), out.numel(), s) == ibp.IBP_ESTATE
    assert L.ibp_gather_decompress_noalloc(hp, ids.ctypes.data, 10, out.data_ptr(), out.numel(), s) == ibp.IBP_ESTATE
    cnt = ctypes.c_uint64(0)
    assert L.ibp_device_errors(hp, ctypes.byref(cnt)) == ibp.IBP_ESTATE
    assert L.ibp_get_stats(hp, ctypes.byref(ibp.ibp_stats())) == ibp.IBP_ESTATE
    assert L.ibp_get_desc(hp, ctypes.byref(ibp.ibp_desc())) == ibp.IBP_ESTATE
    assert L.ibp_reset_stats(hp) == ibp.IBP_ESTATE
    assert L.ibp_cache_destroy(c.value) == ibp.IBP_ESTATE
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == 0xA5).all()
    assert ibp.ibp_memory_usage() == base


def test_two_threads_one_handle(torch):
    """Two threads calling on one handle: a call that finds the handle busy returns
    IBP_ESTATE and does nothing; every call that gets the handle works, and the results
    stay exact. The main thread repeats a long gather (host packing of 600k rows) until six
    have gone through; the other thread loops on short calls meanwhile."""
    L = ibp.lib()
    n, W = 300_000, 100
    rows = structured_rows("floats", n, 4 * W, seed=21)
    stream = ibp.ibp_compress(rows, 32)
    rng = np.random.default_rng(4)
    ids = rng.integers(0, n, size=600_000).astype(np.int64)
    few = np.arange(8, dtype=np.int64)
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST) as h:
        out = torch.empty(ids.size * 4 * W, dtype=torch.uint8, device="cuda")
        side = torch.full((8 * 4 * W,), 0xA5, dtype=torch.uint8, device="cuda")
        stop = threading.Event()
        seen = {"estate": 0, "ok": 0, "other": []}
        s_main = torch.cuda.Stream()
        s_side = torch.cuda.Stream()

        def hammer():
            st_buf = ibp.ibp_stats()
            while not stop.is_set():
                for r in (L.ibp_get_stats(h.ptr, ctypes.byref(st_buf)),
                          L.ibp_gather_decompress(h.ptr, few.ctypes.data, few.size, side.data_ptr(), side.numel(),
                                                  s_side.cuda_stream)):
                    if r == ibp.IBP_ESTATE:
                        seen["estate"] += 1
                    elif r == ibp.IBP_OK:
                        seen["ok"] += 1
                    else:
                        seen["other"].append(r)

        import time
        t = threading.Thread(target=hammer)
        t.start()
        done, main_estate, t0 = 0, 0, time.time()
        try:
            while done < 6 and time.time() - t0 < 60:
                st = L.ibp_gather_decompress(h.ptr, ids.ctypes.data, ids.size, out.data_ptr(), out.numel(),
                                             s_main.cuda_stream)
                if st == ibp.IBP_ESTATE:
                    main_estate += 1
                else:
                    assert st == ibp.IBP_OK, ibp.ibp_last_error()
                    done += 1
        finally:
            stop.set()
            t.join()
        s_main.synchronize()
        s_side.synchronize()
        say(f"[threads] side calls: {seen['estate']} IBP_ESTATE, {seen['ok']} ok; "
            f"main: {done} ok, {main_estate} IBP_ESTATE")
        assert done == 6
        assert not seen["other"], seen["other"]
        assert seen["estate"] > 0
        assert np.array_equal(out.cpu().numpy().reshape(ids.size, 4 * W), rows[ids])
        side_rows = side.cpu().numpy().reshape(8, 4 * W)
        if seen["ok"]:
            assert np.array_equal(side_rows, rows[few])


def _leak_free_failures(torch, call, what, max_n=40):
    """Runs call() with IBP_TEST_FAIL_ALLOC = 1, 2, ... until it succeeds; every failure
    must be IBP_ENOMEM and leave the library's memory as it was. Returns the number of
    failures seen."""
    import os
    base = ibp.ibp_memory_usage()
    fails = 0
    try:
        for n in range(1, max_n):
            os.environ["IBP_TEST_FAIL_ALLOC"] = str(n)
            st = call()
            if st == ibp.IBP_OK:
                return fails
            assert st == ibp.IBP_ENOMEM, (what, n, st, ibp.ibp_last_error())
            assert ibp.ibp_memory_usage() == base, (what, n)
            fails += 1
    finally:
        os.environ.pop("IBP_TEST_FAIL_ALLOC", None)
    raise AssertionError(f"{what}: still failing after {max_n} allocations")


@pytest.mark.parametrize("placement", list(PLACEMENTS))
@pytest.mark.parametrize("scheme", ["clustered", "participation"])
def test_open_allocation_failures(torch, placement, scheme):
    base = ibp.ibp_memory_usage()
    rows = structured_rows("floats", 500, 128, seed=5)
    stream = (oracle.compress(rows, 500, chunk_bytes=8, threshold=(4, 5)) if scheme == "participation"
              else oracle.compress(rows, 32))
    if scheme == "participation" and placement == "zero_copy_aligned":
        # aligned rows hold clustered-scheme streams only: refused before any allocation
        st, hp = _raw_open(stream, PLACEMENTS[placement])
        assert st == ibp.IBP_EINVAL and hp is None and ibp.ibp_memory_usage() == base
        return
    opened = []

    def call():
        st, hp = _raw_open(stream, PLACEMENTS[placement])
        if st == ibp.IBP_OK:
            opened.append(hp)
        else:
            assert hp is None
        return st

    fails = _leak_free_failures(torch, call, f"open {placement} {scheme}")
    say(f"[alloc] open {placement} {scheme}: {fails} allocations failed one by one")
    assert fails >= 3
    assert len(opened) == 1
    h = ibp.Handle(opened[0])
    out = torch.empty(500 * 128, dtype=torch.uint8, device="cuda")
    ibp.ibp_decompress(h, 0, 500, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().reshape(500, 128), rows)
    ibp.ibp_close(h)
    assert ibp.ibp_memory_usage() == base


@pytest.mark.parametrize("placement", ["device", "host", "zero_copy"])
def test_gather_allocation_failures_write_nothing(torch, placement):
    """A host-id gather whose allocation fails returns IBP_ENOMEM before enqueuing
    anything: the output keeps its canary bytes."""
    rows = structured_rows("floats", 2000, 256, seed=6)
    stream = oracle.compress(rows, 32)
    ids = np.random.default_rng(2).integers(0, 2000, size=5000).astype(np.int64)
    with ibp.ibp_open(stream, 0, PLACEMENTS[placement]) as h:
        out = torch.full((ids.size * 256,), 0xA5, dtype=torch.uint8, device="cuda")
        s = torch.cuda.current_stream().cuda_stream

        def call():
            st = ibp.lib().ibp_gather_decompress(h.ptr, ids.ctypes.data, ids.size, out.data_ptr(), out.numel(), s)
            torch.cuda.synchronize()
            if st != ibp.IBP_OK:
                assert (out.cpu().numpy() == 0xA5).all()
            return st

        fails = _leak_free_failures(torch, call, f"gather {placement}")
        say(f"[alloc] gather {placement}: {fails} allocations failed one by one")
        assert fails >= 1
        assert np.array_equal(out.cpu().numpy().reshape(-1, 256), rows[ids])


def test_cache_create_allocation_failures(torch):
    base = ibp.ibp_memory_usage()
    rows = structured_rows("floats", 3000, 256, seed=7)
    stream = oracle.compress(rows, 32)
    hot = np.arange(0, 3000, 3, dtype=np.int64)
    with ibp.ibp_open(stream, 0, ibp.IBP_OPEN_PAYLOAD_HOST_ZERO_COPY) as h:
        made = []

        def call():
            c = ctypes.c_void_p(0)
            st = ibp.lib().ibp_cache_create(h.ptr, hot.ctypes.data, hot.size, ctypes.byref(c))
            if st == ibp.IBP_OK:
                made.append(ibp.Cache(c.value, h))
            return st

        fails = _leak_free_failures(torch, call, "cache create")
        say(f"[alloc] cache create: {fails} allocations failed one by one")
        assert fails >= 3 and len(made) == 1
        d_ids = torch.arange(3000, dtype=torch.int64, device="cuda")
        out = torch.empty(3000 * 256, dtype=torch.uint8, device="cuda")
        ibp.ibp_cache_gather(made[0], d_ids, out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().reshape(-1, 256), rows)
        ibp.ibp_cache_destroy(made[0])
    assert ibp.ibp_memory_usage() == base
