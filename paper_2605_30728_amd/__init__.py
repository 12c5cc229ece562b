"""Python binding of libibp.so, the MI355X Invariant Bit Packing library.

Argument marshalling only: every function here has the name of a C ABI entry point in
include/ibp.h and forwards to it; all compression, validation and decompression runs in
the native library (host C++ and gfx950 HIP kernels). PyTorch is used only for device
memory and streams: device outputs and ids may be given as torch tensors (their
data_ptr() is passed) and streams as torch.cuda.Stream objects (their cuda_stream
handle is passed; None means torch's current stream).

The library must have been built (paper_2605_30728_amd.build); there is no fallback.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libibp.so")

IBP_OK, IBP_EINVAL, IBP_ERANGE, IBP_ENOMEM, IBP_ECORRUPT, IBP_EHIP, IBP_ESTATE = range(7)
STATUS_NAMES = {0: "IBP_OK", 1: "IBP_EINVAL", 2: "IBP_ERANGE", 3: "IBP_ENOMEM", 4: "IBP_ECORRUPT",
                5: "IBP_EHIP", 6: "IBP_ESTATE"}
IBP_OPEN_PAYLOAD_DEVICE = 0
IBP_OPEN_PAYLOAD_HOST = 1
IBP_OPEN_PAYLOAD_HOST_ZERO_COPY = 2
IBP_OPEN_PAYLOAD_HOST_ZERO_COPY_ALIGNED = 3
IBP_STREAM_PARTICIPATION = 1


class IbpError(RuntimeError):
    def __init__(self, status, func, message):
        super().__init__(f"{func}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class ibp_desc(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_uint64), ("n_groups", ctypes.c_uint64),
                ("meta_off", ctypes.c_uint64), ("index_off", ctypes.c_uint64),
                ("payload_off", ctypes.c_uint64), ("payload_bytes", ctypes.c_uint64),
                ("stream_bytes", ctypes.c_uint64), ("row_bytes", ctypes.c_uint32),
                ("group_rows", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("chunk_bytes", ctypes.c_uint32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class ibp_params(ctypes.Structure):
    _fields_ = [("group_rows", ctypes.c_uint32), ("chunk_bytes", ctypes.c_uint32),
                ("threshold_num", ctypes.c_uint32), ("threshold_den", ctypes.c_uint32),
                ("sample_every", ctypes.c_uint32)]


class ibp_stats(ctypes.Structure):
    _fields_ = [("calls", ctypes.c_uint64), ("rows_out", ctypes.c_uint64),
                ("out_bytes", ctypes.c_uint64), ("h2d_bytes", ctypes.c_uint64),
                ("h2d_payload_bytes", ctypes.c_uint64), ("host_pack_ns", ctypes.c_uint64),
                ("gather_meta_bytes", ctypes.c_uint64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class ibp_cache_stats(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_uint64), ("slab_bytes", ctypes.c_uint64), ("table_slots", ctypes.c_uint64),
                ("hits", ctypes.c_uint64), ("misses", ctypes.c_uint64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None
_vp, _u64, _u32, _i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int
_SIGS = {
    "ibp_compress_bound": [_u64, _u32, _u32, ctypes.POINTER(_u64)],
    "ibp_compress": [_vp, _u64, _u32, _u32, _i32, _vp, _u64, ctypes.POINTER(_u64)],
    "ibp_compress_ex": [_vp, _u64, _u32, ctypes.POINTER(ibp_params), _i32, _vp, _u64, ctypes.POINTER(_u64)],
    "ibp_describe": [_vp, _u64, ctypes.POINTER(ibp_desc)],
    "ibp_open": [_vp, _u64, _i32, _u32, ctypes.POINTER(_vp)],
    "ibp_decompress": [_vp, _u64, _u64, _vp, _u64, _vp],
    "ibp_gather_decompress": [_vp, _vp, _u64, _vp, _u64, _vp],
    "ibp_gather_decompress_device": [_vp, _vp, _u64, _vp, _u64, _vp],
    "ibp_gather_decompress_noalloc": [_vp, _vp, _u64, _vp, _u64, _vp],
    "ibp_device_errors": [_vp, ctypes.POINTER(_u64)],
    "ibp_get_desc": [_vp, ctypes.POINTER(ibp_desc)],
    "ibp_get_stats": [_vp, ctypes.POINTER(ibp_stats)],
    "ibp_reset_stats": [_vp],
    "ibp_close": [_vp],
    "ibp_memory_usage": [ctypes.POINTER(_u64), ctypes.POINTER(_u64)],
    "ibp_cache_create": [_vp, _vp, _u64, ctypes.POINTER(_vp)],
    "ibp_cache_gather": [_vp, _vp, _u64, _vp, _u64, _vp],
    "ibp_cache_get_stats": [_vp, ctypes.POINTER(ibp_cache_stats)],
    "ibp_cache_reset_stats": [_vp],
    "ibp_cache_destroy": [_vp],
}
EXPORTS = sorted(list(_SIGS) + ["ibp_last_error", "ibp_version"])


def lib():
    """The loaded library (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2605_30728_amd.build`")
    try:
        import torch  # noqa: F401  -- load torch's HIP runtime first so both share it
    except ImportError:
        pass
    L = ctypes.CDLL(LIB_PATH)
    for name, args in _SIGS.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.ibp_last_error.argtypes = []
    L.ibp_last_error.restype = ctypes.c_char_p
    L.ibp_version.argtypes = []
    L.ibp_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status, func):
    if status != IBP_OK:
        raise IbpError(status, func, lib().ibp_last_error().decode())


def _ptr(x):
    """Device/host address of a tensor, numpy array or integer."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)}")


def _device_tensor(x, what, dtype=None):
    """Checks that a device argument is a contiguous GPU tensor (of `dtype`, if given)
    before its address reaches a kernel; an integer is taken as a raw device address."""
    if isinstance(x, int):
        return
    if isinstance(x, np.ndarray) or not hasattr(x, "is_cuda"):
        raise TypeError(f"{what} must be a GPU tensor (or a raw device address), not {type(x).__name__}")
    if not x.is_cuda:
        raise TypeError(f"{what} must be on the GPU, not on {x.device}")
    if not x.is_contiguous():
        raise TypeError(f"{what} must be contiguous")
    if dtype is not None and x.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, not {x.dtype}")


def _device_ids(x):
    import torch
    _device_tensor(x, "row ids", torch.int64)


def _nbytes(x):
    if hasattr(x, "element_size"):
        return x.numel() * x.element_size()
    if isinstance(x, np.ndarray):
        return x.nbytes
    raise TypeError("give out_cap explicitly for a raw pointer")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _host_bytes(buf):
    a = np.ascontiguousarray(np.frombuffer(buf, np.uint8) if isinstance(buf, (bytes, bytearray)) else buf)
    return a


class Handle:
    """An open stream (ibp_handle*). Close with ibp_close(h) or use as a context manager."""

    def __init__(self, ptr):
        self.ptr = ptr

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        ibp_close(self)


def ibp_version():
    return lib().ibp_version().decode()


def ibp_last_error():
    return lib().ibp_last_error().decode()


def ibp_compress_bound(n_rows, row_bytes, group_rows):
    out = _u64(0)
    _check(lib().ibp_compress_bound(n_rows, row_bytes, group_rows, ctypes.byref(out)), "ibp_compress_bound")
    return out.value


def ibp_compress_ex(rows, group_rows, chunk_bytes=0, threshold=(1, 1), sample_every=1, n_threads=0):
    """Compress with explicit parameters (include/ibp.h ibp_compress_ex): chunk_bytes = 0
    is the clustered scheme; chunk_bytes > 0 the thresholded scheme with participation
    bits, T = threshold[0] / threshold[1] of the counted rows (every sample_every-th)."""
    a = np.ascontiguousarray(rows)
    if a.ndim != 2:
        raise ValueError("rows must be a 2-D array (n_rows, elements)")
    n_rows, row_bytes = a.shape[0], a.shape[1] * a.itemsize
    p = ibp_params(group_rows, chunk_bytes, threshold[0], threshold[1], sample_every)
    got = _u64(0)
    L = lib()
    st = L.ibp_compress_ex(a.ctypes.data, n_rows, row_bytes, ctypes.byref(p), n_threads, None, 0, ctypes.byref(got))
    if st != IBP_ENOMEM or got.value == 0:
        _check(st, "ibp_compress_ex")
    out = np.empty(got.value, np.uint8)
    _check(L.ibp_compress_ex(a.ctypes.data, n_rows, row_bytes, ctypes.byref(p), n_threads, out.ctypes.data,
                             got.value, ctypes.byref(got)), "ibp_compress_ex")
    return out[:got.value]


def ibp_compress(rows, group_rows, n_threads=0):
    """Compress a 2-D host array (n_rows, ...) of any dtype; returns the stream (uint8)."""
    a = np.ascontiguousarray(rows)
    if a.ndim != 2:
        raise ValueError("rows must be a 2-D array (n_rows, elements)")
    n_rows, row_bytes = a.shape[0], a.shape[1] * a.itemsize
    bound = ibp_compress_bound(n_rows, row_bytes, group_rows)
    got = _u64(0)
    L = lib()
    # size first (out_cap 0 reports the size), then the real call
    st = L.ibp_compress(a.ctypes.data, n_rows, row_bytes, group_rows, n_threads, None, 0, ctypes.byref(got))
    if st not in (IBP_OK, IBP_ENOMEM) or (st == IBP_ENOMEM and got.value == 0 and n_rows > 0):
        _check(st, "ibp_compress")
    size = got.value if got.value else bound
    out = np.empty(size, np.uint8)
    _check(L.ibp_compress(a.ctypes.data, n_rows, row_bytes, group_rows, n_threads, out.ctypes.data, size,
                          ctypes.byref(got)), "ibp_compress")
    return out[:got.value]


def ibp_describe(stream):
    s = _host_bytes(stream)
    d = ibp_desc()
    _check(lib().ibp_describe(s.ctypes.data, s.nbytes, ctypes.byref(d)), "ibp_describe")
    return d.as_dict()


def ibp_open(stream, device=0, flags=IBP_OPEN_PAYLOAD_DEVICE):
    s = _host_bytes(stream)
    h = _vp(0)
    _check(lib().ibp_open(s.ctypes.data, s.nbytes, device, flags, ctypes.byref(h)), "ibp_open")
    return Handle(h.value)


def ibp_decompress(h, first_row, n_rows, d_out, out_cap=None, stream=None):
    _device_tensor(d_out, "d_out")
    cap = _nbytes(d_out) if out_cap is None else out_cap
    _check(lib().ibp_decompress(h.ptr, first_row, n_rows, _ptr(d_out), cap, _stream(stream)), "ibp_decompress")


def ibp_gather_decompress(h, row_ids, d_out, out_cap=None, stream=None):
    ids = np.ascontiguousarray(row_ids, dtype=np.int64)
    _device_tensor(d_out, "d_out")
    cap = _nbytes(d_out) if out_cap is None else out_cap
    _check(lib().ibp_gather_decompress(h.ptr, ids.ctypes.data, ids.size, _ptr(d_out), cap, _stream(stream)),
           "ibp_gather_decompress")


def ibp_gather_decompress_noalloc(h, row_ids, d_out, out_cap=None, stream=None):
    ids = np.ascontiguousarray(row_ids, dtype=np.int64)
    _device_tensor(d_out, "d_out")
    cap = _nbytes(d_out) if out_cap is None else out_cap
    _check(lib().ibp_gather_decompress_noalloc(h.ptr, ids.ctypes.data, ids.size, _ptr(d_out), cap,
                                               _stream(stream)), "ibp_gather_decompress_noalloc")


def ibp_gather_decompress_device(h, d_row_ids, d_out, n_ids=None, out_cap=None, stream=None):
    _device_ids(d_row_ids)
    _device_tensor(d_out, "d_out")
    n = d_row_ids.numel() if n_ids is None else n_ids
    cap = _nbytes(d_out) if out_cap is None else out_cap
    _check(lib().ibp_gather_decompress_device(h.ptr, _ptr(d_row_ids), n, _ptr(d_out), cap, _stream(stream)),
           "ibp_gather_decompress_device")


def ibp_device_errors(h):
    c = _u64(0)
    _check(lib().ibp_device_errors(h.ptr, ctypes.byref(c)), "ibp_device_errors")
    return c.value


def ibp_memory_usage():
    """(device bytes, pinned host bytes) the library holds over all handles and caches."""
    dev, pin = _u64(0), _u64(0)
    _check(lib().ibp_memory_usage(ctypes.byref(dev), ctypes.byref(pin)), "ibp_memory_usage")
    return dev.value, pin.value


def ibp_get_desc(h):
    d = ibp_desc()
    _check(lib().ibp_get_desc(h.ptr, ctypes.byref(d)), "ibp_get_desc")
    return d.as_dict()


def ibp_get_stats(h):
    st = ibp_stats()
    _check(lib().ibp_get_stats(h.ptr, ctypes.byref(st)), "ibp_get_stats")
    return st.as_dict()


def ibp_reset_stats(h):
    _check(lib().ibp_reset_stats(h.ptr), "ibp_reset_stats")


def ibp_close(h):
    if h.ptr:
        st = lib().ibp_close(h.ptr)
        if st != IBP_ESTATE:      # the handle is freed on every other outcome
            h.ptr = None
        _check(st, "ibp_close")


class Cache:
    """A compressed device cache (ibp_cache*). Destroy with ibp_cache_destroy(c) or use as
    a context manager."""

    def __init__(self, ptr, handle):
        self.ptr = ptr
        self.handle = handle

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        ibp_cache_destroy(self)


def ibp_cache_create(h, row_ids):
    ids = np.ascontiguousarray(row_ids, dtype=np.int64)
    c = _vp(0)
    _check(lib().ibp_cache_create(h.ptr, ids.ctypes.data, ids.size, ctypes.byref(c)), "ibp_cache_create")
    return Cache(c.value, h)


def ibp_cache_gather(c, d_row_ids, d_out, n_ids=None, out_cap=None, stream=None):
    _device_ids(d_row_ids)
    _device_tensor(d_out, "d_out")
    n = d_row_ids.numel() if n_ids is None else n_ids
    cap = _nbytes(d_out) if out_cap is None else out_cap
    _check(lib().ibp_cache_gather(c.ptr, _ptr(d_row_ids), n, _ptr(d_out), cap, _stream(stream)), "ibp_cache_gather")


def ibp_cache_get_stats(c):
    st = ibp_cache_stats()
    _check(lib().ibp_cache_get_stats(c.ptr, ctypes.byref(st)), "ibp_cache_get_stats")
    return st.as_dict()


def ibp_cache_reset_stats(c):
    _check(lib().ibp_cache_reset_stats(c.ptr), "ibp_cache_reset_stats")


def ibp_cache_destroy(c):
    if c.ptr:
        st = lib().ibp_cache_destroy(c.ptr)
        if st != IBP_ESTATE:      # the cache is freed on every other outcome
            c.ptr = None
        _check(st, "ibp_cache_destroy")
