"""ctypes binding of libumap_layout.so (include/umap_layout.h).

Argument marshalling only: every step of the layout runs in the library's HIP
kernels.  Host arrays are numpy arrays; device arrays may be passed as torch
tensors (their ``data_ptr()``) or raw integer addresses.  Streams are
``torch.cuda.Stream`` objects, raw ``hipStream_t`` integers or None (null
stream).  Errors raise :class:`UmapLayoutError` carrying the C status code and
the library's message.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libumap_layout.so")

UMAP_OK = 0
UMAP_E_INVAL = -1
UMAP_E_ASYMMETRIC = -2
UMAP_E_NOMEM = -3
UMAP_E_DEVICE = -4
UMAP_E_STATE = -5
UMAP_MODE_SYNC = 0
UMAP_MODE_ASYNC = 1
UMAP_MAX_TIMED_EPOCHS = 4096

EXPORTS = (
    "umap_layout_create", "umap_layout_create_device", "umap_transform_create", "umap_layout_run",
    "umap_layout_init", "umap_layout_run_epochs",
    "umap_layout_get", "umap_layout_get_device", "umap_layout_set_embedding", "umap_layout_get_graph",
    "umap_layout_stats", "umap_layout_set_stream", "umap_layout_destroy", "umap_layout_last_error",
    "umap_layout_debug_active", "umap_layout_debug_negatives", "umap_layout_set_kernel", "umap_layout_set_mode",
    "umap_layout_set_rows", "umap_layout_set_epoch_timing", "umap_layout_epoch_ms",
    "umap_fuzzy_graph_device", "umap_fuzzy_graph_device_noalloc", "umap_fit_ab", "umap_probe_copy", "umap_probe_gather",
    "umap_trustworthiness",
)


class umap_layout_stats_t(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64),
        ("n_components", ctypes.c_int32),
        ("n_epochs", ctypes.c_int32),
        ("neg_rate", ctypes.c_int32),
        ("epochs_done", ctypes.c_int32),
        ("nnz_input", ctypes.c_int64),
        ("nnz_kept", ctypes.c_int64),
        ("max_degree", ctypes.c_int32),
        ("w_max", ctypes.c_float),
        ("active_edges", ctypes.c_int64),
        ("edge_updates", ctypes.c_int64),
        ("prep_ms", ctypes.c_double),
        ("init_ms", ctypes.c_double),
        ("epochs_ms", ctypes.c_double),
        ("table_ranges", ctypes.c_int32),
        ("kernel", ctypes.c_int32),
        ("overflow_redone", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("row_first", ctypes.c_int64),
        ("row_last", ctypes.c_int64),
        ("n_waves", ctypes.c_int64),
    ]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class UmapLayoutError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the native library; fail loudly when it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, u64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
        PP = ctypes.POINTER(ctypes.c_void_p)
        sig = {
            "umap_layout_create": [PP, i64, i32, P, P, P, i64, f32, f32, i32, i32],
            "umap_layout_create_device": [PP, i64, i32, P, P, P, i64, f32, f32, i32, i32, P],
            "umap_transform_create": [PP, i64, i32, P, i64, P, P, P, i64, f32, f32, i32, i32],
            "umap_layout_run": [P, u64],
            "umap_layout_init": [P, u64],
            "umap_layout_run_epochs": [P, u64, i32, i32],
            "umap_layout_get": [P, P],
            "umap_layout_get_device": [P, P],
            "umap_layout_set_embedding": [P, P],
            "umap_layout_get_graph": [P, P, P, P, P],
            "umap_layout_stats": [P, ctypes.POINTER(umap_layout_stats_t)],
            "umap_layout_set_stream": [P, P],
            "umap_layout_destroy": [P],
            "umap_layout_last_error": [],
            "umap_layout_debug_active": [P, i32, P],
            "umap_layout_debug_negatives": [P, u64, i32, i64, i64, P],
            "umap_layout_set_kernel": [P, i32],
            "umap_layout_set_mode": [P, i32],
            "umap_layout_set_rows": [P, i64, i64],
            "umap_layout_set_epoch_timing": [P, i32],
            "umap_layout_epoch_ms": [P, P, i32],
            "umap_fuzzy_graph_device": [i64, i32, P, P, P, P, P, P],
            "umap_fuzzy_graph_device_noalloc": [i64, i32, P, P, P, P, P, P],
            "umap_fit_ab": [f32, f32, ctypes.POINTER(f32), ctypes.POINTER(f32)],
            "umap_probe_copy": [P, P, i64, P],
            "umap_probe_gather": [P, i64, i64, i32, P, P],
            "umap_trustworthiness": [P, i64, i32, P, i32, i32, ctypes.POINTER(ctypes.c_double), P],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.umap_layout_destroy.restype = None
        L.umap_layout_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def umap_layout_last_error() -> str:
    return lib().umap_layout_last_error().decode()


def _check(rc: int) -> None:
    if rc != UMAP_OK:
        raise UmapLayoutError(rc, umap_layout_last_error())


def _dev(x, dtype: str | None = None, count: int = 0, name: str = "array") -> int | None:
    """Device address of a torch tensor, checked before it reaches the C ABI:
    a tensor must live on the GPU, be contiguous, hold `dtype` elements
    ("int32" / "float32"; None: any) and at least `count` of them (for an
    untyped buffer, `count` bytes), since the library reads or writes exactly
    that many.  A raw integer address is passed through unchecked (the caller
    vouches for it).  Raises ValueError."""
    if x is None:
        return None
    if not hasattr(x, "data_ptr"):
        return int(x)
    if not getattr(x, "is_cuda", False):
        raise ValueError(f"{name} must be a GPU tensor, got one on {getattr(x, 'device', '?')}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None:
        got = str(x.dtype).replace("torch.", "")
        if got != dtype:
            raise ValueError(f"{name} must hold {dtype}, got {got}")
        if x.numel() < count:
            raise ValueError(f"{name} holds {x.numel()} elements, the call needs {count}")
    elif x.numel() * x.element_size() < count:
        raise ValueError(f"{name} holds {x.numel() * x.element_size()} bytes, the call needs {count}")
    return int(x.data_ptr())


def _stream(s) -> int | None:
    if s is None:
        return None
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream)
    return int(s)


def _host(a: np.ndarray, dtype) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _hp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Handle:
    """Owner of a umap_layout* (destroyed on close / garbage collection)."""

    def __init__(self, ptr: ctypes.c_void_p, n: int, dim: int):
        self.ptr = ptr
        self.n = n
        self.dim = dim

    def close(self) -> None:
        if self.ptr:
            lib().umap_layout_destroy(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def umap_layout_create(n: int, n_components: int, rows, cols, vals, a: float, b: float, n_epochs: int,
                       neg_rate: int) -> Handle:
    r = _host(rows, np.int32)
    c = _host(cols, np.int32)
    v = _host(vals, np.float32)
    if not (r.size == c.size == v.size):
        raise ValueError("rows, cols and vals must have the same length")
    out = ctypes.c_void_p()
    _check(lib().umap_layout_create(ctypes.byref(out), n, n_components, _hp(r), _hp(c), _hp(v), r.size, a, b,
                                    n_epochs, neg_rate))
    return Handle(out, n, n_components)


def umap_transform_create(n_new: int, table, rows, cols, vals, a: float, b: float, n_epochs: int,
                          neg_rate: int) -> Handle:
    t = _host(table, np.float32)
    if t.ndim != 2:
        raise ValueError("table must be an n_table x n_components array")
    r = _host(rows, np.int32)
    c = _host(cols, np.int32)
    v = _host(vals, np.float32)
    if not (r.size == c.size == v.size):
        raise ValueError("rows, cols and vals must have the same length")
    out = ctypes.c_void_p()
    _check(lib().umap_transform_create(ctypes.byref(out), n_new, t.shape[1], _hp(t), t.shape[0], _hp(r), _hp(c),
                                       _hp(v), r.size, a, b, n_epochs, neg_rate))
    return Handle(out, n_new, t.shape[1])


def umap_layout_create_device(n: int, n_components: int, rows, cols, vals, nnz: int, a: float, b: float,
                              n_epochs: int, neg_rate: int, stream=None) -> Handle:
    out = ctypes.c_void_p()
    if nnz < 0:
        raise ValueError("nnz must be >= 0")
    dr = _dev(rows, "int32", nnz, "rows")
    dc = _dev(cols, "int32", nnz, "cols")
    dv = _dev(vals, "float32", nnz, "vals")
    _check(lib().umap_layout_create_device(ctypes.byref(out), n, n_components, dr, dc, dv, nnz, a, b, n_epochs,
                                           neg_rate, _stream(stream)))
    return Handle(out, n, n_components)


def umap_layout_run(h: Handle, seed: int) -> None:
    _check(lib().umap_layout_run(h.ptr, seed))


def umap_layout_init(h: Handle, seed: int) -> None:
    _check(lib().umap_layout_init(h.ptr, seed))


def umap_layout_run_epochs(h: Handle, seed: int, first: int, last: int) -> None:
    _check(lib().umap_layout_run_epochs(h.ptr, seed, first, last))


def umap_layout_get(h: Handle) -> np.ndarray:
    out = np.empty((h.n, h.dim), dtype=np.float32)
    _check(lib().umap_layout_get(h.ptr, _hp(out)))
    return out


def umap_layout_get_device(h: Handle, dev_out) -> None:
    _check(lib().umap_layout_get_device(h.ptr, _dev(dev_out, "float32", h.n * h.dim, "dev_out")))


def umap_layout_set_embedding(h: Handle, E: np.ndarray) -> None:
    e = _host(E, np.float32)
    if e.shape != (h.n, h.dim):
        raise ValueError(f"embedding must have shape {(h.n, h.dim)}")
    _check(lib().umap_layout_set_embedding(h.ptr, _hp(e)))


def umap_layout_set_epoch_timing(h: Handle, enabled: bool) -> None:
    _check(lib().umap_layout_set_epoch_timing(h.ptr, 1 if enabled else 0))


def umap_layout_epoch_ms(h: Handle) -> np.ndarray:
    """Device ms of each epoch the last call timed (empty when timing was off)."""
    n = lib().umap_layout_epoch_ms(h.ptr, None, 0)
    _check(min(n, 0))
    out = np.empty(max(n, 1), dtype=np.float32)
    got = lib().umap_layout_epoch_ms(h.ptr, out.ctypes.data, n)
    _check(min(got, 0))
    return out[:n]


def umap_layout_stats(h: Handle) -> dict:
    s = umap_layout_stats_t()
    _check(lib().umap_layout_stats(h.ptr, ctypes.byref(s)))
    return s.as_dict()


def umap_layout_get_graph(h: Handle):
    st = umap_layout_stats(h)
    nnz = st["nnz_kept"]
    row_ptr = np.empty(h.n + 1, dtype=np.int64)
    col = np.empty(max(nnz, 1), dtype=np.int32)
    eps = np.empty(max(nnz, 1), dtype=np.float32)
    kept = ctypes.c_int64()
    _check(lib().umap_layout_get_graph(h.ptr, _hp(row_ptr), _hp(col), _hp(eps), ctypes.byref(kept)))
    return row_ptr, col[: kept.value].copy(), eps[: kept.value].copy()


def umap_layout_set_stream(h: Handle, stream) -> None:
    _check(lib().umap_layout_set_stream(h.ptr, _stream(stream)))


def umap_layout_set_kernel(h: Handle, which: int) -> None:
    _check(lib().umap_layout_set_kernel(h.ptr, which))


def umap_layout_set_mode(h: Handle, mode: int) -> None:
    _check(lib().umap_layout_set_mode(h.ptr, mode))


def umap_layout_set_rows(h: Handle, row_first: int, row_last: int) -> None:
    _check(lib().umap_layout_set_rows(h.ptr, row_first, row_last))


def umap_layout_destroy(h: Handle) -> None:
    h.close()


def umap_layout_debug_active(h: Handle, epoch: int) -> np.ndarray:
    nnz = umap_layout_stats(h)["nnz_kept"]
    out = np.empty(max(nnz, 1), dtype=np.uint8)
    _check(lib().umap_layout_debug_active(h.ptr, epoch, _hp(out)))
    return out[:nnz].astype(bool)


def umap_layout_debug_negatives(h: Handle, seed: int, epoch: int, e_first: int, count: int) -> np.ndarray:
    R = umap_layout_stats(h)["neg_rate"]
    out = np.empty((max(count, 1), max(R, 1)), dtype=np.uint32)
    _check(lib().umap_layout_debug_negatives(h.ptr, seed, epoch, e_first, count, _hp(out)))
    return out[:count, :R].copy()


def umap_fuzzy_graph_device(n: int, k: int, knn_ids, knn_dists, rows, cols, vals, stream=None) -> None:
    nk = max(n, 0) * max(k, 0)
    _check(lib().umap_fuzzy_graph_device(n, k, _dev(knn_ids, "int32", nk, "knn_ids"),
                                         _dev(knn_dists, "float32", nk, "knn_dists"), _dev(rows, "int32", 2 * nk, "rows"),
                                         _dev(cols, "int32", 2 * nk, "cols"), _dev(vals, "float32", 2 * nk, "vals"),
                                         _stream(stream)))


def umap_fuzzy_graph_device_noalloc(n: int, k: int, knn_ids, knn_dists, rows, cols, vals, stream=None) -> None:
    nk = max(n, 0) * max(k, 0)
    _check(lib().umap_fuzzy_graph_device_noalloc(n, k, _dev(knn_ids, "int32", nk, "knn_ids"),
                                                 _dev(knn_dists, "float32", nk, "knn_dists"),
                                                 _dev(rows, "int32", 2 * nk, "rows"), _dev(cols, "int32", 2 * nk, "cols"),
                                                 _dev(vals, "float32", 2 * nk, "vals"), _stream(stream)))


def umap_fit_ab(spread: float = 1.0, min_dist: float = 0.1) -> tuple[float, float]:
    a = ctypes.c_float()
    b = ctypes.c_float()
    _check(lib().umap_fit_ab(spread, min_dist, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def umap_probe_copy(src, dst, nbytes: int, stream=None) -> None:
    _check(lib().umap_probe_copy(_dev(src, None, nbytes, "src"), _dev(dst, None, nbytes, "dst"), nbytes,
                                 _stream(stream)))


def umap_trustworthiness(X, Y, k: int, stream=None) -> float:
    """T(k) of embedding Y (n x dim) of points X (n x d); both device tensors (fp32, contiguous)."""
    if len(X.shape) != 2 or len(Y.shape) != 2:
        raise ValueError("X and Y must be two-dimensional")
    n, d = int(X.shape[0]), int(X.shape[1])
    dim = int(Y.shape[1])
    if int(Y.shape[0]) != n:
        raise ValueError("X and Y need the same number of rows")
    out = ctypes.c_double()
    _check(lib().umap_trustworthiness(_dev(X, "float32", n * d, "X"), n, d, _dev(Y, "float32", n * dim, "Y"), dim, k,
                                      ctypes.byref(out), _stream(stream)))
    return out.value


def umap_probe_gather(table, entries: int, threads: int, iters: int, out, stream=None) -> None:
    _check(lib().umap_probe_gather(_dev(table, None, 8 * max(entries, 0), "table"), entries, threads, iters,
                                   _dev(out, None, 4 * max(threads, 0), "out"), _stream(stream)))
