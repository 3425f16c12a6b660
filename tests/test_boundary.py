"""C-ABI boundary checks that need no GPU: the library loads, exports every
function its header declares, and rejects invalid arguments before any HIP
call (status codes and messages)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2008_00325_amd import umap_layout as U

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "umap_layout.h")


@pytest.fixture(scope="module")
def L():
    return U.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(umap_\w+)\s*\(", text)))


def test_every_declared_function_is_exported(L):
    names = _declared()
    assert len(names) == 27
    for name in names:
        assert hasattr(L, name), name
        assert name in U.EXPORTS
    assert sorted(U.EXPORTS) == names


def test_status_codes_match_header():
    text = open(HEADER).read()
    codes = dict((m, int(v)) for m, v in re.findall(r"#define (UMAP_\w+) \(?(-?\d+)\)?", text))
    for name, value in codes.items():
        assert getattr(U, name) == value


def _create(n=4, dim=2, rows=(0, 1), cols=(1, 0), vals=(1.0, 1.0), a=1.5, b=0.9, N=10, R=5):
    return U.umap_layout_create(n, dim, np.array(rows), np.array(cols), np.array(vals), a, b, N, R)


@pytest.mark.parametrize("kw,frag", [
    (dict(n=0), "n must be"),
    (dict(n=2**31), "n must be"),
    (dict(dim=0), "n_components"),
    (dict(dim=17), "n_components"),
    (dict(a=0.0), "a must be"),
    (dict(a=float("nan")), "a must be"),
    (dict(b=-1.0), "b must be"),
    (dict(b=float("inf")), "b must be"),
    (dict(N=0), "n_epochs"),
    (dict(N=2**24), "n_epochs"),
    (dict(R=-1), "neg_rate"),
    (dict(R=2**16), "neg_rate"),
    (dict(rows=(0, 4)), "outside"),
    (dict(cols=(-1, 0)), "outside"),
    (dict(vals=(1.0, float("nan"))), "not finite"),
    (dict(vals=(float("inf"), 1.0)), "not finite"),
])
def test_create_rejects_invalid_arguments(kw, frag):
    with pytest.raises(U.UmapLayoutError) as ei:
        _create(**kw)
    assert ei.value.code == U.UMAP_E_INVAL
    assert frag in U.umap_layout_last_error()


def test_create_device_rejects_scalars_without_touching_the_gpu(L):
    out = ctypes.c_void_p(123)
    rc = L.umap_layout_create_device(ctypes.byref(out), 10, 0, None, None, None, 0, 1.0, 1.0, 10, 5, None)
    assert rc == U.UMAP_E_INVAL and out.value is None
    rc = L.umap_layout_create_device(ctypes.byref(out), 10, 2, None, None, None, 5, 1.0, 1.0, 10, 5, None)
    assert rc == U.UMAP_E_INVAL and "NULL" in U.umap_layout_last_error()
    assert L.umap_layout_create(None, 10, 2, None, None, None, 0, 1.0, 1.0, 10, 5) == U.UMAP_E_INVAL


def test_null_handles_are_rejected(L):
    assert L.umap_layout_run(None, 1) == U.UMAP_E_INVAL
    assert L.umap_layout_init(None, 1) == U.UMAP_E_INVAL
    assert L.umap_layout_run_epochs(None, 1, 0, 1) == U.UMAP_E_INVAL
    assert L.umap_layout_get(None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_get_device(None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_set_embedding(None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_get_graph(None, None, None, None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_stats(None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_set_stream(None, None) == U.UMAP_E_INVAL
    assert L.umap_layout_set_kernel(None, 0) == U.UMAP_E_INVAL
    assert L.umap_layout_set_mode(None, U.UMAP_MODE_SYNC) == U.UMAP_E_INVAL
    assert L.umap_layout_set_rows(None, 0, 1) == U.UMAP_E_INVAL
    assert L.umap_layout_set_epoch_timing(None, 1) == U.UMAP_E_INVAL
    assert L.umap_layout_epoch_ms(None, None, 0) == U.UMAP_E_INVAL
    assert L.umap_layout_debug_active(None, 0, None) == U.UMAP_E_INVAL
    assert L.umap_layout_debug_negatives(None, 0, 0, 0, 0, None) == U.UMAP_E_INVAL
    L.umap_layout_destroy(None)  # no-op


def test_fuzzy_graph_and_probe_argument_checks(L):
    p = ctypes.c_void_p(16)
    assert L.umap_fuzzy_graph_device(0, 15, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device(10, 0, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device(10, 1025, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device(2**30, 2, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device(10, 5, None, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device_noalloc(0, 15, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device_noalloc(2**20 + 1, 15, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert "no-allocation" in U.umap_layout_last_error()
    assert L.umap_fuzzy_graph_device_noalloc(10, 0, p, p, p, p, p, None) == U.UMAP_E_INVAL
    assert L.umap_fuzzy_graph_device_noalloc(10, 5, p, p, p, p, None, None) == U.UMAP_E_INVAL
    assert L.umap_probe_copy(p, p, 17, None) == U.UMAP_E_INVAL
    assert L.umap_probe_copy(None, p, 16, None) == U.UMAP_E_INVAL
    assert L.umap_probe_gather(p, 3, 256, 1, p, None) == U.UMAP_E_INVAL
    assert L.umap_probe_gather(p, 4, 100, 1, p, None) == U.UMAP_E_INVAL
    assert L.umap_probe_gather(p, 4, 256, 0, p, None) == U.UMAP_E_INVAL
    assert L.umap_probe_gather(None, 4, 256, 1, p, None) == U.UMAP_E_INVAL
    out = ctypes.c_double(7.0)
    for n, d, dim, k in [(0, 4, 2, 1), (100, 0, 2, 15), (100, 4, 0, 15), (100, 4, 17, 15), (100, 4, 2, 0),
                         (100, 4, 2, 65), (22, 4, 2, 15)]:
        assert L.umap_trustworthiness(p, n, d, p, dim, k, ctypes.byref(out), None) == U.UMAP_E_INVAL
    assert L.umap_trustworthiness(None, 100, 4, p, 2, 15, ctypes.byref(out), None) == U.UMAP_E_INVAL
    assert L.umap_trustworthiness(p, 100, 4, p, 2, 15, None, None) == U.UMAP_E_INVAL
    assert out.value == 7.0


def test_transform_create_argument_checks(L):
    """Every check of umap_transform_create runs before a HIP call."""
    T = np.zeros((5, 2), np.float32)
    r = np.array([0, 1], np.int32)
    c = np.array([4, 4], np.int32)
    v = np.ones(2, np.float32)
    P = ctypes.c_void_p
    out = P()

    def call(n_new=3, table=T, n_table=5, rows=r, cols=c, vals=v, dim=2, nnz=2, a=1.0, b=1.0, N=10, R=5,
             outp=ctypes.byref(out)):
        tp = None if table is None else table.ctypes.data_as(P)
        return L.umap_transform_create(outp, n_new, dim, tp, n_table, rows.ctypes.data_as(P),
                                       cols.ctypes.data_as(P), vals.ctypes.data_as(P), nnz, a, b, N, R)

    assert call(outp=None) == U.UMAP_E_INVAL
    assert call(n_new=0) == U.UMAP_E_INVAL
    assert call(n_table=0) == U.UMAP_E_INVAL
    assert call(table=None) == U.UMAP_E_INVAL
    assert call(dim=17) == U.UMAP_E_INVAL
    assert call(table=np.array([[0, 0], [0, np.inf], [0, 0], [0, 0], [0, 0]], np.float32)) == U.UMAP_E_INVAL
    assert call(cols=np.array([4, 5], np.int32)) == U.UMAP_E_INVAL     # column beyond the table
    assert call(rows=np.array([0, 3], np.int32)) == U.UMAP_E_INVAL     # row beyond the new points
    assert call(vals=np.array([1, np.nan], np.float32)) == U.UMAP_E_INVAL
    assert call(N=0) == U.UMAP_E_INVAL
    assert not out.value


def test_fit_ab_matches_oracle(orc):
    for spread, md in [(1.0, 0.1), (1.0, 0.5), (2.0, 0.05), (0.5, 0.0)]:
        a, b = U.umap_fit_ab(spread, md)
        ra, rb = orc.fit_ab(spread, md)
        assert abs(a - ra) < 1e-5 * ra and abs(b - rb) < 1e-5 * rb
    with pytest.raises(U.UmapLayoutError):
        U.umap_fit_ab(0.0, 0.1)
    with pytest.raises(U.UmapLayoutError):
        U.umap_fit_ab(1.0, 3.5)


def test_create_without_a_gpu_reports_device_error():
    import torch

    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(U.UmapLayoutError) as ei:
        _create()
    assert ei.value.code == U.UMAP_E_DEVICE


# ---------------------------------------------------------------------------
# the Python binding checks device tensors before they reach the C ABI: a
# wrong device, layout, dtype or size would be an out-of-bounds device access
# ---------------------------------------------------------------------------

class _FakeCuda:
    """Stands in for a GPU tensor on a host without one (the checks read only
    these attributes; every case below has at least one bad argument, so the
    library is never called and the null address is never used)."""

    def __init__(self, dtype="float32", numel=16, contiguous=True, itemsize=4, shape=None):
        import torch

        self.shape = shape if shape is not None else (numel,)
        self.is_cuda = True
        self.dtype = getattr(torch, dtype)
        self._n = numel
        self._c = contiguous
        self._s = itemsize
        self.device = "cuda:0"

    def is_contiguous(self):
        return self._c

    def numel(self):
        return self._n

    def element_size(self):
        return self._s

    def data_ptr(self):
        return 0


def test_binding_rejects_bad_device_tensors():
    import torch

    h = U.Handle(None, 10, 2)
    cases = [
        (lambda: U.umap_layout_get_device(h, torch.zeros(20)), "GPU tensor"),
        (lambda: U.umap_layout_get_device(h, _FakeCuda("float32", 19)), "needs 20"),
        (lambda: U.umap_layout_get_device(h, _FakeCuda("float64", 40, itemsize=8)), "float32"),
        (lambda: U.umap_layout_get_device(h, _FakeCuda("float32", 40, contiguous=False)), "contiguous"),
        (lambda: U.umap_layout_create_device(10, 2, _FakeCuda("int32", 7), _FakeCuda("int32", 8),
                                             _FakeCuda("float32", 8), 8, 1.5, 0.9, 10, 5), "rows holds 7"),
        (lambda: U.umap_layout_create_device(10, 2, _FakeCuda("int32", 8), _FakeCuda("int64", 8, itemsize=8),
                                             _FakeCuda("float32", 8), 8, 1.5, 0.9, 10, 5), "cols must hold int32"),
        (lambda: U.umap_layout_create_device(10, 2, _FakeCuda("int32", 8), _FakeCuda("int32", 8),
                                             torch.zeros(8), 8, 1.5, 0.9, 10, 5), "vals must be a GPU tensor"),
        (lambda: U.umap_layout_create_device(10, 2, _FakeCuda("int32", 8), _FakeCuda("int32", 8),
                                             _FakeCuda("float32", 8), -1, 1.5, 0.9, 10, 5), "nnz"),
        (lambda: U.umap_fuzzy_graph_device(5, 3, _FakeCuda("int32", 15), _FakeCuda("float32", 15),
                                           _FakeCuda("int32", 30), _FakeCuda("int32", 30), _FakeCuda("float32", 29)),
         "vals holds 29"),
        (lambda: U.umap_fuzzy_graph_device(5, 3, _FakeCuda("int32", 14), _FakeCuda("float32", 15),
                                           _FakeCuda("int32", 30), _FakeCuda("int32", 30), _FakeCuda("float32", 30)),
         "knn_ids holds 14"),
        (lambda: U.umap_trustworthiness(_FakeCuda("float32", 11), _FakeCuda("float32", 8), 3), "two-dimensional"),
        (lambda: U.umap_trustworthiness(_FakeCuda("float32", 39, shape=(10, 4)), _FakeCuda("float32", 20, shape=(10, 2)), 3),
         "X holds 39"),
        (lambda: U.umap_probe_copy(_FakeCuda("float32", 3), _FakeCuda("float32", 4), 16), "src holds 12 bytes"),
        (lambda: U.umap_probe_gather(_FakeCuda("float32", 15), 8, 256, 1, _FakeCuda("float32", 256)),
         "table holds 60 bytes"),
    ]
    for call, frag in cases:
        with pytest.raises(ValueError) as ei:
            call()
        assert frag in str(ei.value), (frag, str(ei.value))
