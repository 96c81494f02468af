"""The C-ABI library on the host (no GPU): it loads, exports every symbol
that include/spl.h declares, and rejects bad arguments with status codes
before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spl.h")

OK, INVALID, UNSUPPORTED, OVERFLOW = 0, 1, 2, 3


@pytest.fixture(scope="module")
def L():
    from paper_2405_03594_amd import LIB_PATH, build

    if not os.path.exists(LIB_PATH):
        build.build()
    import paper_2405_03594_amd as spl

    return spl.lib()


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spl_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("spl_pack_count", "spl_pack_sparse", "spl_sparse_linear", "spl_sparse_linear_int8",
                     "spl_unpack", "spl_dense_linear", "spl_dense_linear_int8"):
        assert required in names


def test_every_declared_symbol_is_exported(L):
    for name in _declared():
        assert hasattr(L, name), name


def test_status_strings(L):
    for s in range(5):
        assert L.spl_status_string(s)
    assert L.spl_version() >> 16 == 1


def _mat(**kw):
    from paper_2405_03594_amd import _Matrix

    d = dict(rows=4, cols=64, dtype=2, layout=0, nnz=10, bitmask=0x10000, values=0x20000, row_offsets=0x30000,
             tile_offsets=0, values_bytes=1 << 20)
    d.update(kw)
    return _Matrix(**d)


@pytest.mark.parametrize("kw,status", [
    ({}, OK),
    (dict(rows=0), INVALID),
    (dict(cols=-1), INVALID),
    (dict(dtype=9), INVALID),
    (dict(layout=2), INVALID),
    (dict(layout=1), INVALID),                          # tile layout needs tile_offsets
    (dict(layout=1, tile_offsets=0x40000, row_offsets=0), OK),
    (dict(layout=1, tile_offsets=0x40002), INVALID),
    (dict(nnz=-1), INVALID),
    (dict(nnz=257), INVALID),
    (dict(rows=1 << 20, cols=1 << 20, nnz=1 << 31), OVERFLOW),
    (dict(bitmask=0), INVALID),
    (dict(row_offsets=0), INVALID),
    (dict(values=0), INVALID),
    (dict(values=0, nnz=0), INVALID),                   # values always point at an allocation
    (dict(values_bytes=0), INVALID),
    (dict(values_bytes=47), INVALID),                   # 10 bf16 payloads: 20 -> 32, + 16 = 48 bytes
    (dict(values_bytes=48), OK),
    (dict(dtype=3, values_bytes=31), INVALID),          # 10 int8 payloads: 16 + 16
    (dict(dtype=3, values_bytes=32), OK),
    (dict(nnz=0, values_bytes=16), OK),
    (dict(bitmask=0x10004), INVALID),
    (dict(values=0x20008), INVALID),
    (dict(row_offsets=0x30002), INVALID),
])
def test_check_matrix(L, kw, status):
    m = _mat(**kw)
    assert L.spl_check_matrix(ctypes.byref(m)) == status


def test_null_view(L):
    assert L.spl_check_matrix(None) == INVALID


def test_sparse_linear_argument_checks(L):
    m = _mat(layout=1, tile_offsets=0x40000)
    X, Y = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000)
    f = L.spl_sparse_linear_ex
    assert f(None, 2, ctypes.byref(m), Y, 0, None) == INVALID
    assert f(X, 2, ctypes.byref(m), None, 0, None) == INVALID
    assert f(X, -1, ctypes.byref(m), Y, 0, None) == INVALID
    assert f(None, 0, ctypes.byref(m), None, 0, None) == OK            # M = 0 is a no-op
    assert f(ctypes.c_void_p(0x40002), 2, ctypes.byref(m), Y, 0, None) == INVALID
    assert f(X, 2, ctypes.byref(m), Y, 7, None) == INVALID            # unknown algorithm
    assert f(X, 33, ctypes.byref(m), Y, 1, None) == UNSUPPORTED       # decode family is M <= 32
    m8 = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    assert f(X, 2, ctypes.byref(m8), Y, 0, None) == UNSUPPORTED       # int8 view needs the int8 entry
    mr = _mat()
    assert f(X, 2, ctypes.byref(mr), Y, 0, None) == UNSUPPORTED       # row layout: retile first
    mk = _mat(cols=100, layout=1, tile_offsets=0x40000)
    assert f(X, 2, ctypes.byref(mk), Y, 0, None) == UNSUPPORTED       # K % 8 != 0
    assert f(X, 2, None, Y, 0, None) == INVALID


def test_sparse_linear_expanded_argument_checks(L):
    m = _mat(layout=1, tile_offsets=0x40000)
    X, Y, ws = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000), ctypes.c_void_p(0x80000)
    L.spl_sparse_linear_expanded_workspace_bytes.restype = ctypes.c_int64
    need = L.spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(m))
    assert need >= 2 * m.rows * m.cols and need % 256 == 0
    assert L.spl_sparse_linear_expanded_workspace_bytes(None) == -1
    f = L.spl_sparse_linear_expanded
    assert f(X, 2, ctypes.byref(m), Y, None, None) == INVALID              # no workspace
    assert f(X, 2, ctypes.byref(m), Y, ctypes.c_void_p(0x80008), None) == INVALID   # misaligned workspace
    assert f(None, 0, ctypes.byref(m), None, ws, None) == OK               # M = 0 is a no-op
    assert f(X, -1, ctypes.byref(m), Y, ws, None) == INVALID
    m8 = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    assert f(X, 2, ctypes.byref(m8), Y, ws, None) == UNSUPPORTED          # fp16/bf16 only
    mk = _mat(cols=100, layout=1, tile_offsets=0x40000)
    assert f(X, 2, ctypes.byref(mk), Y, ws, None) == UNSUPPORTED          # K % 8 != 0
    assert f(X, 2, None, Y, ws, None) == INVALID


def test_int8_expanded_argument_checks(L):
    m = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    X, Y, s, ws = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000), ctypes.c_void_p(0x60000), ctypes.c_void_p(0x80000)
    L.spl_sparse_linear_expanded_workspace_bytes.restype = ctypes.c_int64
    assert L.spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(m)) >= m.rows * m.cols   # one byte per code
    f = L.spl_sparse_linear_int8_expanded
    assert f(X, s, 2, ctypes.byref(m), s, Y, None, None, None) == INVALID          # no workspace
    assert f(X, s, 2, ctypes.byref(m), s, Y, None, ctypes.c_void_p(0x80004), None) == INVALID
    assert f(X, None, 2, ctypes.byref(m), s, Y, None, ws, None) == INVALID         # no activation scales
    assert f(None, None, 0, ctypes.byref(m), None, None, None, ws, None) == OK     # M = 0 is a no-op
    mb = _mat(layout=1, tile_offsets=0x40000)
    assert f(X, s, 2, ctypes.byref(mb), s, Y, None, ws, None) == UNSUPPORTED      # a bf16 view
    assert f(X, s, 2, None, s, Y, None, ws, None) == INVALID


def test_int8_argument_checks(L):
    m = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    X, Y, s = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000), ctypes.c_void_p(0x60000)
    f = L.spl_sparse_linear_int8
    assert f(X, None, 2, ctypes.byref(m), s, Y, None, None) == INVALID
    assert f(X, s, 2, ctypes.byref(m), None, Y, None, None) == INVALID
    assert f(X, s, 2, ctypes.byref(m), s, Y, ctypes.c_void_p(0x70004), None) == INVALID
    mk = _mat(dtype=3, cols=40, layout=1, tile_offsets=0x40000)
    assert f(X, s, 2, ctypes.byref(mk), s, Y, None, None) == UNSUPPORTED
    mb = _mat(dtype=2, layout=1, tile_offsets=0x40000)
    assert f(X, s, 2, ctypes.byref(mb), s, Y, None, None) == UNSUPPORTED
    assert f(None, None, 0, ctypes.byref(m), None, None, None, None) == OK


@pytest.mark.parametrize("layout", [0, 1])
def test_pack_argument_checks(L, layout):
    W, ro = ctypes.c_void_p(0x10000), ctypes.c_void_p(0x20000)
    bm, v = ctypes.c_void_p(0x30000), ctypes.c_void_p(0x40000)
    nnz = ctypes.c_int64(0)
    assert L.spl_pack_count(None, 2, None, 4, 4, layout, ro, ctypes.byref(nnz), None) == INVALID
    assert L.spl_pack_count(W, 2, None, 4, 4, layout, ro, None, None) == INVALID
    assert L.spl_pack_count(W, 5, None, 4, 4, layout, ro, ctypes.byref(nnz), None) == INVALID
    assert L.spl_pack_count(W, 2, None, 0, 4, layout, ro, ctypes.byref(nnz), None) == INVALID
    assert L.spl_pack_count(W, 2, None, 1 << 31, 4, layout, ro, ctypes.byref(nnz), None) == INVALID
    assert L.spl_pack_count(W, 2, None, 4, 4, 2, ro, ctypes.byref(nnz), None) == INVALID     # unknown layout
    assert L.spl_pack_count(W, 2, None, 4, 4, layout, ctypes.c_void_p(0x20002), ctypes.byref(nnz), None) == INVALID
    assert L.spl_pack_sparse(W, 2, None, 4, 4, layout, ro, None, v, None) == INVALID
    assert L.spl_pack_sparse(W, 2, None, 4, 4, layout, ro, ctypes.c_void_p(0x30004), v, None) == INVALID
    assert L.spl_pack_sparse(W, 2, None, 4, 4, layout, ro, bm, None, None) == INVALID
    assert L.spl_pack_sparse(W, 2, None, 4, 4, layout, ro, bm, ctypes.c_void_p(0x40008), None) == INVALID
    assert L.spl_pack_sparse(W, 2, None, 4, 4, 3, ro, bm, v, None) == INVALID


def test_values_bytes(L):
    assert L.spl_values_bytes(2, 0) == 16 and L.spl_values_bytes(2, 1) == 32 and L.spl_values_bytes(2, 8) == 32
    assert L.spl_values_bytes(2, 9) == 48 and L.spl_values_bytes(1, 8) == 32
    assert L.spl_values_bytes(3, 16) == 32 and L.spl_values_bytes(3, 17) == 48
    assert L.spl_values_bytes(4, 32) == 32 and L.spl_values_bytes(4, 33) == 48
    assert L.spl_values_bytes(9, 8) == 0 and L.spl_values_bytes(2, -1) == 0


def test_validate_rejects_bad_views_on_the_host(L):
    assert L.spl_validate(None, None) == INVALID
    m = _mat(values_bytes=0)
    assert L.spl_validate(ctypes.byref(m), None) == INVALID            # fails spl_check_matrix: no device access


def test_dense_argument_checks(L):
    X, Y, W = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000), ctypes.c_void_p(0x10000)
    assert L.spl_dense_linear_ex(X, 2, None, 2, 8, 8, Y, 0, None) == INVALID
    assert L.spl_dense_linear_ex(X, 2, W, 3, 8, 8, Y, 0, None) == INVALID
    assert L.spl_dense_linear_ex(X, 2, W, 2, 8, 12, Y, 0, None) == UNSUPPORTED
    assert L.spl_dense_linear_ex(X, 40, W, 2, 8, 8, Y, 1, None) == UNSUPPORTED
    assert L.spl_dense_linear_int8(X, None, 2, W, X, 8, 16, Y, None, None) == INVALID
    assert L.spl_dense_linear_int8(X, X, 2, W, X, 8, 24, Y, None, None) == UNSUPPORTED


def test_tile_count_and_retile_checks(L):
    assert L.spl_tile16_count(4096, 4096) == 256 * 128
    assert L.spl_tile16_count(17, 33) == 2 * 2
    assert L.spl_tile16_count(0, 4) == 0
    rows = _mat()
    tiles = _mat(layout=1, tile_offsets=0x40000)
    B, V, T = ctypes.c_void_p(0x50000), ctypes.c_void_p(0x60000), ctypes.c_void_p(0x70000)
    assert L.spl_retile16(ctypes.byref(tiles), B, V, T, None) == INVALID       # input must be the row layout
    assert L.spl_retile16(ctypes.byref(rows), None, V, T, None) == INVALID
    assert L.spl_retile16(ctypes.byref(rows), B, V, None, None) == INVALID
    assert L.spl_retile16(ctypes.byref(rows), B, ctypes.c_void_p(0x20000), T, None) == INVALID  # aliasing


def test_group_argument_checks(L):
    from paper_2405_03594_amd import MAX_GROUP, _DenseTask, _SparseTask

    m = _mat(layout=1, tile_offsets=0x40000)
    m16 = _mat(dtype=1, layout=1, tile_offsets=0x40000)
    X, Y = 0x40000, 0x50000

    def tasks(*mats):
        arr = (_SparseTask * max(1, len(mats)))()
        for i, mm in enumerate(mats):
            arr[i].X, arr[i].Y = X, Y + 0x1000 * i
            arr[i].W = ctypes.pointer(mm) if mm is not None else None
        return arr

    f = L.spl_sparse_linear_group
    assert f(tasks(m, m), 2, 0, 0, None) == OK                    # M = 0: checked, then a no-op
    assert f(tasks(m), 0, 2, 0, None) == INVALID                  # empty group
    assert f(None, 1, 2, 0, None) == INVALID
    assert f(tasks(*([m] * (MAX_GROUP + 1))), MAX_GROUP + 1, 2, 0, None) == INVALID
    assert f(tasks(m, None), 2, 2, 0, None) == INVALID            # missing matrix
    assert f(tasks(m, m16), 2, 0, 0, None) == INVALID             # mixed dtypes
    assert f(tasks(m, _mat(layout=1, tile_offsets=0x40000, rows=0)), 2, 0, 0, None) == INVALID
    assert f(tasks(m), 1, -1, 0, None) == INVALID
    assert f(tasks(m), 1, 33, 1, None) == UNSUPPORTED             # decode family is M <= 32

    g = L.spl_dense_linear_group
    d = (_DenseTask * 2)()
    for i in range(2):
        d[i].X, d[i].W, d[i].N, d[i].K, d[i].Y = X, 0x60000, 8, 64, Y
    assert g(d, 2, 0, 2, 0, None) == OK
    assert g(d, 2, 2, 3, 0, None) == INVALID                      # int8 has its own entry point
    assert g(d, 0, 2, 2, 0, None) == INVALID
    d[1].K = 60
    assert g(d, 2, 2, 2, 0, None) == UNSUPPORTED                  # K % 8 != 0
    d[1].K, d[1].W = 64, 0x60008
    assert g(d, 2, 2, 2, 0, None) == INVALID                      # misaligned W


def test_int8_group_argument_checks(L):
    from paper_2405_03594_amd import MAX_GROUP, _DenseInt8Task, _Int8Task

    m = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    mbf = _mat(dtype=2, layout=1, tile_offsets=0x40000)
    X, Y, s = 0x40000, 0x50000, 0x60000

    def tasks(*mats, scales=s):
        arr = (_Int8Task * max(1, len(mats)))()
        for i, mm in enumerate(mats):
            arr[i].Xq, arr[i].x_scales, arr[i].w_scales = X, scales, scales
            arr[i].Y = Y + 0x1000 * i
            arr[i].Wq = ctypes.pointer(mm) if mm is not None else None
        return arr

    f = L.spl_sparse_linear_int8_group
    assert f(tasks(m, m), 2, 0, None) == OK                       # M = 0: checked, then a no-op
    assert f(tasks(m, m, scales=None), 2, 0, None) == OK          # M = 0 reads no scales
    assert f(tasks(m), 0, 2, None) == INVALID                     # empty group
    assert f(None, 1, 2, None) == INVALID
    assert f(tasks(*([m] * (MAX_GROUP + 1))), MAX_GROUP + 1, 2, None) == INVALID
    assert f(tasks(m, None), 2, 0, None) == INVALID               # missing matrix
    assert f(tasks(m, mbf), 2, 0, None) == UNSUPPORTED            # a bf16 matrix in an int8 group
    assert f(tasks(m, m, scales=None), 2, 2, None) == INVALID     # scales required when M > 0
    assert f(tasks(m), 1, -1, None) == INVALID
    bad = tasks(m, m)
    bad[1].acc_out = 0x70004                                       # misaligned int32 output
    assert f(bad, 2, 2, None) == INVALID

    g = L.spl_dense_linear_int8_group
    d = (_DenseInt8Task * 2)()
    for i in range(2):
        d[i].Xq, d[i].x_scales, d[i].Wq, d[i].w_scales = X, s, 0x10000, s
        d[i].N, d[i].K, d[i].Y = 8, 64, Y + 0x1000 * i
    assert g(d, 2, 0, None) == OK
    assert g(d, 0, 2, None) == INVALID
    d[1].K = 24
    assert g(d, 2, 2, None) == UNSUPPORTED                        # K % 16 != 0
    d[1].K, d[1].Wq = 64, 0x10008
    assert g(d, 2, 2, None) == INVALID                            # misaligned W


def test_quantize_rows_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    f = L.spl_quantize_rows_i8
    X, Q, s = 0x40000, 0x50000, 0x60000
    assert f(X, 2, 0, 64, Q, s, None) == OK                       # M = 0: a no-op
    assert f(X, 2, -1, 64, Q, s, None) == INVALID
    assert f(X, 3, 4, 64, Q, s, None) == UNSUPPORTED              # int8 input
    assert f(X, 2, 4, 60, Q, s, None) == UNSUPPORTED              # K % 8 != 0
    assert f(None, 2, 4, 64, Q, s, None) == INVALID
    assert f(X, 2, 4, 64, None, s, None) == INVALID
    assert f(X, 2, 4, 64, Q, None, None) == INVALID
    assert f(X + 8, 2, 4, 64, Q, s, None) == INVALID              # misaligned X
    assert f(X, 1, 4, 64, Q + 4, s, None) == INVALID              # misaligned codes
    assert f(X, 2, 4, 0, Q, s, None) == INVALID                   # K = 0


def test_silu_mul_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    g = _mat(layout=1, tile_offsets=0x40000)
    u = _mat(layout=1, tile_offsets=0x40000)
    X, Y = ctypes.c_void_p(0x40000), ctypes.c_void_p(0x50000)
    f = L.spl_sparse_linear_silu_mul
    assert f(None, 0, ctypes.byref(g), ctypes.byref(u), None, 0, None) == OK       # M = 0 is a no-op
    assert f(X, -1, ctypes.byref(g), ctypes.byref(u), Y, 0, None) == INVALID
    assert f(X, 2, None, ctypes.byref(u), Y, 0, None) == INVALID
    assert f(X, 2, ctypes.byref(g), None, Y, 0, None) == INVALID
    assert f(X, 2, ctypes.byref(g), ctypes.byref(u), None, 0, None) == INVALID
    assert f(X, 2, ctypes.byref(g), ctypes.byref(u), Y, 7, None) == INVALID        # unknown algorithm
    assert f(X, 17, ctypes.byref(g), ctypes.byref(u), Y, 1, None) == UNSUPPORTED   # paired decode is M <= 16
    for bad in (_mat(rows=8, layout=1, tile_offsets=0x40000), _mat(cols=128, layout=1, tile_offsets=0x40000),
                _mat(dtype=1, layout=1, tile_offsets=0x40000)):
        assert f(X, 2, ctypes.byref(g), ctypes.byref(bad), Y, 0, None) == INVALID  # shape or dtype mismatch
    i8 = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    assert f(X, 2, ctypes.byref(i8), ctypes.byref(i8), Y, 0, None) == UNSUPPORTED
    rows = _mat()
    assert f(X, 2, ctypes.byref(rows), ctypes.byref(rows), Y, 0, None) == UNSUPPORTED   # row layout


def test_magnitude_mask_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    f = L.spl_magnitude_mask
    W, m, ws = 0x40000, 0x50000, 0x60000
    assert L.spl_magnitude_mask_workspace_bytes() >= 4 * (1 << 15)
    assert f(None, 2, 4, 64, 10, m, ws, None) == INVALID
    assert f(W, 2, 4, 64, 10, None, ws, None) == INVALID
    assert f(W, 2, 4, 64, 10, m, None, None) == INVALID
    assert f(W, 3, 4, 64, 10, m, ws, None) == UNSUPPORTED                  # int8 payloads
    assert f(W, 2, 4, 60, 10, m, ws, None) == UNSUPPORTED                  # K % 8 != 0
    assert f(W, 2, 1 << 16, 1 << 15, 10, m, ws, None) == UNSUPPORTED       # N K >= 2^31
    assert f(W, 2, 4, 64, -1, m, ws, None) == INVALID
    assert f(W, 2, 4, 64, 257, m, ws, None) == INVALID                     # prune > N K
    assert f(W + 8, 2, 4, 64, 10, m, ws, None) == INVALID                  # misaligned W
    assert f(W, 2, 4, 64, 10, m + 4, ws, None) == INVALID                  # misaligned mask
    assert f(W, 2, 0, 64, 10, m, ws, None) == INVALID                      # N = 0
    g = L.spl_magnitude_mask_noalloc                                       # the same checks, no workspace
    assert g(None, 2, 4, 64, 10, m, None) == INVALID
    assert g(W, 2, 4, 64, 10, None, None) == INVALID
    assert g(W, 3, 4, 64, 10, m, None) == UNSUPPORTED
    assert g(W, 2, 4, 60, 10, m, None) == UNSUPPORTED
    assert g(W, 2, 1 << 16, 1 << 15, 10, m, None) == UNSUPPORTED           # N K >= 2^31: past the maximum
    assert g(W, 2, 262144, 8192, 10, m, None) == UNSUPPORTED               # N K == 2^31
    assert g(W, 2, 4, 64, 257, m, None) == INVALID
    assert g(W + 8, 2, 4, 64, 10, m, None) == INVALID
    assert g(W, 2, 4, 64, 10, m + 4, None) == INVALID


def test_training_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    m = _mat(layout=1, tile_offsets=0x40000)
    A, B, G, ws = 0x40000, 0x50000, 0x60000, 0x70000
    t = L.spl_transpose16
    assert t(A, 0, 5, B, None) == OK and t(A, 5, 0, B, None) == OK
    assert t(A, -1, 5, B, None) == INVALID
    assert t(None, 4, 4, B, None) == INVALID and t(A, 4, 4, None, None) == INVALID
    assert t(A, 64 * 65536, 4, B, None) == UNSUPPORTED
    g = L.spl_gather_tiled
    assert g(None, ctypes.byref(m), G, None) == INVALID
    assert g(A + 8, ctypes.byref(m), G, None) == INVALID                       # misaligned dense rows
    assert g(A, ctypes.byref(_mat()), G, None) == UNSUPPORTED                 # row layout
    assert g(A, ctypes.byref(_mat(dtype=3, layout=1, tile_offsets=0x40000)), G, None) == UNSUPPORTED
    w = L.spl_sparse_weight_grad
    a256 = lambda b: -(-b // 256) * 256
    # the transposes of dY [16][4] and X [16][64] only: no dense [4][64] gradient
    assert L.spl_sparse_weight_grad_workspace_bytes(16, 4, 64) == a256(2 * 4 * 16) + a256(2 * 64 * 16)
    assert L.spl_sparse_weight_grad_workspace_bytes(2048, 11008, 4096) == 2 * 2048 * (11008 + 4096)
    assert L.spl_sparse_weight_grad_workspace_bytes(-1, 4, 64) < 0
    assert w(A, B, 0, ctypes.byref(m), G, ws, None) == UNSUPPORTED             # no tokens
    assert w(A, B, 12, ctypes.byref(m), G, ws, None) == UNSUPPORTED            # M % 8 != 0
    assert w(A, B, 16, ctypes.byref(m), G, ws + 16, None) == INVALID           # workspace alignment
    assert w(None, B, 16, ctypes.byref(m), G, ws, None) == INVALID
    assert w(A, B, 16, ctypes.byref(m), None, ws, None) == INVALID
    from paper_2405_03594_amd import _WeightGradTask
    gg = L.spl_sparse_weight_grad_group
    task = lambda mm, dY=A, X=B, out=G: _WeightGradTask(dY, X, ctypes.pointer(mm), out)
    two = (_WeightGradTask * 2)(task(m), task(m))
    assert gg(two, 0, 16, ws, None) == INVALID and gg(None, 1, 16, ws, None) == INVALID
    assert gg(two, 17, 16, ws, None) == INVALID                                # past SPL_MAX_GROUP
    assert gg(two, 2, 0, ws, None) == UNSUPPORTED                              # no tokens
    assert gg(two, 2, 12, ws, None) == UNSUPPORTED                             # M % 8 != 0
    assert gg(two, 2, 16, ws + 16, None) == INVALID                            # workspace alignment
    f16 = _mat(dtype=1, layout=1, tile_offsets=0x40000)
    assert gg((_WeightGradTask * 2)(task(m), task(f16)), 2, 16, ws, None) == INVALID   # mixed dtypes
    assert gg((_WeightGradTask * 2)(task(m), task(m, out=None)), 2, 16, ws, None) == INVALID
    assert gg((_WeightGradTask * 1)(task(_mat())), 1, 16, ws, None) == UNSUPPORTED     # row layout
    ig, wb = L.spl_sparse_input_grad, L.spl_sparse_input_grad_workspace_bytes
    big = _mat(rows=4096, cols=4096, layout=1, tile_offsets=0x40000)
    assert wb(2048, ctypes.byref(big)) == 0                                    # W's tiles read in the product
    assert wb(2000, ctypes.byref(big)) == 2 * a256(2 * 4096 * 4096)            # decoded, transposed copies
    assert wb(256, ctypes.byref(big)) == 2 * a256(2 * 4096 * 4096)            # 16 x 1 blocks: fewer than CUs
    assert wb(-1, ctypes.byref(big)) < 0 and wb(16, ctypes.byref(_mat())) < 0  # row layout
    m8 = _mat(rows=8, cols=64, layout=1, tile_offsets=0x40000)
    assert ig(A, 0, ctypes.byref(m8), G, None, None) == OK                     # no tokens
    assert ig(A, -1, ctypes.byref(m8), G, ws, None) == INVALID
    assert ig(None, 16, ctypes.byref(m8), G, ws, None) == INVALID
    assert ig(A, 16, ctypes.byref(m8), None, ws, None) == INVALID
    assert ig(A + 8, 16, ctypes.byref(m8), G, ws, None) == INVALID             # misaligned dY rows
    assert ig(A, 16, ctypes.byref(m8), G, None, None) == INVALID               # the fallback needs a workspace
    assert ig(A, 16, ctypes.byref(m8), G, ws + 16, None) == INVALID            # workspace alignment
    assert ig(A, 16, ctypes.byref(m), G, ws, None) == UNSUPPORTED              # N % 8 != 0 (dense fallback)
    assert ig(A, 16, ctypes.byref(_mat(rows=8)), G, ws, None) == UNSUPPORTED   # row layout
    s = L.spl_sparse_sgd_update
    assert s(ctypes.byref(m), None, 0.1, None) == INVALID                      # nnz > 0 needs a gradient
    assert s(ctypes.byref(_mat()), G, 0.1, None) == UNSUPPORTED                # row layout


def test_transpose_perm_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    w = _mat(rows=8, cols=64, layout=1, tile_offsets=0x40000)
    t = _mat(rows=64, cols=8, layout=1, tile_offsets=0x40000)
    f = L.spl_transpose_perm
    P, ws = 0x50000, 0x60000
    assert f(ctypes.byref(w), ctypes.byref(w), P, ws, None) == INVALID        # not the transposed shape
    assert f(ctypes.byref(w), ctypes.byref(_mat(rows=64, cols=8, nnz=9, layout=1, tile_offsets=0x40000)), P, ws,
             None) == INVALID                                                  # nnz differs
    assert f(ctypes.byref(w), ctypes.byref(t), None, ws, None) == INVALID
    assert f(ctypes.byref(w), ctypes.byref(t), P, ws + 16, None) == INVALID   # workspace alignment
    odd = _mat(rows=4, cols=64, layout=1, tile_offsets=0x40000)
    assert f(ctypes.byref(odd), ctypes.byref(_mat(rows=64, cols=4, layout=1, tile_offsets=0x40000)), P, ws,
             None) == UNSUPPORTED                                              # N % 8 != 0
    p = L.spl_permute_values
    assert p(0x40000, P, 0, 0x70000, None) == OK
    assert p(0x40000, P, -1, 0x70000, None) == INVALID
    assert p(None, P, 5, 0x70000, None) == INVALID
    assert p(0x40000, P + 2, 5, 0x70000, None) == INVALID                    # misaligned perm


def test_int4_argument_checks(L):
    """Checks that return before any HIP call (no device needed)."""
    w8 = _mat(dtype=3, layout=1, tile_offsets=0x40000)
    w4 = _mat(dtype=4, layout=1, tile_offsets=0x40000)
    X, s, Y = 0x40000, 0x50000, 0x60000
    assert L.spl_int4_values_bytes(5) >= 3 + 16
    assert L.spl_check_matrix(ctypes.byref(w4)) == INVALID                # only the int4 entry takes SPL_I4
    p = L.spl_pack_int4
    assert p(ctypes.byref(w4), 0x70000, None, None) == INVALID            # the source must be an int8 view
    assert p(ctypes.byref(_mat(layout=1, tile_offsets=0x40000)), 0x70000, None, None) == UNSUPPORTED   # bf16
    assert p(ctypes.byref(w8), 0x70008, None, None) == INVALID            # misaligned output
    assert p(ctypes.byref(w8), 0x70000, 0x80002, None) == INVALID         # misaligned count word
    f = L.spl_sparse_linear_int4
    assert f(X, s, 0, ctypes.byref(w4), s, Y, None, None) == OK           # M = 0
    assert f(X, s, 17, ctypes.byref(w4), s, Y, None, None) == UNSUPPORTED # decode batches only
    assert f(X, s, 2, ctypes.byref(w8), s, Y, None, None) == UNSUPPORTED  # an int8 view
    assert f(X, None, 2, ctypes.byref(w4), s, Y, None, None) == INVALID
    assert f(X, s, 2, ctypes.byref(_mat(dtype=4, cols=40, layout=1, tile_offsets=0x40000)), s, Y, None,
             None) == UNSUPPORTED                                          # K % 16 != 0


def _cpu_matrix(N=8, K=64, dtype=None):
    import torch

    import paper_2405_03594_amd as spl

    dtype = dtype or torch.bfloat16
    return spl.SparseMatrix(torch.zeros(16 * ((N + 15) // 16) * ((K + 31) // 32), dtype=torch.int32),
                            torch.zeros(64, dtype=dtype), None, torch.zeros(((N + 15) // 16) * ((K + 31) // 32) + 1,
                                                                           dtype=torch.int32), N, K, 0, "tile16")


def test_wrappers_reject_mismatched_tensors_before_any_launch():
    """The Python binding checks shapes, dtypes, lengths and contiguity before
    it calls the C ABI (which sees only pointers)."""
    import torch

    import paper_2405_03594_amd as spl

    Wc = _cpu_matrix()
    X = torch.zeros((2, 64), dtype=torch.bfloat16)
    cases = [
        (lambda: spl.sparse_linear(torch.zeros((2, 63), dtype=torch.bfloat16), Wc), "shape"),
        (lambda: spl.sparse_linear(torch.zeros((2, 64), dtype=torch.float16), Wc), "dtype"),
        (lambda: spl.sparse_linear(X, Wc, out=torch.zeros((2, 9), dtype=torch.bfloat16)), "shape"),
        (lambda: spl.sparse_linear(X, Wc, out=torch.zeros((8, 2), dtype=torch.bfloat16).t()), "contiguous"),
        (lambda: spl.sparse_linear(torch.zeros(64, dtype=torch.bfloat16), Wc), "2-D"),
        (lambda: spl.sparse_linear_group([X, torch.zeros((2, 32), dtype=torch.bfloat16)], [Wc, Wc]), "shape"),
        (lambda: spl.sparse_linear_silu_mul(torch.zeros((2, 60), dtype=torch.bfloat16), Wc, Wc), "shape"),
        (lambda: spl.sparse_linear_silu_mul(X, Wc, _cpu_matrix(N=9)), "share"),
        (lambda: spl.dense_linear(X, torch.zeros((8, 60), dtype=torch.bfloat16)), "shape"),
    ]
    W8 = _cpu_matrix(dtype=torch.int8)
    Xq = torch.zeros((2, 64), dtype=torch.int8)
    sx, sw = torch.zeros(2, dtype=torch.float32), torch.zeros(8, dtype=torch.float32)
    cases += [
        (lambda: spl.sparse_linear_int8(Xq.to(torch.int16), sx, W8, sw), "dtype"),
        (lambda: spl.sparse_linear_int8(torch.zeros((2, 48), dtype=torch.int8), sx, W8, sw), "shape"),
        (lambda: spl.sparse_linear_int8(Xq, torch.zeros(1, dtype=torch.float32), W8, sw), "x_scales"),
        (lambda: spl.sparse_linear_int8(Xq, sx, W8, torch.zeros(7, dtype=torch.float32)), "w_scales"),
        (lambda: spl.sparse_linear_int8(Xq, sx.double(), W8, sw), "dtype"),
        (lambda: spl.sparse_linear_int8(Xq, sx, W8, sw, acc_out=torch.zeros((2, 8), dtype=torch.int64)), "dtype"),
        (lambda: spl.sparse_linear_int8(Xq, sx, W8, sw, out=torch.zeros((2, 8), dtype=torch.float32)), "dtype"),
        (lambda: spl.sparse_linear_int8_group([Xq], [sx[:1]], [W8], [sw]), "x_scales"),
        (lambda: spl.sparse_linear_int4(torch.zeros((2, 16), dtype=torch.int8), sx, W8, sw), "shape"),
        (lambda: spl.dense_linear_int8(Xq, sx, torch.zeros((8, 64), dtype=torch.int8), sw[:4]), "w_scales"),
        (lambda: spl.quantize_rows_i8(X, scales=torch.zeros(1, dtype=torch.float32)), "scales"),
    ]
    dY = torch.zeros((2, 8), dtype=torch.bfloat16)                      # Wc is [8][64]
    Wn = _cpu_matrix()
    Wn.nnz = 40
    cases += [
        (lambda: spl.sparse_weight_grad(torch.zeros((2, 9), dtype=torch.bfloat16), X, Wc), "shape"),
        (lambda: spl.sparse_weight_grad(dY, torch.zeros((3, 64), dtype=torch.bfloat16), Wc), "shape"),
        (lambda: spl.sparse_weight_grad(dY, X.half(), Wc), "dtype"),
        (lambda: spl.sparse_weight_grad(dY, X, Wn, out=torch.zeros(39, dtype=torch.bfloat16)), "at least 40"),
        (lambda: spl.sparse_weight_grad_group([dY, dY], [X, X], [Wc]), "one entry per task"),
        (lambda: spl.sparse_weight_grad_group([dY], [torch.zeros((2, 63), dtype=torch.bfloat16)], [Wc]), "shape"),
        (lambda: spl.sparse_weight_grad_group([dY], [X], [Wn], outs=[torch.zeros(8, dtype=torch.bfloat16)]),
         "at least 40"),
        (lambda: spl.sparse_input_grad(torch.zeros((2, 7), dtype=torch.bfloat16), Wc), "shape"),
        (lambda: spl.sparse_input_grad(dY.half(), Wc), "dtype"),
        (lambda: spl.sparse_input_grad(dY, Wc, out=torch.zeros((2, 63), dtype=torch.bfloat16)), "shape"),
    ]
    for fn, what in cases:
        with pytest.raises(ValueError, match=what):
            fn()
