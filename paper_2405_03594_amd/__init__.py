"""Python binding of libspl, the gfx950 sparse linear library (C ABI in ``include/spl.h``).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libspl.so``.  PyTorch supplies device memory and the stream.
There is no fallback: if the library is missing or a call fails, an
exception is raised.

Names follow the C ABI without its ``spl_`` prefix:

* ``pack_sparse(W, mask)`` -> :class:`SparseMatrix` (bitmask, packed values,
  row offsets; paper section 2.4.1);
* ``sparse_linear(X, Wc)`` -> ``Y = X (W . Mask)^T`` for fp16/bf16 (section 2.4.2);
* ``sparse_linear_int8(Xq, x_scales, Wqc, w_scales)`` -> fp16 ``Y`` (section 3.4);
* ``sparse_linear_group`` / ``dense_linear_group``: several independent
  linears (e.g. q, k, v) of one batch size in one launch;
* ``unpack``, ``dense_linear``, ``dense_linear_int8``: decoder and dense comparators;
* ``sparse_weight_grad[_group]``, ``sparse_input_grad``, ``sparse_sgd_update``:
  the training step with the mask held fixed (Algorithm 1).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspl.so")

F16, BF16, I8 = 1, 2, 3
LAYOUT = {"rows": 0, "tile16": 1}
ALGO = {"auto": 0, "decode": 1, "prefill": 2}
_STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "overflow", 4: "HIP runtime error"}
I4 = 4                                  # 4-bit codes, two per byte (values held as uint8)
_TORCH_DTYPE = {torch.float16: F16, torch.bfloat16: BF16, torch.int8: I8, torch.uint8: I4}
_CODE_DTYPE = {F16: torch.float16, BF16: torch.bfloat16, I8: torch.int8, I4: torch.uint8}


class SplError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {_STATUS.get(status, status)} (status {status})")
        self.status = status


class _Matrix(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64),
        ("cols", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("layout", ctypes.c_int32),
        ("nnz", ctypes.c_int64),
        ("bitmask", ctypes.c_void_p),
        ("values", ctypes.c_void_p),
        ("row_offsets", ctypes.c_void_p),
        ("tile_offsets", ctypes.c_void_p),
        ("values_bytes", ctypes.c_int64),
    ]


class _SparseTask(ctypes.Structure):
    _fields_ = [("X", ctypes.c_void_p), ("W", ctypes.POINTER(_Matrix)), ("Y", ctypes.c_void_p)]


class _DenseTask(ctypes.Structure):
    _fields_ = [("X", ctypes.c_void_p), ("W", ctypes.c_void_p), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("Y", ctypes.c_void_p)]


class _Int8Task(ctypes.Structure):
    _fields_ = [("Xq", ctypes.c_void_p), ("x_scales", ctypes.c_void_p), ("Wq", ctypes.POINTER(_Matrix)),
                ("w_scales", ctypes.c_void_p), ("Y", ctypes.c_void_p), ("acc_out", ctypes.c_void_p)]


class _WeightGradTask(ctypes.Structure):
    _fields_ = [("dY", ctypes.c_void_p), ("X", ctypes.c_void_p), ("W", ctypes.POINTER(_Matrix)),
                ("grad_values", ctypes.c_void_p)]


class _DenseInt8Task(ctypes.Structure):
    _fields_ = [("Xq", ctypes.c_void_p), ("x_scales", ctypes.c_void_p), ("Wq", ctypes.c_void_p),
                ("w_scales", ctypes.c_void_p), ("N", ctypes.c_int64), ("K", ctypes.c_int64), ("Y", ctypes.c_void_p),
                ("acc_out", ctypes.c_void_p)]


MAX_GROUP = 16
_lib = None


def lib() -> ctypes.CDLL:
    """Load libspl.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    MP = ctypes.POINTER(_Matrix)
    sigs = {
        "spl_version": (I32, []),
        "spl_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "spl_read_probe": (ctypes.c_int, [P, I64, P, P]),
        "spl_check_matrix": (ctypes.c_int, [MP]),
        "spl_validate": (ctypes.c_int, [MP, P]),
        "spl_values_bytes": (I64, [I32, I64]),
        "spl_tile16_count": (I64, [I64, I64]),
        "spl_retile16": (ctypes.c_int, [MP, P, P, P, P]),
        "spl_pack_count": (ctypes.c_int, [P, I32, P, I64, I64, I32, P, ctypes.POINTER(I64), P]),
        "spl_pack_sparse": (ctypes.c_int, [P, I32, P, I64, I64, I32, P, P, P, P]),
        "spl_unpack": (ctypes.c_int, [MP, P, P]),
        "spl_sparse_linear": (ctypes.c_int, [P, I64, MP, P, P]),
        "spl_sparse_linear_ex": (ctypes.c_int, [P, I64, MP, P, I32, P]),
        "spl_sparse_linear_expanded_workspace_bytes": (I64, [MP]),
        "spl_sparse_linear_expanded": (ctypes.c_int, [P, I64, MP, P, P, P]),
        "spl_sparse_linear_int8": (ctypes.c_int, [P, P, I64, MP, P, P, P, P]),
        "spl_sparse_linear_int8_expanded": (ctypes.c_int, [P, P, I64, MP, P, P, P, P, P]),
        "spl_quantize_rows_i8": (ctypes.c_int, [P, ctypes.c_int32, I64, I64, P, P, P]),
        "spl_sparse_linear_silu_mul": (ctypes.c_int, [P, I64, MP, MP, P, I32, P]),
        "spl_magnitude_mask_workspace_bytes": (I64, []),
        "spl_magnitude_mask": (ctypes.c_int, [P, I32, I64, I64, I64, P, P, P]),
        "spl_magnitude_mask_noalloc": (ctypes.c_int, [P, I32, I64, I64, I64, P, P]),
        "spl_transpose16": (ctypes.c_int, [P, I64, I64, P, P]),
        "spl_int4_values_bytes": (I64, [I64]),
        "spl_pack_int4": (ctypes.c_int, [MP, P, P, P]),
        "spl_sparse_linear_int4": (ctypes.c_int, [P, P, I64, MP, P, P, P, P]),
        "spl_gather_tiled": (ctypes.c_int, [P, MP, P, P]),
        "spl_sparse_weight_grad_workspace_bytes": (I64, [I64, I64, I64]),
        "spl_sparse_weight_grad": (ctypes.c_int, [P, P, I64, MP, P, P, P]),
        "spl_sparse_weight_grad_group": (ctypes.c_int, [ctypes.POINTER(_WeightGradTask), I32, I64, P, P]),
        "spl_sparse_input_grad_workspace_bytes": (I64, [I64, MP]),
        "spl_sparse_input_grad": (ctypes.c_int, [P, I64, MP, P, P, P]),
        "spl_sparse_sgd_update": (ctypes.c_int, [MP, P, ctypes.c_float, P]),
        "spl_transpose_perm_workspace_bytes": (I64, [I64, I64, I64]),
        "spl_transpose_perm": (ctypes.c_int, [MP, MP, P, P, P]),
        "spl_permute_values": (ctypes.c_int, [P, P, I64, P, P]),
        "spl_dense_linear": (ctypes.c_int, [P, I64, P, I32, I64, I64, P, P]),
        "spl_dense_linear_ex": (ctypes.c_int, [P, I64, P, I32, I64, I64, P, I32, P]),
        "spl_dense_linear_int8": (ctypes.c_int, [P, P, I64, P, P, I64, I64, P, P, P]),
        "spl_sparse_linear_group": (ctypes.c_int, [ctypes.POINTER(_SparseTask), I32, I64, I32, P]),
        "spl_dense_linear_group": (ctypes.c_int, [ctypes.POINTER(_DenseTask), I32, I64, I32, I32, P]),
        "spl_sparse_linear_int8_group": (ctypes.c_int, [ctypes.POINTER(_Int8Task), I32, I64, P]),
        "spl_dense_linear_int8_group": (ctypes.c_int, [ctypes.POINTER(_DenseInt8Task), I32, I64, P]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise SplError(fn, status)


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev_tensor(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _arg(t, name: str, shape=None, dtype=None, min_numel: int | None = None, device: bool = True) -> torch.Tensor:
    """An argument tensor's shape, dtype, length and contiguity, checked before
    its device: the C ABI sees only pointers, so a mismatch here would make a
    kernel read or write past a buffer."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if min_numel is not None and (t.dim() != 1 or t.numel() < min_numel):
        raise ValueError(f"{name} must be 1-D with at least {min_numel} entries")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return _dev_tensor(t, name) if device else t


def _q_args(Xq, x_scales, N: int, K: int, w_scales, M: int, device: bool = True) -> None:
    """int8 activations [M][K] and their per-row scales, per-channel weight scales [N]."""
    _arg(Xq, "Xq", shape=(M, K), dtype=torch.int8, device=False)
    _arg(x_scales, "x_scales", dtype=torch.float32, min_numel=M, device=False)
    _arg(w_scales, "w_scales", dtype=torch.float32, min_numel=N, device=False)
    if device:
        for t, nm in ((Xq, "Xq"), (x_scales, "x_scales"), (w_scales, "w_scales")):
            _dev_tensor(t, nm)


def _q_outs(out, acc_out, M: int, N: int, device: bool = True) -> None:
    _arg(out, "out", shape=(M, N), dtype=torch.float16, device=False)
    if acc_out is not None:
        _arg(acc_out, "acc_out", shape=(M, N), dtype=torch.int32, device=False)
    if device:
        _dev_tensor(out, "out")
        if acc_out is not None:
            _dev_tensor(acc_out, "acc_out")


def _rows_of(X, name: str) -> int:
    if not isinstance(X, torch.Tensor) or X.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    return X.shape[0]


@dataclass
class SparseMatrix:
    """A compressed [N][K] matrix in one of the two layouts of include/spl.h:
    "rows" (row-layout bitmask, values, row_offsets) or "tile16" (16 x 32
    submatrices: tile-major bitmask, values, tile_offsets)."""

    bitmask: torch.Tensor              # int32 view of the uint32 bitmask words
    values: torch.Tensor               # payloads (fp16 / bf16 / int8), length >= nnz (+16 bytes of tail)
    row_offsets: torch.Tensor | None   # int32 [N+1] (rows layout)
    tile_offsets: torch.Tensor | None  # int32 [B*S+1] (tile16 layout)
    rows: int
    cols: int
    nnz: int
    layout: str = "rows"

    @property
    def dtype(self) -> torch.dtype:
        return self.values.dtype

    def view(self) -> _Matrix:
        return _Matrix(self.rows, self.cols, _TORCH_DTYPE[self.values.dtype], LAYOUT[self.layout], self.nnz,
                       self.bitmask.data_ptr(), self.values.data_ptr(),
                       self.row_offsets.data_ptr() if self.row_offsets is not None else 0,
                       self.tile_offsets.data_ptr() if self.tile_offsets is not None else 0,
                       self.values.numel() * self.values.element_size())

    def compressed_bytes(self) -> int:
        """Bytes of the encoding: payloads + bitmask + offsets."""
        offs = self.row_offsets if self.layout == "rows" else self.tile_offsets
        payload = (self.nnz + 1) // 2 if self.values.dtype == torch.uint8 else self.nnz * self.values.element_size()
        return payload + self.bitmask.numel() * 4 + offs.numel() * 4


def _values_buffer(nnz: int, dtype: torch.dtype, device) -> torch.Tensor:
    # spl_values_bytes: payloads rounded up to 16 bytes plus 16 readable bytes of
    # tail (kernels may read, never write, up to 16 bytes past the last payload)
    esz = torch.empty((), dtype=dtype).element_size()
    return torch.zeros(int(lib().spl_values_bytes(_TORCH_DTYPE[dtype], nnz)) // esz, dtype=dtype, device=device)


def pack_sparse(W: torch.Tensor, mask: torch.Tensor | None = None, layout: str = "tile16",
                stream=None) -> SparseMatrix:
    """Compress W [N][K] (fp16/bf16/int8) under `mask` (uint8/bool, non-zero = kept;
    None = keep the non-zero payloads) with spl_pack_count + spl_pack_sparse.
    layout="tile16" (default) is the layout the linear kernels read; "rows" is
    the row-layout interchange format."""
    L = lib()
    if not isinstance(W, torch.Tensor) or W.dim() != 2 or W.dtype not in _TORCH_DTYPE or W.dtype == torch.uint8:
        raise ValueError("W must be a 2-D fp16/bf16/int8 tensor")
    if layout not in LAYOUT:
        raise ValueError(f"unknown layout {layout!r}")
    N, K = W.shape
    if mask is not None:
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        _arg(mask, "mask", shape=(N, K), dtype=torch.uint8)
    _dev_tensor(W, "W")
    code = _TORCH_DTYPE[W.dtype]
    if layout == "rows":
        blocks = N
        bitmask = torch.empty((N, (K + 31) // 32), dtype=torch.int32, device=W.device)
    else:
        blocks = int(L.spl_tile16_count(N, K))
        bitmask = torch.empty(blocks * 16, dtype=torch.int32, device=W.device)
    offsets = torch.empty(blocks + 1, dtype=torch.int32, device=W.device)
    nnz = ctypes.c_int64(0)
    s = _stream(stream)
    _check("spl_pack_count", L.spl_pack_count(_ptr(W), code, _ptr(mask), N, K, LAYOUT[layout], _ptr(offsets),
                                              ctypes.byref(nnz), s))
    values = _values_buffer(nnz.value, W.dtype, W.device)
    _check("spl_pack_sparse", L.spl_pack_sparse(_ptr(W), code, _ptr(mask), N, K, LAYOUT[layout], _ptr(offsets),
                                                _ptr(bitmask), _ptr(values), s))
    if layout == "rows":
        return SparseMatrix(bitmask, values, offsets, None, N, K, nnz.value, "rows")
    return SparseMatrix(bitmask, values, None, offsets, N, K, nnz.value, "tile16")


def validate(Wc: SparseMatrix, stream=None) -> bool:
    """Device check of the view's format (spl_validate): True if consistent."""
    view = Wc.view()
    st = lib().spl_validate(ctypes.byref(view), _stream(stream))
    if st == 1:
        return False
    _check("spl_validate", st)
    return True


def retile16(Wc: SparseMatrix, stream=None) -> SparseMatrix:
    """Row layout -> tile layout (16 x 32 submatrices)."""
    L = lib()
    if Wc.layout != "rows":
        raise ValueError("retile16 expects the row layout")
    T = int(L.spl_tile16_count(Wc.rows, Wc.cols))
    dev = Wc.values.device
    bitmask = torch.empty(T * 16, dtype=torch.int32, device=dev)
    tile_offsets = torch.empty(T + 1, dtype=torch.int32, device=dev)
    values = _values_buffer(Wc.nnz, Wc.dtype, dev)
    view = Wc.view()
    _check("spl_retile16", L.spl_retile16(ctypes.byref(view), _ptr(bitmask), _ptr(values), _ptr(tile_offsets),
                                          _stream(stream)))
    return SparseMatrix(bitmask, values, None, tile_offsets, Wc.rows, Wc.cols, Wc.nnz, "tile16")


def unpack(Wc: SparseMatrix, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    L = lib()
    if out is None:
        out = torch.empty((Wc.rows, Wc.cols), dtype=Wc.dtype, device=Wc.values.device)
    view = Wc.view()
    _check("spl_unpack", L.spl_unpack(ctypes.byref(view), _ptr(out), _stream(stream)))
    return out


def sparse_linear(X: torch.Tensor, Wc: SparseMatrix, out: torch.Tensor | None = None, algo: str = "auto",
                  stream=None) -> torch.Tensor:
    """Y [M][N] = X [M][K] (W . Mask)^T, fp32 accumulation, output in X's dtype."""
    L = lib()
    M = _rows_of(X, "X")
    _arg(X, "X", shape=(M, Wc.cols), dtype=Wc.dtype, device=False)
    if out is None:
        out = torch.empty((M, Wc.rows), dtype=X.dtype, device=X.device)
    _arg(out, "out", shape=(M, Wc.rows), dtype=Wc.dtype)
    _dev_tensor(X, "X")
    view = Wc.view()
    _check("spl_sparse_linear_ex", L.spl_sparse_linear_ex(_ptr(X), M, ctypes.byref(view), _ptr(out), ALGO[algo],
                                                          _stream(stream)))
    return out


def sparse_linear_expanded(X: torch.Tensor, Wc: SparseMatrix, out: torch.Tensor | None = None,
                           workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """sparse_linear through a decoded copy of W in `workspace` (see
    spl_sparse_linear_expanded): for large batches."""
    L = lib()
    M = _rows_of(X, "X")
    _arg(X, "X", shape=(M, Wc.cols), dtype=Wc.dtype, device=False)
    if out is None:
        out = torch.empty((M, Wc.rows), dtype=X.dtype, device=X.device)
    _arg(out, "out", shape=(M, Wc.rows), dtype=Wc.dtype)
    _dev_tensor(X, "X")
    view = Wc.view()
    need = L.spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(view))
    if need < 0:
        raise ValueError("spl_sparse_linear_expanded: the matrix view is invalid")
    if workspace is None:
        workspace = torch.empty((need,), dtype=torch.uint8, device=X.device)
    _dev_tensor(workspace, "workspace")
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace holds {workspace.numel() * workspace.element_size()} bytes, needs {need}")
    _check("spl_sparse_linear_expanded", L.spl_sparse_linear_expanded(_ptr(X), M, ctypes.byref(view), _ptr(out),
                                                                      _ptr(workspace), _stream(stream)))
    return out


def sparse_linear_silu_mul(X: torch.Tensor, Wgate: SparseMatrix, Wup: SparseMatrix, out: torch.Tensor | None = None,
                           algo: str = "auto", stream=None) -> torch.Tensor:
    """Y [M][N] = silu(X Wgate^T) * (X Wup^T): the gated half of a Llama MLP in
    one launch (see spl_sparse_linear_silu_mul)."""
    L = lib()
    if (Wup.rows, Wup.cols, Wup.dtype) != (Wgate.rows, Wgate.cols, Wgate.dtype):
        raise ValueError("gate and up must share shape and dtype")
    M = _rows_of(X, "X")
    _arg(X, "X", shape=(M, Wgate.cols), dtype=Wgate.dtype, device=False)
    if out is None:
        out = torch.empty((M, Wgate.rows), dtype=X.dtype, device=X.device)
    _arg(out, "out", shape=(M, Wgate.rows), dtype=Wgate.dtype)
    _dev_tensor(X, "X")
    vg, vu = Wgate.view(), Wup.view()
    _check("spl_sparse_linear_silu_mul", L.spl_sparse_linear_silu_mul(_ptr(X), M, ctypes.byref(vg), ctypes.byref(vu),
                                                                      _ptr(out), ALGO[algo], _stream(stream)))
    return out


def read_probe(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """Stream-read every byte of `buf` (a measurement helper; see spl_read_probe)."""
    L = lib()
    _dev_tensor(buf, "buf")
    _dev_tensor(sink, "sink")
    nbytes = buf.numel() * buf.element_size()
    if sink.numel() * sink.element_size() < 4:
        raise ValueError("sink needs 4 bytes")
    _check("spl_read_probe", L.spl_read_probe(_ptr(buf), nbytes, _ptr(sink), _stream(stream)))


def magnitude_mask(W: torch.Tensor, prune: int, out: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Keep-mask (uint8 [N][K]) zeroing exactly `prune` entries of smallest |w|,
    ties by ascending row-major index (see spl_magnitude_mask)."""
    L = lib()
    _dev_tensor(W, "W")
    N, K = W.shape
    if out is None:
        out = torch.empty((N, K), dtype=torch.uint8, device=W.device)
    if workspace is None:
        workspace = torch.empty((L.spl_magnitude_mask_workspace_bytes(),), dtype=torch.uint8, device=W.device)
    _check("spl_magnitude_mask", L.spl_magnitude_mask(_ptr(W), _TORCH_DTYPE[W.dtype], N, K, int(prune), _ptr(out),
                                                      _ptr(workspace), _stream(stream)))
    return out


def magnitude_mask_noalloc(W: torch.Tensor, prune: int, out: torch.Tensor, stream=None) -> torch.Tensor:
    """magnitude_mask through the entry point that allocates nothing (see
    spl_magnitude_mask_noalloc): the caller passes the uint8 [N][K] output;
    the scratch is the library's own, shared by every call on the device."""
    L = lib()
    if W.dim() != 2:
        raise ValueError(f"W: expected a 2-D tensor, got shape {tuple(W.shape)}")
    N, K = W.shape
    if W.dtype not in (torch.float16, torch.bfloat16):
        raise ValueError(f"W has dtype {W.dtype}, expected float16 or bfloat16")
    _arg(out, "out", shape=(N, K), dtype=torch.uint8, device=False)
    _dev_tensor(W, "W")
    _dev_tensor(out, "out")
    _check("spl_magnitude_mask_noalloc", L.spl_magnitude_mask_noalloc(_ptr(W), _TORCH_DTYPE[W.dtype], N, K,
                                                                      int(prune), _ptr(out), _stream(stream)))
    return out


def transpose16(A: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """out [C][R] = A [R][C]^T for a 16-bit matrix (see spl_transpose16)."""
    L = lib()
    _dev_tensor(A, "A")
    R, C = A.shape
    if out is None:
        out = torch.empty((C, R), dtype=A.dtype, device=A.device)
    _check("spl_transpose16", L.spl_transpose16(_ptr(A), R, C, _ptr(out), _stream(stream)))
    return out


def gather_tiled(W: torch.Tensor, pattern: SparseMatrix, out: torch.Tensor | None = None, stream=None):
    """The entries of dense W [N][K] at the kept positions of `pattern`, in its value order."""
    L = lib()
    _dev_tensor(W, "W")
    if out is None:
        out = torch.empty_like(pattern.values)
    view = pattern.view()
    _check("spl_gather_tiled", L.spl_gather_tiled(_ptr(W), ctypes.byref(view), _ptr(out), _stream(stream)))
    return out


def _wgrad_args(dY, X, Wc: SparseMatrix, out, M: int, name: str = "") -> None:
    _arg(dY, "dY" + name, shape=(M, Wc.rows), dtype=Wc.dtype, device=False)
    _arg(X, "X" + name, shape=(M, Wc.cols), dtype=Wc.dtype, device=False)
    if out is not None:
        _arg(out, "out" + name, dtype=Wc.dtype, min_numel=Wc.nnz, device=False)


def _workspace(L, workspace, need: int, device) -> torch.Tensor:
    if need < 0:
        raise ValueError("the workspace-size function rejected the shape")
    if workspace is None:
        return torch.empty((max(need, 1),), dtype=torch.uint8, device=device)
    _dev_tensor(workspace, "workspace")
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace holds {workspace.numel() * workspace.element_size()} bytes, needs {need}")
    return workspace


def sparse_weight_grad(dY: torch.Tensor, X: torch.Tensor, Wc: SparseMatrix, out: torch.Tensor | None = None,
                       workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Kept entries of dY^T X in Wc's value order (see spl_sparse_weight_grad)."""
    L = lib()
    M = _rows_of(X, "X")
    _wgrad_args(dY, X, Wc, out, M)
    _dev_tensor(dY, "dY")
    _dev_tensor(X, "X")
    if out is None:
        out = torch.empty_like(Wc.values)
    _dev_tensor(out, "out")
    workspace = _workspace(L, workspace, L.spl_sparse_weight_grad_workspace_bytes(M, Wc.rows, Wc.cols), X.device)
    view = Wc.view()
    _check("spl_sparse_weight_grad", L.spl_sparse_weight_grad(_ptr(dY), _ptr(X), M, ctypes.byref(view), _ptr(out),
                                                              _ptr(workspace), _stream(stream)))
    return out


def sparse_weight_grad_group(dYs, Xs, mats, outs=None, workspace: torch.Tensor | None = None,
                             stream=None) -> list:
    """Weight gradients of several layers of one batch in one call (see
    spl_sparse_weight_grad_group); outs[i] gets mats[i]'s kept entries."""
    L = lib()
    if not (len(dYs) == len(Xs) == len(mats)) or not 1 <= len(mats) <= MAX_GROUP:
        raise ValueError("dYs, Xs and mats: one entry per task, 1..MAX_GROUP tasks")
    if outs is not None and len(outs) != len(mats):
        raise ValueError("outs: one entry per task")
    M = _rows_of(Xs[0], "X")
    for i, (dY, X, Wc) in enumerate(zip(dYs, Xs, mats)):
        _wgrad_args(dY, X, Wc, outs[i] if outs is not None else None, M, f"[{i}]")
    for i, (dY, X) in enumerate(zip(dYs, Xs)):
        _dev_tensor(dY, f"dY[{i}]")
        _dev_tensor(X, f"X[{i}]")
    if outs is None:
        outs = [torch.empty_like(Wc.values) for Wc in mats]
    for i, o in enumerate(outs):
        _dev_tensor(o, f"out[{i}]")
    need = max(L.spl_sparse_weight_grad_workspace_bytes(M, Wc.rows, Wc.cols) for Wc in mats)
    workspace = _workspace(L, workspace, need, Xs[0].device)
    views = [Wc.view() for Wc in mats]
    tasks = (_WeightGradTask * len(mats))(*[
        _WeightGradTask(dY.data_ptr(), X.data_ptr(), ctypes.pointer(v), o.data_ptr())
        for dY, X, v, o in zip(dYs, Xs, views, outs)])
    _check("spl_sparse_weight_grad_group", L.spl_sparse_weight_grad_group(tasks, len(mats), M, _ptr(workspace),
                                                                          _stream(stream)))
    return outs


def sparse_input_grad(dY: torch.Tensor, Wc: SparseMatrix, out: torch.Tensor | None = None,
                      workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """dX [M][K] = dY [M][N] (W . Mask) from W's packed tiles (see spl_sparse_input_grad)."""
    L = lib()
    M = _rows_of(dY, "dY")
    _arg(dY, "dY", shape=(M, Wc.rows), dtype=Wc.dtype, device=False)
    if out is not None:
        _arg(out, "out", shape=(M, Wc.cols), dtype=Wc.dtype, device=False)
    _dev_tensor(dY, "dY")
    if out is None:
        out = torch.empty((M, Wc.cols), dtype=dY.dtype, device=dY.device)
    _dev_tensor(out, "out")
    view = Wc.view()
    need = L.spl_sparse_input_grad_workspace_bytes(M, ctypes.byref(view))
    if need < 0:
        raise ValueError("spl_sparse_input_grad_workspace_bytes rejected the shape")
    if need > 0 or workspace is not None:
        workspace = _workspace(L, workspace, need, dY.device)
    _check("spl_sparse_input_grad", L.spl_sparse_input_grad(_ptr(dY), M, ctypes.byref(view), _ptr(out),
                                                            _ptr(workspace), _stream(stream)))
    return out


def sparse_sgd_update(Wc: SparseMatrix, grad_values: torch.Tensor, lr: float, stream=None) -> None:
    """Wc.values <- Wc.values - lr * grad_values in place (see spl_sparse_sgd_update)."""
    L = lib()
    view = Wc.view()
    _check("spl_sparse_sgd_update", L.spl_sparse_sgd_update(ctypes.byref(view), _ptr(grad_values), float(lr),
                                                            _stream(stream)))


def transpose_perm(W: SparseMatrix, Wt: SparseMatrix, stream=None) -> torch.Tensor:
    """perm (int32 [nnz]): value i of Wt is value perm[i] of W (see spl_transpose_perm)."""
    L = lib()
    perm = torch.empty((max(W.nnz, 1),), dtype=torch.int32, device=W.values.device)
    ws = torch.empty((max(L.spl_transpose_perm_workspace_bytes(W.rows, W.cols, W.nnz), 1),), dtype=torch.uint8,
                     device=W.values.device)
    vw, vt = W.view(), Wt.view()
    _check("spl_transpose_perm", L.spl_transpose_perm(ctypes.byref(vw), ctypes.byref(vt), _ptr(perm), _ptr(ws),
                                                      _stream(stream)))
    return perm


def permute_values(src: torch.Tensor, perm: torch.Tensor, nnz: int, out: torch.Tensor, stream=None) -> torch.Tensor:
    """out[i] = src[perm[i]] for i < nnz (see spl_permute_values)."""
    L = lib()
    _check("spl_permute_values", L.spl_permute_values(_ptr(src), _ptr(perm), int(nnz), _ptr(out), _stream(stream)))
    return out


def pack_int4(W8: SparseMatrix, stream=None, check: bool = True) -> SparseMatrix:
    """The 4-bit form of an int8 tile-layout matrix whose codes lie in [-8, 7]
    (see spl_pack_int4): same pattern, values as uint8 bytes of two nibbles.
    With check, the library counts codes outside [-8, 7] and a nonzero count
    raises ValueError (this waits for the stream)."""
    L = lib()
    if W8.dtype != torch.int8 or W8.layout != "tile16":
        raise ValueError("pack_int4 takes an int8 matrix in the tile layout")
    dev = W8.values.device
    v4 = torch.zeros((L.spl_int4_values_bytes(W8.nnz),), dtype=torch.uint8, device=dev)
    bad = torch.zeros((1,), dtype=torch.int32, device=dev) if check else None
    view = W8.view()
    _check("spl_pack_int4", L.spl_pack_int4(ctypes.byref(view), _ptr(v4), _ptr(bad), _stream(stream)))
    if check:
        (stream if stream is not None else torch.cuda.current_stream()).synchronize()
        n = int(bad.item())
        if n:
            raise ValueError(f"pack_int4: {n} codes outside [-8, 7]")
    return SparseMatrix(W8.bitmask, v4, None, W8.tile_offsets, W8.rows, W8.cols, W8.nnz, "tile16")


def sparse_linear_int4(Xq: torch.Tensor, x_scales: torch.Tensor, W4: SparseMatrix, w_scales: torch.Tensor,
                       out: torch.Tensor | None = None, acc_out: torch.Tensor | None = None,
                       stream=None) -> torch.Tensor:
    """fp16 Y from 4-bit sparse weights and int8 activations, M <= 16 (see spl_sparse_linear_int4)."""
    L = lib()
    M = _rows_of(Xq, "Xq")
    _q_args(Xq, x_scales, W4.rows, W4.cols, w_scales, M, device=False)
    if out is None:
        out = torch.empty((M, W4.rows), dtype=torch.float16, device=Xq.device)
    _q_outs(out, acc_out, M, W4.rows)
    _q_args(Xq, x_scales, W4.rows, W4.cols, w_scales, M)
    view = W4.view()
    _check("spl_sparse_linear_int4", L.spl_sparse_linear_int4(_ptr(Xq), _ptr(x_scales), M, ctypes.byref(view),
                                                              _ptr(w_scales), _ptr(out), _ptr(acc_out),
                                                              _stream(stream)))
    return out


def quantize_rows_i8(X: torch.Tensor, out: torch.Tensor | None = None, scales: torch.Tensor | None = None,
                     stream=None):
    """Per-token int8 codes and binary32 scales of fp16/bf16 activations X [M][K]
    (section 3.4; see spl_quantize_rows_i8).  Returns (Xq int8 [M][K], x_scales f32 [M])."""
    L = lib()
    M = _rows_of(X, "X")
    K = X.shape[1]
    if X.dtype not in (torch.float16, torch.bfloat16):
        raise ValueError("X must be fp16 or bf16")
    if out is None:
        out = torch.empty((M, K), dtype=torch.int8, device=X.device)
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=X.device)
    _arg(out, "out", shape=(M, K), dtype=torch.int8, device=False)
    _arg(scales, "scales", dtype=torch.float32, min_numel=M, device=False)
    for t, nm in ((X, "X"), (out, "out"), (scales, "scales")):
        _dev_tensor(t, nm)
    _check("spl_quantize_rows_i8", L.spl_quantize_rows_i8(_ptr(X), _TORCH_DTYPE[X.dtype], M, K, _ptr(out),
                                                          _ptr(scales), _stream(stream)))
    return out, scales


def sparse_linear_int8(Xq: torch.Tensor, x_scales: torch.Tensor, Wqc: SparseMatrix, w_scales: torch.Tensor,
                       out: torch.Tensor | None = None, acc_out: torch.Tensor | None = None,
                       stream=None) -> torch.Tensor:
    """fp16 Y = dequant(int32 Xq (Wq . Mask)^T) with per-token and per-channel scales."""
    L = lib()
    M = _rows_of(Xq, "Xq")
    _q_args(Xq, x_scales, Wqc.rows, Wqc.cols, w_scales, M, device=False)
    if out is None:
        out = torch.empty((M, Wqc.rows), dtype=torch.float16, device=Xq.device)
    _q_outs(out, acc_out, M, Wqc.rows)
    _q_args(Xq, x_scales, Wqc.rows, Wqc.cols, w_scales, M)
    view = Wqc.view()
    _check("spl_sparse_linear_int8", L.spl_sparse_linear_int8(_ptr(Xq), _ptr(x_scales), M, ctypes.byref(view),
                                                              _ptr(w_scales), _ptr(out), _ptr(acc_out),
                                                              _stream(stream)))
    return out


def sparse_linear_int8_expanded(Xq: torch.Tensor, x_scales: torch.Tensor, Wqc: SparseMatrix, w_scales: torch.Tensor,
                                out: torch.Tensor | None = None, acc_out: torch.Tensor | None = None,
                                workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """sparse_linear_int8 through a decoded copy of the codes in `workspace`
    (see spl_sparse_linear_int8_expanded): for large batches."""
    L = lib()
    M = _rows_of(Xq, "Xq")
    _q_args(Xq, x_scales, Wqc.rows, Wqc.cols, w_scales, M, device=False)
    if out is None:
        out = torch.empty((M, Wqc.rows), dtype=torch.float16, device=Xq.device)
    _q_outs(out, acc_out, M, Wqc.rows)
    _q_args(Xq, x_scales, Wqc.rows, Wqc.cols, w_scales, M)
    view = Wqc.view()
    need = L.spl_sparse_linear_expanded_workspace_bytes(ctypes.byref(view))
    if need < 0:
        raise ValueError("spl_sparse_linear_int8_expanded: the matrix view is invalid")
    if workspace is None:
        workspace = torch.empty((need,), dtype=torch.uint8, device=Xq.device)
    _dev_tensor(workspace, "workspace")
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace holds {workspace.numel() * workspace.element_size()} bytes, needs {need}")
    _check("spl_sparse_linear_int8_expanded",
           L.spl_sparse_linear_int8_expanded(_ptr(Xq), _ptr(x_scales), M, ctypes.byref(view), _ptr(w_scales),
                                             _ptr(out), _ptr(acc_out), _ptr(workspace), _stream(stream)))
    return out


def dense_linear(X: torch.Tensor, W: torch.Tensor, out: torch.Tensor | None = None, algo: str = "auto",
                 stream=None) -> torch.Tensor:
    """Dense comparator: Y = X W^T with the same kernel families."""
    L = lib()
    M = _rows_of(X, "X")
    _rows_of(W, "W")
    N, K = W.shape
    _arg(X, "X", shape=(M, K), dtype=W.dtype, device=False)
    _arg(W, "W", shape=(N, K), device=False)
    if out is None:
        out = torch.empty((M, N), dtype=X.dtype, device=X.device)
    _arg(out, "out", shape=(M, N), dtype=W.dtype)
    _dev_tensor(X, "X")
    _dev_tensor(W, "W")
    _check("spl_dense_linear_ex", L.spl_dense_linear_ex(_ptr(X), M, _ptr(W), _TORCH_DTYPE[W.dtype], N, K,
                                                        _ptr(out), ALGO[algo], _stream(stream)))
    return out


def dense_linear_int8(Xq: torch.Tensor, x_scales: torch.Tensor, Wq: torch.Tensor, w_scales: torch.Tensor,
                      out: torch.Tensor | None = None, acc_out: torch.Tensor | None = None,
                      stream=None) -> torch.Tensor:
    L = lib()
    M = _rows_of(Xq, "Xq")
    _rows_of(Wq, "Wq")
    N, K = Wq.shape
    _arg(Wq, "Wq", shape=(N, K), dtype=torch.int8, device=False)
    _q_args(Xq, x_scales, N, K, w_scales, M, device=False)
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    _q_outs(out, acc_out, M, N)
    _dev_tensor(Wq, "Wq")
    _q_args(Xq, x_scales, N, K, w_scales, M)
    _check("spl_dense_linear_int8", L.spl_dense_linear_int8(_ptr(Xq), _ptr(x_scales), M, _ptr(Wq),
                                                            _ptr(w_scales), N, K, _ptr(out), _ptr(acc_out),
                                                            _stream(stream)))
    return out


def sparse_linear_group(Xs, Wcs, outs=None, algo: str = "auto", stream=None):
    """Y_i = X_i (W_i . Mask_i)^T for up to MAX_GROUP independent layers sharing the
    batch size and dtype, in one launch (decode) or one launch per layer (prefill)."""
    L = lib()
    n = len(Xs)
    if n != len(Wcs) or not 1 <= n <= MAX_GROUP:
        raise ValueError("need 1..MAX_GROUP (X, W) pairs")
    M = _rows_of(Xs[0], "X")
    if outs is None:
        outs = [torch.empty((M, W.rows), dtype=X.dtype, device=X.device) for X, W in zip(Xs, Wcs)]
    if len(outs) != n:
        raise ValueError("one output per layer")
    views = [W.view() for W in Wcs]
    tasks = (_SparseTask * n)()
    for i, (X, W, Y) in enumerate(zip(Xs, Wcs, outs)):
        if W.dtype != Wcs[0].dtype:
            raise ValueError("every layer of a group shares M and the fp16/bf16 dtype")
        _arg(X, "X", shape=(M, W.cols), dtype=W.dtype, device=False)
        _arg(Y, "out", shape=(M, W.rows), dtype=W.dtype, device=False)
    for i, (X, W, Y) in enumerate(zip(Xs, Wcs, outs)):
        _dev_tensor(X, "X")
        _dev_tensor(Y, "out")
        tasks[i].X = X.data_ptr()
        tasks[i].W = ctypes.pointer(views[i])
        tasks[i].Y = Y.data_ptr()
    _check("spl_sparse_linear_group", L.spl_sparse_linear_group(tasks, n, M, ALGO[algo], _stream(stream)))
    return outs


def dense_linear_group(Xs, Ws, outs=None, algo: str = "auto", stream=None):
    """Dense comparator of :func:`sparse_linear_group`."""
    L = lib()
    n = len(Xs)
    if n != len(Ws) or not 1 <= n <= MAX_GROUP:
        raise ValueError("need 1..MAX_GROUP (X, W) pairs")
    M = _rows_of(Xs[0], "X")
    if outs is None:
        outs = [torch.empty((M, W.shape[0]), dtype=X.dtype, device=X.device) for X, W in zip(Xs, Ws)]
    if len(outs) != n:
        raise ValueError("one output per layer")
    tasks = (_DenseTask * n)()
    for i, (X, W, Y) in enumerate(zip(Xs, Ws, outs)):
        _rows_of(W, "W")
        if W.dtype != Xs[0].dtype:
            raise ValueError("every layer of a group shares M and the fp16/bf16 dtype")
        _arg(W, "W", device=False)
        _arg(X, "X", shape=(M, W.shape[1]), dtype=W.dtype, device=False)
        _arg(Y, "out", shape=(M, W.shape[0]), dtype=W.dtype, device=False)
    for i, (X, W, Y) in enumerate(zip(Xs, Ws, outs)):
        for t, nm in ((X, "X"), (W, "W"), (Y, "out")):
            _dev_tensor(t, nm)
        tasks[i].X = X.data_ptr()
        tasks[i].W = W.data_ptr()
        tasks[i].N, tasks[i].K = W.shape
        tasks[i].Y = Y.data_ptr()
    _check("spl_dense_linear_group", L.spl_dense_linear_group(tasks, n, M, _TORCH_DTYPE[Xs[0].dtype], ALGO[algo],
                                                              _stream(stream)))
    return outs


def sparse_linear_int8_group(Xqs, x_scales, Wqcs, w_scales, outs=None, acc_outs=None, stream=None):
    """fp16 Y_i = dequant(int32 Xq_i (Wq_i . Mask_i)^T) for up to MAX_GROUP independent
    int8 layers sharing the batch size, in one launch."""
    L = lib()
    n = len(Xqs)
    if not (n == len(x_scales) == len(Wqcs) == len(w_scales)) or not 1 <= n <= MAX_GROUP:
        raise ValueError("need 1..MAX_GROUP (Xq, x_scales, Wq, w_scales) tuples")
    M = _rows_of(Xqs[0], "Xq")
    if outs is None:
        outs = [torch.empty((M, W.rows), dtype=torch.float16, device=X.device) for X, W in zip(Xqs, Wqcs)]
    accs = acc_outs if acc_outs is not None else [None] * n
    if len(outs) != n or len(accs) != n:
        raise ValueError("one output per layer")
    views = [W.view() for W in Wqcs]
    tasks = (_Int8Task * n)()
    for i in range(n):
        _q_args(Xqs[i], x_scales[i], Wqcs[i].rows, Wqcs[i].cols, w_scales[i], M, device=False)
        _q_outs(outs[i], accs[i], M, Wqcs[i].rows, device=False)
    for i in range(n):
        _q_args(Xqs[i], x_scales[i], Wqcs[i].rows, Wqcs[i].cols, w_scales[i], M)
        _q_outs(outs[i], accs[i], M, Wqcs[i].rows)
        tasks[i].Xq, tasks[i].x_scales = Xqs[i].data_ptr(), x_scales[i].data_ptr()
        tasks[i].Wq = ctypes.pointer(views[i])
        tasks[i].w_scales, tasks[i].Y = w_scales[i].data_ptr(), outs[i].data_ptr()
        tasks[i].acc_out = None if accs[i] is None else accs[i].data_ptr()
    _check("spl_sparse_linear_int8_group", L.spl_sparse_linear_int8_group(tasks, n, M, _stream(stream)))
    return outs


def dense_linear_int8_group(Xqs, x_scales, Wqs, w_scales, outs=None, acc_outs=None, stream=None):
    """Dense comparator of :func:`sparse_linear_int8_group`."""
    L = lib()
    n = len(Xqs)
    if not (n == len(x_scales) == len(Wqs) == len(w_scales)) or not 1 <= n <= MAX_GROUP:
        raise ValueError("need 1..MAX_GROUP (Xq, x_scales, Wq, w_scales) tuples")
    M = _rows_of(Xqs[0], "Xq")
    if outs is None:
        outs = [torch.empty((M, W.shape[0]), dtype=torch.float16, device=X.device) for X, W in zip(Xqs, Wqs)]
    accs = acc_outs if acc_outs is not None else [None] * n
    if len(outs) != n or len(accs) != n:
        raise ValueError("one output per layer")
    tasks = (_DenseInt8Task * n)()
    for i in range(n):
        _rows_of(Wqs[i], "Wq")
        _arg(Wqs[i], "Wq", dtype=torch.int8, device=False)
        _q_args(Xqs[i], x_scales[i], Wqs[i].shape[0], Wqs[i].shape[1], w_scales[i], M, device=False)
        _q_outs(outs[i], accs[i], M, Wqs[i].shape[0], device=False)
    for i in range(n):
        _dev_tensor(Wqs[i], "Wq")
        _q_args(Xqs[i], x_scales[i], Wqs[i].shape[0], Wqs[i].shape[1], w_scales[i], M)
        _q_outs(outs[i], accs[i], M, Wqs[i].shape[0])
        tasks[i].Xq, tasks[i].x_scales, tasks[i].Wq = Xqs[i].data_ptr(), x_scales[i].data_ptr(), Wqs[i].data_ptr()
        tasks[i].w_scales, tasks[i].Y = w_scales[i].data_ptr(), outs[i].data_ptr()
        tasks[i].N, tasks[i].K = Wqs[i].shape
        tasks[i].acc_out = None if accs[i] is None else accs[i].data_ptr()
    _check("spl_dense_linear_int8_group", L.spl_dense_linear_int8_group(tasks, n, M, _stream(stream)))
    return outs
