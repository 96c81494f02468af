"""CPU oracle for the bitmask-compressed sparse linear layers.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library and
its Python binding never import, load or call it, and the two share no code.

The arithmetic lives in ``spl_oracle.c`` (plain C, binary64, every step
written out in the paper's order); this module only marshals numpy arrays
into it.  Paper: arXiv 2405.03594, section 2.4.1 (bitmask expansion and its
worked example), section 2.4.2 (the GPU variant: compressed submatrices that
are decompressed before the matrix units use them), section 3.4 (int8
weights and activations).

Parity pins for every function here are in ``tests/test_oracle.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spl_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

DTYPES = {"f16": 1, "bf16": 2, "i8": 3}

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (binary64, no contraction of products)."""
    if not force and os.path.exists(_LIB_PATH) and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I32 = ctypes.c_int32
    sig = {
        "orc_words_per_row": (I64, [I64]),
        "orc_pack_nnz": (I64, [P, I32, P, I64, I64]),
        "orc_pack": (None, [P, I32, P, I64, I64, P, P, P]),
        "orc_unpack": (None, [P, P, P, I32, I64, I64, P]),
        "orc_linear_f64": (None, [P, I64, I64, I32, P, P, P, I64, P, ctypes.c_int]),
        "orc_linear_f64_pairs": (None, [P, I64, I64, I32, P, P, P, I64, P, P, I64, P, ctypes.c_int]),
        "orc_dense_f64": (None, [P, I64, I64, I32, P, I64, P, ctypes.c_int]),
        "orc_linear_i8": (ctypes.c_int, [P, P, I64, I64, P, P, P, P, I64, P, P, ctypes.c_int]),
        "orc_dense_i8": (ctypes.c_int, [P, P, I64, I64, P, P, I64, P, P, ctypes.c_int]),
        "orc_quantize_rows_i8": (None, [P, I32, I64, I64, P, P]),
        "orc_tile_blocks": (I64, [I64]),
        "orc_tile_ksteps": (I64, [I64]),
        "orc_pack_tiled": (None, [P, I32, P, I64, I64, P, P, P]),
        "orc_unpack_tiled": (None, [P, P, P, I32, I64, I64, P]),
        "orc_f16_to_f64_array": (None, [P, I64, P]),
        "orc_bf16_to_f64_array": (None, [P, I64, P]),
        "orc_f32_to_f16_array": (None, [P, I64, P]),
        "orc_dequant_f16_array": (None, [P, P, P, I64, P]),
        "orc_max_threads": (ctypes.c_int, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _code(dtype: str) -> int:
    return DTYPES[dtype]


def max_threads() -> int:
    return int(_load().orc_max_threads())


@dataclass
class Packed:
    """The canonical encoding (see spl_oracle.c for the exact bit layout)."""

    bitmask: np.ndarray      # uint32 [N][ceil(K/32)]
    values: np.ndarray       # uint16 (fp16/bf16 payloads) or int8 [nnz]
    row_offsets: np.ndarray  # int32 [N+1]
    N: int
    K: int
    dtype: str

    @property
    def nnz(self) -> int:
        return int(self.row_offsets[-1])


def _payload_dtype(dtype: str):
    return np.int8 if dtype == "i8" else np.uint16


def pack(W: np.ndarray, dtype: str, mask: np.ndarray | None = None) -> Packed:
    """Bitmask expansion encoder (section 2.4.1): naive column-order walk."""
    lib = _load()
    W = np.ascontiguousarray(W)
    assert W.dtype == _payload_dtype(dtype), (W.dtype, dtype)
    N, K = W.shape
    if mask is not None:
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        assert mask.shape == W.shape
    nnz = int(lib.orc_pack_nnz(_ptr(W), _code(dtype), _ptr(mask), N, K))
    words = int(lib.orc_words_per_row(K))
    bitmask = np.zeros((N, words), dtype=np.uint32)
    values = np.zeros(max(nnz, 1), dtype=_payload_dtype(dtype))
    row_offsets = np.zeros(N + 1, dtype=np.int32)
    lib.orc_pack(_ptr(W), _code(dtype), _ptr(mask), N, K, _ptr(bitmask), _ptr(values), _ptr(row_offsets))
    return Packed(bitmask, values[:nnz], row_offsets, N, K, dtype)


@dataclass
class Tiled:
    """The GPU tile layout: 16 x 32 submatrices, each with its own 16 bitmask
    words and its kept values (see spl_oracle.c for the exact definition)."""

    bitmask: np.ndarray       # uint32 [B*S*16]
    values: np.ndarray        # payloads [nnz]
    tile_offsets: np.ndarray  # int32 [B*S + 1]
    N: int
    K: int
    dtype: str

    @property
    def nnz(self) -> int:
        return int(self.tile_offsets[-1])


def pack_tiled(W: np.ndarray, dtype: str, mask: np.ndarray | None = None) -> Tiled:
    """Submatrix encoder of section 2.4.2 with 16 x 32 tiles."""
    lib = _load()
    W = np.ascontiguousarray(W)
    assert W.dtype == _payload_dtype(dtype)
    N, K = W.shape
    if mask is not None:
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
    nnz = int(lib.orc_pack_nnz(_ptr(W), _code(dtype), _ptr(mask), N, K))
    B, S = int(lib.orc_tile_blocks(N)), int(lib.orc_tile_ksteps(K))
    bitmask = np.zeros(B * S * 16, dtype=np.uint32)
    values = np.zeros(max(nnz, 1), dtype=_payload_dtype(dtype))
    offs = np.zeros(B * S + 1, dtype=np.int32)
    lib.orc_pack_tiled(_ptr(W), _code(dtype), _ptr(mask), N, K, _ptr(bitmask), _ptr(values), _ptr(offs))
    return Tiled(bitmask, values[:nnz], offs, N, K, dtype)


def unpack_tiled(p: Tiled) -> np.ndarray:
    lib = _load()
    out = np.zeros((p.N, p.K), dtype=_payload_dtype(p.dtype))
    vals = p.values if p.values.size else np.zeros(1, dtype=_payload_dtype(p.dtype))
    lib.orc_unpack_tiled(_ptr(p.bitmask), _ptr(np.ascontiguousarray(vals)), _ptr(p.tile_offsets), _code(p.dtype),
                         p.N, p.K, _ptr(out))
    return out


def unpack(p: Packed) -> np.ndarray:
    """Decoder: kept positions take their stored payload, the rest +0."""
    lib = _load()
    out = np.zeros((p.N, p.K), dtype=_payload_dtype(p.dtype))
    vals = p.values if p.values.size else np.zeros(1, dtype=_payload_dtype(p.dtype))
    lib.orc_unpack(_ptr(p.bitmask), _ptr(np.ascontiguousarray(vals)), _ptr(p.row_offsets), _code(p.dtype),
                   p.N, p.K, _ptr(out))
    return out


def linear_f64(X: np.ndarray, p: Packed, nthreads: int = 0) -> np.ndarray:
    """Y = X (W.Mask)^T in binary64 from the packed weight; X is [M][K] fp16/bf16 bits."""
    lib = _load()
    X = np.ascontiguousarray(X, dtype=np.uint16)
    M, K = X.shape
    assert K == p.K and p.dtype in ("f16", "bf16")
    Y = np.zeros((M, p.N), dtype=np.float64)
    vals = p.values if p.values.size else np.zeros(1, dtype=np.uint16)
    lib.orc_linear_f64(_ptr(X), M, K, _code(p.dtype), _ptr(p.bitmask), _ptr(np.ascontiguousarray(vals)),
                       _ptr(p.row_offsets), p.N, _ptr(Y), nthreads)
    return Y


def linear_f64_pairs(X: np.ndarray, p: Packed, ms: np.ndarray, ns: np.ndarray, nthreads: int = 0) -> np.ndarray:
    """The same definition at selected output positions (ms[i], ns[i])."""
    lib = _load()
    X = np.ascontiguousarray(X, dtype=np.uint16)
    M, K = X.shape
    ms = np.ascontiguousarray(ms, dtype=np.int64)
    ns = np.ascontiguousarray(ns, dtype=np.int64)
    assert ms.shape == ns.shape
    assert (ms >= 0).all() and (ms < M).all() and (ns >= 0).all() and (ns < p.N).all()
    out = np.zeros(ms.shape, dtype=np.float64)
    vals = p.values if p.values.size else np.zeros(1, dtype=np.uint16)
    lib.orc_linear_f64_pairs(_ptr(X), M, K, _code(p.dtype), _ptr(p.bitmask), _ptr(np.ascontiguousarray(vals)),
                             _ptr(p.row_offsets), p.N, _ptr(ms), _ptr(ns), ms.size, _ptr(out), nthreads)
    return out


def _silu_mul(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    """silu(g) * u = g / (1 + e^-g) * u in binary64 (e^-g overflowing to inf gives -0)."""
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g)) * u


def silu_mul_f64(X: np.ndarray, pg: Packed, pu: Packed, nthreads: int = 0) -> np.ndarray:
    """The gated half of a Llama MLP on two sparse weights that share X:
    Y = silu(X (Wg.Mg)^T) * (X (Wu.Mu)^T), elementwise, in binary64, with
    silu(z) = z / (1 + e^-z).  Both products are the plain definition above."""
    assert pg.N == pu.N and pg.K == pu.K
    return _silu_mul(linear_f64(X, pg, nthreads), linear_f64(X, pu, nthreads))


def silu_mul_f64_pairs(X: np.ndarray, pg: Packed, pu: Packed, ms: np.ndarray, ns: np.ndarray,
                       nthreads: int = 0) -> np.ndarray:
    """The same at selected output positions (ms[i], ns[i])."""
    assert pg.N == pu.N and pg.K == pu.K
    return _silu_mul(linear_f64_pairs(X, pg, ms, ns, nthreads), linear_f64_pairs(X, pu, ms, ns, nthreads))

def dense_f64(X: np.ndarray, W: np.ndarray, dtype: str, nthreads: int = 0) -> np.ndarray:
    """Plain dense product in binary64: Y = X W^T, W is [N][K]."""
    lib = _load()
    X = np.ascontiguousarray(X, dtype=np.uint16)
    W = np.ascontiguousarray(W, dtype=np.uint16)
    M, K = X.shape
    N, K2 = W.shape
    assert K == K2
    Y = np.zeros((M, N), dtype=np.float64)
    lib.orc_dense_f64(_ptr(X), M, K, _code(dtype), _ptr(W), N, _ptr(Y), nthreads)
    return Y


def linear_i8(Xq: np.ndarray, sx: np.ndarray, p: Packed, sw: np.ndarray, nthreads: int = 0):
    """Sparse-quantized linear (section 3.4): exact int32 accumulators and fp16 outputs (bits)."""
    lib = _load()
    Xq = np.ascontiguousarray(Xq, dtype=np.int8)
    sx = np.ascontiguousarray(sx, dtype=np.float32)
    sw = np.ascontiguousarray(sw, dtype=np.float32)
    M, K = Xq.shape
    assert K == p.K and p.dtype == "i8" and sx.shape == (M,) and sw.shape == (p.N,)
    acc = np.zeros((M, p.N), dtype=np.int32)
    Y = np.zeros((M, p.N), dtype=np.uint16)
    vals = p.values if p.values.size else np.zeros(1, dtype=np.int8)
    rc = lib.orc_linear_i8(_ptr(Xq), _ptr(sx), M, K, _ptr(p.bitmask), _ptr(np.ascontiguousarray(vals)),
                           _ptr(p.row_offsets), _ptr(sw), p.N, _ptr(acc), _ptr(Y), nthreads)
    if rc != 0:
        raise OverflowError("int8 accumulator outside the int32 range")
    return acc, Y


def dense_i8(Xq: np.ndarray, sx: np.ndarray, Wq: np.ndarray, sw: np.ndarray, nthreads: int = 0):
    """Dense int8 reference with the same epilogue."""
    lib = _load()
    Xq = np.ascontiguousarray(Xq, dtype=np.int8)
    Wq = np.ascontiguousarray(Wq, dtype=np.int8)
    sx = np.ascontiguousarray(sx, dtype=np.float32)
    sw = np.ascontiguousarray(sw, dtype=np.float32)
    M, K = Xq.shape
    N = Wq.shape[0]
    acc = np.zeros((M, N), dtype=np.int32)
    Y = np.zeros((M, N), dtype=np.uint16)
    rc = lib.orc_dense_i8(_ptr(Xq), _ptr(sx), M, K, _ptr(Wq), _ptr(sw), N, _ptr(acc), _ptr(Y), nthreads)
    if rc != 0:
        raise OverflowError("int8 accumulator outside the int32 range")
    return acc, Y


def quantize_rows_i8(X: np.ndarray, dtype: str):
    """Per-token int8 codes and binary32 scales of fp16/bf16 activation bits
    (the reading of section 3.4 in orc_quantize_rows_i8)."""
    lib = _load()
    X = np.ascontiguousarray(X, dtype=np.uint16)
    M, K = X.shape
    Xq = np.zeros((M, K), dtype=np.int8)
    sx = np.zeros(M, dtype=np.float32)
    lib.orc_quantize_rows_i8(_ptr(X), _code(dtype), M, K, _ptr(Xq), _ptr(sx))
    return Xq, sx


def magnitude_mask(W: np.ndarray, dtype: str, prune: int) -> np.ndarray:
    """Keep-mask (uint8 [N][K], 1 = kept) of one matrix after one-shot
    magnitude pruning (section 2: the smallest-magnitude weights are removed).
    Reading: exactly `prune` entries are zeroed per matrix, those of smallest
    |w| as decoded from the fp16/bf16 payload, ties in ascending row-major
    index.  The plain definition: a stable sort of |w| (binary64, exact);
    NaN payloads have no magnitude and are rejected."""
    mag = np.abs(to_f64(np.ascontiguousarray(W, dtype=np.uint16), dtype)).ravel()
    assert not np.isnan(mag).any(), "NaN payloads have no magnitude"
    assert 0 <= prune <= mag.size
    order = np.argsort(mag, kind="stable")
    keep = np.ones(mag.size, dtype=np.uint8)
    keep[order[:prune]] = 0
    return keep.reshape(np.shape(W))

def weight_grad_f64(dY: np.ndarray, X: np.ndarray, dtype: str, p: Packed) -> np.ndarray:
    """Gradient of a sparse linear layer Y = X (W.Mask)^T with respect to its
    kept weights (Algorithm 1 trains with the mask held fixed, so pruned
    entries get no gradient): G[n][k] = Mask[n][k] * sum_m dY[m][n] X[m][k],
    dense [N][K] binary64 (zeros off the mask)."""
    g = to_f64(dY, dtype).T @ to_f64(X, dtype)
    return g * mask_of(p)


def input_grad_f64(dY: np.ndarray, dtype: str, p: Packed) -> np.ndarray:
    """Gradient with respect to the activations: dX = dY (W.Mask), [M][K] binary64."""
    return to_f64(dY, dtype) @ to_f64(unpack(p), dtype)


def sgd_f64(w: np.ndarray, g: np.ndarray, lr: float) -> np.ndarray:
    """One masked SGD step on the kept weights (Algorithm 1: theta <- theta - lr grad,
    then masked; the kept values are the only ones stored): w - lr g in binary64."""
    return np.asarray(w, dtype=np.float64) - float(lr) * np.asarray(g, dtype=np.float64)


def mask_of(p: Packed) -> np.ndarray:
    """The keep-mask [N][K] (0/1 float64) of a row-layout pack, from its bitmask."""
    words = (p.K + 31) // 32
    bm = np.ascontiguousarray(p.bitmask, dtype=np.uint32).reshape(p.N, words)
    bits = (bm[:, :, None] >> np.arange(32, dtype=np.uint32)[None, None, :]) & 1
    return bits.reshape(p.N, words * 32)[:, :p.K].astype(np.float64)

def pack_i4(codes: np.ndarray) -> np.ndarray:
    """4-bit payload storage (section 4 names lower-bit payloads as future
    work; the reading taken): value i of a matrix's value array - an int8 code
    in [-8, 7] - is the two's-complement nibble at byte i // 2, the low nibble
    for even i.  An odd count leaves the last high nibble 0.  The value order
    is that of the int8 tile layout, so the products and the epilogue are
    those of the int8 path on the same integers (linear_i8)."""
    c = np.ascontiguousarray(codes, dtype=np.int8).ravel()
    assert c.size == 0 or (c.min() >= -8 and c.max() <= 7)
    nib = (c.astype(np.int16) & 0xF).astype(np.uint8)
    out = np.zeros((c.size + 1) // 2, dtype=np.uint8)
    for i, v in enumerate(nib):                        # value by value, as defined
        out[i // 2] |= v << (4 * (i % 2))
    return out


def unpack_i4(b: np.ndarray, count: int) -> np.ndarray:
    """Inverse of pack_i4: the first `count` codes (int8, sign-extended nibbles)."""
    b = np.ascontiguousarray(b, dtype=np.uint8)
    out = np.empty(count, dtype=np.int8)
    for i in range(count):
        v = (int(b[i // 2]) >> (4 * (i % 2))) & 0xF
        out[i] = v - 16 if v >= 8 else v
    return out

def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    lib = _load()
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.zeros(bits.shape, dtype=np.float64)
    lib.orc_f16_to_f64_array(_ptr(bits), bits.size, _ptr(out))
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    lib = _load()
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.zeros(bits.shape, dtype=np.float64)
    lib.orc_bf16_to_f64_array(_ptr(bits), bits.size, _ptr(out))
    return out


def to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    return f16_to_f64(bits) if dtype == "f16" else bf16_to_f64(bits)


def f32_to_f16(x: np.ndarray) -> np.ndarray:
    lib = _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.zeros(x.shape, dtype=np.uint16)
    lib.orc_f32_to_f16_array(_ptr(x), x.size, _ptr(out))
    return out


def dequant_f16(acc: np.ndarray, sx: np.ndarray, sw: np.ndarray) -> np.ndarray:
    """Element-wise epilogue on broadcast-compatible arrays; returns fp16 bits."""
    lib = _load()
    acc, sx, sw = np.broadcast_arrays(np.asarray(acc, np.int32), np.asarray(sx, np.float32), np.asarray(sw, np.float32))
    acc = np.ascontiguousarray(acc)
    sx = np.ascontiguousarray(sx)
    sw = np.ascontiguousarray(sw)
    out = np.zeros(acc.shape, dtype=np.uint16)
    lib.orc_dequant_f16_array(_ptr(acc), _ptr(sx), _ptr(sw), acc.size, _ptr(out))
    return out


def tolerance_ok(y: np.ndarray, ref: np.ndarray, abs_tol: float = 2e-2, rel_tol: float = 1e-2) -> np.ndarray:
    """Per-element acceptance for fp16/bf16 outputs: |y - ref| <= max(abs_tol, rel_tol * |ref|)."""
    return np.abs(y - ref) <= np.maximum(abs_tol, rel_tol * np.abs(ref))
