"""Seeded synthetic inputs for the sparse linear layers.

The one module that both sides of every parity check use.  It holds none of
the method's arithmetic (no packing, no products, no dequantisation): it
draws Gaussian weights and activations, rounds the draws to their storage
types, builds magnitude-pruning masks and quantises *inputs* to int8.

Workload recipe (stands in for the trained sparse Llama-2-7B checkpoints the
paper measures on, which are not available here):

* weights ``W[N][K]`` ~ N(0, 0.02^2) drawn in binary32 from NumPy's PCG64 with
  the given seed, rounded to fp16 / bf16 with round-to-nearest-even;
* the mask zeroes exactly ``floor(s * N * K)`` entries per matrix (integer
  arithmetic), the smallest ``|w|`` of the *rounded* values; equal magnitudes
  are zeroed in ascending row-major order;
* activations ``X[M][K]`` ~ N(0, 1), rounded the same way;
* int8: per-output-channel scale ``max_kept |w| / 127`` and per-token scale
  ``max |x| / 127`` (binary32), codes ``clamp(rne(v / scale), -127, 127)``;
  an all-zero row gets scale 1 and zero codes.

Llama-2-7B linear shapes (out features N x in features K):
q, k, v, o: 4096 x 4096; gate, up: 11008 x 4096; down: 4096 x 11008.
"""
from __future__ import annotations

import numpy as np

LLAMA2_7B_LINEARS = (
    ("q", 4096, 4096),
    ("k", 4096, 4096),
    ("v", 4096, 4096),
    ("o", 4096, 4096),
    ("gate", 11008, 4096),
    ("up", 11008, 4096),
    ("down", 4096, 11008),
)
LLAMA2_7B_LAYERS = 32
WEIGHT_STD = 0.02


def weight_seed(layer: int, j: int) -> int:
    """Seed of matrix j (q=0 ... down=6) of decoder layer `layer`."""
    return 1000 + 10 * layer + j


def activation_seed(j: int) -> int:
    """Seed of the activations that feed matrix j."""
    return 9000 + j


_CHUNK = 1 << 20


def normal_f32(seed: int, shape, std: float = 1.0, out: np.ndarray | None = None) -> np.ndarray:
    """N(0, std^2) binary32 draws from PCG64(seed), in row-major order.  Filled
    in chunks from one stream, so a larger draw extends a smaller one."""
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(n, dtype=np.float32)
    flat = out.reshape(-1)
    assert flat.size == n and flat.dtype == np.float32
    rng = np.random.Generator(np.random.PCG64(seed))
    for i in range(0, n, _CHUNK):
        rng.standard_normal(dtype=np.float32, out=flat[i:i + _CHUNK])
    if std != 1.0:
        flat *= np.float32(std)
    return out.reshape(shape)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """binary32 -> bfloat16 bits, round to nearest even (finite inputs)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.reshape(-1).view(np.uint32)
    out = np.empty(u.size, dtype=np.uint16)
    for i in range(0, u.size, _CHUNK):
        c = u[i:i + _CHUNK]
        bias = (c >> np.uint32(16)) & np.uint32(1)
        bias += np.uint32(0x7FFF)
        bias += c
        bias >>= np.uint32(16)
        out[i:i + _CHUNK] = bias
    return out.reshape(x.shape)


def round_f16(x: np.ndarray) -> np.ndarray:
    """binary32 -> fp16 bits, round to nearest even (NumPy's conversion)."""
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f16":
        return round_f16(x)
    raise ValueError(dtype)


def bits_to_f32(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Storage bits -> binary32 values (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float32)
    raise ValueError(dtype)


def parse_sparsity(s) -> tuple[int, int]:
    """0.7 / "70%" / (7, 10) -> (numerator, denominator) in lowest terms of a decimal."""
    if isinstance(s, tuple):
        return int(s[0]), int(s[1])
    if isinstance(s, str):
        s = s.strip().rstrip("%")
        num = round(float(s) * 100)
        return num, 10000
    num = round(float(s) * 10000)
    return num, 10000


def magnitude_mask(bits: np.ndarray, sparsity) -> np.ndarray:
    """uint8 keep-mask of a 16-bit float matrix: zero exactly floor(s*numel)
    entries of smallest |w|, ties in ascending row-major order."""
    num, den = parse_sparsity(sparsity)
    flat = np.ascontiguousarray(bits, dtype=np.uint16).reshape(-1)
    numel = flat.size
    z = numel * num // den
    if z <= 0:
        return np.ones(bits.shape, dtype=np.uint8)
    if z >= numel:
        return np.zeros(bits.shape, dtype=np.uint8)
    counts = np.zeros(0x8000, dtype=np.int64)
    for i in range(0, numel, _CHUNK):
        counts += np.bincount(flat[i:i + _CHUNK] & np.uint16(0x7FFF), minlength=0x8000)
    cum = np.cumsum(counts)
    t = int(np.searchsorted(cum, z, side="right"))   # first magnitude key whose cumulative count exceeds z
    below = int(cum[t - 1]) if t > 0 else 0          # entries strictly smaller than t: all zeroed
    tie_zero = z - below                             # entries equal to t zeroed, lowest indices first
    mask = np.empty(numel, dtype=np.uint8)
    for i in range(0, numel, _CHUNK):
        key = flat[i:i + _CHUNK] & np.uint16(0x7FFF)
        m = mask[i:i + _CHUNK]
        np.greater(key, t, out=m.view(np.bool_))
        ties = np.flatnonzero(key == t)
        if tie_zero >= ties.size:
            tie_zero -= ties.size                    # all of these ties are zeroed
        else:
            m[ties[tie_zero:]] = 1                   # the remaining ties are kept
            tie_zero = 0
    return mask.reshape(bits.shape)


def weight(seed: int, N: int, K: int, dtype: str, sparsity) -> tuple[np.ndarray, np.ndarray]:
    """(W bits [N][K], keep-mask uint8 [N][K]); W is *not* multiplied by the mask."""
    w = round_to(normal_f32(seed, (N, K), WEIGHT_STD), dtype)
    return w, magnitude_mask(w, sparsity)


def activations(seed: int, M: int, K: int, dtype: str) -> np.ndarray:
    """X bits [M][K] ~ N(0, 1); rows are a prefix of the rows drawn at larger M."""
    return round_to(normal_f32(seed, (M, K), 1.0), dtype)


def quantize_rows_int8(v: np.ndarray, keep: np.ndarray | None = None, qmax: int = 127) -> tuple[np.ndarray, np.ndarray]:
    """Symmetric per-row integer codes in [-qmax, qmax] of a binary32 matrix
    (only `keep` entries count and are coded; the rest become 0): 127 for
    int8, 7 for int4.  Returns (codes int8, scales f32)."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    if keep is not None:
        v = np.where(keep.astype(bool), v, np.float32(0))
    amax = np.max(np.abs(v), axis=1)
    scale = (amax / np.float32(qmax)).astype(np.float32)
    scale = np.where(amax == 0, np.float32(1.0), scale).astype(np.float32)
    q = np.rint((v / scale[:, None]).astype(np.float32))
    q = np.clip(q, -qmax, qmax).astype(np.int8)
    return q, scale


def int8_weight(seed: int, N: int, K: int, sparsity) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(Wq int8 [N][K] (0 outside the mask), keep-mask, sw f32 [N]) from the bf16 pruned weight."""
    w, mask = weight(seed, N, K, "bf16", sparsity)
    q, sw = quantize_rows_int8(bits_to_f32(w, "bf16"), mask)
    return q, mask, sw


def int4_weight(seed: int, N: int, K: int, sparsity) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(Wq int8 codes in [-7, 7] [N][K] (0 outside the mask), keep-mask, sw f32 [N]):
    4-bit per-row symmetric codes of the bf16 pruned weight, held in int8."""
    w, mask = weight(seed, N, K, "bf16", sparsity)
    q, sw = quantize_rows_int8(bits_to_f32(w, "bf16"), mask, qmax=7)
    return q, mask, sw


def int4_weight_full_range(seed: int, N: int, K: int, sparsity) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """int4_weight with the codes' edges planted: every kept code of row 0 and
    of row N - 1 set to -8 (the one code without a positive twin), row N // 2
    set to 7, and a seeded eighth of the other kept codes set to -8."""
    q, mask, sw = int4_weight(seed, N, K, sparsity)
    q = q.copy()
    keep = mask.astype(bool)
    rng = np.random.default_rng(seed ^ 0x1F4B)
    q[keep & (rng.random(q.shape) < 0.125)] = -8
    for r, v in ((N // 2, 7), (0, -8), (N - 1, -8)):
        q[r, keep[r]] = v
    return q, mask, sw


def int8_activations(seed: int, M: int, K: int) -> tuple[np.ndarray, np.ndarray]:
    """(Xq int8 [M][K], sx f32 [M]) from bf16 N(0,1) activations."""
    x = activations(seed, M, K, "bf16")
    return quantize_rows_int8(bits_to_f32(x, "bf16"))
