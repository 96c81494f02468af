"""Shared test helpers: host <-> device marshalling of raw payload bits and
the comparison rules of the parity tests.  No method arithmetic here."""
from __future__ import annotations

import numpy as np

TORCH_DT = {}


def _torch():
    import torch

    if not TORCH_DT:
        TORCH_DT.update({"bf16": torch.bfloat16, "f16": torch.float16})
    return torch


def to_dev(bits: np.ndarray, dtype: str):
    """uint16 payload bits (fp16/bf16) or int8 codes -> device tensor of that dtype."""
    torch = _torch()
    if dtype == "i8":
        return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.int8)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    return t.view(TORCH_DT[dtype]).cuda()


def from_dev_bits(t) -> np.ndarray:
    """Device fp16/bf16 tensor -> uint16 payload bits on the host."""
    torch = _torch()
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def from_dev_f64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_pack_equal(Wc, ref) -> None:
    """Bit-exact comparison of a device SparseMatrix with the oracle's Packed
    (row layout) or Tiled (tile layout)."""
    assert Wc.nnz == ref.nnz, (Wc.nnz, ref.nnz)
    if Wc.layout == "rows":
        assert np.array_equal(Wc.row_offsets.cpu().numpy(), ref.row_offsets)
    else:
        assert np.array_equal(Wc.tile_offsets.cpu().numpy(), ref.tile_offsets)
    assert np.array_equal(Wc.bitmask.cpu().numpy().view(np.uint32).reshape(-1), ref.bitmask.reshape(-1))
    vals = Wc.values[: Wc.nnz].cpu()
    if ref.dtype == "i8":
        got = vals.numpy()
    else:
        got = vals.view(_torch().int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref.values)


def assert_close(y: np.ndarray, ref: np.ndarray, what: str = "") -> None:
    """fp16/bf16 acceptance: |y - ref| <= max(2e-2, 1e-2 |ref|) element by element."""
    import oracle

    ok = oracle.tolerance_ok(y, ref)
    if not ok.all():
        bad = np.argwhere(~ok)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {ok.size} outside tolerance; first at {i}: "
                             f"got {y[i]!r}, oracle {ref[i]!r}; max abs err {np.max(np.abs(y - ref)):.3g}")
