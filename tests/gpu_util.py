"""Helpers for the GPU parity tests: device transfer, layout conversions of
test inputs, and the parity bars (bf16: max-abs 2e-2 with fp32 accumulation;
fp32: normwise relative error 1e-5)."""
from __future__ import annotations

import numpy as np

BF16_MAX_ABS = 2e-2
F32_NORMWISE = 1e-5


def torch_mod():
    import torch
    return torch


def dev(x, dtype: str):
    torch = torch_mod()
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.float32)))
    return t.to(device="cuda", dtype=td)


def dev_f32(x):
    return dev(x, "f32")


def host(t) -> np.ndarray:
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.detach().to(device="cpu", dtype=torch.float64).numpy()


def check(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "", equal_nan: bool = False):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if equal_nan:
        nan_g, nan_r = np.isnan(got), np.isnan(ref)
        assert np.array_equal(nan_g, nan_r), f"{what}: NaN pattern differs"
        got, ref = np.where(nan_g, 0.0, got), np.where(nan_r, 0.0, ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU output"
    if got.size == 0:
        return 0.0
    if dtype == "bf16":
        err = float(np.max(np.abs(got - ref)))
        assert err <= BF16_MAX_ABS, f"{what}: max-abs error {err:.4g} > {BF16_MAX_ABS}"
    else:
        denom = float(np.max(np.abs(ref)))
        err = float(np.max(np.abs(got - ref))) / (denom if denom > 0 else 1.0)
        assert err <= F32_NORMWISE, f"{what}: normwise relative error {err:.3g} > {F32_NORMWISE}"
    return err


def pair_padded(x: np.ndarray, lengths, transposed: bool = False, ld: int | None = None,
                fill: float = 0.0) -> np.ndarray:
    """Channel-major pair-padded operand layout of a [sum N^2, C] pair tensor:
    channel c of cell (i,a,b) at c*ld + P_i + a*n8 + b (or b*n8 + a); padding
    entries hold `fill` (NaN checks that a kernel never reads them as data)."""
    C = x.shape[1]
    n8 = [(int(n) + 7) // 8 * 8 for n in lengths]
    P = np.concatenate([[0], np.cumsum([int(n) * m for n, m in zip(lengths, n8)])]).astype(np.int64)
    ld = int(P[-1]) if ld is None else ld
    ld = max(8, (ld + 7) // 8 * 8)
    out = np.full((C, ld), fill, np.float64)
    off = 0
    for i, n in enumerate(lengths):
        n = int(n)
        blk = x[off:off + n * n].reshape(n, n, C)
        if transposed:
            blk = blk.transpose(1, 0, 2)
        pad = np.full((n, n8[i], C), fill)
        pad[:, :n] = blk
        out[:, P[i]:P[i] + n * n8[i]] = pad.reshape(n * n8[i], C).T
        off += n * n
    return out


def unpad_pair(y: np.ndarray, lengths, transposed: bool = False) -> np.ndarray:
    """Inverse of pair_padded: [C, ld] -> [sum N^2, C] (padding dropped)."""
    C = y.shape[0]
    n8 = [(int(n) + 7) // 8 * 8 for n in lengths]
    rows, P = [], 0
    for i, n in enumerate(lengths):
        n = int(n)
        blk = y[:, P:P + n * n8[i]].T.reshape(n, n8[i], C)[:, :n]
        if transposed:
            blk = blk.transpose(1, 0, 2)
        rows.append(blk.reshape(n * n, C))
        P += n * n8[i]
    return np.concatenate(rows) if rows else np.zeros((0, C))
