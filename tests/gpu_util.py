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


# Every comparison is recorded here as (what, error, bar, max |reference|);
# the test session prints them at its end (tests/conftest.py), so the margin of
# each case is visible in the log, not only its pass/fail.
PARITY_LOG: list = []

# bf16 values below this magnitude have a half-ulp of at most 2^-6 < 2e-2, so
# one rounding of the stored output stays inside the bar; inputs are scaled so
# every compared bf16 tensor stays below it.
BF16_MAX_MAGNITUDE = 8.0


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
    amax = float(np.max(np.abs(ref)))
    if dtype == "bf16":
        err = float(np.max(np.abs(got - ref)))
        PARITY_LOG.append((what, err, BF16_MAX_ABS, amax))
        assert err <= BF16_MAX_ABS, f"{what}: max-abs error {err:.4g} > {BF16_MAX_ABS}"
        assert amax < BF16_MAX_MAGNITUDE, f"{what}: reference magnitude {amax:.3g} beyond the bf16 range of the bar"
    else:
        err = float(np.max(np.abs(got - ref))) / (amax if amax > 0 else 1.0)
        PARITY_LOG.append((what, err, F32_NORMWISE, amax))
        assert err <= F32_NORMWISE, f"{what}: normwise relative error {err:.3g} > {F32_NORMWISE}"
    return err


def ulp_bf16(x) -> np.ndarray:
    """Spacing of bf16 values at |x| (8 significant bits): 2^(floor(log2 |x|) - 7)."""
    a = np.maximum(np.abs(np.asarray(x, np.float64)), 2.0 ** -126)
    return np.ldexp(1.0, np.floor(np.log2(a)).astype(np.int64) - 7)


# Chained comparisons (several bf16-stored steps run from the same input on
# both sides).  Every stored update rounds on both sides, the GPU from its
# fp32 value and the oracle from the exact one; where the two straddle a
# rounding boundary the stored values land one ulp apart, and the residual
# stream carries that ulp into every later step.  After R stored updates of
# a tensor the two can therefore differ by R ulps without any step being
# wrong (each step on its own stored inputs is held to the 2e-2 bar by the
# per-kernel checks).  A gated triangle update counts twice: its LayerNorm
# over t turns a one-ulp flip of t into up to one more ulp of the update.
# Flips are rare events (the fp32 and exact values must straddle a boundary),
# so besides the R-ulp bound at most CHAIN_FRACTION of the elements may
# differ by more than one ulp (or 2e-2): a mistake that shifts many elements
# by a little fails that even where it stays inside the bound.
CHAIN_FRACTION = 1e-4


def chain_updates(steps, blocks: int = 1) -> int:
    """Stored updates of the pair state along `blocks` blocks of `steps`
    (every step but the single update writes z; "lin" only in the first
    block)."""
    total = 0
    for b in range(blocks):
        for t in steps:
            if t == "single" or (t == "lin" and b > 0):
                continue
            total += 2 if t in ("tri_out_g", "tri_in_g") else 1
    return total


# the single state: the stored column mean entering the single update, and
# the update itself, per block
SINGLE_UPDATES = 2


def check_chained(got: np.ndarray, ref: np.ndarray, what: str = "", updates: int = 2):
    """Chained bf16 comparison after `updates` stored updates: every element
    within max(2e-2, updates ulps of the larger of the two values), and at
    most CHAIN_FRACTION of them beyond max(2e-2, one ulp)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU output"
    if got.size == 0:
        return 0.0
    d = np.abs(got - ref)
    ulp = ulp_bf16(np.maximum(np.abs(got), np.abs(ref)))
    bound = np.maximum(BF16_MAX_ABS, updates * ulp)
    err = float(np.max(d))
    ratio = float(np.max(d / bound))
    frac = float(np.mean(d > np.maximum(BF16_MAX_ABS, ulp)))
    amax = float(np.max(np.abs(ref)))
    PARITY_LOG.append((what + f" [chained; {ratio:.2f} of max(2e-2, {updates} ulp); beyond 1 ulp {frac:.1e}]",
                       err, BF16_MAX_ABS, amax))
    worst = int(np.argmax(d / bound))
    assert ratio <= 1.0, (f"{what}: chained error {d.flat[worst]:.4g} at |ref| {abs(ref.flat[worst]):.3g} "
                          f"exceeds max(2e-2, {updates} ulp)")
    assert frac <= CHAIN_FRACTION, f"{what}: {frac:.2e} of the elements are more than one ulp (and 2e-2) off"
    assert amax < BF16_MAX_MAGNITUDE, f"{what}: reference magnitude {amax:.3g} beyond the bf16 range of the bar"
    return err


def _tiled_plane_index(n: int, transposed: bool) -> np.ndarray:
    """Offsets inside one pair-tiled plane of every cell (a, b), a-major: plane
    element (r, k) of a 16 x 32 tile grid (row tiles outer, ceil(n/32) tiles
    per row), stored in fragment lane order ((k%32)//8 * 16 + r%16) * 8 + k%8;
    the plain variant puts cell (a, b) at (r, k) = (a, b), the transposed one
    at (b, a)."""
    a, b = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    r, k = (b, a) if transposed else (a, b)
    nkt = -(-n // 32)
    return (((r // 16) * nkt + k // 32) * 512 + ((k % 32) // 8 * 16 + r % 16) * 8 + k % 8).reshape(-1)


def tiled_offsets(lengths) -> np.ndarray:
    sizes = [(-(-int(n) // 16) * 16) * (-(-int(n) // 32) * 32) for n in lengths]
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


def pair_tiled(x: np.ndarray, lengths, transposed: bool = False, ld: int | None = None,
               fill: float = 0.0) -> np.ndarray:
    """Channel-major pair-tiled operand layout of a [sum N^2, C] pair tensor;
    padding entries hold `fill` (NaN checks that a kernel never reads them as
    data)."""
    C = x.shape[1]
    P = tiled_offsets(lengths)
    ld = int(P[-1]) if ld is None else ld
    ld = max(8, (ld + 7) // 8 * 8)
    out = np.full((C, ld), fill, np.float64)
    off = 0
    for i, n in enumerate(lengths):
        n = int(n)
        idx = P[i] + _tiled_plane_index(n, transposed)
        out[:, idx] = x[off:off + n * n].T
        off += n * n
    return out


def untile_pair(y: np.ndarray, lengths, transposed: bool = False) -> np.ndarray:
    """Inverse of pair_tiled: [C, ld] -> [sum N^2, C] (padding dropped)."""
    C = y.shape[0]
    P = tiled_offsets(lengths)
    rows = [y[:, P[i] + _tiled_plane_index(int(n), transposed)].T for i, n in enumerate(lengths)]
    return np.concatenate(rows) if rows else np.zeros((0, C))
