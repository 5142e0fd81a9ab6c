"""Parity of the backward calls (through the C ABI) against the oracle's
float64 gradients on the same seeded inputs.

Bars: fp32 outputs of fp32 arithmetic on exact inputs (broadcast and reduce
gradients, the fp32 triangle) are held to the fp32 normwise 1e-5.  Gradients
of the bf16 path (bf16 operands, fp32 accumulation, bf16 intermediates the
oracle keeps exact) are held to a normwise relative 1e-2, i.e. a few bf16
roundings (2^-9 relative each) along the chain; their magnitudes follow the
loss scale, so an absolute bar would not carry over between cases."""
import numpy as np
import pytest

from oracle import grads as G
from oracle import ops as O
from oracle.numerics import round_bf16
from paper_2609_30379_amd import synth
from tests.gpu_util import PARITY_LOG, check, dev, host

pytestmark = pytest.mark.gpu

GRAD_NORMWISE = 1e-2


def check_grad(got, ref, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU output"
    if got.size == 0:
        return 0.0
    denom = float(np.max(np.abs(ref)))
    err = float(np.max(np.abs(got - ref))) / (denom if denom > 0 else 1.0)
    PARITY_LOG.append((what + " [gradient, normwise]", err, GRAD_NORMWISE, denom))
    assert err <= GRAD_NORMWISE, f"{what}: normwise relative error {err:.3g} > {GRAD_NORMWISE}"
    return err


@pytest.fixture(scope="module")
def B():
    from paper_2609_30379_amd import binding
    binding.load()
    return binding


def _n(seed, name, shape, scale=1.0, dtype="bf16"):
    return synth.normal(seed, name, shape, scale, dtype)


LSETS = {"ragged": [5, 0, 1, 37, 64, 3, 70], "tiny": [15, 12, 10, 7],
         "bench": synth.lengths_for(synth.WORKLOADS["pair_b8_n208_224_bf16"]).tolist()}


# ------------------------------------------------------------------ broadcast / reduce
@pytest.mark.parametrize("lname", ["ragged", "tiny", "bench"])
@pytest.mark.parametrize("dtype,C", [("bf16", 128), ("f32", 16)])
@pytest.mark.parametrize("accumulate", [False, True])
def test_broadcast_backward(B, lname, dtype, C, accumulate):
    import torch
    L = LSETS[lname]
    lay = B.NestedLayout(L)
    S, R = sum(L), sum(n * n for n in L)
    dz = _n(60, "dz", (R, C), 1.0, dtype)
    du0 = _n(61, "du0", (S, C), 1.0, "f32") if accumulate else np.zeros((S, C))
    dv0 = _n(62, "dv0", (S, C), 1.0, "f32") if accumulate else np.zeros((S, C))
    du = dev(du0, "f32") if accumulate else torch.full((S, C), float("nan"), device="cuda")
    dv = dev(dv0, "f32") if accumulate else torch.full((S, C), float("nan"), device="cuda")
    B.nt_pair_broadcast_backward(lay, dev(dz, dtype), du, dv, accumulate=accumulate)
    ru, rv = G.pair_broadcast_backward(dz, L)
    check(host(du), du0 + ru, "f32", f"broadcast backward du {lname} {dtype} acc={accumulate}")
    check(host(dv), dv0 + rv, "f32", f"broadcast backward dv {lname} {dtype} acc={accumulate}")


@pytest.mark.parametrize("level", ["pairs", "pairs_first", "singles"])
@pytest.mark.parametrize("op", ["sum", "mean"])
@pytest.mark.parametrize("dtype,C", [("bf16", 128), ("f32", 36)])
def test_segment_reduce_backward_and_first_axis_reduce(B, level, op, dtype, C):
    import torch
    L = LSETS["ragged"]
    lay = B.NestedLayout(L)
    rows = sum(n * n for n in L) if level != "singles" else sum(L)
    out_rows = sum(L) if level != "singles" else len(L)
    olevel = {"pairs": "pair_cols", "pairs_first": "pair_rows", "singles": "samples"}[level]
    dy = _n(63, "dy", (out_rows, C), 1.0, "f32")
    dx0 = _n(64, "dx0", (rows, C), 1.0, dtype)
    for acc in (False, True):
        dx = dev(dx0, dtype) if acc else torch.full((rows, C), float("nan"), dtype=dev(dx0, dtype).dtype, device="cuda")
        B.nt_segment_reduce_backward(lay, level, op, dev(dy, "f32"), dx, accumulate=acc)
        ref = G.segment_reduce_backward(dy, L, olevel, op) + (dx0 if acc else 0.0)
        check(host(dx), ref, dtype, f"reduce backward {level} {op} {dtype} acc={acc}")
    # the forward over the first pair axis
    if level == "pairs_first":
        x = _n(65, "x", (rows, C), 0.7, dtype)
        y = torch.full((out_rows, C), 7.0, dtype=torch.float32, device="cuda")
        B.nt_segment_reduce(lay, "pairs_first", op, dev(x, dtype), y)
        check(host(y), O.segment_reduce(x, L, "pair_rows", op), "f32", f"first-axis reduce {op} {dtype}")


# ------------------------------------------------------------------ triangle
@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("dtype,C,L", [("bf16", 64, [5, 0, 1, 37, 64, 3, 70]), ("bf16", 128, [222, 130, 1]),
                                       ("f32", 16, [15, 12, 10, 7, 0, 1])])
def test_triangle_backward(B, direction, dtype, C, L):
    lay = B.NestedLayout(L)
    R = sum(n * n for n in L)
    sc = float(np.sqrt(0.5 / np.sqrt(max(L))))
    ab = _n(66, "ab", (R, 2 * C), sc, dtype)
    dt = _n(67, "dt", (R, C), 1.0, dtype)
    da0, db0 = _n(68, "da0", (R, C), 1.0, dtype), _n(69, "db0", (R, C), 1.0, dtype)
    abd = dev(ab, dtype)
    da, db = dev(da0, dtype), dev(db0, dtype)
    direc = "outgoing" if direction == 0 else "incoming"
    B.nt_triangle_mul_backward(lay, direction, abd[:, :C], abd[:, C:], dev(dt, dtype), da, db)
    ra, rb = G.triangle_mul_backward(ab[:, :C], ab[:, C:], dt, L, direc)
    what = f"triangle backward {direc} {dtype} C={C} L={L}"
    if dtype == "f32":
        check(host(da), da0 + ra, "f32", what + " da")
        check(host(db), db0 + rb, "f32", what + " db")
    else:
        check_grad(host(da), da0 + ra, what + " da")
        check_grad(host(db), db0 + rb, what + " db")


# ------------------------------------------------------------------ LayerNorm + Linear
LIN_BWD = [
    # rows, K, N, ln, epilogue, x dtype, dx dtype
    (1000, 128, 388, True, "none", "bf16", "bf16"),      # attention projection shape
    (777, 128, 128, True, "residual", "bf16", "bf16"),
    (500, 64, 256, True, "gelu", "bf16", "bf16"),
    (1000, 128, 128, True, "swiglu_residual", "bf16", "bf16"),   # SwiGLU transition, F = 512
    (300, 384, 256, False, "none", "bf16", "f32"),      # single projection u|v (no LayerNorm)
    (300, 128, 384, False, "residual", "f32", "f32"),   # single update from an fp32 column mean
    (130, 136, 40, True, "none", "f32", "bf16"),
    (70001, 128, 256, True, "none", "bf16", "bf16"),   # weight gradient over 244 row ranges, 17-row tail
    (7, 128, 128, True, "swiglu_residual", "bf16", "bf16"),   # fewer rows than one tile / one 32-row step
    (9, 128, 256, True, "none", "bf16", "f32"),
    (5, 64, 128, True, "none", "bf16", "bf16"),
]


@pytest.mark.parametrize("R,K,N,ln,epi,xdt,dxdt", LIN_BWD)
def test_layernorm_linear_backward(B, R, K, N, ln, epi, xdt, dxdt):
    import torch
    F = 4 * K if epi == "swiglu_residual" else 0
    Nw = 2 * F if F else N
    x = _n(70, "x", (R, K), 0.5, xdt)
    w = _n(71, "w", (Nw, K), 1.0 / np.sqrt(K), "bf16")
    b = _n(72, "b", (Nw,), 0.1, "f32")
    g, be = _n(73, "g", (K,), 0.1, "f32") + 1.0, _n(74, "be", (K,), 0.1, "f32")
    w2 = _n(75, "w2", (N, F), 0.5 / np.sqrt(F), "bf16") if F else None
    dy = _n(76, "dy", (R, N), 1.0, "bf16")
    dw = torch.zeros((Nw, K), device="cuda")
    db = torch.zeros((Nw,), device="cuda")
    dg = torch.zeros((K,), device="cuda")
    dbe = torch.zeros((K,), device="cuda")
    dw2 = torch.zeros((N, F), device="cuda") if F else None
    db2 = torch.zeros((N,), device="cuda") if F else None
    dx = torch.full((R, K), float("nan"), dtype=torch.bfloat16 if dxdt == "bf16" else torch.float32, device="cuda")
    B.nt_layernorm_linear_backward(dev(x, xdt), dev(w, "bf16"), dev(dy, "bf16"),
                                   ln=(dev(g, "f32"), dev(be, "f32")) if ln else None, bias=dev(b, "f32"),
                                   epilogue=epi, w2=dev(w2, "bf16") if F else None, hidden=F, dx=dx, dw=dw, db=db,
                                   dgamma=dg if ln else None, dbeta=dbe if ln else None, dw2=dw2, db2=db2)
    ref = G.layernorm_linear_backward(x, w, b, dy, ln=(g, be) if ln else None, epilogue=epi, w2=w2,
                                      xn_store=round_bf16, h_store=round_bf16)
    if not ln and xdt == "f32":
        # the forward product consumed x rounded to bf16
        ref = G.layernorm_linear_backward(round_bf16(x), w, b, dy, epilogue=epi)
    what = f"linear backward {R}x{K}->{N} ln={ln} {epi}"
    check_grad(host(dx), ref["dx"], what + " dx")
    check_grad(host(dw), ref["dw"], what + " dw")
    check_grad(host(db), ref["db"], what + " db")
    if ln:
        check_grad(host(dg), ref["dgamma"], what + " dgamma")
        check_grad(host(dbe), ref["dbeta"], what + " dbeta")
    if F:
        check_grad(host(dw2), ref["dw2"], what + " dw2")
        check_grad(host(db2), ref["db2"], what + " db2")


@pytest.mark.parametrize("K", [64, 128, 136])
def test_layernorm_linear_backward_without_dx(B, K):
    """dx not wanted (NULL): the LayerNorm and weight gradients alone, equal
    to those of a call that also writes dx (fused and general LayerNorm paths)."""
    import torch
    R, N = 3001, 256
    x = _n(83, "x", (R, K), 0.5, "bf16")
    w = _n(84, "w", (N, K), 1.0 / np.sqrt(K), "bf16")
    g, be = _n(85, "g", (K,), 0.1, "f32") + 1.0, _n(86, "be", (K,), 0.1, "f32")
    dy = _n(87, "dy", (R, N), 1.0, "bf16")
    outs = []
    for with_dx in (False, True):
        dw, dg, dbe = (torch.zeros((N, K), device="cuda"), torch.zeros((K,), device="cuda"),
                       torch.zeros((K,), device="cuda"))
        dx = torch.empty((R, K), dtype=torch.bfloat16, device="cuda") if with_dx else None
        B.nt_layernorm_linear_backward(dev(x, "bf16"), dev(w, "bf16"), dev(dy, "bf16"),
                                       ln=(dev(g, "f32"), dev(be, "f32")), dx=dx, dw=dw, dgamma=dg, dbeta=dbe)
        outs.append((host(dw), host(dg), host(dbe)))
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)
    ref = G.layernorm_linear_backward(x, w, None, dy, ln=(g, be), xn_store=round_bf16)
    check_grad(outs[0][1], ref["dgamma"], f"linear backward without dx K={K} dgamma")
    check_grad(outs[0][2], ref["dbeta"], f"linear backward without dx K={K} dbeta")


@pytest.mark.parametrize("epi,K,N,ln", [("swiglu_residual", 128, 128, True), ("none", 128, 256, True),
                                        ("none", 64, 128, True), ("gelu", 128, 384, False)])
def test_layernorm_linear_backward_strided(B, epi, K, N, ln):
    """x, dy and dx as column views of wider buffers (row strides K + 8, N + 16,
    K + 24): the weight-gradient kernel reads strided operands, the fused
    SwiGLU and d(LN x) kernels strided rows; padding is never written."""
    import torch
    R = 4099
    F = 4 * K if epi == "swiglu_residual" else 0
    Nw = 2 * F if F else N
    x = _n(100, "x", (R, K), 0.5, "bf16")
    w = _n(101, "w", (Nw, K), 1.0 / np.sqrt(K), "bf16")
    b = _n(102, "b", (Nw,), 0.1, "f32")
    g, be = _n(103, "g", (K,), 0.1, "f32") + 1.0, _n(104, "be", (K,), 0.1, "f32")
    w2 = _n(105, "w2", (N, F), 0.5 / np.sqrt(F), "bf16") if F else None
    dy = _n(106, "dy", (R, N), 1.0, "bf16")
    xw = torch.zeros((R, K + 8), dtype=torch.bfloat16, device="cuda")
    xw[:, :K] = dev(x, "bf16")
    dyw = torch.zeros((R, N + 16), dtype=torch.bfloat16, device="cuda")
    dyw[:, :N] = dev(dy, "bf16")
    dxw = torch.full((R, K + 24), float("nan"), dtype=torch.bfloat16, device="cuda")
    dw, db = torch.zeros((Nw, K), device="cuda"), torch.zeros((Nw,), device="cuda")
    dg, dbe = torch.zeros((K,), device="cuda"), torch.zeros((K,), device="cuda")
    dw2 = torch.zeros((N, F), device="cuda") if F else None
    db2 = torch.zeros((N,), device="cuda") if F else None
    B.nt_layernorm_linear_backward(xw[:, :K], dev(w, "bf16"), dyw[:, :N],
                                   ln=(dev(g, "f32"), dev(be, "f32")) if ln else None, bias=dev(b, "f32"),
                                   epilogue=epi, w2=dev(w2, "bf16") if F else None, hidden=F, dx=dxw[:, :K], dw=dw,
                                   db=db, dgamma=dg if ln else None, dbeta=dbe if ln else None, dw2=dw2, db2=db2)
    ref = G.layernorm_linear_backward(x, w, b, dy, ln=(g, be) if ln else None, epilogue=epi, w2=w2,
                                      xn_store=round_bf16, h_store=round_bf16)
    what = f"strided linear backward {R}x{K}->{N} {epi}"
    check_grad(host(dxw[:, :K]), ref["dx"], what + " dx")
    check_grad(host(dw), ref["dw"], what + " dw")
    check_grad(host(db), ref["db"], what + " db")
    if ln:
        check_grad(host(dg), ref["dgamma"], what + " dgamma")
        check_grad(host(dbe), ref["dbeta"], what + " dbeta")
    if F:
        check_grad(host(dw2), ref["dw2"], what + " dw2")
        check_grad(host(db2), ref["db2"], what + " db2")
    assert torch.isnan(dxw[:, K:]).all(), what + ": padding of dx written"


def test_layernorm_linear_backward_full_size(B):
    """The attention projection of the near-uniform block (364k rows,
    128 -> 388) and a second call that accumulates the weight gradients."""
    import torch
    L = LSETS["bench"]
    R = sum(n * n for n in L)
    K, N = 128, 388
    x = _n(77, "x", (R, K), 0.5, "bf16")
    w = _n(78, "w", (N, K), 1.0 / np.sqrt(K), "bf16")
    b = _n(79, "b", (N,), 0.1, "f32")
    g, be = _n(80, "g", (K,), 0.1, "f32") + 1.0, _n(81, "be", (K,), 0.1, "f32")
    dy = _n(82, "dy", (R, N), 1.0, "bf16")
    dw = torch.zeros((N, K), device="cuda")
    dg = torch.zeros((K,), device="cuda")
    dx = torch.empty((R, K), dtype=torch.bfloat16, device="cuda")
    args = (dev(x, "bf16"), dev(w, "bf16"), dev(dy, "bf16"))
    for _ in range(2):
        B.nt_layernorm_linear_backward(*args, ln=(dev(g, "f32"), dev(be, "f32")), bias=dev(b, "f32"), dx=dx, dw=dw,
                                       dgamma=dg)
    ref = G.layernorm_linear_backward(x, w, b, dy, ln=(g, be), xn_store=round_bf16)
    check_grad(host(dx), ref["dx"], "linear backward full size dx")
    check_grad(host(dw), 2 * ref["dw"], "linear backward full size dw (two calls)")
    check_grad(host(dg), 2 * ref["dgamma"], "linear backward full size dgamma (two calls)")


# ------------------------------------------------------------------ attention
ATT_BWD = [
    ([5, 0, 1, 37, 64, 3, 70], 4, "cells"),
    ([5, 0, 1, 37, 64, 3, 70], 2, "heads"),
    ([5, 0, 1, 37, 64, 3, 70], 2, None),
    ([300, 17, 1, 256], 2, "cells"),             # the N <= 512 instance
]


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("L,H,bias_layout", ATT_BWD)
def test_pair_attention_backward(B, axis, L, H, bias_layout):
    import torch
    D = 32
    lay = B.NestedLayout(L)
    R = sum(n * n for n in L)
    c = H * D
    qkv = _n(83, "qkv", (R, 3 * c), 1.0, "bf16")
    bias = _n(84, "bias", (R, H), 1.0, "bf16") if bias_layout else None
    dout = _n(85, "dout", (R, c), 1.0, "bf16")
    qd = dev(qkv, "bf16")
    if bias_layout == "heads":
        bd = dev(np.ascontiguousarray(bias.T), "bf16")
        dbias = torch.full((H, R), float("nan"), device="cuda")
    elif bias_layout == "cells":
        bd = dev(bias, "bf16")
        dbias = torch.full((R, H), float("nan"), device="cuda")
    else:
        bd, dbias = None, None
    dq, dk, dv = (torch.full((R, c), float("nan"), dtype=torch.bfloat16, device="cuda") for _ in range(3))
    B.nt_pair_row_attention_backward(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], dev(dout, "bf16"),
                                     dq, dk, dv, bias=bd, dbias=dbias, bias_layout=bias_layout or "cells")
    rq, rk, rv, rb = G.pair_row_attention_backward(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], bias, dout, L, H, D,
                                                   axis=axis)
    what = f"attention backward axis {axis} L={L} H={H} bias {bias_layout}"
    check_grad(host(dq), rq, what + " dq")
    check_grad(host(dk), rk, what + " dk")
    check_grad(host(dv), rv, what + " dv")
    if bias_layout:
        got = host(dbias)
        check_grad(got.T if bias_layout == "heads" else got, rb, what + " dbias")


# ------------------------------------------------------------------ rectangular pairs
@pytest.mark.parametrize("dtype,C", [("bf16", 128), ("f32", 16)])
def test_rectangular_pair_ops(B, dtype, C):
    """Broadcast, both pair reductions and their backward on N_i x M_i pairs
    (ragged rows and columns, an empty row track and an empty column track)."""
    import torch
    rows, cols = [5, 0, 37, 64, 3, 7, 1], [9, 4, 1, 70, 0, 13, 2]
    lay = B.NestedLayout(rows, cols=cols)
    assert lay.rect and lay.sum_m == sum(cols) and lay.sum_n2 == sum(n * m for n, m in zip(rows, cols))
    S, M, R = sum(rows), sum(cols), lay.sum_n2
    u, v = _n(90, "u", (S, C), 0.7, dtype), _n(91, "v", (M, C), 0.7, dtype)
    z = torch.full((R, C), float("nan"), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")
    B.nt_pair_broadcast(lay, dev(u, dtype), dev(v, dtype), z)
    check(host(z), O.pair_broadcast(u, v, rows, cols=cols), dtype, f"rect broadcast {dtype}")
    x = _n(92, "x", (R, C), 0.7, dtype)
    for level, olevel, out_rows in (("pairs", "pair_cols", S), ("pairs_first", "pair_rows", M)):
        for op in ("sum", "mean"):
            y = torch.full((out_rows, C), 7.0, dtype=torch.float32, device="cuda")
            B.nt_segment_reduce(lay, level, op, dev(x, dtype), y)
            check(host(y), O.segment_reduce(x, rows, olevel, op, cols=cols), "f32", f"rect reduce {level} {op}",
                  equal_nan=True)
            dy = _n(93, "dy", (out_rows, C), 1.0, "f32")
            dx = torch.full((R, C), float("nan"), dtype=z.dtype, device="cuda")
            B.nt_segment_reduce_backward(lay, level, op, dev(dy, "f32"), dx)
            check(host(dx), G.segment_reduce_backward(dy, rows, olevel, op, cols=cols), dtype,
                  f"rect reduce backward {level} {op}")
    dz = _n(94, "dz", (R, C), 1.0, dtype)
    du = torch.full((S, C), float("nan"), device="cuda")
    dv = torch.full((M, C), float("nan"), device="cuda")
    B.nt_pair_broadcast_backward(lay, dev(dz, dtype), du, dv)
    ru, rv = G.pair_broadcast_backward(dz, rows, cols)
    check(host(du), ru, "f32", f"rect broadcast backward du {dtype}")
    check(host(dv), rv, "f32", f"rect broadcast backward dv {dtype}")
    # square-only calls reject rectangular layouts
    with pytest.raises(B.NtError):
        B.nt_triangle_mul(lay, 0, z, z, z)


# ------------------------------------------------------------------ diagnostic loss
@pytest.mark.parametrize("level", ["pairs", "singles"])
@pytest.mark.parametrize("xdt,dxdt,C,pad", [("bf16", "bf16", 128, 0), ("bf16", "f32", 384, 0), ("f32", "f32", 128, 0),
                                            ("f32", "bf16", 64, 0), ("bf16", "bf16", 384, 2), ("f32", "f32", 16, 1),
                                            ("bf16", "bf16", 2056, 0)])
def test_weighted_square_loss(B, level, xdt, dxdt, C, pad):
    """One term of the joint diagnostic loss and its gradient (App. A), on
    16-byte aligned gradient rows (vector stores) and on padded rows (element
    stores), for narrow and wide rows."""
    import torch
    L = LSETS["ragged"] if C <= 384 else [5, 0, 1, 37, 3]
    lay = B.NestedLayout(L)
    rows = sum(n * n for n in L) if level == "pairs" else sum(L)
    x = _n(90, "x", (rows, C), 0.7, xdt)
    w = np.linspace(0.5, 2.0, len(L))
    loss = torch.full((len(L),), float("nan"), device="cuda")
    tdt = torch.bfloat16 if dxdt == "bf16" else torch.float32
    dx_full = torch.full((rows, C + pad), float("nan"), dtype=tdt, device="cuda")
    dx = dx_full[:, :C]
    B.nt_weighted_square_loss(lay, level, dev(x, xdt), torch.tensor(w, dtype=torch.float32, device="cuda"), 0.25,
                              loss, dx=dx)
    counts = [n * n for n in L] if level == "pairs" else L
    ref_loss, ref_g = O.weighted_square_loss(x, counts, w, 0.25)
    what = f"loss {level} x={xdt} dx={dxdt} C={C} pad={pad}"
    got = host(loss)
    assert np.allclose(got, ref_loss, rtol=1e-4, atol=1e-6), (what, got, ref_loss)
    # dx = 2 scale w x: one rounding to dx's dtype
    check(host(dx), ref_g, dxdt, what + " dx")
    if pad:
        assert torch.isnan(dx_full[:, C:]).all(), what + ": padding written"
