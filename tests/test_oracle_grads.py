"""Pins of the oracle's gradients (oracle/grads.py): every backward agrees with
central finite differences of its own forward (directional derivatives along
random directions, so every input element takes part), and with torch
autograd of an independent torch forward on a masked padded batch."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import grads, layout, ops
from oracle.numerics import layernorm

RNG = np.random.default_rng(2609)


def _r(*shape, s=1.0):
    return s * RNG.standard_normal(shape)


def _fd(f, args, i, direction, eps=1e-6):
    """Central difference of f along `direction` in argument i."""
    a = list(args)
    a[i] = args[i] + eps * direction
    hi = f(*a)
    a[i] = args[i] - eps * direction
    lo = f(*a)
    return (hi - lo) / (2 * eps)


def _check_directional(loss, args, grads_, names, rtol=1e-6):
    for i, (g, name) in enumerate(zip(grads_, names)):
        if g is None:
            continue
        for _ in range(2):
            dirn = RNG.standard_normal(np.shape(args[i]))
            want = _fd(loss, args, i, dirn)
            got = float(np.sum(g * dirn))
            assert abs(got - want) <= rtol * max(1.0, abs(want)), (name, got, want)


# ---------------------------------------------------------------- broadcast / reduce
def test_broadcast_backward_finite_differences_and_sums():
    L, C = [3, 0, 4, 1], 5
    S, R = sum(L), sum(n * n for n in L)
    u, v, G = _r(S, C), _r(S, C), _r(R, C)
    du, dv = grads.pair_broadcast_backward(G, L)
    loss = lambda uu, vv: float(np.sum(G * ops.pair_broadcast(uu, vv, L)))  # noqa: E731
    _check_directional(loss, (u, v), (du, dv), ("du", "dv"))
    # worked example: lengths (2, 3) and dz = 1 give the lengths themselves
    du1, dv1 = grads.pair_broadcast_backward(np.ones((13, 1)), [2, 3])
    assert du1[:, 0].tolist() == [2, 2, 3, 3, 3] and dv1[:, 0].tolist() == [2, 2, 3, 3, 3]


@pytest.mark.parametrize("level,op", [("pair_cols", "sum"), ("pair_cols", "mean"), ("pair_rows", "sum"),
                                      ("pair_rows", "mean"), ("samples", "sum"), ("samples", "mean")])
def test_reduce_backward_finite_differences(level, op):
    L, C = [3, 1, 4], 3
    rows = sum(n * n for n in L) if level != "samples" else sum(L)
    out_rows = sum(L) if level != "samples" else len(L)
    x, G = _r(rows, C), _r(out_rows, C)

    def fwd(xx):
        if level == "pair_rows":          # the sum over the first pair axis: transpose, then the column sum
            t = np.concatenate([blk.transpose(1, 0, 2).reshape(-1, C)
                                for blk in layout.unpack(xx, layout.pair_offsets(L), [(n, n) for n in L])])
            return ops.segment_reduce(t, L, "pair_cols", op)
        return ops.segment_reduce(xx, L, level, op)

    dx = grads.segment_reduce_backward(G, L, level, op)
    _check_directional(lambda xx: float(np.sum(G * fwd(xx))), (x,), (dx,), ("dx",))


# ---------------------------------------------------------------- LayerNorm + Linear
@pytest.mark.parametrize("epilogue,ln", [("none", True), ("none", False), ("residual", True), ("gelu", True),
                                         ("swiglu_residual", True)])
def test_layernorm_linear_backward_finite_differences(epilogue, ln):
    R, K, N, Fh = 7, 6, 5, 4
    x = _r(R, K)
    if epilogue == "swiglu_residual":
        w, b, w2, b2 = _r(2 * Fh, K, s=0.5), _r(2 * Fh, s=0.1), _r(K, Fh, s=0.5), _r(K, s=0.1)
        G = _r(R, K)
    else:
        w, b, w2, b2 = _r(N, K, s=0.5), _r(N, s=0.1), None, None
        G = _r(R, N)
    gam, bet = 1 + _r(K, s=0.1), _r(K, s=0.1)
    res = _r(R, N) if epilogue == "residual" else None

    def fwd(xx, ww, bb, gg, be, w2_=None, b2_=None):
        y = ops.layernorm_linear(xx, ww, bb, ln=(gg, be) if ln else None,
                                 epilogue="none" if epilogue == "residual" else epilogue, w2=w2_, b2=b2_)
        return y

    out = grads.layernorm_linear_backward(x, w, b, G, ln=(gam, bet) if ln else None, epilogue=epilogue, w2=w2, b2=b2)
    args = [x, w, b, gam, bet] + ([w2, b2] if w2 is not None else [])
    names = ["dx", "dw", "db", "dgamma", "dbeta"] + (["dw2", "db2"] if w2 is not None else [])
    got = [out.get(n) if (ln or n not in ("dgamma", "dbeta")) else None for n in names]
    _check_directional(lambda *a: float(np.sum(G * fwd(*a))), args, got, names)
    if epilogue == "residual":
        assert np.array_equal(out["dresidual"], G)


def test_layernorm_backward_matches_torch_autograd(torch_cpu):
    x, g, b, G = _r(9, 12), 1 + _r(12, s=0.2), _r(12, s=0.2), _r(9, 12)
    dx, dg, db = grads.layernorm_backward(x, g, G)
    xt, gt, bt = (torch.tensor(t, requires_grad=True) for t in (x, g, b))
    F.layer_norm(xt, (12,), gt, bt, 1e-5).backward(torch.from_numpy(G))
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(layernorm(x, g, b), F.layer_norm(xt, (12,), gt, bt, 1e-5).detach().numpy(), atol=1e-12)


# ---------------------------------------------------------------- attention
def _attn_inputs(L, H, d):
    R = sum(n * n for n in L)
    return _r(R, H * d), _r(R, H * d), _r(R, H * d), _r(R, H), _r(R, H * d)


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("with_bias", [True, False])
def test_attention_backward_finite_differences(axis, with_bias):
    L, H, d = [3, 1, 4], 2, 3
    q, k, v, bias, G = _attn_inputs(L, H, d)
    bias = bias if with_bias else None
    dq, dk, dv, db = grads.pair_row_attention_backward(q, k, v, bias, G, L, H, d, axis=axis, scale=0.6)
    def loss(qq, kk, vv, bb):
        o = ops.pair_row_attention(qq, kk, vv, bb if with_bias else None, L, H, d, axis=axis, scale=0.6)
        return float(np.sum(G * o))
    assert (db is None) == (not with_bias)
    _check_directional(loss, (q, k, v, bias if with_bias else np.zeros(1)), (dq, dk, dv, db),
                       ("dq", "dk", "dv", "dbias"))


@pytest.mark.parametrize("axis", [0, 1])
def test_attention_backward_from_the_exact_output_is_unchanged(axis):
    """D taken from the forward output equals D from the softmax when the
    output is exact (rowsum(dO * O) = rowsum(dP * P))."""
    L, H, d = [4, 2, 0, 3], 2, 3
    q, k, v, bias, G = _attn_inputs(L, H, d)
    o = ops.pair_row_attention(q, k, v, bias, L, H, d, axis=axis)
    a = grads.pair_row_attention_backward(q, k, v, bias, G, L, H, d, axis=axis)
    b = grads.pair_row_attention_backward(q, k, v, bias, G, L, H, d, axis=axis, o=o)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-12)


def test_attention_backward_matches_torch_autograd_on_a_padded_batch(torch_cpu):
    """Masked padded row attention in torch (valid keys only), differentiated
    by autograd; the packed gradients equal its valid cells."""
    L, H, d = [4, 2, 3], 2, 4
    q, k, v, bias, G = _attn_inputs(L, H, d)
    dq, dk, dv, db = grads.pair_row_attention_backward(q, k, v, bias, G, L, H, d, axis=0)
    B, N = len(L), max(L)
    po = layout.pair_offsets(L)

    def pad(x, c):
        out = np.zeros((B, N, N, c))
        for i, n in enumerate(L):
            out[i, :n, :n] = x[po[i]:po[i + 1]].reshape(n, n, c)
        return torch.tensor(out, requires_grad=True)

    qt, kt, vt, bt = pad(q, H * d), pad(k, H * d), pad(v, H * d), pad(bias, H)
    Gt = pad(G, H * d).detach()
    logits = torch.einsum("brjhd,brkhd->brhjk", qt.reshape(B, N, N, H, d), kt.reshape(B, N, N, H, d)) / np.sqrt(d)
    logits = logits + bt.permute(0, 3, 1, 2)[:, None]
    keyok = torch.tensor([[kk < n for kk in range(N)] for n in L])
    logits = logits.masked_fill(~keyok[:, None, None, None, :], float("-inf"))
    o = torch.einsum("brhjk,brkhd->brjhd", torch.softmax(logits, -1), vt.reshape(B, N, N, H, d)).reshape(B, N, N, H * d)
    cell = torch.tensor([[[a < n and c < n for c in range(N)] for a in range(N)] for n in L])
    (o * Gt * cell[..., None]).sum().backward()

    def unpad(t, c):
        return np.concatenate([t[i, :n, :n].reshape(n * n, c).numpy() for i, n in enumerate(L)])

    for got, t, c in ((dq, qt, H * d), (dk, kt, H * d), (dv, vt, H * d), (db, bt, H)):
        np.testing.assert_allclose(got, unpad(t.grad, c), rtol=1e-9, atol=1e-11)


# ---------------------------------------------------------------- triangle
@pytest.mark.parametrize("direction", ["outgoing", "incoming"])
def test_triangle_backward_finite_differences_and_autograd(direction, torch_cpu):
    L, C = [3, 0, 4, 2], 3
    R = sum(n * n for n in L)
    a, b, G = _r(R, C), _r(R, C), _r(R, C)
    da, db = grads.triangle_mul_backward(a, b, G, L, direction)
    loss = lambda aa, bb: float(np.sum(G * ops.triangle_mul(aa, bb, L, direction)))  # noqa: E731
    _check_directional(loss, (a, b), (da, db), ("da", "db"))
    po = layout.pair_offsets(L)
    eq = "xkc,ykc->xyc" if direction == "outgoing" else "kxc,kyc->xyc"
    for i, n in enumerate(L):
        if not n:
            continue
        sl = slice(po[i], po[i + 1])
        at = torch.tensor(a[sl].reshape(n, n, C), requires_grad=True)
        bt = torch.tensor(b[sl].reshape(n, n, C), requires_grad=True)
        (torch.einsum(eq, at, bt) * torch.from_numpy(G[sl].reshape(n, n, C))).sum().backward()
        np.testing.assert_allclose(da[sl], at.grad.reshape(n * n, C).numpy(), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(db[sl], bt.grad.reshape(n * n, C).numpy(), rtol=1e-10, atol=1e-12)
