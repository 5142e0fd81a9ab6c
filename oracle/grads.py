"""Analytic gradients of the packed pair-state operations, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's measured step is forward, loss and backward through the packed
representation (Sec. 3.4 "Gradients across representations"; Sec. 4.1
"Measurement"): a gradient carries the same partitions and dimension order
as the value it belongs to.  Every function here returns gradients in the
packed layout of the corresponding input, computed per sample on its dense
element (the reference-semantics contract of Appendix A applied to the
derivative: the logical view of a packed gradient is the dense gradient of
the logical view).

Each backward takes the forward's inputs and the gradient of a scalar loss
with respect to the forward's output, and returns the gradients with respect
to every input.  The formulas are the chain rule written out; the pins
(tests/test_oracle_grads.py) check them against central finite differences
and against torch autograd of independent torch forwards.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from . import layout
from .numerics import LN_EPS, linear, softmax
from .ops import _pair_elements, _single_elements


def _f64(x):
    return np.asarray(x, dtype=np.float64)


# ----------------------------------------------------------------- broadcast
def pair_broadcast_backward(dz, lengths, cols=None):
    """z[o_i + a M_i + b] = u[eta_i + a] + v[kappa_i + b] (Eq. running-block,
    first line; M_i = N_i for square pairs).  du[eta_i + a] = sum_b dz[a, b]
    (the column sum of Eq. pair-reduction), dv[kappa_i + b] = sum_a dz[a, b]
    (the sum over the first pair axis).  Returns (du [sum N, C], dv [sum M, C])."""
    C = _f64(dz).shape[1]
    du, dv = [], []
    for P in _pair_elements(dz, lengths, cols):
        du.append(P.sum(axis=1))
        dv.append(P.sum(axis=0))
    return layout.pack(du, (C,)), layout.pack(dv, (C,))


# ----------------------------------------------------------------- reduce
def segment_reduce_backward(dy, lengths, level="pair_cols", op="sum", cols=None):
    """Backward of segment_reduce: the gradient of every reduced position is
    the gradient of its group, divided by the group size for the mean.
      pair_cols  dx[o_i + a M_i + b] = dy[eta_i + a]   (/ M_i)
      pair_rows  dx[o_i + a M_i + b] = dy[kappa_i + b] (/ N_i)   (sum over the first pair axis)
      samples    dx[eta_i + t] = dy[i] (/ N_i)
    (square pairs: M_i = N_i, kappa = eta)."""
    dy = _f64(dy)
    C = dy.shape[1]
    outs = []
    if level in ("pair_cols", "pair_rows"):
        cols = lengths if cols is None else cols
        group = lengths if level == "pair_cols" else cols
        for Y, n, m in zip(_single_elements(dy, group), lengths, cols):
            n, m = int(n), int(m)
            cnt = m if level == "pair_cols" else n
            g = Y / cnt if (op == "mean" and cnt) else Y
            P = np.repeat(g[:, None, :], m, axis=1) if level == "pair_cols" else np.repeat(g[None, :, :], n, axis=0)
            outs.append(P)
        return layout.pack(outs, (C,))
    if level == "samples":
        for i, n in enumerate(lengths):
            n = int(n)
            g = dy[i] / n if (op == "mean" and n) else dy[i]
            outs.append(np.repeat(g[None, :], n, axis=0))
        return layout.pack(outs, (C,))
    raise ValueError(level)


# ----------------------------------------------------------------- LayerNorm + Linear
def layernorm_backward(x, gamma, dxhat_affine, eps=LN_EPS):
    """y = (x - mu) / sqrt(var + eps) * gamma + beta over the feature axis
    (biased variance).  Given dy, returns (dx, dgamma, dbeta):
      xhat = (x - mu) * rstd,  g = dy * gamma,
      dx = rstd * (g - mean(g) - xhat * mean(g * xhat)),
      dgamma = sum_rows dy * xhat,  dbeta = sum_rows dy."""
    x = _f64(x)
    dy = _f64(dxhat_affine)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    g = dy * _f64(gamma)
    dx = rstd * (g - g.mean(axis=-1, keepdims=True) - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    return dx, (dy * xhat).sum(axis=0), dy.sum(axis=0)


def _gelu_grad(x):
    """d/dx of x * Phi(x) = Phi(x) + x * phi(x) (exact erf GELU)."""
    return 0.5 * (1.0 + erf(x / np.sqrt(2.0))) + x * np.exp(-0.5 * x * x) / np.sqrt(2.0 * np.pi)


def _silu_grad(x):
    s = 1.0 / (1.0 + np.exp(-x))
    return s * (1.0 + x * (1.0 - s))


def layernorm_linear_backward(x, w, b, dy, ln=None, eps=LN_EPS, epilogue="none", w2=None, b2=None,
                              residual_is_x=True, xn_store=None, h_store=None):
    """Backward of ops.layernorm_linear (Sec. 3.3: V' = V W^T + b, after an
    optional LayerNorm on each row's features).

    x [R, K], w [N_w, K], dy [R, N].  ln = (gamma, beta) or None.
    epilogue "none" / "residual": y = LN(x) W^T + b (+ residual); the
        residual's gradient is dy itself and is returned as "dresidual".
    "gelu": y = gelu(p), p = LN(x) W^T + b.
    "swiglu_residual": y = residual + (silu(g) * u) W2^T + b2 with
        [g | u] = LN(x) W^T + b; with residual_is_x (the forward's default,
        residual = x) dx includes dy, otherwise dy is returned as "dresidual".
    xn_store / h_store: storage rounding applied to the normalised rows and
    to the gated hidden where the GPU path stores them (identity by default).
    Returns a dict with dx, dw, db and, as they apply, dgamma, dbeta, dw2,
    db2, dresidual."""
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    keep_xn = xn_store or (lambda t: t)
    keep_h = h_store or (lambda t: t)
    out = {}
    if ln is not None:
        mu = x.mean(axis=-1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
        xn = keep_xn((x - mu) / np.sqrt(var + eps) * _f64(ln[0]) + _f64(ln[1]))
    else:
        xn = x
    if epilogue in ("none", "residual"):
        dp = dy
        if epilogue == "residual":
            out["dresidual"] = dy.copy()
    elif epilogue == "gelu":
        dp = dy * _gelu_grad(linear(xn, w, b))
    elif epilogue == "swiglu_residual":
        gu = linear(xn, w, b)
        F = gu.shape[1] // 2
        g, u = gu[:, :F], gu[:, F:]
        h = keep_h(g / (1.0 + np.exp(-g)) * u)
        w2 = _f64(w2)
        out["dw2"] = dy.T @ h
        out["db2"] = dy.sum(axis=0)
        dh = dy @ w2
        silu_g = g / (1.0 + np.exp(-g))
        dp = np.concatenate([dh * u * _silu_grad(g), dh * silu_g], axis=1)
        if not residual_is_x:
            out["dresidual"] = dy.copy()
    else:
        raise ValueError(epilogue)
    out["dw"] = dp.T @ xn
    out["db"] = dp.sum(axis=0)
    dxn = dp @ w
    if ln is not None:
        dx, out["dgamma"], out["dbeta"] = layernorm_backward(x, ln[0], dxn, eps)
    else:
        dx = dxn
    if epilogue == "swiglu_residual" and residual_is_x:
        dx = dx + dy
    out["dx"] = dx
    return out


# ----------------------------------------------------------------- attention
def _attention_rows_backward(Q, K, V, Bm, dO, scale, Os=None):
    """One sample, starting-node form (ops._row_attention_sample): Q, K, V, dO
    [N, N, H, d], Bm [N, N, H] or None.  For every pair row r and head h:
      S = scale Q_r K_r^T + B,  P = softmax_k(S),  O_r = P V_r
      dV_r = P^T dO_r,  dP = dO_r V_r^T,  dS = P * (dP - D),
      D = rowsum(dP * P) = rowsum(dO_r * O_r),
      dQ_r = scale dS K_r,  dK_r = scale dS^T Q_r,  dB += dS (summed over r).
    Os: the forward output as stored ([N, N, H, d]); when given, D is taken
    from it (rowsum(dO * O)), as a backward that reads the stored output does."""
    N, _, H, d = Q.shape
    dQ, dK, dV = np.zeros_like(Q), np.zeros_like(K), np.zeros_like(V)
    dB = np.zeros((N, N, H))
    for r in range(N):
        for h in range(H):
            s = scale * (Q[r, :, h, :] @ K[r, :, h, :].T)
            if Bm is not None:
                s = s + Bm[:, :, h]
            P = softmax(s, axis=-1)
            g = dO[r, :, h, :]
            dV[r, :, h, :] = P.T @ g
            dP = g @ V[r, :, h, :].T
            D = (dP * P).sum(axis=-1, keepdims=True) if Os is None else (g * Os[r, :, h, :]).sum(-1, keepdims=True)
            dS = P * (dP - D)
            dQ[r, :, h, :] = scale * (dS @ K[r, :, h, :])
            dK[r, :, h, :] = scale * (dS.T @ Q[r, :, h, :])
            dB[:, :, h] += dS
    return dQ, dK, dV, dB


def pair_row_attention_backward(q, k, v, bias, do, lengths, heads, head_dim, axis=0, scale=None, o=None):
    """Backward of ops.pair_row_attention.  Returns (dq, dk, dv, dbias) in the
    packed layouts of q, k, v ([sum N^2, H*d]) and of the bias ([sum N^2, H];
    None without a bias).  Axis 1 is axis 0 on each sample's transpose, so its
    gradients are transposed back the same way.  o: the stored forward output
    (e.g. rounded to bf16), from which D = rowsum(do * o) is taken; None uses
    the exact softmax."""
    H, d = int(heads), int(head_dim)
    scale = 1.0 / np.sqrt(d) if scale is None else float(scale)
    Qs, Ks, Vs, Gs = (_pair_elements(t, lengths) for t in (q, k, v, do))
    Bs = _pair_elements(bias, lengths) if bias is not None else [None] * len(lengths)
    Os = _pair_elements(o, lengths) if o is not None else [None] * len(lengths)
    outs = ([], [], [], [])
    for Q, K, V, G, Bm, Om in zip(Qs, Ks, Vs, Gs, Bs, Os):
        N = Q.shape[0]
        Q, K, V, G = (t.reshape(N, N, H, d) for t in (Q, K, V, G))
        Om = None if Om is None else Om.reshape(N, N, H, d)
        if axis == 1:
            Q, K, V, G = (t.transpose(1, 0, 2, 3) for t in (Q, K, V, G))
            Om = None if Om is None else Om.transpose(1, 0, 2, 3)
            Bm = None if Bm is None else Bm.transpose(1, 0, 2)
        dQ, dK, dV, dB = _attention_rows_backward(Q, K, V, Bm, G, scale, Om)
        if axis == 1:
            dQ, dK, dV = (t.transpose(1, 0, 2, 3) for t in (dQ, dK, dV))
            dB = dB.transpose(1, 0, 2)
        for lst, t in zip(outs, (dQ, dK, dV)):
            lst.append(t.reshape(N, N, H * d))
        outs[3].append(dB)
    dq, dk, dv = (layout.pack(o, (H * d,)) for o in outs[:3])
    db = layout.pack(outs[3], (H,)) if bias is not None else None
    return dq, dk, dv, db


# ----------------------------------------------------------------- triangle
def triangle_mul_backward(a, b, dt, lengths, direction="outgoing"):
    """Backward of ops.triangle_mul, per sample and channel c:
      outgoing  T_c = A_c B_c^T:   dA_c = dT_c B_c,    dB_c = dT_c^T A_c
      incoming  T_c = A_c^T B_c:   dA_c = B_c dT_c^T,  dB_c = A_c dT_c
    Returns (da, db) in the packed layout of a and b."""
    if direction not in ("outgoing", "incoming"):
        raise ValueError(direction)
    As, Bs, Gs = (_pair_elements(t, lengths) for t in (a, b, dt))
    da, db = [], []
    for A, Bm, G in zip(As, Bs, Gs):
        Ac, Bc, Gc = (np.ascontiguousarray(np.moveaxis(t, 2, 0)) for t in (A, Bm, G))
        tr = lambda t: np.swapaxes(t, 1, 2)     # noqa: E731
        if direction == "outgoing":
            dA, dB = Gc @ Bc, tr(Gc) @ Ac
        else:
            dA, dB = Bc @ tr(Gc), Ac @ Gc
        da.append(np.moveaxis(dA, 0, 2))
        db.append(np.moveaxis(dB, 0, 2))
    C = _f64(a).shape[1]
    return layout.pack(da, (C,)), layout.pack(db, (C,))
