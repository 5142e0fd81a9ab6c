"""Per-operation oracle: every op loops over samples and runs dense float64 math
on each sample's own element.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Packed layouts used here are the paper's (Sec. 3.1, Eq. packing, ragged axes
first, features last): singles are [sum N_i, C]; square pairs are
[sum N_i^2, C] with cell (i, a, b) at row o_i + a N_i + b (Eq. coordinate).
Attention tensors are [rows, H*d] (head-major within a row) and the pair bias
is [sum N_i^2, H].
"""
from __future__ import annotations

import numpy as np

from . import layout
from .numerics import layernorm, linear, silu, gelu, sigmoid, softmax, LN_EPS


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _pair_elements(x, lengths, cols=None):
    """Logical view of a pair tensor: list of [N_i, M_i, C...] arrays (square
    pairs: M_i = N_i; rectangular pairs pack (N_i, M_i, C) as N_i M_i rows,
    Eq. packing)."""
    cols = lengths if cols is None else cols
    o = layout.rect_pair_offsets(lengths, cols)
    return layout.unpack(_f64(x), o, [(int(n), int(m)) for n, m in zip(lengths, cols)])


def _single_elements(x, lengths):
    o = layout.single_offsets(lengths)
    return layout.unpack(_f64(x), o, [(int(n),) for n in lengths])


# --------------------------------------------------------------------------- A2
def pair_broadcast(u, v, lengths, z_in=None, cols=None):
    """Pair construction by broadcasting (Eq. running-block, first line; Sec. 3.2
    "Creating axes through broadcasting"): element shapes (N_i,1,C) + (1,M_i,C)
    give (N_i,M_i,C) with P_i[a,b,:] = U_i[a,:] + V_i[b,:].  Square pairs take
    M_i = N_i and both operands from one single track; rectangular pairs take
    v from a column track of M_i rows per sample (cols).  No activation is
    applied (Appendix A.1).  With z_in the result is added to an existing pair
    state of the same layout.
    Pins: worked example (2,3), gather form of Fig. "program", numpy
    broadcasting for equal lengths, fp32 exactness, a rectangular worked
    example."""
    cols = lengths if cols is None else cols
    U, V = _single_elements(u, lengths), _single_elements(v, cols)
    elems = [Ui[:, None, :] + Vi[None, :, :] for Ui, Vi in zip(U, V)]
    C = _f64(u).shape[1]
    P = layout.pack(elems, (C,))
    if z_in is not None:
        P = P + _f64(z_in)
    return P


# --------------------------------------------------------------------------- A3
def layernorm_linear(x, w, b=None, ln=None, eps=LN_EPS, epilogue="none",
                     w2=None, b2=None, residual=None, gate=None):
    """Feature transform on packed rows (Sec. 3.3: V' = V W^T + b, normalisation
    on each row's feature tail; Sec. 3.2: feature transforms retain structure).
    Rows are independent, so the packed computation is the dense one on V.

    ln        (gamma, beta) for a LayerNorm before the projection, or None.
    epilogue  "none"            y = LN(x) W^T + b
              "residual"        y = residual + LN(x) W^T + b
              "gelu"            y = gelu(LN(x) W^T + b)   (exact erf form)
              "gated_residual"  y = residual + sigmoid(gate) * (LN(x) W^T + b),
                                the output gate of the AlphaFold 3 triangle
                                update that Sec. 4.3 cites (gate [rows, N])
              "swiglu_residual" the pre-normalised SwiGLU transition of
                                Eq. running-block (second line, h_theta):
                                W stacks [W_gate; W_up] (2F x C), then
                                y = residual + (silu(LN(x)W_g^T+b_g) * (LN(x)W_u^T+b_u)) W2^T + b2
                                (residual defaults to x).
    """
    x = _f64(x)
    xn = layernorm(x, *ln, eps=eps) if ln is not None else x
    y = linear(xn, w, b)
    if epilogue == "none":
        return y
    if epilogue == "residual":
        return _f64(residual) + y
    if epilogue == "gated_residual":
        return _f64(residual) + sigmoid(gate) * y
    if epilogue == "gelu":
        return gelu(y)
    if epilogue == "swiglu_residual":
        F = y.shape[1] // 2
        h = silu(y[:, :F]) * y[:, F:]
        res = x if residual is None else _f64(residual)
        return res + linear(h, w2, b2)
    raise ValueError(f"unknown epilogue {epilogue!r}")


# --------------------------------------------------------------------------- A4
def _row_attention_sample(Q, K, V, Bias, scale):
    """One sample, starting-node form: Q,K,V [N,N,H,d], Bias [N,N,H].
    O[r,j,h] = sum_k softmax_k(scale * Q[r,j,h].K[r,k,h] + Bias[j,k,h]) V[r,k,h]."""
    N, _, H, d = Q.shape
    O = np.zeros_like(Q)
    for r in range(N):
        for h in range(H):
            s = scale * (Q[r, :, h, :] @ K[r, :, h, :].T)        # [j, k]
            if Bias is not None:
                s = s + Bias[:, :, h]
            O[r, :, h, :] = softmax(s, axis=-1) @ V[r, :, h, :]
    return O


def pair_row_attention(q, k, v, bias, lengths, heads, head_dim, axis=0, scale=None, gate=None):
    """Row (axis=0, around the starting node) or column (axis=1, around the
    ending node) attention with pair bias over a square pair state
    (Sec. 4.3 "A larger pair application", which cites the AlphaFold 3
    Pairformer; the paper gives no formula, see the design notes for this
    reading).  Axis 1 is axis 0 applied to every sample's transpose
    (P'[a,b] = P[b,a] for q, k, v and the bias), transposed back.
    gate: [sum N^2, H*d] logits of the output gate of the AlphaFold 3 form
    (the cited method), o <- sigmoid(gate) * o per cell and channel; None:
    no gate.
    Parity: the formula is a reading; pinned by special cases (zero queries,
    one dominant bias entry, equal lengths = dense batch, masked padded
    attention) and brute force."""
    H, d = int(heads), int(head_dim)
    scale = 1.0 / np.sqrt(d) if scale is None else float(scale)
    Qs, Ks, Vs = (_pair_elements(t, lengths) for t in (q, k, v))
    Bs = _pair_elements(bias, lengths) if bias is not None else [None] * len(lengths)
    outs = []
    for Q, K, V, Bm in zip(Qs, Ks, Vs, Bs):
        N = Q.shape[0]
        Q, K, V = (t.reshape(N, N, H, d) for t in (Q, K, V))
        if axis == 1:
            Q, K, V = (t.transpose(1, 0, 2, 3) for t in (Q, K, V))
            Bm = None if Bm is None else Bm.transpose(1, 0, 2)
        O = _row_attention_sample(Q, K, V, Bm, scale)
        if axis == 1:
            O = O.transpose(1, 0, 2, 3)
        outs.append(O.reshape(N, N, H * d))
    out = layout.pack(outs, (H * d,))
    return out if gate is None else sigmoid(gate) * out


def single_attention_pair_bias(q, k, v, bias, lengths, heads, head_dim, scale=None):
    """Attention over each sample's single rows with a bias read from its pair
    state (the Pairformer's single attention with pair bias, which Sec. 4.3
    cites for its pair application): for sample i, query t and key k,
      o[t] = sum_k softmax_k(scale * q[t].k[k] + bias[cell(i,t,k)]) v[k],
    with q, k, v, o token-major [sum N, H*d] and bias [sum N^2, H] (None: no
    bias, which is plain per-sample self-attention).  This is
    the row-attention step with one row per sample, in the single index
    space.  Parity: a reading of a cited method; pinned by zero queries, one
    dominant bias entry, masked padded attention and brute force."""
    H, d = int(heads), int(head_dim)
    scale = 1.0 / np.sqrt(d) if scale is None else float(scale)
    Qs, Ks, Vs = (_single_elements(t, lengths) for t in (q, k, v))
    Bs = _pair_elements(bias, lengths) if bias is not None else [None] * len(lengths)
    outs = []
    for Q, K, V, Bm in zip(Qs, Ks, Vs, Bs):
        N = Q.shape[0]
        Q, K, V = (t.reshape(N, H, d) for t in (Q, K, V))
        O = np.zeros_like(Q)
        for h in range(H):
            if N:
                s = scale * (Q[:, h, :] @ K[:, h, :].T)
                if Bm is not None:
                    s = s + Bm[:, :, h]
                O[:, h, :] = softmax(s, axis=-1) @ V[:, h, :]
        outs.append(O.reshape(N, H * d))
    return layout.pack(outs, (H * d,))


def attention_1d(q, k, v, lengths, heads, head_dim, scale=None, kv_lengths=None):
    """Variable-length attention on packed token-major [T, H*d] buffers with
    cumulative lengths (Sec. 3.3 "Attention through packed blocks"): queries
    of sample i attend to the keys of sample i only; no mask otherwise.
    kv_lengths: cross-attention, where sample i has its own number of keys and
    values (k, v packed by kv_lengths) and the output adopts the query
    structure; a query with no keys gets 0 (the empty sum)."""
    H, d = int(heads), int(head_dim)
    scale = 1.0 / np.sqrt(d) if scale is None else float(scale)
    kv_lengths = lengths if kv_lengths is None else kv_lengths
    Qs = _single_elements(q, lengths)
    Ks, Vs = (_single_elements(t, kv_lengths) for t in (k, v))
    outs = []
    for Q, K, V in zip(Qs, Ks, Vs):
        N, M = Q.shape[0], K.shape[0]
        Q = Q.reshape(N, H, d)
        K, V = K.reshape(M, H, d), V.reshape(M, H, d)
        O = np.zeros_like(Q)
        for h in range(H):
            if N and M:
                s = scale * (Q[:, h, :] @ K[:, h, :].T)
                O[:, h, :] = softmax(s, axis=-1) @ V[:, h, :]
        outs.append(O.reshape(N, H * d))
    return layout.pack(outs, (H * d,))


# --------------------------------------------------------------------------- A5
def triangle_mul(a, b, lengths, direction="outgoing"):
    """Triangle multiplicative update on a square pair state, channelwise
    (Sec. 4.3, after AlphaFold 3; the paper gives no formula, see the design
    notes for this reading):
      outgoing  T[x,y,c] = sum_k A[x,k,c] B[y,k,c]
      incoming  T[x,y,c] = sum_k A[k,x,c] B[k,y,c]
    with A, B the sample's [N,N,C] elements.  No gates and no output
    projection: the caller adds T to the pair state.
    Parity: reading; pinned by b = 1 (row sums), a = b (symmetry), incoming =
    outgoing of transposes, equal lengths = dense einsum and brute force."""
    As, Bs = _pair_elements(a, lengths), _pair_elements(b, lengths)
    if direction not in ("outgoing", "incoming"):
        raise ValueError(direction)
    outs = []
    for A, Bm in zip(As, Bs):
        # one N x N matrix product per channel c: A_c B_c^T (outgoing) or
        # A_c^T B_c (incoming), on channel-first copies of the planes
        Ac = np.ascontiguousarray(np.moveaxis(A, 2, 0))
        Bc = np.ascontiguousarray(np.moveaxis(Bm, 2, 0))
        if direction == "outgoing":
            Tc = Ac @ np.swapaxes(Bc, 1, 2)
        else:
            Tc = np.swapaxes(Ac, 1, 2) @ Bc
        outs.append(np.moveaxis(Tc, 0, 2))
    C = _f64(a).shape[1]
    return layout.pack(outs, (C,))


def gated_operand(proj, gate_logits):
    """sigmoid(gate) * proj, elementwise: the gated projection that forms the
    operands a and b of the AlphaFold 3 triangle multiplicative update cited
    in Sec. 4.3 (gated variant; the plain update uses proj directly)."""
    return sigmoid(gate_logits) * _f64(proj)


# --------------------------------------------------------------------------- A6
def segment_reduce(x, lengths, level="pair_cols", op="sum", cols=None):
    """Reductions that consume a ragged axis.

    level "pair_cols": Eq. pair-reduction, V_Y[eta_i + a] = sum_b V_P[o_i + a M_i + b];
        "mean" divides each group by M_i (N_i for square pairs: Eq.
        running-block, third line; the rectangular variant divides by M_i).
    level "pair_rows": the same over the other pair axis,
        V_Y[kappa_i + b] = sum_a V_P[o_i + a M_i + b], mean over N_i (the
        broadcast's gradient with respect to its column operand).
    cols: M_i of rectangular pairs (None: square).
    level "samples":   complete reduction within each single-axis element,
        y_i = sum_t X_i[t] (Appendix A: sum(dim=0) of [1,2] and [3,4] is [3,7]);
        "mean" divides by N_i.  An empty element sums to 0 and its mean is NaN,
        as the dense mean of an empty array.
    """
    if op not in ("sum", "mean"):
        raise ValueError(op)
    outs = []
    if level in ("pair_cols", "pair_rows"):
        for P in _pair_elements(x, lengths, cols):
            ax = 1 if level == "pair_cols" else 0
            cnt = P.shape[ax]
            Y = P.sum(axis=ax)
            if op == "mean":                   # an empty group's mean is NaN, as the dense mean of nothing
                Y = Y / cnt if cnt else np.full_like(Y, np.nan)
            outs.append(Y)
        C = _f64(x).shape[1]
        return layout.pack(outs, (C,))
    if level == "samples":
        for X in _single_elements(x, lengths):
            N = X.shape[0]
            y = X.sum(axis=0)
            if op == "mean":
                y = y / N if N else np.full_like(y, np.nan)
            outs.append(y)
        return np.stack(outs, 0) if outs else np.zeros((0, _f64(x).shape[1]))
    raise ValueError(level)


# --------------------------------------------------------------------------- loss
def weighted_square_loss(x, counts, weights, scale):
    """The diagnostic loss of the measured single-pair-single program (App. A,
    Eq. joint-diagnostic-loss), one term: sample i owns the next counts[i]
    packed rows of x, and contributes scale * weights[i] * ||x_i||_F^2.
    Returns (per-sample losses [B], gradient dL/dx = 2 scale w_i x)."""
    x = _f64(x)
    o = layout.offsets(counts)
    loss = np.array([scale * w * float(np.sum(x[o[i]:o[i + 1]] ** 2)) for i, w in enumerate(weights)])
    g = np.concatenate([2.0 * scale * w * x[o[i]:o[i + 1]] for i, w in enumerate(weights)]) if len(x) else x
    return loss, g
