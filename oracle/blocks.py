"""Block compositions of the oracle, with the storage rounding points of the
bf16 execution: the paper measures with BF16 parameters and inputs (Sec. 4.1
"Measurement"), so every tensor a step produces is a bf16 value -- the
normalised features entering a projection, the gated SwiGLU hidden, every
projection output and every pair/single state.  Those points are rounded here
(numerics.store); all arithmetic between them is float64.  For the fp32
workloads nothing is rounded.

Each kernel-sized piece of a block is its own function (`ref_*`), returning
its output unrounded; the block composes them and rounds every output that a
later piece consumes.  The per-kernel parity tests call the same functions on
the GPU's own stored inputs.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

from . import ops
from .numerics import gelu, layernorm, linear, sigmoid, silu, store


def _ln_linear(x, w, b, ln, st):
    """LN(x) stored in the working precision, then V W^T + b (Sec. 3.3)."""
    return linear(st(layernorm(x, *ln)), w, b)


def _ln(p, key):
    return (p[key + ".ln_g"], p[key + ".ln_b"])


# ------------------------------------------------------------ kernel pieces
# Every function takes stored (already rounded) inputs and returns its output
# unrounded; `st` is the storage rounding of values inside the piece (the
# normalised features, the gated SwiGLU hidden).

def ref_single_proj(s, p):
    """[u|v] = s W_uv^T + b_uv (Eq. running-block, first line: u_theta, v_theta)."""
    return linear(s, p["uv.w"], p["uv.b"])


def ref_broadcast(uv, C, lengths, z=None):
    """z (+)= u_a + v_b over every sample's pair cells (Eq. running-block, first line)."""
    return ops.pair_broadcast(uv[:, :C], uv[:, C:], lengths, z_in=z)


def ref_ln_linear(z, p, key, st):
    """LN(z) W^T + b with LN(z) stored (Sec. 3.3)."""
    return _ln_linear(z, p[key + ".w"], p[key + ".b"], _ln(p, key), st)


def ref_bcast_ln_linear(uv, C, lengths, p, key, st):
    """The broadcast, stored, then LN+Linear (the pair construction followed
    by the block's configuration step)."""
    return ref_ln_linear(st(ref_broadcast(uv, C, lengths)), p, key, st)


def ref_attention(qkv, beta, lengths, C, H, d, axis):
    """Row (axis 0) or column (axis 1) attention with pair bias on stored q|k|v
    ([R, 3C]) and bias ([R, H])."""
    return ops.pair_row_attention(qkv[:, :C], qkv[:, C:2 * C], qkv[:, 2 * C:3 * C], beta, lengths, H, d, axis=axis)


def ref_attn_out(o, z, p, key):
    """z + o W_o^T + b_o."""
    return z + linear(o, p[key + ".wo"], p[key + ".bo"])


def ref_triangle(ab, z, C, lengths, direction):
    """z + triangle(a, b), direction "outgoing" or "incoming"."""
    return z + ops.triangle_mul(ab[:, :C], ab[:, C:], lengths, direction)


def ref_attention_gated(qkvg, beta, lengths, C, H, d, axis):
    """Gated attention (the AlphaFold 3 form of the cited method): on stored
    [q|k|v|g] ([R, 4C]) and bias, o = sigmoid(g) * attention(q, k, v, bias)."""
    return ops.pair_row_attention(qkvg[:, :C], qkvg[:, C:2 * C], qkvg[:, 2 * C:3 * C], beta, lengths, H, d,
                                  axis=axis, gate=qkvg[:, 3 * C:4 * C])


def ref_gated_operands(proj, C):
    """a = sigmoid(a_g) * a_p, b = sigmoid(b_g) * b_p from the projection
    [a_p | a_g | b_p | b_g | g] ([R, 5C])."""
    return (ops.gated_operand(proj[:, :C], proj[:, C:2 * C]),
            ops.gated_operand(proj[:, 2 * C:3 * C], proj[:, 3 * C:4 * C]))


def ref_triangle_t(a, b, lengths, direction):
    """t = triangle(a, b) alone (the gated update normalises t before adding it)."""
    return ops.triangle_mul(a, b, lengths, direction)


def ref_gated_out(t, g, z, p, key, st):
    """z + sigmoid(g) * (LN(t) W_o^T + b_o) with LN(t) stored: the output of
    the gated triangle update."""
    return ops.layernorm_linear(st(layernorm(t, *_ln(p, key + ".out"))), p[key + ".wo"], p[key + ".bo"],
                                epilogue="gated_residual", residual=z, gate=g)


def ref_transition(z, p, st):
    """z + SwiGLU(LN(z)) with LN(z) and the gated hidden stored (Eq.
    running-block, second line)."""
    gu = _ln_linear(z, p["trans.w"], p["trans.b"], _ln(p, "trans"), st)
    F = gu.shape[1] // 2
    h = st(silu(gu[:, :F]) * gu[:, F:])
    return z + linear(h, p["trans.w2"], p["trans.b2"])


def ref_column_mean(z, lengths):
    """(1/N_i) sum_b z[a, b] (Eq. running-block, third line; Eq. pair-reduction)."""
    return ops.segment_reduce(z, lengths, "pair_cols", "mean")


def ref_single_update(m, s, p, st):
    """s + m W_s^T + b_s with the column mean m stored (g_theta)."""
    return s + linear(st(m), p["single.w"], p["single.b"])


PAIR_ORDER_BLOCK = ("bcast", "lin", "att_row", "tri_out", "trans", "single")
PAIR_ORDER_STACK = ("bcast", "tri_out", "tri_in", "att_row", "att_col", "trans", "single")
PAIR_ORDER_STACK_GATED = ("bcast", "tri_out_g", "tri_in_g", "att_row_g", "att_col_g", "trans", "single")


def pair_block(s, lengths, p, dims, order, z=None, dtype="bf16", round_last=True):
    """One single-pair-single block (Eq. running-block generalised with the
    Pairformer-style steps of Sec. 4.3).

    s       [sum N, C_s] single track;  z: [sum N^2, C_z] pair state or None.
    p       weights (see the input generator), dims: dict(c_z, heads, head_dim).
    order   sequence of steps:
      bcast    z = [z +] bcast(u, v), [u|v] = s W_uv^T + b_uv     (Eq. running-block l.1)
      lin      z = LN(z) W^T + b                                   (Sec. 3.3)
      att_row  [q|k|v|beta] = LN(z) W^T + b; o = attention axis 0; z += o W_o^T + b_o
      att_col  the same around the ending node (axis 1)
      tri_out  [a|b] = LN(z) W^T + b; z += triangle_outgoing(a, b)
      tri_in   [a|b] = LN(z) W^T + b; z += triangle_incoming(a, b)
      tri_out_g, tri_in_g   the gated update of AlphaFold 3 (the method Sec.
               4.3 cites): [a_p|a_g|b_p|b_g|g] = LN(z) W^T + b,
               a = sigmoid(a_g) a_p, b = sigmoid(b_g) b_p, t = triangle(a, b),
               z += sigmoid(g) * (LN(t) W_o^T + b_o)
      att_row_g, att_col_g  gated attention: [q|k|v|g|beta] = LN(z) W^T + b,
               o = sigmoid(g) * attention, z += o W_o^T + b_o
      trans    z = z + SwiGLU(LN(z))                                (Eq. running-block l.2)
      single   m = mean_b z[.,b];  s = s + m W_s^T + b_s            (Eq. running-block l.3)
    round_last=False returns the output of the final step unrounded (the
    exact value the last store of the GPU path rounds); every value a later
    step consumes is still stored.
    Returns (s, z, trace) where trace maps step names to intermediate values.
    """
    C, H, d = dims["c_z"], dims["heads"], dims["head_dim"]
    keep = lambda t: store(t, dtype)        # noqa: E731
    trace = {}
    s = np.asarray(s, np.float64)
    for k, step in enumerate(order):
        last = k == len(order) - 1
        st = keep if (round_last or not last) else (lambda t: np.asarray(t, np.float64))
        if step == "bcast":
            uv = keep(ref_single_proj(s, p))
            trace["uv"] = uv
            z = st(ref_broadcast(uv, C, lengths, z))
        elif step == "lin":
            z = st(ref_ln_linear(z, p, "lin", keep))
        elif step in ("att_row", "att_col"):
            proj = keep(ref_ln_linear(z, p, step, keep))
            qkv, beta = proj[:, :3 * C], proj[:, 3 * C:3 * C + H]
            o = keep(ref_attention(qkv, beta, lengths, C, H, d, 0 if step == "att_row" else 1))
            trace[step + ".o"] = o
            z = st(ref_attn_out(o, z, p, step))
        elif step in ("att_row_g", "att_col_g"):
            proj = keep(ref_ln_linear(z, p, step, keep))
            qkvg, beta = proj[:, :4 * C], proj[:, 4 * C:4 * C + H]
            o = keep(ref_attention_gated(qkvg, beta, lengths, C, H, d, 0 if step == "att_row_g" else 1))
            trace[step + ".o"] = o
            z = st(ref_attn_out(o, z, p, step))
        elif step in ("tri_out_g", "tri_in_g"):
            # the gated operands are formed from the projection before it is
            # stored; the output gate logits are stored
            proj = ref_ln_linear(z, p, step, keep)
            a, b = (keep(t) for t in ref_gated_operands(proj, C))
            proj = keep(proj)
            t = keep(ref_triangle_t(a, b, lengths, "outgoing" if step == "tri_out_g" else "incoming"))
            trace[step + ".t"] = t
            z = st(ref_gated_out(t, proj[:, 4 * C:5 * C], z, p, step, keep))
        elif step in ("tri_out", "tri_in"):
            ab = keep(ref_ln_linear(z, p, step, keep))
            z = st(ref_triangle(ab, z, C, lengths, "outgoing" if step == "tri_out" else "incoming"))
        elif step == "trans":
            z = st(ref_transition(z, p, keep))
        elif step == "single":
            m = ref_column_mean(z, lengths)
            trace["col_mean"] = m
            s = st(ref_single_update(m, s, p, keep))
        else:
            raise ValueError(f"unknown step {step!r}")
        trace[step] = z
    return s, z, trace


def encoder_layer(x, lengths, p, heads, head_dim, dtype="bf16", round_last=True):
    """Pre-LayerNorm Transformer encoder layer on packed tokens followed by a
    per-sample mean pool (the 1-D token path: Sec. 3.3 "Attention through
    packed blocks"; BERT-Base shape of Appendix C).  The pool reads the stored
    layer output; round_last=False returns that output unrounded.
    Returns (x_out, pooled, trace)."""
    st = lambda t: store(t, dtype)          # noqa: E731
    c = heads * head_dim
    x = np.asarray(x, np.float64)
    qkv = st(_ln_linear(x, p["qkv.w"], p["qkv.b"], (p["ln1_g"], p["ln1_b"]), st))
    o = st(ops.attention_1d(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], lengths, heads, head_dim))
    x = st(x + linear(o, p["o.w"], p["o.b"]))
    h = st(gelu(_ln_linear(x, p["ffn1.w"], p["ffn1.b"], (p["ln2_g"], p["ln2_b"]), st)))
    x_exact = x + linear(h, p["ffn2.w"], p["ffn2.b"])
    x = st(x_exact)
    pooled = ops.segment_reduce(x, lengths, "samples", "mean")
    return (x if round_last else x_exact), pooled, {"qkv": qkv, "o": o, "h": h}


def mechanism_weights(B):
    """Sample weights of Eq. joint-diagnostic-loss: alpha_i = 1 + i/B, beta_i = 1.5 - i/(2B)."""
    return (np.array([1.0 + i / B for i in range(B)]), np.array([1.5 - i / (2.0 * B) for i in range(B)]))


def mechanism_step(x, lengths, p, dtype="bf16", y=None, cols=None, S=1):
    """One training step of the measured single-pair-single program (Eq.
    running-block; App. A "Measured single-pair-single program"): forward,
    the joint diagnostic loss, and the backward of every parameter and input.

    Square (y, cols None): X_i [N_i, C] gives both pair operands,
      P_i[a,b] = u(X_i[a]) + v(X_i[b]).
    Rectangular: rows from x (N_i) and columns from y (M_i = cols[i]),
      P_i[a,b] = u(X_i[a]) + v(Y_i[b]), and the column mean divides by M_i.
    Then  Pt = P + SwiGLU(LN(P)),  Xt[a] = X[a] + g(mean_b Pt[a, b]),
      L = sum_i alpha_i ||Xt_i||^2 / (S C sum N) + sum_i beta_i ||Pt_i||^2 / (S C_p sum N M).
    p: u.w/u.b, v.w/v.b ([C_p, C]), trans.* (as the pair block), g.w/g.b ([C, C_p]).
    bf16: every tensor that one kernel stores and another reads is rounded
    (u, v, P, LN(P), the gated hidden, Pt, the column mean as consumed, Xt, and
    the gradients handed between kernels as bf16: dXt, dPt, dP, du, dv); all
    arithmetic between them is float64.
    Returns dict: xt, pt, loss (total), loss_s, loss_p (per sample), and
    gradients d_<param> and dx (and dy for rectangular)."""
    from . import grads as G
    from .numerics import round_bf16
    keep = (lambda t: round_bf16(t)) if dtype == "bf16" else (lambda t: np.asarray(t, np.float64))  # noqa: E731
    rect = y is not None
    cols = lengths if cols is None else cols
    x = np.asarray(x, np.float64)
    yy = np.asarray(y, np.float64) if rect else x
    B = len(lengths)
    C, Cp = x.shape[1], p["u.w"].shape[0]
    alpha, beta = mechanism_weights(B)
    sum_n = int(np.sum(lengths))
    cells = int(sum(int(n) * int(m) for n, m in zip(lengths, cols)))
    # forward
    u = keep(linear(x, p["u.w"], p["u.b"]))
    v = keep(linear(yy, p["v.w"], p["v.b"]))
    P = keep(ops.pair_broadcast(u, v, lengths, cols=cols))
    Pt = keep(ref_transition(P, p, keep))
    m = ops.segment_reduce(Pt, lengths, "pair_cols", "mean", cols=cols)
    mk = keep(m)
    xt = keep(x + linear(mk, p["g.w"], p["g.b"]))
    ls, dxt = ops.weighted_square_loss(xt, lengths, alpha, 1.0 / (S * C * sum_n))
    lp, dpt = ops.weighted_square_loss(Pt, [int(n) * int(mm) for n, mm in zip(lengths, cols)], beta,
                                       1.0 / (S * Cp * cells))
    out = {"xt": xt, "pt": Pt, "loss_s": ls, "loss_p": lp, "loss": float(ls.sum() + lp.sum())}
    # backward
    gs = G.layernorm_linear_backward(mk, p["g.w"], p["g.b"], keep(dxt), epilogue="residual")
    out["d_g.w"], out["d_g.b"] = gs["dw"], gs["db"]
    dm = gs["dx"]                                           # fp32 on the GPU, kept exact
    dpt_total = keep(keep(dpt) + G.segment_reduce_backward(dm, lengths, "pair_cols", "mean", cols=cols))
    gt = G.layernorm_linear_backward(P, p["trans.w"], p["trans.b"], dpt_total, ln=(p["trans.ln_g"], p["trans.ln_b"]),
                                     epilogue="swiglu_residual", w2=p["trans.w2"], b2=p["trans.b2"],
                                     xn_store=keep, h_store=keep)
    for k_out, k_in in (("d_trans.w", "dw"), ("d_trans.b", "db"), ("d_trans.w2", "dw2"), ("d_trans.b2", "db2"),
                        ("d_trans.ln_g", "dgamma"), ("d_trans.ln_b", "dbeta")):
        out[k_out] = gt[k_in]
    dP = keep(gt["dx"])
    du, dv = G.pair_broadcast_backward(dP, lengths, cols)
    du, dv = keep(du), keep(dv)
    gu = G.layernorm_linear_backward(x, p["u.w"], p["u.b"], du)
    gv = G.layernorm_linear_backward(yy, p["v.w"], p["v.b"], dv)
    out["d_u.w"], out["d_u.b"], out["d_v.w"], out["d_v.b"] = gu["dw"], gu["db"], gv["dw"], gv["db"]
    dx = dxt + gu["dx"]                                     # the residual path, then the u projection
    if rect:
        out["dy"] = gv["dx"]
    else:
        dx = dx + gv["dx"]
    out["dx"] = dx
    return out


def mechanism_step_nonleading(x, lengths, p, S, dtype="bf16"):
    """The single-pair-single training step in the non-leading layout (Eq.
    packing: an element (S, N_i, C) packs as (N_i, S, C), so x is
    [sum N, S*C] with X_i[s] = x[eta_i:eta_{i+1}, s*C:(s+1)*C]; App. A runs
    the program with S = 3).  Every op acts on the feature axis or on the
    ragged axes of one s, so the program on X_i is the leading program on
    each X_i[s] with shared weights: the pair state is (S, N_i, N_i, C_p),
    packed [sum N^2, S*C_p]; the loss of Eq. joint-diagnostic-loss sums over
    all S slices with S in both denominators; weight gradients sum over s.
    Returns the keys of mechanism_step, with xt, pt, dx in the packed
    non-leading layout."""
    x = np.asarray(x, np.float64)
    C = x.shape[1] // S
    outs = [mechanism_step(x[:, s * C:(s + 1) * C], lengths, p, dtype=dtype, S=S) for s in range(S)]
    res = {"xt": np.concatenate([o["xt"] for o in outs], 1),
           "pt": np.concatenate([o["pt"] for o in outs], 1),
           "dx": np.concatenate([o["dx"] for o in outs], 1),
           "loss_s": sum(o["loss_s"] for o in outs), "loss_p": sum(o["loss_p"] for o in outs),
           "loss": float(sum(o["loss"] for o in outs))}
    for k in outs[0]:
        if k.startswith("d_"):
            res[k] = sum(o[k] for o in outs)
    return res
