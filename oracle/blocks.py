"""Block compositions of the oracle, with the storage rounding points of the
bf16 execution: the paper measures with BF16 parameters and inputs (Sec. 4.1
"Measurement"), so every tensor a step produces is a bf16 value -- the
normalised features entering a projection, the gated SwiGLU hidden, every
projection output and every pair/single state.  Those points are rounded here
(numerics.store); all arithmetic between them is float64.  For the fp32
workloads nothing is rounded.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

from . import ops
from .numerics import gelu, layernorm, linear, silu, store


def _ln_linear(x, w, b, ln, st):
    """LN(x) stored in the working precision, then V W^T + b (Sec. 3.3)."""
    return linear(st(layernorm(x, *ln)), w, b)


def _swiglu(x, p, st):
    """x + SwiGLU(LN(x)) with bf16 storage of LN(x) and of the gated hidden
    (Eq. running-block, second line)."""
    gu = _ln_linear(x, p["trans.w"], p["trans.b"], (p["trans.ln_g"], p["trans.ln_b"]), st)
    F = gu.shape[1] // 2
    h = st(silu(gu[:, :F]) * gu[:, F:])
    return x + linear(h, p["trans.w2"], p["trans.b2"])


PAIR_ORDER_BLOCK = ("bcast", "lin", "att_row", "tri_out", "trans", "single")
PAIR_ORDER_STACK = ("bcast", "tri_out", "tri_in", "att_row", "att_col", "trans", "single")


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
            uv = keep(linear(s, p["uv.w"], p["uv.b"]))
            trace["uv"] = uv
            z = st(ops.pair_broadcast(uv[:, :C], uv[:, C:], lengths, z_in=z))
        elif step == "lin":
            z = st(_ln_linear(z, p["lin.w"], p["lin.b"], (p["lin.ln_g"], p["lin.ln_b"]), keep))
        elif step in ("att_row", "att_col"):
            key = step
            proj = _ln_linear(z, p[key + ".w"], p[key + ".b"], (p[key + ".ln_g"], p[key + ".ln_b"]), keep)
            q, kk, v = keep(proj[:, :C]), keep(proj[:, C:2 * C]), keep(proj[:, 2 * C:3 * C])
            beta = keep(proj[:, 3 * C:3 * C + H])
            o = keep(ops.pair_row_attention(q, kk, v, beta, lengths, H, d,
                                            axis=0 if step == "att_row" else 1))
            trace[step + ".o"] = o
            z = st(z + linear(o, p[key + ".wo"], p[key + ".bo"]))
        elif step in ("tri_out", "tri_in"):
            ab = keep(_ln_linear(z, p[step + ".w"], p[step + ".b"], (p[step + ".ln_g"], p[step + ".ln_b"]), keep))
            t = ops.triangle_mul(ab[:, :C], ab[:, C:], lengths,
                                 "outgoing" if step == "tri_out" else "incoming")
            z = st(z + t)
        elif step == "trans":
            z = st(_swiglu(z, p, keep))
        elif step == "single":
            m = ops.segment_reduce(z, lengths, "pair_cols", "mean")
            trace["col_mean"] = m
            s = st(s + linear(keep(m), p["single.w"], p["single.b"]))
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
