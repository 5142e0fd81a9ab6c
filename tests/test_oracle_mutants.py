"""The pins must be able to fail: plant plausible mistakes in the oracle (on the
CPU only) and check that at least one pin catches each of them."""
import numpy as np
import pytest

import oracle.ops as ops
import oracle.numerics as numerics
from oracle import layout
from tests import test_oracle_ops as T_ops
from tests import test_oracle_blocks as T_blk
from tests import test_oracle_layout as T_lay
from tests import test_oracle_grads as T_grads
import oracle.grads as grads


def _fails(fn, *a, **k):
    try:
        fn(*a, **k)
    except AssertionError:
        return True
    return False


def _mut_broadcast_swapped(u, v, lengths, z_in=None):
    return _orig["pair_broadcast"](v, u, lengths, z_in)


def _mut_ln_unbiased(x, gamma, beta, eps=1e-5):
    x = np.asarray(x, np.float64)
    return (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * gamma + beta


def _mut_attention_bias_transposed(q, k, v, bias, lengths, heads, head_dim, axis=0, scale=None):
    if bias is not None:
        bias = np.array(bias, np.float64)
        for off, n in zip(layout.pair_offsets(lengths), lengths):
            blk = bias[off:off + n * n].reshape(n, n, -1)
            bias[off:off + n * n] = blk.transpose(1, 0, 2).reshape(n * n, -1)
    return _orig["pair_row_attention"](q, k, v, bias, lengths, heads, head_dim, axis, scale)


def _mut_attention_no_scale(q, k, v, bias, lengths, heads, head_dim, axis=0, scale=None):
    return _orig["pair_row_attention"](q, k, v, bias, lengths, heads, head_dim, axis, 1.0)


def _mut_single_attention_bias_transposed(q, k, v, bias, lengths, heads, head_dim, scale=None):
    bias = np.array(bias, np.float64)
    for off, n in zip(layout.pair_offsets(lengths), lengths):
        blk = bias[off:off + n * n].reshape(n, n, -1)
        bias[off:off + n * n] = blk.transpose(1, 0, 2).reshape(n * n, -1)
    return _orig["single_attention_pair_bias"](q, k, v, bias, lengths, heads, head_dim, scale)


def _mut_single_attention_no_bias(q, k, v, bias, lengths, heads, head_dim, scale=None):
    return _orig["single_attention_pair_bias"](q, k, v, np.zeros_like(np.asarray(bias, np.float64)), lengths, heads, head_dim, scale)


def _mut_triangle_transposed(a, b, lengths, direction="outgoing"):
    return _orig["triangle_mul"](b, a, lengths, direction)


def _mut_triangle_direction(a, b, lengths, direction="outgoing"):
    other = {"outgoing": "incoming", "incoming": "outgoing"}[direction]
    return _orig["triangle_mul"](a, b, lengths, other)


def _mut_reduce_rows(x, lengths, level="pair_cols", op="sum"):
    if level != "pair_cols":
        return _orig["segment_reduce"](x, lengths, level, op)
    outs = []
    for off, n in zip(layout.pair_offsets(lengths), lengths):
        P = np.asarray(x[off:off + n * n], np.float64).reshape(n, n, -1)
        Y = P.sum(axis=0)                       # reduces over rows instead of columns
        outs.append(Y / n if op == "mean" and n else Y)
    return np.concatenate(outs, 0)


def _mut_pair_offsets(lengths):
    return layout.offsets([int(n) * int(n) + (1 if i == 0 else 0) for i, n in enumerate(lengths)])


def _mut_triangle_bwd_transposed(a, b, dt, lengths, direction="outgoing"):
    # uses dT^T where dT belongs (and the reverse)
    tr = np.concatenate([blk.transpose(1, 0, 2).reshape(-1, blk.shape[2])
                         for blk in layout.unpack(np.asarray(dt, np.float64), layout.pair_offsets(lengths),
                                                  [(n, n) for n in lengths])]) if len(dt) else dt
    return _orig_g["triangle_mul_backward"](a, b, tr, lengths, direction)


def _mut_ln_bwd_no_mean(x, gamma, dy, eps=1e-5):
    x, dy = np.asarray(x, np.float64), np.asarray(dy, np.float64)
    mu = x.mean(-1, keepdims=True)
    rstd = 1 / np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + eps)
    xhat = (x - mu) * rstd
    g = dy * gamma
    return rstd * (g - xhat * (g * xhat).mean(-1, keepdims=True)), (dy * xhat).sum(0), dy.sum(0)


def _mut_attn_bwd_no_bias_grad_sum(q, k, v, bias, do, lengths, heads, head_dim, axis=0, scale=None):
    dq, dk, dv, db = _orig_g["pair_row_attention_backward"](q, k, v, bias, do, lengths, heads, head_dim, axis, scale)
    return dq, dk, dv, (None if db is None else db / max(1, max(lengths)))


def _mut_broadcast_bwd_swapped(dz, lengths):
    du, dv = _orig_g["pair_broadcast_backward"](dz, lengths)
    return dv, du


_orig_g = {k: getattr(grads, k) for k in ("triangle_mul_backward", "layernorm_backward",
                                          "pair_row_attention_backward", "pair_broadcast_backward")}

_orig = {k: getattr(ops, k) for k in ("pair_broadcast", "pair_row_attention", "triangle_mul", "segment_reduce",
                                        "single_attention_pair_bias")}

MUTANTS = [
    ("broadcast_swapped", ops, "pair_broadcast", _mut_broadcast_swapped,
     [(T_ops.test_broadcast_worked_example, ())]),
    ("layernorm_unbiased", numerics, "layernorm", _mut_ln_unbiased,
     [(T_ops.test_layernorm_linear_brute_force, ())]),
    ("attention_bias_transposed", ops, "pair_row_attention", _mut_attention_bias_transposed,
     [(T_ops.test_attention_brute_force, ()), (T_ops.test_attention_dominant_bias_selects_value, ())]),
    ("attention_no_scale", ops, "pair_row_attention", _mut_attention_no_scale,
     [(T_ops.test_attention_brute_force, ())]),
    ("single_attention_bias_transposed", ops, "single_attention_pair_bias", _mut_single_attention_bias_transposed,
     [(T_ops.test_single_attention_brute_force, ()), (T_ops.test_single_attention_dominant_bias_selects_value, ())]),
    ("single_attention_no_bias", ops, "single_attention_pair_bias", _mut_single_attention_no_bias,
     [(T_ops.test_single_attention_brute_force, ())]),
    ("triangle_operands_swapped", ops, "triangle_mul", _mut_triangle_transposed,
     [(T_ops.test_triangle_masked_padded_and_brute_force, ())]),
    ("triangle_direction", ops, "triangle_mul", _mut_triangle_direction,
     [(T_ops.test_triangle_masked_padded_and_brute_force, ())]),
    ("reduce_over_rows", ops, "segment_reduce", _mut_reduce_rows,
     [(T_ops.test_pair_column_sum_equation, ())]),
    ("pair_offsets_off_by_one", layout, "pair_offsets", _mut_pair_offsets,
     [(T_lay.test_worked_example_offsets_and_splits, ())]),
    ("triangle_backward_transposed_cotangent", grads, "triangle_mul_backward", _mut_triangle_bwd_transposed,
     [(T_grads.test_triangle_backward_finite_differences_and_autograd, ("outgoing", None))]),
    ("layernorm_backward_without_mean_term", grads, "layernorm_backward", _mut_ln_bwd_no_mean,
     [(T_grads.test_layernorm_backward_matches_torch_autograd, (None,))]),
    ("attention_backward_bias_gradient_averaged", grads, "pair_row_attention_backward", _mut_attn_bwd_no_bias_grad_sum,
     [(T_grads.test_attention_backward_finite_differences, (0, True))]),
    ("broadcast_backward_swapped", grads, "pair_broadcast_backward", _mut_broadcast_bwd_swapped,
     [(T_grads.test_broadcast_backward_finite_differences_and_sums, ())]),
]


@pytest.mark.parametrize("name,mod,attr,mutant,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mod, attr, mutant, pins):
    monkeypatch.setattr(mod, attr, mutant)
    if mod is numerics:          # ops imported the name directly
        monkeypatch.setattr(ops, attr, mutant)
    caught = [_fails(fn, *args) for fn, args in pins]
    assert any(caught), f"no pin caught the planted mistake {name}"


def test_padded_block_pin_catches_a_triangle_mistake(monkeypatch):
    monkeypatch.setattr(ops, "triangle_mul", _mut_triangle_transposed)
    from oracle import blocks
    assert _fails(T_blk.test_pair_block_equals_masked_padded, [4, 6, 2], blocks.PAIR_ORDER_STACK)


def _mut_gated_operand_roles_swapped(proj, gate_logits):
    return numerics.sigmoid(proj) * np.asarray(gate_logits, np.float64)


def _mut_attention_gate_ignored(q, k, v, bias, lengths, heads, head_dim, axis=0, scale=None, gate=None):
    return _orig["pair_row_attention"](q, k, v, bias, lengths, heads, head_dim, axis, scale)


def _mut_gated_residual_ungated(x, w, b=None, ln=None, eps=1e-5, epilogue="none", w2=None, b2=None, residual=None,
                                gate=None):
    if epilogue == "gated_residual":
        epilogue, gate = "residual", None
    return _orig_lin(x, w, b, ln, eps, epilogue, w2, b2, residual, gate)


_orig_lin = ops.layernorm_linear


@pytest.mark.parametrize("attr,mutant", [("gated_operand", _mut_gated_operand_roles_swapped),
                                         ("pair_row_attention", _mut_attention_gate_ignored),
                                         ("layernorm_linear", _mut_gated_residual_ungated)])
def test_padded_block_pin_catches_gated_step_mistakes(monkeypatch, attr, mutant):
    """Swapped gate and projection roles, an ignored attention gate and an
    ungated triangle output each fail the masked padded pin of the gated stack."""
    monkeypatch.setattr(ops, attr, mutant)
    from oracle import blocks
    assert _fails(T_blk.test_pair_block_equals_masked_padded, [4, 6, 2, 1], blocks.PAIR_ORDER_STACK_GATED)
