"""Pins of the per-op oracle: worked examples, closed forms, special cases that
reduce to library routines, masked padded computations and brute force."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import layout, ops

GOLD = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


def _rand(*shape):
    return RNG.standard_normal(shape)


def _pad_pairs(x, lengths):
    """Independent padded view [B, Nmax, Nmax, C] plus validity mask (true = valid)."""
    B, nmax, C = len(lengths), max(lengths), x.shape[1]
    out = np.zeros((B, nmax, nmax, C))
    mask = np.zeros((B, nmax, nmax), bool)
    pos = 0
    for i, n in enumerate(lengths):
        for a in range(n):
            out[i, a, :n] = x[pos:pos + n]
            mask[i, a, :n] = True
            pos += n
    return out, mask


def _unpad_pairs(p, lengths):
    return np.concatenate([p[i, :n, :n].reshape(n * n, -1) for i, n in enumerate(lengths)], 0)


# ---------------------------------------------------------------- broadcast
def test_broadcast_worked_example():
    g = json.load(open(os.path.join(GOLD, "worked_example_2_3.json")))
    L = g["lengths"]
    u = np.arange(5, dtype=float)[:, None] * 10.0      # row features 0,10,20,30,40
    v = np.arange(5, dtype=float)[:, None]              # column features 0..4
    z = ops.pair_broadcast(u, v, L)
    assert z.shape == (13, 1)
    expect = [10 * r + c for r, c in zip(g["rows"], g["columns"])]
    assert z[:, 0].tolist() == expect


def test_broadcast_equals_gather_form():
    L = [3, 1, 0, 5]
    u, v = _rand(9, 6), _rand(9, 6)
    rows, cols = layout.pair_gather_indices(L)
    np.testing.assert_array_equal(ops.pair_broadcast(u, v, L), u[rows] + v[cols])


def test_broadcast_equal_lengths_is_numpy_broadcasting():
    B, N, C = 3, 4, 5
    u, v = _rand(B * N, C), _rand(B * N, C)
    dense = u.reshape(B, N, 1, C) + v.reshape(B, 1, N, C)
    np.testing.assert_array_equal(ops.pair_broadcast(u, v, [N] * B), dense.reshape(-1, C))


def test_broadcast_accumulate_and_fp32_exact():
    L = [2, 3]
    u = _rand(5, 4).astype(np.float32)
    v = _rand(5, 4).astype(np.float32)
    z0 = _rand(13, 4)
    z = ops.pair_broadcast(u, v, L, z_in=z0)
    np.testing.assert_allclose(z - z0, ops.pair_broadcast(u, v, L), rtol=0, atol=1e-12)
    # one add of float32 inputs: the fp32 GPU result is the correctly rounded sum
    one = ops.pair_broadcast(u, v, L)
    assert np.array_equal(one.astype(np.float32), (u[layout.pair_gather_indices(L)[0]].astype(np.float32)
                                                   + v[layout.pair_gather_indices(L)[1]].astype(np.float32)))


# ---------------------------------------------------------------- LN + Linear
def _torch_ln_linear(x, w, b, g=None, beta=None):
    t = torch.from_numpy(x)
    if g is not None:
        t = torch.nn.functional.layer_norm(t, (x.shape[1],), torch.from_numpy(g), torch.from_numpy(beta), 1e-5)
    return torch.nn.functional.linear(t, torch.from_numpy(w), torch.from_numpy(b))


def test_layernorm_linear_matches_torch(torch_cpu):
    x, w, b, g, be = _rand(23, 16), _rand(7, 16), _rand(7), _rand(16), _rand(16)
    ref = _torch_ln_linear(x, w, b, g, be).numpy()
    np.testing.assert_allclose(ops.layernorm_linear(x, w, b, ln=(g, be)), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ops.layernorm_linear(x, w, b), _torch_ln_linear(x, w, b).numpy(), rtol=1e-12, atol=1e-12)


def test_layernorm_linear_brute_force():
    x, w, b, g, be = _rand(3, 5), _rand(2, 5), _rand(2), _rand(5), _rand(5)
    y = ops.layernorm_linear(x, w, b, ln=(g, be))
    for r in range(3):
        mu = sum(x[r]) / 5
        var = sum((x[r][k] - mu) ** 2 for k in range(5)) / 5
        xn = [(x[r][k] - mu) / (var + 1e-5) ** 0.5 * g[k] + be[k] for k in range(5)]
        for n in range(2):
            assert y[r, n] == pytest.approx(sum(xn[k] * w[n][k] for k in range(5)) + b[n], rel=1e-12, abs=1e-12)


def test_layernorm_linear_epilogues(torch_cpu):
    x, g, be = _rand(11, 8), _rand(8), _rand(8)
    w, b = _rand(6, 8), _rand(6)
    res = _rand(11, 6)
    np.testing.assert_allclose(ops.layernorm_linear(x, w, b, ln=(g, be), epilogue="residual", residual=res),
                               res + _torch_ln_linear(x, w, b, g, be).numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ops.layernorm_linear(x, w, b, ln=(g, be), epilogue="gelu"),
                               torch.nn.functional.gelu(_torch_ln_linear(x, w, b, g, be)).numpy(),
                               rtol=1e-12, atol=1e-12)
    # SwiGLU transition: gate rows first, up rows second, then the down projection
    F = 5
    wg, bg, wu, bu = _rand(F, 8), _rand(F), _rand(F, 8), _rand(F)
    w2, b2 = _rand(8, F), _rand(8)
    t = torch.nn.functional.layer_norm(torch.from_numpy(x), (8,), torch.from_numpy(g), torch.from_numpy(be), 1e-5)
    h = torch.nn.functional.silu(t @ torch.from_numpy(wg).T + torch.from_numpy(bg)) * (t @ torch.from_numpy(wu).T + torch.from_numpy(bu))
    ref = torch.from_numpy(x) + h @ torch.from_numpy(w2).T + torch.from_numpy(b2)
    got = ops.layernorm_linear(x, np.concatenate([wg, wu]), np.concatenate([bg, bu]), ln=(g, be),
                               epilogue="swiglu_residual", w2=w2, b2=b2)
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_layernorm_linear_packed_equals_padded_rows():
    # rows are independent: packed result = padded result on valid rows (Sec. 3.3)
    L = [3, 1, 4]
    x = _rand(8, 6)
    w, b, g, be = _rand(5, 6), _rand(5), _rand(6), _rand(6)
    padded = np.zeros((3, 4, 6))
    o = layout.single_offsets(L)
    for i, n in enumerate(L):
        padded[i, :n] = x[o[i]:o[i + 1]]
    yp = ops.layernorm_linear(padded.reshape(-1, 6), w, b, ln=(g, be)).reshape(3, 4, 5)
    yv = np.concatenate([yp[i, :n] for i, n in enumerate(L)])
    np.testing.assert_allclose(ops.layernorm_linear(x, w, b, ln=(g, be)), yv, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- reductions
def test_batch_sum_worked_example():
    g = json.load(open(os.path.join(GOLD, "batch_sum_example.json")))
    x = np.array([v for e in g["elements"] for v in e], float)[:, None]
    y = ops.segment_reduce(x, [len(e) for e in g["elements"]], "samples", "sum")
    assert y[:, 0].tolist() == g["sum"]


def test_pair_column_sum_equation():
    # Eq. pair-reduction written out for lengths (2,3), C=1
    L = [2, 3]
    z = np.arange(13, dtype=float)[:, None]
    y = ops.segment_reduce(z, L, "pair_cols", "sum")
    assert y[:, 0].tolist() == [0 + 1, 2 + 3, 4 + 5 + 6, 7 + 8 + 9, 10 + 11 + 12]
    m = ops.segment_reduce(z, L, "pair_cols", "mean")
    np.testing.assert_allclose(m[:, 0], [0.5, 2.5, 5.0, 8.0, 11.0])


def test_mean_of_broadcast_closed_form():
    # mean_b (u_a + v_b) = u_a + mean_b v_b
    L = [4, 1, 6]
    u, v = _rand(11, 3), _rand(11, 3)
    m = ops.segment_reduce(ops.pair_broadcast(u, v, L), L, "pair_cols", "mean")
    o = layout.single_offsets(L)
    expect = np.concatenate([u[o[i]:o[i + 1]] + v[o[i]:o[i + 1]].mean(0) for i in range(3)])
    np.testing.assert_allclose(m, expect, rtol=1e-13, atol=1e-13)


def test_segment_sums_add_to_total_and_empty_samples():
    L = [3, 0, 2]
    x = _rand(5, 4)
    s = ops.segment_reduce(x, L, "samples", "sum")
    np.testing.assert_allclose(s.sum(0), x.sum(0), rtol=1e-13)
    assert np.all(s[1] == 0)
    m = ops.segment_reduce(x, L, "samples", "mean")
    assert np.all(np.isnan(m[1]))
    np.testing.assert_allclose(m[0], x[:3].mean(0))
    z = _rand(13, 2)
    assert ops.segment_reduce(z, L, "pair_cols", "sum").shape == (5, 2)


# ---------------------------------------------------------------- attention
def _attn_inputs(L, H, d, bias=True):
    R = sum(n * n for n in L)
    q, k, v = _rand(R, H * d), _rand(R, H * d), _rand(R, H * d)
    b = _rand(R, H) if bias else None
    return q, k, v, b


def test_attention_zero_queries_average_values():
    L, H, d = [3, 5], 2, 4
    q, k, v, _ = _attn_inputs(L, H, d)
    o = ops.pair_row_attention(np.zeros_like(q), k, v, np.zeros((q.shape[0], H)), L, H, d)
    # softmax of a constant row is uniform: o[r,j] = mean_k v[r,k]
    for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
        V = v[off:off + n * n].reshape(n, n, H * d)
        expect = np.repeat(V.mean(1, keepdims=True), n, axis=1)
        np.testing.assert_allclose(o[off:off + n * n].reshape(n, n, -1), expect, rtol=1e-12, atol=1e-12)


def test_attention_dominant_bias_selects_value():
    L, H, d = [4, 2], 2, 3
    q, k, v, _ = _attn_inputs(L, H, d)
    R = q.shape[0]
    bias = np.zeros((R, H))
    pick = {}
    for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
        for j in range(n):
            for h in range(H):
                kk = (j + 1 + h) % n
                bias[off + j * n + kk, h] = 1e4     # bias[j, kk] dominates row j
                pick[(i, j, h)] = kk
    o = ops.pair_row_attention(q, k, v, bias, L, H, d)
    for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
        for r in range(n):
            for j in range(n):
                for h in range(H):
                    kk = pick[(i, j, h)]
                    np.testing.assert_allclose(o[off + r * n + j, h * d:(h + 1) * d],
                                               v[off + r * n + kk, h * d:(h + 1) * d], rtol=1e-9, atol=1e-9)


def test_attention_equals_masked_padded_sdpa(torch_cpu):
    L, H, d = [5, 2, 4], 2, 4
    q, k, v, b = _attn_inputs(L, H, d)
    o = ops.pair_row_attention(q, k, v, b, L, H, d)
    qp, m = _pad_pairs(q, L)
    kp, _ = _pad_pairs(k, L)
    vp, _ = _pad_pairs(v, L)
    bp, _ = _pad_pairs(b, L)
    B, N = len(L), max(L)
    # [B, r, j, h, d] -> [B*r, h, j, d]
    tq = torch.from_numpy(qp.reshape(B, N, N, H, d)).permute(0, 1, 3, 2, 4).reshape(B * N, H, N, d)
    tk = torch.from_numpy(kp.reshape(B, N, N, H, d)).permute(0, 1, 3, 2, 4).reshape(B * N, H, N, d)
    tv = torch.from_numpy(vp.reshape(B, N, N, H, d)).permute(0, 1, 3, 2, 4).reshape(B * N, H, N, d)
    # additive mask: bias[j,k,h] on valid keys, -inf on padded keys
    keymask = np.zeros((B, N), bool)
    for i, n in enumerate(L):
        keymask[i, :n] = True
    add = np.where(keymask[:, None, None, :], bp.transpose(0, 3, 1, 2), -np.inf)   # [B, h, j, k]
    add = np.where(keymask[:, None, :, None], add, 0.0)                               # padded queries: harmless
    tadd = torch.from_numpy(np.repeat(add[:, None], N, axis=1).reshape(B * N, H, N, N))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=tadd)
    ref = ref.reshape(B, N, H, N, d).permute(0, 1, 3, 2, 4).reshape(B, N, N, H * d).numpy()
    np.testing.assert_allclose(o, _unpad_pairs(ref, L), rtol=1e-11, atol=1e-11)


def test_attention_axis1_is_transposed_axis0():
    L, H, d = [3, 4], 2, 2
    q, k, v, b = _attn_inputs(L, H, d)

    def T(x):
        out = np.empty_like(x)
        for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
            out[off:off + n * n] = x[off:off + n * n].reshape(n, n, -1).transpose(1, 0, 2).reshape(n * n, -1)
        return out

    o1 = ops.pair_row_attention(q, k, v, b, L, H, d, axis=1)
    o0 = ops.pair_row_attention(T(q), T(k), T(v), T(b), L, H, d, axis=0)
    np.testing.assert_allclose(o1, T(o0), rtol=1e-13, atol=1e-13)
    assert not np.allclose(o1, ops.pair_row_attention(q, k, v, b, L, H, d, axis=0))


def test_attention_brute_force():
    L, H, d = [3, 2], 2, 2
    q, k, v, b = _attn_inputs(L, H, d)
    o = ops.pair_row_attention(q, k, v, b, L, H, d, scale=0.7)
    for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
        cell = lambda x, y: off + x * n + y   # noqa: E731
        for r in range(n):
            for j in range(n):
                for h in range(H):
                    sl = slice(h * d, (h + 1) * d)
                    logits = [0.7 * sum(q[cell(r, j), sl] * k[cell(r, kk), sl]) + b[cell(j, kk), h] for kk in range(n)]
                    mx = max(logits)
                    w = [np.exp(t - mx) for t in logits]
                    acc = sum(w[kk] * v[cell(r, kk), sl] for kk in range(n)) / sum(w)
                    np.testing.assert_allclose(o[cell(r, j), sl], acc, rtol=1e-12, atol=1e-12)


def test_attention_1d_matches_masked_padded_sdpa(torch_cpu):
    L, H, d = [4, 1, 6], 3, 4
    T = sum(L)
    q, k, v = _rand(T, H * d), _rand(T, H * d), _rand(T, H * d)
    o = ops.attention_1d(q, k, v, L, H, d)
    B, N = len(L), max(L)
    pad = lambda x: np.stack([np.pad(x[s:e], ((0, N - (e - s)), (0, 0))) for s, e in zip(layout.single_offsets(L)[:-1], layout.single_offsets(L)[1:])])  # noqa: E731
    t = lambda x: torch.from_numpy(pad(x).reshape(B, N, H, d)).transpose(1, 2)  # noqa: E731
    mask = torch.from_numpy(np.array([[kk < n for kk in range(N)] for n in L]))[:, None, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=mask)
    ref = ref.transpose(1, 2).reshape(B, N, H * d).numpy()
    np.testing.assert_allclose(o, np.concatenate([ref[i, :n] for i, n in enumerate(L)]), rtol=1e-12, atol=1e-12)


# ------------------------------------------------- single attention, pair bias
def _single_attn_inputs(L, H, d):
    T, R = sum(L), sum(n * n for n in L)
    return _rand(T, H * d), _rand(T, H * d), _rand(T, H * d), _rand(R, H)


def test_single_attention_zero_queries_average_values():
    L, H, d = [3, 0, 5], 2, 4
    q, k, v, _ = _single_attn_inputs(L, H, d)
    o = ops.single_attention_pair_bias(np.zeros_like(q), k, v, np.zeros((sum(n * n for n in L), H)), L, H, d)
    for s, e in zip(layout.single_offsets(L)[:-1], layout.single_offsets(L)[1:]):
        if e > s:
            np.testing.assert_allclose(o[s:e], np.repeat(v[s:e].mean(0, keepdims=True), e - s, axis=0), rtol=1e-12, atol=1e-12)


def test_single_attention_dominant_bias_selects_value():
    L, H, d = [4, 2, 3], 2, 3
    q, k, v, _ = _single_attn_inputs(L, H, d)
    bias = np.zeros((sum(n * n for n in L), H))
    pick = {}
    for n, po, so in zip(L, layout.pair_offsets(L), layout.single_offsets(L)):
        for t in range(n):
            for h in range(H):
                kk = (t + 1 + h) % n
                bias[po + t * n + kk, h] = 1e4          # bias[t, kk] dominates query t
                pick[(so, t, h)] = kk
    o = ops.single_attention_pair_bias(q, k, v, bias, L, H, d)
    for (so, t, h), kk in pick.items():
        np.testing.assert_allclose(o[so + t, h * d:(h + 1) * d], v[so + kk, h * d:(h + 1) * d], rtol=1e-9, atol=1e-9)


def test_single_attention_equals_masked_padded_sdpa(torch_cpu):
    L, H, d = [5, 1, 3], 3, 4
    q, k, v, b = _single_attn_inputs(L, H, d)
    o = ops.single_attention_pair_bias(q, k, v, b, L, H, d)
    B, N = len(L), max(L)
    so = layout.single_offsets(L)
    pad = lambda x: np.stack([np.pad(x[s:e], ((0, N - (e - s)), (0, 0))) for s, e in zip(so[:-1], so[1:])])  # noqa: E731
    t = lambda x: torch.from_numpy(pad(x).reshape(B, N, H, d)).transpose(1, 2)  # noqa: E731
    bp, _ = _pad_pairs(b, L)                                           # [B, N, N, H]
    keymask = np.array([[kk < n for kk in range(N)] for n in L])
    add = np.where(keymask[:, None, None, :], bp.transpose(0, 3, 1, 2), -np.inf)
    add = np.where(keymask[:, None, :, None], add, 0.0)
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=torch.from_numpy(add))
    ref = ref.transpose(1, 2).reshape(B, N, H * d).numpy()
    np.testing.assert_allclose(o, np.concatenate([ref[i, :n] for i, n in enumerate(L)]), rtol=1e-11, atol=1e-11)


def test_single_attention_without_bias_is_masked_padded_sdpa(torch_cpu):
    """bias=None: plain per-sample self-attention, i.e. padded SDPA with the
    padded keys masked (no pair term)."""
    L, H, d = [4, 1, 6, 0], 2, 3
    q, k, v, _ = _single_attn_inputs(L, H, d)
    o = ops.single_attention_pair_bias(q, k, v, None, L, H, d)
    B, N = len(L), max(L)
    so = layout.single_offsets(L)
    pad = lambda x: np.stack([np.pad(x[s:e], ((0, N - (e - s)), (0, 0))) for s, e in zip(so[:-1], so[1:])])  # noqa: E731
    t = lambda x: torch.from_numpy(pad(x).reshape(B, N, H, d)).transpose(1, 2)  # noqa: E731
    keymask = np.array([[kk < n for kk in range(N)] for n in L])
    add = np.where(keymask[:, None, None, :], 0.0, -np.inf)
    add = np.where(keymask[:, None, :, None], add, 0.0)
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=torch.from_numpy(add))
    ref = ref.transpose(1, 2).reshape(B, N, H * d).numpy()
    np.testing.assert_allclose(o, np.concatenate([ref[i, :n] for i, n in enumerate(L)]), rtol=1e-11, atol=1e-11)


def test_single_attention_brute_force():
    L, H, d = [3, 2], 2, 2
    q, k, v, b = _single_attn_inputs(L, H, d)
    o = ops.single_attention_pair_bias(q, k, v, b, L, H, d, scale=0.7)
    for n, po, so in zip(L, layout.pair_offsets(L), layout.single_offsets(L)):
        for t in range(n):
            for h in range(H):
                sl = slice(h * d, (h + 1) * d)
                logits = [0.7 * sum(q[so + t, sl] * k[so + kk, sl]) + b[po + t * n + kk, h] for kk in range(n)]
                mx = max(logits)
                w = [np.exp(x - mx) for x in logits]
                acc = sum(w[kk] * v[so + kk, sl] for kk in range(n)) / sum(w)
                np.testing.assert_allclose(o[so + t, sl], acc, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- triangle
def test_triangle_ones_gives_row_sums():
    L, C = [4, 2, 3], 3
    R = sum(n * n for n in L)
    a = _rand(R, C)
    t = ops.triangle_mul(a, np.ones((R, C)), L, "outgoing")
    rs = ops.segment_reduce(a, L, "pair_cols", "sum")          # sum_k a[x,k]
    for (i, n), off, eo in zip(enumerate(L), layout.pair_offsets(L), layout.single_offsets(L)):
        T = t[off:off + n * n].reshape(n, n, C)
        np.testing.assert_allclose(T, np.repeat(rs[eo:eo + n][:, None], n, axis=1), rtol=1e-12, atol=1e-12)


def test_triangle_symmetric_when_a_equals_b():
    L, C = [5, 3], 2
    R = sum(n * n for n in L)
    a = _rand(R, C)
    for direction in ("outgoing", "incoming"):
        t = ops.triangle_mul(a, a, L, direction)
        for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
            T = t[off:off + n * n].reshape(n, n, C)
            np.testing.assert_allclose(T, T.transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_triangle_incoming_is_outgoing_of_transposes():
    L, C = [3, 4], 2
    R = sum(n * n for n in L)
    a, b = _rand(R, C), _rand(R, C)

    def T(x):
        out = np.empty_like(x)
        for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
            out[off:off + n * n] = x[off:off + n * n].reshape(n, n, -1).transpose(1, 0, 2).reshape(n * n, -1)
        return out

    np.testing.assert_allclose(ops.triangle_mul(a, b, L, "incoming"),
                               ops.triangle_mul(T(a), T(b), L, "outgoing"), rtol=1e-13, atol=1e-13)
    assert not np.allclose(ops.triangle_mul(a, b, L, "incoming"), ops.triangle_mul(a, b, L, "outgoing"))


def test_triangle_masked_padded_and_brute_force():
    L, C = [4, 1, 3], 3
    R = sum(n * n for n in L)
    a, b = _rand(R, C), _rand(R, C)
    ap, _ = _pad_pairs(a, L)          # padded cells are zero, so they add nothing
    bp, _ = _pad_pairs(b, L)
    out_ref = _unpad_pairs(np.einsum("bxkc,bykc->bxyc", ap, bp), L)
    in_ref = _unpad_pairs(np.einsum("bkxc,bkyc->bxyc", ap, bp), L)
    np.testing.assert_allclose(ops.triangle_mul(a, b, L, "outgoing"), out_ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ops.triangle_mul(a, b, L, "incoming"), in_ref, rtol=1e-12, atol=1e-12)
    t = ops.triangle_mul(a, b, L, "outgoing")
    for (i, n), off in zip(enumerate(L), layout.pair_offsets(L)):
        for x in range(n):
            for y in range(n):
                for c in range(C):
                    s = sum(a[off + x * n + kk, c] * b[off + y * n + kk, c] for kk in range(n))
                    assert t[off + x * n + y, c] == pytest.approx(s, rel=1e-12, abs=1e-12)


def test_pair_row_sum_is_the_column_sum_of_the_transposes():
    """Sum over the first pair axis: for lengths (2, 3) and cells numbered in
    packed order, sample 0 gives [0+2, 1+3] and sample 1 gives the column sums
    of [[4,5,6],[7,8,9],[10,11,12]]; in general it equals the Eq. pair-reduction
    of each sample's transpose."""
    x = np.arange(13, dtype=np.float64)[:, None]
    y = ops.segment_reduce(x, [2, 3], "pair_rows", "sum")
    assert y[:, 0].tolist() == [2, 4, 21, 24, 27]
    L, C = [4, 0, 3, 1], 3
    x = np.random.default_rng(3).standard_normal((sum(n * n for n in L), C))
    t = np.concatenate([b.transpose(1, 0, 2).reshape(-1, C)
                        for b in layout.unpack(x, layout.pair_offsets(L), [(n, n) for n in L])])
    for op in ("sum", "mean"):
        np.testing.assert_allclose(ops.segment_reduce(x, L, "pair_rows", op), ops.segment_reduce(t, L, "pair_cols", op),
                                   rtol=1e-13, atol=1e-13)


def test_rectangular_broadcast_and_column_mean_worked_example():
    """Rows (2, 1) and columns (3, 2): sample 0 holds u0+v0 .. u1+v2 in row-major
    cell order (o = [0, 6, 8]), sample 1 holds u2+v3, u2+v4; the column mean
    of a pair row divides by its M_i (Eq. pair-reduction, rectangular variant)."""
    u = np.array([[1.0], [2.0], [3.0]])
    v = np.array([[10.0], [20.0], [30.0], [40.0], [50.0]])
    z = ops.pair_broadcast(u, v, [2, 1], cols=[3, 2])
    assert z[:, 0].tolist() == [11, 21, 31, 12, 22, 32, 43, 53]
    assert layout.rect_pair_offsets([2, 1], [3, 2]).tolist() == [0, 6, 8]
    m = ops.segment_reduce(z, [2, 1], "pair_cols", "mean", cols=[3, 2])
    assert m[:, 0].tolist() == [21.0, 22.0, 48.0]
    r = ops.segment_reduce(z, [2, 1], "pair_rows", "sum", cols=[3, 2])
    assert r[:, 0].tolist() == [23.0, 43.0, 63.0, 43.0, 53.0]
    # square pairs are the special case cols = lengths
    L = [3, 0, 2]
    uu = np.random.default_rng(4).standard_normal((5, 2))
    np.testing.assert_array_equal(ops.pair_broadcast(uu, uu, L, cols=L), ops.pair_broadcast(uu, uu, L))


def test_weighted_square_loss_is_its_definition():
    x = np.arange(10.0).reshape(5, 2)
    loss, g = ops.weighted_square_loss(x, [2, 3], [1.0, 2.0], 0.5)
    assert loss.tolist() == [0.5 * (0 + 1 + 4 + 9), 0.5 * 2.0 * (16 + 25 + 36 + 49 + 64 + 81)]
    np.testing.assert_array_equal(g, np.concatenate([x[:2], 2.0 * x[2:]]))


def test_rectangular_mean_of_an_empty_group_is_nan():
    """A pair row with no columns (M_i = 0) has an empty column mean: NaN, the
    dense mean of an empty array; its sum is 0."""
    x = np.ones((2, 1))
    m = ops.segment_reduce(x, [2, 3], "pair_cols", "mean", cols=[1, 0])
    assert m[:2, 0].tolist() == [1.0, 1.0] and np.all(np.isnan(m[2:]))
    assert ops.segment_reduce(x, [2, 3], "pair_cols", "sum", cols=[1, 0])[2:, 0].tolist() == [0.0, 0.0, 0.0]


def test_cross_attention_equals_masked_padded_sdpa(torch_cpu):
    """Cross-attention with different query and key lengths per sample equals
    padded SDPA with the padded keys masked, on the valid queries; the
    self-attention case kv_lengths = lengths is attention_1d itself; a sample
    with queries but no keys gives 0."""
    Lq, Lk, H, d = [3, 5, 1, 2], [4, 1, 6, 0], 2, 3
    rng = np.random.default_rng(12)
    q = rng.standard_normal((sum(Lq), H * d))
    k, v = rng.standard_normal((sum(Lk), H * d)), rng.standard_normal((sum(Lk), H * d))
    o = ops.attention_1d(q, k, v, Lq, H, d, kv_lengths=Lk)
    B, Nq, Nk = len(Lq), max(Lq), max(Lk)
    qo, ko = layout.single_offsets(Lq), layout.single_offsets(Lk)

    def pad(x, off, n_max):
        return torch.from_numpy(np.stack([np.pad(x[a:b], ((0, n_max - (b - a)), (0, 0)))
                                          for a, b in zip(off[:-1], off[1:])]).reshape(B, n_max, H, d)).transpose(1, 2)
    mask = torch.from_numpy(np.array([[kk < m for kk in range(Nk)] for m in Lk]))[:, None, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(pad(q, qo, Nq), pad(k, ko, Nk), pad(v, ko, Nk),
                                                           attn_mask=mask.expand(B, H, Nq, Nk))
    ref = ref.transpose(1, 2).reshape(B, Nq, H * d).numpy()
    for i, n in enumerate(Lq):
        want = ref[i, :n] if Lk[i] else np.zeros((n, H * d))
        np.testing.assert_allclose(o[qo[i]:qo[i + 1]], want, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(ops.attention_1d(q, q, q, Lq, H, d, kv_lengths=Lq), ops.attention_1d(q, q, q, Lq, H, d),
                               rtol=0, atol=0)
