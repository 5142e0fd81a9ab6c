"""Per-kernel parity of the HIP path (through the C ABI) against the CPU oracle
on identical seeded inputs.  Shapes span several tiles, ragged tails, empty
and length-1 samples."""
import numpy as np
import pytest

from oracle import ops as O
from paper_2609_30379_amd import synth
from tests.gpu_util import check, dev, host, pair_tiled, untile_pair

pytestmark = pytest.mark.gpu

LENGTHS = {
    "tiny": [15, 12, 10, 7],
    "ragged": [5, 0, 1, 37, 64, 3, 70],
    "one": [1],
}


@pytest.fixture(scope="module")
def B():
    from paper_2609_30379_amd import binding
    binding.load()
    return binding


def _layout(B, L):
    return B.NestedLayout(L)


def _n(seed, name, shape, scale=1.0, dtype="bf16"):
    return synth.normal(seed, name, shape, scale, dtype)


# ------------------------------------------------------------------ broadcast
@pytest.mark.parametrize("lname", list(LENGTHS))
@pytest.mark.parametrize("dtype,C", [("bf16", 128), ("bf16", 64), ("f32", 16)])
@pytest.mark.parametrize("accumulate", [False, True])
def test_pair_broadcast(B, lname, dtype, C, accumulate):
    L = LENGTHS[lname]
    lay = _layout(B, L)
    S, R = sum(L), sum(n * n for n in L)
    uv = _n(1, "uv", (S, 2 * C), 0.6, dtype)
    z0 = _n(2, "z0", (R, C), 0.6, dtype)
    uvd = dev(uv, dtype)
    z = dev(z0, dtype)
    B.nt_pair_broadcast(lay, uvd[:, :C], uvd[:, C:], z, accumulate=accumulate)
    ref = O.pair_broadcast(uv[:, :C], uv[:, C:], L, z_in=z0 if accumulate else None)
    check(host(z), ref, dtype, f"broadcast {lname} {dtype} C={C} acc={accumulate}")


def test_pair_broadcast_full_size(B):
    w = synth.WORKLOADS["pair_b8_n208_224_bf16"]
    L = synth.lengths_for(w).tolist()
    lay = _layout(B, L)
    S, R, C = sum(L), sum(n * n for n in L), w.c_z
    uv = _n(3, "uv", (S, 2 * C), 0.5)
    uvd = dev(uv, "bf16")
    import torch
    z = torch.empty((R, C), dtype=torch.bfloat16, device="cuda")
    B.nt_pair_broadcast(lay, uvd[:, :C], uvd[:, C:], z)
    check(host(z), O.pair_broadcast(uv[:, :C], uv[:, C:], L), "bf16", "broadcast full size")


# ------------------------------------------------------------------ reduce
@pytest.mark.parametrize("lname", list(LENGTHS))
@pytest.mark.parametrize("dtype,C", [("bf16", 128), ("bf16", 768), ("f32", 16), ("f32", 36)])
@pytest.mark.parametrize("level", ["pairs", "singles"])
@pytest.mark.parametrize("op", ["sum", "mean"])
def test_segment_reduce(B, lname, dtype, C, level, op):
    import torch
    L = LENGTHS[lname]
    lay = _layout(B, L)
    rows = sum(n * n for n in L) if level == "pairs" else sum(L)
    out_rows = sum(L) if level == "pairs" else len(L)
    x = _n(4, "x", (rows, C), 0.7, dtype)
    y = torch.full((out_rows, C), 123.0, dtype=torch.float32, device="cuda")
    B.nt_segment_reduce(lay, level, op, dev(x, dtype), y)
    ref = O.segment_reduce(x, L, "pair_cols" if level == "pairs" else "samples", op)
    check(host(y), ref, "f32", f"reduce {lname} {level} {op} {dtype}", equal_nan=True)


def test_segment_reduce_empty_sample_mean_is_nan(B):
    import torch
    lay = _layout(B, [3, 0, 2])
    x = dev(np.ones((5, 8)), "bf16")
    y = torch.zeros((3, 8), dtype=torch.float32, device="cuda")
    B.nt_segment_reduce(lay, "singles", "mean", x, y)
    out = host(y)
    assert np.all(out[0] == 1.0) and np.all(np.isnan(out[1])) and np.all(out[2] == 1.0)
    B.nt_segment_reduce(lay, "singles", "sum", x, y)
    assert np.all(host(y)[1] == 0.0)


# ------------------------------------------------------------------ LN + Linear
LIN_CASES = [
    # rows, K, N, ln, epilogue, x dtype, dtype, n_tail
    (1000, 128, 128, True, "none", "bf16", "bf16", 0),
    (777, 128, 388, True, "none", "bf16", "bf16", 4),
    (500, 128, 176, True, "none", "bf16", "bf16", 48),      # tail of 3 column tiles: not the wave kernel
    (333, 64, 512, True, "gelu", "bf16", "bf16", 0),        # wave kernel, four column groups
    (95, 128, 128, True, "residual", "bf16", "bf16", 0),    # wave kernel, residual, last tile of 15 rows
    (300, 384, 256, False, "none", "bf16", "bf16", 0),
    (600, 768, 2304, True, "none", "bf16", "bf16", 0),       # large-K path (LayerNorm rows in the workspace)
    (600, 768, 3072, True, "gelu", "bf16", "bf16", 0),
    (600, 3072, 768, False, "residual", "bf16", "bf16", 0),  # no LayerNorm, <= 8192 rows: small-row kernel
    (8500, 3072, 768, False, "residual", "bf16", "bf16", 0), # no LayerNorm, > 8192 rows: large-K path
    (200, 416, 136, True, "gelu", "bf16", "bf16", 0),        # large-K path: 13 k-steps, part of a channel tile
    (257, 1024, 520, True, "residual", "bf16", "bf16", 0),   # large-K path: one row past a row tile
    (1000, 256, 256, True, "none", "bf16", "bf16", 0),       # K = 256 without SwiGLU: row-tile kernel
    (9000, 256, 128, False, "gelu", "bf16", "bf16", 0),      # K = 256, no LayerNorm, > 8192 rows: row-tile kernel
    (700, 128, 600, True, "none", "bf16", "bf16", 0),        # K = 128, > 512 outputs: row-tile kernel
    (333, 64, 520, True, "residual", "bf16", "bf16", 0),     # K = 64, > 512 outputs with a residual: row-tile kernel
    (300, 128, 384, False, "residual", "f32", "bf16", 0),
    (129, 136, 40, True, "residual", "bf16", "bf16", 0),
    (100, 16, 50, True, "none", "f32", "f32", 2),
    (100, 32, 32, False, "residual", "f32", "f32", 0),
    (100, 16, 16, True, "gelu", "f32", "f32", 0),
]


@pytest.mark.parametrize("R,K,N,ln,epi,xdt,dtype,n_tail", LIN_CASES)
def test_layernorm_linear(B, R, K, N, ln, epi, xdt, dtype, n_tail):
    import torch
    x = _n(5, "x", (R, K), 0.5, xdt)
    w = _n(6, "w", (N, K), 0.5 / np.sqrt(K), dtype)
    b = _n(7, "b", (N,), 0.1, "f32")
    g = _n(8, "g", (K,), 0.1, "f32") + 1.0
    be = _n(9, "be", (K,), 0.1, "f32")
    res = _n(10, "res", (R, N - n_tail), 0.5, dtype) if epi == "residual" else None
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    y = torch.full((R, N - n_tail), float("nan"), dtype=td, device="cuda")
    yt = torch.full((max(n_tail, 1), R + 8), float("nan"), dtype=td, device="cuda") if n_tail else None
    B.nt_layernorm_linear(dev(x, xdt), dev(w, dtype), dev(b, "f32"), y,
                          ln=(dev(g, "f32"), dev(be, "f32")) if ln else None, epilogue=epi,
                          residual=dev(res, dtype) if res is not None else None, n_tail=n_tail, y_tail=yt)
    ref = O.layernorm_linear(x, w, b, ln=(g, be) if ln else None,
                             epilogue=epi if epi != "residual" else "none")
    main = ref[:, :N - n_tail] + (res if res is not None else 0.0)
    check(host(y), main, dtype, f"linear main {R}x{K}->{N} {epi}")
    if n_tail:
        check(host(yt)[:, :R].T, ref[:, N - n_tail:], dtype, "linear tail")


GATED_LIN_CASES = [
    # rows, K, N, ln, x dtype, dtype: the output of the gated triangle update
    (1000, 128, 128, True, "bf16", "bf16"),     # wave kernel
    (777, 64, 64, True, "bf16", "bf16"),        # wave kernel, K = 64, last tile of 9 rows
    (5000, 128, 128, False, "bf16", "bf16"),    # wave kernel without LayerNorm
    (300, 136, 40, True, "bf16", "bf16"),       # generic tile kernel
    (129, 128, 256, True, "bf16", "bf16"),      # more than 128 outputs: generic tile kernel
    (100, 16, 16, True, "f32", "f32"),
]


@pytest.mark.parametrize("R,K,N,ln,xdt,dtype", GATED_LIN_CASES)
def test_layernorm_linear_gated_residual(B, R, K, N, ln, xdt, dtype):
    """y = residual + sigmoid(gate) * (LN(x) W^T + b); the gate and the
    residual are column slices of wider buffers."""
    import torch
    x = _n(40, "x", (R, K), 0.5, xdt)
    w = _n(41, "w", (N, K), 1.0 / np.sqrt(K), dtype)
    b = _n(42, "b", (N,), 0.1, "f32")
    g = _n(43, "g", (K,), 0.1, "f32") + 1.0
    be = _n(44, "be", (K,), 0.1, "f32")
    wide = _n(45, "gate_res", (R, 2 * N + 8), 0.5, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    wd = dev(wide, dtype)
    gate, res = wd[:, :N], wd[:, N + 8:]
    y = torch.full((R, N), float("nan"), dtype=td, device="cuda")
    B.nt_layernorm_linear(dev(x, xdt), dev(w, dtype), dev(b, "f32"), y,
                          ln=(dev(g, "f32"), dev(be, "f32")) if ln else None, epilogue="gated_residual",
                          residual=res, gate=gate)
    ref = O.layernorm_linear(x, w, b, ln=(g, be) if ln else None, epilogue="gated_residual",
                             residual=wide[:, N + 8:], gate=wide[:, :N])
    check(host(y), ref, dtype, f"linear gated residual {R}x{K}->{N} ln={ln}")


@pytest.mark.parametrize("lname,C,N,epi", [("ragged", 128, 128, "none"), ("tiny", 64, 64, "none"),
                                           ("ragged", 64, 96, "gelu"), ("one", 128, 128, "none"),
                                           ("small_mix", 128, 256, "none"), ("wide", 128, 128, "none")])
def test_layernorm_linear_broadcast_rows(B, lname, C, N, epi):
    """LN+Linear over the pair broadcast of u and v, built as the rows are read:
    equals the broadcast (stored in bf16) followed by LN+Linear, and the
    plain two-call path bit for bit."""
    import torch
    L = {"small_mix": [1, 2, 3, 17, 0, 5, 16, 15, 33], "wide": [230, 7, 300, 1, 64]}.get(lname) or LENGTHS[lname]
    lay = _layout(B, L)
    S, R = sum(L), sum(n * n for n in L)
    uv = _n(31, "uv", (S, 2 * C), 0.6, "bf16")
    w = _n(32, "w", (N, C), 0.5 / np.sqrt(C), "bf16")
    b = _n(33, "b", (N,), 0.1, "f32")
    g, be = _n(34, "g", (C,), 0.1, "f32") + 1, _n(35, "be", (C,), 0.1, "f32")
    uvd = dev(uv, "bf16")
    wd, bd, lnd = dev(w, "bf16"), dev(b, "f32"), (dev(g, "f32"), dev(be, "f32"))
    y = torch.full((R, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.nt_layernorm_linear(None, wd, bd, y, ln=lnd, epilogue=epi, layout=lay, level="pairs",
                          bcast=(uvd[:, :C], uvd[:, C:]))
    from oracle.numerics import round_bf16
    zb = round_bf16(O.pair_broadcast(uv[:, :C], uv[:, C:], L))
    ref = O.layernorm_linear(zb, w, b, ln=(g, be), epilogue=epi)
    check(host(y), ref, "bf16", f"broadcast rows {lname} C={C} N={N} {epi}")
    z = torch.empty((R, C), dtype=torch.bfloat16, device="cuda")
    B.nt_pair_broadcast(lay, uvd[:, :C], uvd[:, C:], z)
    y2 = torch.full((R, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.nt_layernorm_linear(z, wd, bd, y2, ln=lnd, epilogue=epi, layout=lay, level="pairs")
    torch.cuda.synchronize()
    assert torch.equal(y, y2), "broadcast rows differ from broadcast + LN+Linear"


@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("dtype,C", [("bf16", 64), ("f32", 16)])
def test_layernorm_linear_pair_tiled_tail(B, transposed, dtype, C):
    import torch
    L = LENGTHS["ragged"]
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    x = _n(11, "x", (R, C), 0.5, dtype)
    w = _n(12, "w", (2 * C, C), 0.5 / np.sqrt(C), dtype)
    b = _n(13, "b", (2 * C,), 0.1, "f32")
    g, be = _n(14, "g", (C,), 0.1, "f32") + 1, _n(15, "be", (C,), 0.1, "f32")
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    ld = (lay.sum_pad + 7) // 8 * 8
    yt = torch.full((2 * C, ld), float("nan"), dtype=td, device="cuda")
    B.nt_layernorm_linear(dev(x, dtype), dev(w, dtype), dev(b, "f32"), None, ln=(dev(g, "f32"), dev(be, "f32")),
                          n_tail=2 * C, y_tail=yt, tail_layout="pair_tiled_t" if transposed else "pair_tiled",
                          layout=lay, level="pairs", c_out=2 * C)
    ref = O.layernorm_linear(x, w, b, ln=(g, be))
    check(untile_pair(host(yt), L, transposed), ref, dtype, "pair-tiled tail")


@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("lname", ["ragged", "tiny", "one"])
def test_layernorm_linear_sigmoid_glu_pair_tiled(B, transposed, lname):
    """Gated operands sigmoid(a_g) a_p | sigmoid(b_g) b_p of [a_p; a_g; b_p; b_g]
    rows written straight into pair-tiled planes (C = 128), and contracted by
    the gated triangle call on those planes."""
    import torch
    from oracle import blocks as OB
    from oracle.numerics import store
    L, C = LENGTHS[lname], 128
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    x = _n(50, "x", (R, C), 0.5, "bf16")
    w = _n(51, "w", (4 * C, C), 1.0 / np.sqrt(C), "bf16")
    w[:C] = synth.snap_bf16(0.3 * w[:C])                 # projections a_p, b_p scaled so |t| stays below 8
    w[2 * C:3 * C] = synth.snap_bf16(0.3 * w[2 * C:3 * C])
    b = _n(52, "b", (4 * C,), 0.1, "f32")
    g, be = _n(53, "g", (C,), 0.1, "f32") + 1, _n(54, "be", (C,), 0.1, "f32")
    ld = (lay.sum_pad + 7) // 8 * 8
    yt = torch.full((2 * C, ld), float("nan"), dtype=torch.bfloat16, device="cuda")
    variant = "pair_tiled_t" if transposed else "pair_tiled"
    B.nt_layernorm_linear(dev(x, "bf16"), dev(w, "bf16"), dev(b, "f32"), None, ln=(dev(g, "f32"), dev(be, "f32")),
                          epilogue="sigmoid_glu", hidden=C, n_tail=2 * C, y_tail=yt, tail_layout=variant,
                          layout=lay, level="pairs", c_out=2 * C)
    proj = O.layernorm_linear(x, w, b, ln=(g, be))
    a_ref, b_ref = OB.ref_gated_operands(np.concatenate([proj, np.zeros((R, C))], 1), C)
    got = untile_pair(host(yt), L, transposed)
    check(got, np.concatenate([a_ref, b_ref], 1), "bf16", f"sigmoid GLU pair-tiled {lname} transposed={transposed}")
    t = torch.full((R, C), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.nt_triangle_mul_gated(lay, 1 if transposed else 0, yt[:C], yt[C:], t, operands=variant)
    ref = O.triangle_mul(store(got[:, :C], "bf16"), store(got[:, C:], "bf16"), L,
                         "incoming" if transposed else "outgoing")
    check(host(t), ref, "bf16", f"gated triangle on GLU planes {lname} transposed={transposed}")


@pytest.mark.parametrize("R,K,F,dtype", [(1000, 128, 512, "bf16"), (333, 64, 256, "bf16"), (65, 256, 96, "bf16"),
                                         (100, 16, 64, "f32"),
                                         # several 256-row passes per workgroup, ragged last pass
                                         (140001, 128, 512, "bf16"),
                                         # two hidden chunks; hidden width not a multiple of 64
                                         (1000, 128, 64, "bf16"), (500, 128, 96, "bf16"), (777, 64, 128, "bf16")])
def test_swiglu_transition(B, R, K, F, dtype):
    import torch
    x = _n(16, "x", (R, K), 0.5, dtype)
    w = _n(17, "w", (2 * F, K), 1.0 / np.sqrt(K), dtype)
    b = _n(18, "b", (2 * F,), 0.1, "f32")
    w2 = _n(19, "w2", (K, F), 0.25 / np.sqrt(F), dtype)
    b2 = _n(20, "b2", (K,), 0.1, "f32")
    g, be = _n(21, "g", (K,), 0.1, "f32") + 1, _n(22, "be", (K,), 0.1, "f32")
    xd = dev(x, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    y = torch.full((R, K), float("nan"), dtype=td, device="cuda")
    B.nt_layernorm_linear(xd, dev(w, dtype), dev(b, "f32"), y, ln=(dev(g, "f32"), dev(be, "f32")),
                          epilogue="swiglu_residual", w2=dev(w2, dtype), bias2=dev(b2, "f32"), hidden=F)
    ref = O.layernorm_linear(x, w, b, ln=(g, be), epilogue="swiglu_residual", w2=w2, b2=b2)
    check(host(y), ref, dtype, f"swiglu {R}x{K} F={F}")
    # in place (y aliases x), as the pair block runs it
    B.nt_layernorm_linear(xd, dev(w, dtype), dev(b, "f32"), xd, ln=(dev(g, "f32"), dev(be, "f32")),
                          epilogue="swiglu_residual", w2=dev(w2, dtype), bias2=dev(b2, "f32"), hidden=F)
    check(host(xd), ref, dtype, "swiglu in place")


# ------------------------------------------------------------------ attention
ATT_LENGTHS = [5, 0, 1, 37, 64, 3, 70, 130, 17]


def _head_major(bias_cells):
    return np.ascontiguousarray(bias_cells.T)


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("dtype,H,D,lset", [("bf16", 4, 32, "att"), ("bf16", 2, 64, "att"), ("f32", 2, 8, "tiny"),
                                            ("bf16", 3, 32, "att"), ("bf16", 4, 32, "few"),
                                            ("bf16", 2, 32, "long"), ("bf16", 2, 32, "edge256"),
                                            ("bf16", 2, 32, "mid"), ("bf16", 2, 32, "mid512")])
@pytest.mark.parametrize("bias_layout", ["heads", "cells", None])
def test_pair_attention(B, axis, dtype, H, D, lset, bias_layout):
    import torch
    # head_dim 32: samples up to 256 take the persistent short-row kernel, one
    # workgroup per CU with an equal share of all rows, crossing sample
    # boundaries ("att", also with 3 heads, which do not divide the
    # workgroups of an XCD; "few": fewer rows than workgroups, an empty
    # sample; "edge256": the longest sample, whole key chunks only, one full
    # query block), up to 512 its work-list instance ("mid": a short tail
    # chunk; "mid512": the longest sample, a sample just past 256 and one of
    # length 1); "long" (a sample above 512) and head_dim 64 take the per-row
    # path
    L = {"att": ATT_LENGTHS, "tiny": LENGTHS["tiny"], "long": [530, 7, 64], "edge256": [256, 128, 2, 192, 65],
         "mid": [300, 64, 3], "mid512": [512, 257, 1, 100], "few": [3, 0, 2]}[lset]
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    qkv = _n(23, "qkv", (R, 3 * H * D), 1.0, dtype)
    qkv[:, 2 * H * D:] *= 0.5
    if dtype == "bf16":
        qkv = synth.snap_bf16(qkv)
    bias = _n(24, "bias", (R, H), 1.0, dtype)
    qd = dev(qkv, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    o = torch.full((R, H * D), float("nan"), dtype=td, device="cuda")
    c = H * D
    if bias_layout == "heads":
        bd = dev(_head_major(bias), dtype)
    elif bias_layout == "cells":               # [sum N^2, H] as a column slice of a wider buffer (row stride H + 5)
        wide = np.zeros((R, H + 5))
        wide[:, 2:2 + H] = bias
        bd = dev(wide, dtype)[:, 2:2 + H]
    else:
        bd, bias = None, None
    B.nt_pair_row_attention(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o, bias=bd,
                            bias_layout=bias_layout or "cells")
    first = host(o)
    # a second call over whatever the first left in LDS must give the same bits
    B.nt_pair_row_attention(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o, bias=bd,
                            bias_layout=bias_layout or "cells")
    assert np.array_equal(host(o), first, equal_nan=True), "pair attention is not deterministic"
    ref = O.pair_row_attention(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], bias, L, H, D, axis=axis)
    check(first, ref, dtype, f"pair attention axis {axis} {dtype} {lset} H={H} d={D} bias {bias_layout}")


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("L", [ATT_LENGTHS, [300, 64, 3], [512, 257, 1, 100]], ids=["att", "mid", "mid512"])
def test_pair_attention_masking_bias(B, axis, L):
    """A bias that masks keys with -inf (and with huge finite negatives) on
    valid cells: the masked keys get probability zero exactly as in the
    oracle.  Diagonal cells are never masked, so every query keeps a key."""
    import torch
    H, D = 2, 32
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    qkv = synth.snap_bf16(_n(25, "qkv", (R, 3 * H * D), 1.0, "bf16"))
    bias = _n(26, "bias", (R, H), 1.0, "bf16")
    u = np.random.default_rng(27).random((R, H))
    diag = np.zeros(R, bool)
    for off, n in zip(np.cumsum([0] + [n * n for n in L[:-1]]), L):
        diag[off + np.arange(n) * (n + 1)] = True
    bias[(u < 0.3) & ~diag[:, None]] = -np.inf
    bias[(u > 0.97) & ~diag[:, None]] = -1e35
    c = H * D
    qd = dev(qkv, "bf16")
    o = torch.full((R, c), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.nt_pair_row_attention(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o,
                            bias=dev(_head_major(bias), "bf16"), bias_layout="heads")
    got = host(o)
    assert np.isfinite(got).all()
    ref = O.pair_row_attention(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], bias, L, H, D, axis=axis)
    check(got, ref, "bf16", f"pair attention axis {axis} masking bias {L}")


@pytest.mark.parametrize("axis", [0, 1])
@pytest.mark.parametrize("dtype,H,D,lset", [("bf16", 4, 32, "att"), ("bf16", 2, 32, "mid512"),
                                            ("bf16", 2, 32, "long"), ("bf16", 2, 64, "tiny"),
                                            ("f32", 2, 8, "tiny")])
def test_pair_attention_gated(B, axis, dtype, H, D, lset):
    """o = sigmoid(g) * attention with the gate a column slice of the q|k|v|g
    projection: the persistent and work-list instances of the head_dim 32
    kernel (N <= 256, <= 512), the per-row path (N > 512, head_dim 64) and
    fp32; a second call repeats bit for bit."""
    import torch
    L = {"att": ATT_LENGTHS, "tiny": LENGTHS["tiny"], "long": [530, 7, 64], "mid512": [512, 257, 1, 100]}[lset]
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    c = H * D
    qkvg = _n(46, "qkvg", (R, 4 * c), 1.0, dtype)
    qkvg[:, 2 * c:3 * c] *= 0.5
    if dtype == "bf16":
        qkvg = synth.snap_bf16(qkvg)
    bias = _n(47, "bias", (R, H), 1.0, dtype)
    qd = dev(qkvg, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    o = torch.full((R, c), float("nan"), dtype=td, device="cuda")
    bd = dev(_head_major(bias), dtype)
    call = lambda: B.nt_pair_row_attention(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:3 * c], o,  # noqa: E731
                                           bias=bd, bias_layout="heads", gate=qd[:, 3 * c:])
    call()
    first = host(o)
    call()
    assert np.array_equal(host(o), first, equal_nan=True), "gated pair attention is not deterministic"
    ref = O.pair_row_attention(qkvg[:, :c], qkvg[:, c:2 * c], qkvg[:, 2 * c:3 * c], bias, L, H, D, axis=axis,
                               gate=qkvg[:, 3 * c:])
    check(first, ref, dtype, f"gated pair attention axis {axis} {dtype} {lset} H={H} d={D}")


@pytest.mark.parametrize("H,lset", [(4, "att"), (12, "att"), (12, "mid512"), (4, "one")])
@pytest.mark.parametrize("bias_layout", ["heads", "cells", None])
def test_single_attention_pair_bias(B, H, lset, bias_layout):
    """Axis 3: attention over each sample's tokens with the bias read from the
    pair state (bf16, d = 32), against the oracle; plus its argument errors."""
    import torch
    D = 32
    L = {"att": ATT_LENGTHS, "mid512": [512, 257, 1, 100], "one": [1, 1, 2]}[lset]
    lay = _layout(B, L)
    T, R = sum(L), sum(n * n for n in L)
    qkv = synth.snap_bf16(_n(41, "qkv1", (T, 3 * H * D), 1.0, "bf16"))
    bias = _n(42, "bias1", (R, H), 1.0, "bf16")
    c = H * D
    qd = dev(qkv, "bf16")
    o = torch.full((T, c), float("nan"), dtype=torch.bfloat16, device="cuda")
    if bias_layout == "heads":
        bd = dev(_head_major(bias), "bf16")
    elif bias_layout == "cells":
        bd = dev(bias, "bf16")
    else:
        bd, bias = None, None
    call = lambda: B.nt_pair_row_attention(lay, 3, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o, bias=bd,  # noqa: E731
                                           bias_layout=bias_layout or "cells")
    call()
    first = host(o)
    call()                                       # a second call must give the same bits
    assert np.array_equal(host(o), first, equal_nan=True), "single attention is not deterministic"
    ref = O.single_attention_pair_bias(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], bias, L, H, D)
    check(first, ref, "bf16", f"single attention with pair bias H={H} {lset} bias {bias_layout}")
    with pytest.raises(B.NtError):              # f32 is not supported on axis 3
        of = torch.zeros((T, c), dtype=torch.float32, device="cuda")
        qf = torch.zeros((T, 3 * c), dtype=torch.float32, device="cuda")
        B.nt_pair_row_attention(lay, 3, H, D, qf[:, :c], qf[:, c:2 * c], qf[:, 2 * c:], of)
    with pytest.raises(B.NtError):
        B.nt_pair_row_attention(lay, 4, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o)


@pytest.mark.parametrize("dtype,H,D,L", [("bf16", 3, 64, [1, 5, 64, 65, 130, 512, 0, 200]),
                                         ("bf16", 2, 64, [256, 17, 1, 100, 33, 0]),
                                         ("bf16", 2, 32, [33, 1, 97]),
                                         ("f32", 2, 8, [15, 12, 10, 7, 0, 1])])
def test_attention_1d(B, dtype, H, D, L):
    import torch
    lay = _layout(B, L)
    T = sum(L)
    c = H * D
    qkv = _n(25, "qkv", (T, 3 * c), 1.0, dtype)
    qd = dev(qkv, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    o = torch.full((T, c), float("nan"), dtype=td, device="cuda")
    B.nt_pair_row_attention(lay, 2, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o)
    ref = O.attention_1d(qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], L, H, D)
    check(host(o), ref, dtype, f"1-D attention {dtype}")


CROSS_CASES = [("bf16", 3, 64, [1, 5, 64, 130, 0, 200, 77], [3, 0, 64, 512, 10, 1, 256]),
               ("bf16", 2, 32, [33, 1, 97, 300], [100, 7, 0, 256]),
               ("bf16", 4, 32, [130, 16, 2], [257, 511, 33]),
               ("f32", 2, 8, [15, 12, 10, 7, 0, 1], [3, 20, 0, 7, 5, 1]),
               ("f32", 1, 64, [65, 3], [0, 130])]


@pytest.mark.parametrize("dtype,H,D,Lq,Lk", CROSS_CASES)
def test_cross_attention(B, dtype, H, D, Lq, Lk):
    """Queries and keys ragged differently (the output takes the query
    structure); samples with keys but no queries, queries but no keys (the
    empty sum, 0), up to 512 keys; a second call repeats bit for bit."""
    import torch
    lq, lk = _layout(B, Lq), _layout(B, Lk)
    c = H * D
    q = _n(26, "q", (sum(Lq), c), 1.0, dtype)
    kv = _n(27, "kv", (sum(Lk), 2 * c), 1.0, dtype)
    qd, kvd = dev(q, dtype), dev(kv, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    o = torch.full((sum(Lq), c), float("nan"), dtype=td, device="cuda")
    B.nt_cross_attention(lq, lk, H, D, qd, kvd[:, :c], kvd[:, c:], o)
    ref = O.attention_1d(q, kv[:, :c], kv[:, c:], Lq, H, D, kv_lengths=Lk)
    check(host(o), ref, dtype, f"cross-attention {dtype} H={H} d={D} Lq={Lq} Lk={Lk}")
    o2 = torch.full_like(o, float("nan"))
    B.nt_cross_attention(lq, lk, H, D, qd, kvd[:, :c], kvd[:, c:], o2)
    assert torch.equal(o, o2)


def test_cross_attention_with_equal_lengths_is_self_attention(B):
    """kv layout = q layout gives the bits of the 1-D self-attention call."""
    import torch
    L, H, D = [1, 64, 65, 300, 0, 17], 2, 64
    lay, lay2 = _layout(B, L), _layout(B, L)
    c = H * D
    qkv = dev(_n(28, "qkv", (sum(L), 3 * c)), "bf16")
    o1 = torch.empty((sum(L), c), dtype=torch.bfloat16, device="cuda")
    o2 = torch.empty_like(o1)
    B.nt_pair_row_attention(lay, 2, H, D, qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], o1)
    B.nt_cross_attention(lay, lay2, H, D, qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], o2)
    assert torch.equal(o1, o2)


def test_cross_attention_rejects_mismatched_batches_and_long_keys(B):
    import torch
    H, D = 2, 32
    q = torch.zeros((10, H * D), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((600, 2 * H * D), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros_like(q)
    with pytest.raises(B.NtError) as e:
        B.nt_cross_attention(_layout(B, [4, 6]), _layout(B, [600]), H, D, q, kv[:, :64], kv[:, 64:], o)
    assert e.value.status == B.NT_ERR_LAYOUT_MISMATCH
    with pytest.raises(B.NtError) as e:
        B.nt_cross_attention(_layout(B, [4, 6]), _layout(B, [0, 600]), H, D, q, kv[:, :64], kv[:, 64:], o)
    assert e.value.status == B.NT_ERR_UNSUPPORTED


# ------------------------------------------------------------------ triangle
@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("dtype,C,lname", [("bf16", 64, "ragged"), ("bf16", 32, "tiny"), ("f32", 16, "tiny"),
                                           ("f32", 16, "ragged")])
def test_triangle_pair_tiled(B, direction, dtype, C, lname):
    """Operands already pair-tiled (the plain variant for outgoing, the
    transposed one for incoming), padding filled with NaN."""
    L = LENGTHS[lname]
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    a = _n(26, "a", (R, C), 0.3, dtype)
    b = _n(27, "b", (R, C), 0.3, dtype)
    z0 = _n(28, "z0", (R, C), 0.5, dtype)
    tr = direction == 1
    ld = (lay.sum_pad + 7) // 8 * 8
    ap = dev(pair_tiled(a, L, tr, ld, fill=np.nan), dtype)
    bp = dev(pair_tiled(b, L, tr, ld, fill=np.nan), dtype)
    z = dev(z0, dtype)
    B.nt_triangle_mul(lay, direction, ap, bp, z, operands="pair_tiled_t" if tr else "pair_tiled")
    ref = z0 + O.triangle_mul(a, b, L, "outgoing" if direction == 0 else "incoming")
    check(host(z), ref, dtype, f"triangle pair-tiled dir {direction} {dtype} {lname}")
    # the other variant does not match this direction: rejected before any work
    with pytest.raises(B.NtError):
        B.nt_triangle_mul(lay, direction, ap, bp, z, operands="pair_tiled" if tr else "pair_tiled_t")


TRI_PACKED = [
    ("bf16", 64, [5, 0, 1, 37, 64, 3, 70]),
    ("bf16", 128, [489, 420, 257, 1, 0]),        # the longest pair states of the workloads, full width
    ("bf16", 128, [222, 208, 33]),
    ("f32", 16, [15, 12, 10, 7]),
    ("f32", 12, [5, 0, 1, 37, 3]),
]


@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("dtype,C,L", TRI_PACKED)
def test_triangle_packed(B, direction, dtype, C, L):
    """Operands as packed [sum N^2, C] pair tensors (Eq. packing), the call
    re-tiling them into its workspace; a and b are column slices of one
    [sum N^2, 2C] projection, as a producer writes them."""
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    nmax = max(L)
    ab = _n(29, "ab", (R, 2 * C), float(np.sqrt(0.5 / np.sqrt(nmax))), dtype)    # t = sum_k a b of std ~0.5
    z0 = _n(30, "z0", (R, C), 0.5, dtype)
    abd = dev(ab, dtype)
    z = dev(z0, dtype)
    B.nt_triangle_mul(lay, direction, abd[:, :C], abd[:, C:], z, operands="packed")
    direc = "outgoing" if direction == 0 else "incoming"
    cu = np.concatenate([[0], np.cumsum([n * n for n in L])])
    got = host(z)
    for i, n in enumerate(L):                   # per sample: the oracle on one sample at a time
        if n == 0:
            continue
        sl = slice(int(cu[i]), int(cu[i + 1]))
        ref = z0[sl] + O.triangle_mul(ab[sl, :C], ab[sl, C:], [n], direc)
        check(got[sl], ref, dtype, f"triangle packed dir {direction} {dtype} C={C} sample N={n}")

TRI_GATED = [("bf16", 64, [5, 0, 1, 37, 64, 3, 70], 0.5), ("bf16", 128, [257, 130, 1], 0.35),
             ("f32", 16, [15, 12, 10, 7], 0.5)]


@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("dtype,C,L,gain", TRI_GATED)
def test_triangle_gated(B, direction, dtype, C, L, gain):
    """t = triangle(sigmoid(a_g) a_p, sigmoid(b_g) b_p) from one [a_p|a_g|b_p|b_g]
    projection; t is overwritten (NaN before the call), never read."""
    import torch
    from oracle.numerics import store
    lay = _layout(B, L)
    R = sum(n * n for n in L)
    p4 = _n(48, "p4", (R, 4 * C), 1.0, dtype)
    p4[:, 0:C] *= gain
    p4[:, 2 * C:3 * C] *= gain
    if dtype == "bf16":
        p4 = synth.snap_bf16(p4)
    pd = dev(p4, dtype)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    t = torch.full((R, C), float("nan"), dtype=td, device="cuda")
    B.nt_triangle_mul_gated(lay, direction, pd[:, :2 * C], pd[:, 2 * C:], t)
    a = store(O.gated_operand(p4[:, :C], p4[:, C:2 * C]), dtype)
    b = store(O.gated_operand(p4[:, 2 * C:3 * C], p4[:, 3 * C:]), dtype)
    ref = O.triangle_mul(a, b, L, "outgoing" if direction == 0 else "incoming")
    check(host(t), ref, dtype, f"gated triangle {dtype} C={C} L={L} direction {direction}")

