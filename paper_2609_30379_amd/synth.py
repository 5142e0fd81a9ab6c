"""Seeded synthetic workloads: length vectors, activations and weights.

This module only draws random numbers and describes workload shapes.  It holds
none of the packed-tensor arithmetic, so the GPU path and the CPU oracle can be
fed byte-identical inputs without sharing any of the computation.

Length distributions follow the pair workloads of the paper's evaluation
(square pair regimes of Table "regimes", Appendix C) and a BERT-Base-shaped
token batch (IMDB / BERT, Appendix C, B=64); no dataset is read.  Values are
drawn in float64, converted to float32 and, for bf16 workloads, snapped to the
nearest bf16 value (round to nearest even) so that every input is exactly
representable in the storage type of both sides.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "lengths_for", "tensor_rng", "snap_bf16",
    "pair_block_params", "encoder_layer_params", "normal", "cols_for", "mechanism_params", "mechanism_gains",
]


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: batch geometry, widths and storage dtype."""
    name: str
    kind: str                  # "pair" (pair block / stack) or "tokens"
    batch: int
    dist: tuple                # ("uniform", lo, hi) or ("lognormal", mu, sigma, lo, hi)
    seed: int
    dtype: str                 # "f32" or "bf16"
    c_s: int = 0               # single width
    c_z: int = 0               # pair width
    heads: int = 0
    head_dim: int = 0
    hidden: int = 0            # transition / FFN hidden width
    blocks: int = 1
    transition: bool = True
    tri_incoming: bool = False
    col_attention: bool = False
    single_update: bool = True
    gains: dict = field(default_factory=dict, compare=False, hash=False)
    steps: tuple = ()          # ordered steps of one block (pair workloads)
    s_scale: float = 1.0       # std of the initial single track
    col_dist: tuple = ()       # rectangular pairs: distribution of the column lengths M_i
    s_axis: int = 1            # non-leading layout: static axis S of elements (S, N_i, C), packed (N_i, S, C)


def _pair_gains(n_max: int, blocks: int = 1) -> dict:
    # Gains keep every bf16 tensor that crosses a kernel boundary inside
    # |v| < 8 (pair state std ~0.5-0.6), where one bf16 half-ulp is at most
    # 2^-6 and so inside the 2e-2 bar of a single rounding.
    damp = 1.0 / np.sqrt(blocks)
    return {
        "uv": 0.35 * damp,        # z = u_a + v_b has std ~0.5
        "lin": 0.5,               # LayerNorm+Linear that replaces z
        "qkv": 0.5, "bias": 0.6,  # attention projections
        "o": 0.5 * damp,          # attention output projection (residual)
        # pair states built by broadcasting are rank-structured, so the
        # triangle sum over k is coherent and grows like N: a, b get gain
        # sqrt(0.3 / n_max) to keep t = sum_k a b of order 0.3
        "ab": float(np.sqrt(0.3 / n_max)) * np.sqrt(damp),
        "gu": 1.0, "d": 0.25 * damp,   # SwiGLU transition
        "s": 0.5,                 # single update from the column mean
        "gate": 1.0,              # gate logits of the gated (AlphaFold 3 form) steps
        # gated triangle: t is normalised before use, so a_p, b_p are scaled
        # to give t of order 0.3 (sigmoid gates halve each operand)
        "ab_g": float(np.sqrt(0.3 / n_max)) * 4.0 * np.sqrt(damp),
    }


# Block step sequences: the tiny block (broadcast, LayerNorm+Linear, row
# attention, triangle), the single pair block (plus the SwiGLU transition) and
# the Pairformer-style stack block; every block ends with the column mean back
# to the single track (Eq. running-block, third line).
_TINY = ("bcast", "lin", "att_row", "tri_out", "single")
_BLOCK = ("bcast", "lin", "att_row", "tri_out", "trans", "single")
_STACK = ("bcast", "tri_out", "tri_in", "att_row", "att_col", "trans", "single")
# the same stack with the gated triangle and attention steps of AlphaFold 3
_STACK_GATED = ("bcast", "tri_out_g", "tri_in_g", "att_row_g", "att_col_g", "trans", "single")

def mechanism_gains() -> dict:
    """Gains of the single-pair-single program: pair state std ~0.5, the
    SwiGLU update and the single update of the same order as their inputs."""
    return {"uv": 0.35, "gu": 1.0, "d": 0.25, "g": 0.5}


WORKLOADS = {
    w.name: w for w in [
        Workload("pair_tiny_f32_b4", "pair", 4, ("uniform", 4, 16), 0, "f32",
                 c_s=32, c_z=16, heads=2, head_dim=8, hidden=64,
                 transition=False, gains=_pair_gains(16), steps=_TINY),
        Workload("pair_b8_n208_224_bf16", "pair", 8, ("uniform", 208, 224), 0, "bf16",
                 c_s=384, c_z=128, heads=4, head_dim=32, hidden=512,
                 gains=_pair_gains(224), steps=_BLOCK),
        Workload("pair_b8_n32_512_bf16", "pair", 8, ("uniform", 32, 512), 1, "bf16",
                 c_s=384, c_z=128, heads=4, head_dim=32, hidden=512,
                 gains=_pair_gains(512), steps=_BLOCK),
        Workload("pairformer4_b16_lognormal192_bf16", "pair", 16,
                 ("lognormal", 192.0, 0.6, 16, 768), 0, "bf16",
                 c_s=384, c_z=128, heads=4, head_dim=32, hidden=512, blocks=4,
                 tri_incoming=True, col_attention=True,
                 gains=_pair_gains(768, blocks=4), steps=_STACK),
        Workload("pairformer4_gated_b16_lognormal192_bf16", "pair", 16,
                 ("lognormal", 192.0, 0.6, 16, 768), 0, "bf16",
                 c_s=384, c_z=128, heads=4, head_dim=32, hidden=512, blocks=4,
                 tri_incoming=True, col_attention=True,
                 gains=_pair_gains(768, blocks=4), steps=_STACK_GATED),
        # the measured single-pair-single program (App. A): B=8, C=384,
        # C_p=128, expansion 4; square lengths 66..317, rectangular
        # 66..307 x 66..309 (Table "regimes")
        Workload("mechanism_square_b8_n66_317_bf16", "mechanism", 8, ("uniform", 66, 317), 2, "bf16",
                 c_s=384, c_z=128, hidden=512, gains=mechanism_gains()),
        Workload("mechanism_rect_b8_n66_307_m66_309_bf16", "mechanism", 8, ("uniform", 66, 307), 3, "bf16",
                 c_s=384, c_z=128, hidden=512, gains=mechanism_gains(), col_dist=("uniform", 66, 309)),
        # the non-leading layout of the same program: elements (S=3, N_i, C),
        # lengths 40..182 (Table "regimes")
        Workload("mechanism_nonleading_s3_b8_n40_182_bf16", "mechanism", 8, ("uniform", 40, 182), 4, "bf16",
                 c_s=384, c_z=128, hidden=512, gains=mechanism_gains(), s_axis=3),
        Workload("tokens_b64_lognormal230_bf16", "tokens", 64,
                 ("lognormal", 230.0, 0.5, 16, 512), 0, "bf16",
                 c_s=768, heads=12, head_dim=64, hidden=3072,
                 gains={"qkv": 0.5, "o": 0.5, "ffn1": 0.5, "ffn2": 0.5}),
    ]
}


def _draw(rng, dist, batch):
    if dist[0] == "uniform":
        _, lo, hi = dist
        n = rng.integers(lo, hi, size=batch, endpoint=True)
    elif dist[0] == "lognormal":
        _, mu, sigma, lo, hi = dist
        n = np.clip(np.rint(rng.lognormal(np.log(mu), sigma, size=batch)), lo, hi)
    else:
        raise ValueError(f"unknown length distribution {dist[0]!r}")
    return np.asarray(n, dtype=np.int32)


def lengths_for(w: Workload, seed: int | None = None) -> np.ndarray:
    """Per-sample lengths N_i (int32) of a workload, from its own seed (or the
    given one, for a second ragged axis drawn from the same distribution)."""
    return _draw(np.random.default_rng(w.seed if seed is None else seed), w.dist, w.batch)


def cols_for(w: Workload):
    """Column lengths M_i of a rectangular-pair workload (drawn after the row
    lengths from the same generator), or None for square pairs."""
    if not w.col_dist:
        return None
    rng = np.random.default_rng(w.seed)
    _draw(rng, w.dist, w.batch)
    return _draw(rng, w.col_dist, w.batch)


def tensor_rng(seed: int, name: str) -> np.random.Generator:
    """An independent generator per named tensor, stable across runs."""
    return np.random.default_rng(np.random.SeedSequence([seed, zlib.crc32(name.encode())]))


def snap_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (round to nearest, ties to even), returned as float32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    out = u.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(f), f, out)


def normal(seed: int, name: str, shape, scale: float = 1.0, dtype: str = "f32",
           loc: float = 0.0) -> np.ndarray:
    """loc + scale * N(0,1) draws for one named tensor, stored as float32."""
    x = (loc + scale * tensor_rng(seed, name).standard_normal(shape)).astype(np.float32)
    return snap_bf16(x) if dtype == "bf16" else x


def _linear(seed, name, n_out, n_in, gain, dtype):
    w = normal(seed, name + ".w", (n_out, n_in), gain / np.sqrt(n_in), dtype)
    b = normal(seed, name + ".b", (n_out,), 0.1 * gain)          # fp32 always
    return w, b


def _ln(seed, name, c):
    return (normal(seed, name + ".gamma", (c,), 0.1, loc=1.0),
            normal(seed, name + ".beta", (c,), 0.1))


def pair_block_params(w: Workload, block: int = 0, seed: int | None = None) -> dict:
    """Random-init weights of one pair block (see the block recipe in the
    oracle).  Matrices are [out, in] (y = x W^T + b), stored in the workload
    dtype; biases and LayerNorm affine parameters are float32."""
    seed = w.seed if seed is None else seed
    g, dt, cz, cs, H = w.gains, w.dtype, w.c_z, w.c_s, w.heads
    p = {}
    pre = f"blk{block}."
    p["uv.w"], p["uv.b"] = _linear(seed, pre + "uv", 2 * cz, cs, g["uv"], dt)
    if block == 0:
        p["lin.ln_g"], p["lin.ln_b"] = _ln(seed, pre + "lin", cz)
        p["lin.w"], p["lin.b"] = _linear(seed, pre + "lin", cz, cz, g["lin"], dt)
    gated = any(s.endswith("_g") for s in w.steps)
    attn = [] if gated else ["row"] + (["col"] if w.col_attention else [])
    for a in attn:
        p[f"att_{a}.ln_g"], p[f"att_{a}.ln_b"] = _ln(seed, pre + "att_" + a, cz)
        wq, bq = _linear(seed, pre + f"att_{a}.qkv", 3 * cz, cz, g["qkv"], dt)
        wb, bb = _linear(seed, pre + f"att_{a}.bias", H, cz, g["bias"], dt)
        p[f"att_{a}.w"] = np.concatenate([wq, wb], 0)
        p[f"att_{a}.b"] = np.concatenate([bq, bb], 0)
        p[f"att_{a}.wo"], p[f"att_{a}.bo"] = _linear(seed, pre + f"att_{a}.o", cz, cz, g["o"], dt)
    for key in [s for s in w.steps if s.startswith("att_") and s.endswith("_g")]:
        # [q | k | v | g | bias]: the gate logits before the bias tail
        p[f"{key}.ln_g"], p[f"{key}.ln_b"] = _ln(seed, pre + key, cz)
        parts = [_linear(seed, pre + f"{key}.qkv", 3 * cz, cz, g["qkv"], dt),
                 _linear(seed, pre + f"{key}.gate", cz, cz, g["gate"], dt),
                 _linear(seed, pre + f"{key}.bias", H, cz, g["bias"], dt)]
        p[f"{key}.w"] = np.concatenate([a for a, _ in parts], 0)
        p[f"{key}.b"] = np.concatenate([b for _, b in parts], 0)
        p[f"{key}.wo"], p[f"{key}.bo"] = _linear(seed, pre + f"{key}.o", cz, cz, g["o"], dt)
    for key in [s for s in w.steps if s.startswith("tri_") and s.endswith("_g")]:
        # [a_p | a_g | b_p | b_g | g], then LN(t) and the output projection
        p[f"{key}.ln_g"], p[f"{key}.ln_b"] = _ln(seed, pre + key, cz)
        parts = [_linear(seed, pre + f"{key}.{nm}", cz, cz, g["ab_g"] if nm in ("ap", "bp") else g["gate"], dt)
                 for nm in ("ap", "ag", "bp", "bg", "g")]
        p[f"{key}.w"] = np.concatenate([a for a, _ in parts], 0)
        p[f"{key}.b"] = np.concatenate([b for _, b in parts], 0)
        p[f"{key}.out.ln_g"], p[f"{key}.out.ln_b"] = _ln(seed, pre + key + ".out", cz)
        p[f"{key}.wo"], p[f"{key}.bo"] = _linear(seed, pre + f"{key}.o", cz, cz, g["o"], dt)
    tri = [] if gated else ["out"] + (["in"] if w.tri_incoming else [])
    for t in tri:
        p[f"tri_{t}.ln_g"], p[f"tri_{t}.ln_b"] = _ln(seed, pre + "tri_" + t, cz)
        p[f"tri_{t}.w"], p[f"tri_{t}.b"] = _linear(seed, pre + f"tri_{t}", 2 * cz, cz, g["ab"], dt)
    if w.transition:
        p["trans.ln_g"], p["trans.ln_b"] = _ln(seed, pre + "trans", cz)
        p["trans.w"], p["trans.b"] = _linear(seed, pre + "trans.gu", 2 * w.hidden, cz, g["gu"], dt)
        p["trans.w2"], p["trans.b2"] = _linear(seed, pre + "trans.d", cz, w.hidden, g["d"], dt)
    if w.single_update:
        p["single.w"], p["single.b"] = _linear(seed, pre + "single", cs, cz, g["s"], dt)
    return p


def encoder_layer_params(w: Workload, seed: int | None = None) -> dict:
    """Random-init weights of one pre-LayerNorm encoder layer (token path)."""
    seed = w.seed if seed is None else seed
    g, dt, c = w.gains, w.dtype, w.c_s
    p = {}
    p["ln1_g"], p["ln1_b"] = _ln(seed, "enc.ln1", c)
    p["qkv.w"], p["qkv.b"] = _linear(seed, "enc.qkv", 3 * c, c, g["qkv"], dt)
    p["o.w"], p["o.b"] = _linear(seed, "enc.o", c, c, g["o"], dt)
    p["ln2_g"], p["ln2_b"] = _ln(seed, "enc.ln2", c)
    p["ffn1.w"], p["ffn1.b"] = _linear(seed, "enc.ffn1", w.hidden, c, g["ffn1"], dt)
    p["ffn2.w"], p["ffn2.b"] = _linear(seed, "enc.ffn2", c, w.hidden, g["ffn2"], dt)
    return p


def mechanism_params(w: Workload, seed: int | None = None) -> dict:
    """Random-init weights of the single-pair-single program: u, v (C -> C_p),
    the pre-normalised SwiGLU transition of width C_p with expansion
    hidden / C_p, and g (C_p -> C).  Matrices in the workload dtype, vectors fp32."""
    seed = w.seed if seed is None else seed
    g, dt, C, Cp = w.gains, w.dtype, w.c_s, w.c_z
    p = {}
    p["u.w"], p["u.b"] = _linear(seed, "mech.u", Cp, C, g["uv"], dt)
    p["v.w"], p["v.b"] = _linear(seed, "mech.v", Cp, C, g["uv"], dt)
    p["trans.ln_g"], p["trans.ln_b"] = _ln(seed, "mech.trans", Cp)
    p["trans.w"], p["trans.b"] = _linear(seed, "mech.trans.gu", 2 * w.hidden, Cp, g["gu"], dt)
    p["trans.w2"], p["trans.b2"] = _linear(seed, "mech.trans.d", Cp, w.hidden, g["d"], dt)
    p["g.w"], p["g.b"] = _linear(seed, "mech.g", C, Cp, g["g"], dt)
    return p
