"""Block compositions on the GPU path: every step is one call into libnt.so.

pair block      the single-pair-single block of Eq. running-block, extended with
                the Pairformer-style steps of Sec. 4.3 (row/column attention
                with pair bias, outgoing/incoming triangle update, SwiGLU
                transition), over a packed [sum N_i^2, C] pair state.
encoder layer   a pre-LayerNorm encoder layer on packed [sum N_i, C] tokens
                with segmented attention and a per-sample mean pool.

Workspaces (activation buffers and the ops' scratch) are allocated once per
(layout, dims); a step allocates nothing.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import binding as B

ORDER_BLOCK = ("bcast", "lin", "att_row", "tri_out", "trans", "single")
ORDER_STACK = ("bcast", "tri_out", "tri_in", "att_row", "att_col", "trans", "single")


def _round8(n: int) -> int:
    return (int(n) + 7) // 8 * 8


class OpTimer:
    """Records a pair of events on the current stream around every op of a
    block, to attribute device time per op (used by the benchmark)."""

    def __init__(self):
        self.events = []          # (name, start, end)

    def __call__(self, name):
        return _OpSpan(self, name)

    def summary(self):
        """{op: (launches, median microseconds per launch)} after a device
        synchronisation.  An event span also holds any time the device waits
        for the host to issue the op's launches; the median over launches
        keeps an occasional host stall out of the op's figure."""
        torch.cuda.synchronize()
        acc = {}
        for name, a, b in self.events:
            acc.setdefault(name, []).append(a.elapsed_time(b) * 1e3)
        return {k: (len(v), float(np.median(v))) for k, v in acc.items()}


class _OpSpan:
    def __init__(self, timer, name):
        self.timer, self.name = timer, name

    def __enter__(self):
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)
        self.a.record()

    def __exit__(self, *exc):
        self.b.record()
        self.timer.events.append((self.name, self.a, self.b))


class _NoSpan:
    def __enter__(self):
        return None

    def __exit__(self, *exc):
        return False


_NOSPAN = _NoSpan()
timer = None                      # set to an OpTimer to record per-op events


def _op(name):
    return timer(name) if timer is not None else _NOSPAN


def to_device(params: dict, dtype: str, device="cuda") -> dict:
    """Weights as device tensors: matrices in the storage dtype, vectors in fp32."""
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = {}
    for k, v in params.items():
        t = torch.from_numpy(np.ascontiguousarray(v))
        out[k] = t.to(device=device, dtype=td if t.dim() == 2 else torch.float32).contiguous()
    return out


class PairWorkspace:
    """Device buffers of one pair block for a given layout and widths."""

    def __init__(self, layout: B.NestedLayout, c_s: int, c_z: int, heads: int, dtype: str, device="cuda",
                 gated: bool = False):
        td = torch.bfloat16 if dtype == "bf16" else torch.float32
        R, S = layout.sum_n2, layout.sum_n
        self.td = td
        self.uv = torch.empty((S, 2 * c_z), dtype=td, device=device)
        self.z = [torch.empty((R, c_z), dtype=td, device=device) for _ in range(2)]
        self.qkv = torch.empty((R, 3 * c_z), dtype=td, device=device)
        self.bias = torch.empty((heads, max(_round8(R), 8)), dtype=td, device=device)
        self.o = torch.empty((R, c_z), dtype=td, device=device)
        self.ab = torch.empty((2 * c_z, max(_round8(layout.sum_pad), 8)), dtype=td, device=device)
        self.m = torch.empty((S, c_z), dtype=torch.float32, device=device)
        # op scratch: the attention bias image (both axes) and the
        # transition's weight image, used one op at a time on one stream
        need = max(B.attention_workspace_bytes(layout, ax, heads, c_z // heads, dtype, True) for ax in (0, 1))
        need = max(need, B.layernorm_linear_workspace_bytes(R, c_z, c_z, dtype, epilogue="swiglu_residual",
                                                            hidden=4 * c_z))
        if gated:
            # gated steps: [q|k|v|g] or [a_p|a_g|b_p|b_g] rows, the gate logits
            # of the triangle output and the contraction t; the gated operands
            # are re-tiled into the scratch
            self.p4 = torch.empty((R, 4 * c_z), dtype=td, device=device)
            self.g = torch.empty((R, c_z), dtype=td, device=device)
            self.t = torch.empty((R, c_z), dtype=td, device=device)
            need = max(need, B.triangle_workspace_bytes(layout, c_z, "packed", dtype))
        self.scratch = B.workspace_tensor(need, device)
        self.cur = 0


fuse_broadcast = True             # the pair block fuses broadcast -> LayerNorm+Linear when it can


def fuse_bcast(ws: PairWorkspace, C: int) -> bool:
    return fuse_broadcast and ws.td == torch.bfloat16 and C in (64, 128)


def glu_tiled(ws: PairWorkspace, C: int) -> bool:
    """The gated triangle operands go straight into pair-tiled planes (bf16,
    C = 128); otherwise the projection is stored and gated while re-tiled."""
    return ws.td == torch.bfloat16 and C == 128


def pair_block(layout: B.NestedLayout, s, W: dict, dims: dict, order, ws: PairWorkspace, z=None, tap=None):
    """Runs one pair block.  s ([sum N, C_s]) is updated in place by the
    "single" step; returns the pair state tensor (a workspace buffer, or z).
    tap(op, **outputs), when given, is called after every op with the device
    tensors that op wrote (the per-kernel parity tests read them)."""
    C, H, d = dims["c_z"], dims["heads"], dims["head_dim"]
    tap = tap or (lambda op, **t: None)
    order = list(order)
    k = 0
    while k < len(order):
        step = order[k]
        k += 1
        if step == "bcast" and z is None and k < len(order) and order[k] == "lin" and fuse_bcast(ws, C):
            # broadcast feeding the LayerNorm+Linear directly: the broadcast
            # pair tensor is never written (its rows are built as they are read)
            with _op("single_proj"):
                B.nt_layernorm_linear(s, W["uv.w"], W["uv.b"], ws.uv, layout=layout, level="singles")
            tap("single_proj", uv=ws.uv)
            z = ws.z[ws.cur]
            with _op("bcast_ln_linear"):
                B.nt_layernorm_linear(None, W["lin.w"], W["lin.b"], z, ln=(W["lin.ln_g"], W["lin.ln_b"]),
                                      layout=layout, level="pairs", bcast=(ws.uv[:, :C], ws.uv[:, C:]))
            tap("bcast_ln_linear", z=z)
            k += 1
        elif step == "bcast":
            with _op("single_proj"):
                B.nt_layernorm_linear(s, W["uv.w"], W["uv.b"], ws.uv, layout=layout, level="singles")
            tap("single_proj", uv=ws.uv)
            acc = z is not None
            z = ws.z[ws.cur] if z is None else z
            with _op("pair_broadcast"):
                B.nt_pair_broadcast(layout, ws.uv[:, :C], ws.uv[:, C:], z, accumulate=acc)
            tap("pair_broadcast", z=z)
        elif step == "lin":
            out = ws.z[1 - ws.cur] if z is ws.z[ws.cur] else ws.z[ws.cur]
            with _op("ln_linear"):
                B.nt_layernorm_linear(z, W["lin.w"], W["lin.b"], out, ln=(W["lin.ln_g"], W["lin.ln_b"]),
                                      layout=layout, level="pairs")
            tap("lin", z=out)
            if out is ws.z[1 - ws.cur]:
                ws.cur = 1 - ws.cur
            z = out
        elif step in ("att_row", "att_col"):
            with _op("attn_proj"):
                B.nt_layernorm_linear(z, W[step + ".w"], W[step + ".b"], ws.qkv,
                                      ln=(W[step + ".ln_g"], W[step + ".ln_b"]), n_tail=H, y_tail=ws.bias,
                                      tail_layout="channel_major", layout=layout, level="pairs")
            tap(step + ".proj", qkv=ws.qkv, bias=ws.bias)
            with _op("attention_" + step[4:]):
                B.nt_pair_row_attention(layout, 0 if step == "att_row" else 1, H, d, ws.qkv[:, :C],
                                        ws.qkv[:, C:2 * C], ws.qkv[:, 2 * C:], ws.o, bias=ws.bias, bias_layout="heads",
                                        workspace=ws.scratch)
            tap(step + ".attention", o=ws.o)
            with _op("attn_out_residual"):
                B.nt_layernorm_linear(ws.o, W[step + ".wo"], W[step + ".bo"], z, epilogue="residual", residual=z,
                                      layout=layout, level="pairs", residual_layout=layout)
            tap(step + ".out", z=z)
        elif step in ("att_row_g", "att_col_g"):
            ln = (W[step + ".ln_g"], W[step + ".ln_b"])
            with _op("attn_proj_g"):
                # [q|k|v] with the bias tail, then the gate logits: the weight
                # rows [q; k; v; g; bias] regrouped once on the device
                B.nt_layernorm_linear(z, W[step + ".w_qkvb"], W[step + ".b_qkvb"], ws.qkv, ln=ln, n_tail=H,
                                      y_tail=ws.bias, tail_layout="channel_major", layout=layout, level="pairs")
                B.nt_layernorm_linear(z, W[step + ".w"][3 * C:4 * C], W[step + ".b"][3 * C:4 * C], ws.g, ln=ln,
                                      layout=layout, level="pairs")
            tap(step + ".proj", qkv=ws.qkv, g=ws.g, bias=ws.bias)
            with _op("attention_" + step[4:7] + "_g"):
                B.nt_pair_row_attention(layout, 0 if step == "att_row_g" else 1, H, d, ws.qkv[:, :C],
                                        ws.qkv[:, C:2 * C], ws.qkv[:, 2 * C:], ws.o, bias=ws.bias,
                                        bias_layout="heads", workspace=ws.scratch, gate=ws.g)
            tap(step + ".attention", o=ws.o)
            with _op("attn_out_residual"):
                B.nt_layernorm_linear(ws.o, W[step + ".wo"], W[step + ".bo"], z, epilogue="residual", residual=z,
                                      layout=layout, level="pairs", residual_layout=layout)
            tap(step + ".out", z=z)
        elif step in ("tri_out_g", "tri_in_g"):
            ln = (W[step + ".ln_g"], W[step + ".ln_b"])
            tiled = "pair_tiled" if step == "tri_out_g" else "pair_tiled_t"
            with _op("tri_proj_g"):
                # gated operands sigmoid(a_g) a_p | sigmoid(b_g) b_p straight
                # into pair-tiled planes, then the output gate logits g
                if glu_tiled(ws, C):
                    B.nt_layernorm_linear(z, W[step + ".w"][:4 * C], W[step + ".b"][:4 * C], None, ln=ln,
                                          epilogue="sigmoid_glu", hidden=C, n_tail=2 * C, y_tail=ws.ab,
                                          tail_layout=tiled, layout=layout, level="pairs", c_out=2 * C)
                else:
                    B.nt_layernorm_linear(z, W[step + ".w"][:4 * C], W[step + ".b"][:4 * C], ws.p4, ln=ln,
                                          layout=layout, level="pairs")
                B.nt_layernorm_linear(z, W[step + ".w"][4 * C:], W[step + ".b"][4 * C:], ws.g, ln=ln,
                                      layout=layout, level="pairs")
            if glu_tiled(ws, C):
                tap(step + ".proj", ab=ws.ab, g=ws.g)
            else:
                tap(step + ".proj", p4=ws.p4, g=ws.g)
            with _op("triangle_" + step[4:-2] + "_g"):
                if glu_tiled(ws, C):
                    B.nt_triangle_mul_gated(layout, 0 if step == "tri_out_g" else 1, ws.ab[:C], ws.ab[C:], ws.t,
                                            operands=tiled)
                else:
                    B.nt_triangle_mul_gated(layout, 0 if step == "tri_out_g" else 1, ws.p4[:, :2 * C],
                                            ws.p4[:, 2 * C:], ws.t, workspace=ws.scratch)
            tap(step + ".triangle", t=ws.t)
            with _op("tri_out_gated_residual"):
                B.nt_layernorm_linear(ws.t, W[step + ".wo"], W[step + ".bo"], z,
                                      ln=(W[step + ".out.ln_g"], W[step + ".out.ln_b"]), epilogue="gated_residual",
                                      residual=z, gate=ws.g, layout=layout, level="pairs", residual_layout=layout)
            tap(step + ".out", z=z)
        elif step in ("tri_out", "tri_in"):
            with _op("tri_proj"):
                B.nt_layernorm_linear(z, W[step + ".w"], W[step + ".b"], None,
                                      ln=(W[step + ".ln_g"], W[step + ".ln_b"]), n_tail=2 * C, y_tail=ws.ab,
                                      tail_layout="pair_tiled" if step == "tri_out" else "pair_tiled_t",
                                      layout=layout, level="pairs", c_out=2 * C)
            tap(step + ".proj", ab=ws.ab)
            with _op("triangle_" + step[4:]):
                B.nt_triangle_mul(layout, 0 if step == "tri_out" else 1, ws.ab[:C], ws.ab[C:], z,
                                  operands="pair_tiled" if step == "tri_out" else "pair_tiled_t")
            tap(step + ".triangle", z=z)
        elif step == "trans":
            with _op("transition"):
                B.nt_layernorm_linear(z, W["trans.w"], W["trans.b"], z, ln=(W["trans.ln_g"], W["trans.ln_b"]),
                                      epilogue="swiglu_residual", w2=W["trans.w2"], bias2=W["trans.b2"],
                                      hidden=W["trans.w2"].shape[1], layout=layout, level="pairs",
                                      workspace=ws.scratch)
            tap("transition", z=z)
        elif step == "single":
            with _op("segment_mean"):
                B.nt_segment_reduce(layout, "pairs", "mean", z, ws.m)
            tap("segment_mean", m=ws.m)
            with _op("single_update"):
                B.nt_layernorm_linear(ws.m, W["single.w"], W["single.b"], s, epilogue="residual", residual=s,
                                      layout=layout, level="singles", residual_layout=layout)
            tap("single_update", s=s)
        else:
            raise ValueError(f"unknown step {step!r}")
    return z


class TokenWorkspace:
    def __init__(self, layout: B.NestedLayout, c: int, hidden: int, dtype: str, device="cuda"):
        td = torch.bfloat16 if dtype == "bf16" else torch.float32
        T = layout.sum_n
        self.qkv = torch.empty((T, 3 * c), dtype=td, device=device)
        self.o = torch.empty((T, c), dtype=td, device=device)
        self.h = torch.empty((T, hidden), dtype=td, device=device)
        self.pooled = torch.empty((layout.batch, c), dtype=torch.float32, device=device)
        # op scratch: the LayerNorm rows of the large-K products
        need = max(B.layernorm_linear_workspace_bytes(T, c, 3 * c, dtype, ln=True),
                   B.layernorm_linear_workspace_bytes(T, c, hidden, dtype, ln=True, epilogue="gelu"))
        self.scratch = B.workspace_tensor(need, device)


def encoder_layer(layout: B.NestedLayout, x, W: dict, heads: int, head_dim: int, ws: TokenWorkspace):
    """Pre-LN encoder layer on packed tokens, in place on x; returns the pooled means."""
    c = heads * head_dim
    with _op("qkv_proj"):
        B.nt_layernorm_linear(x, W["qkv.w"], W["qkv.b"], ws.qkv, ln=(W["ln1_g"], W["ln1_b"]),
                              layout=layout, level="singles", workspace=ws.scratch)
    with _op("attention_1d"):
        B.nt_pair_row_attention(layout, 2, heads, head_dim, ws.qkv[:, :c], ws.qkv[:, c:2 * c], ws.qkv[:, 2 * c:],
                                ws.o, scale=1.0 / math.sqrt(head_dim))
    with _op("out_proj_residual"):
        B.nt_layernorm_linear(ws.o, W["o.w"], W["o.b"], x, epilogue="residual", residual=x, layout=layout,
                              level="singles")
    with _op("ffn_up_gelu"):
        B.nt_layernorm_linear(x, W["ffn1.w"], W["ffn1.b"], ws.h, ln=(W["ln2_g"], W["ln2_b"]), epilogue="gelu",
                              layout=layout, level="singles", workspace=ws.scratch)
    with _op("ffn_down_residual"):
        B.nt_layernorm_linear(ws.h, W["ffn2.w"], W["ffn2.b"], x, epilogue="residual", residual=x, layout=layout,
                              level="singles")
    with _op("sample_mean"):
        B.nt_segment_reduce(layout, "singles", "mean", x, ws.pooled)
    return ws.pooled


class PairRun:
    """A pair workload prepared on the device: layout, weights of every block,
    the initial single track and the workspaces.  step() runs all blocks."""

    def __init__(self, w, lengths=None, device="cuda"):
        from . import synth
        self.w = w
        self.lengths = [int(n) for n in (synth.lengths_for(w) if lengths is None else lengths)]
        self.layout = B.NestedLayout(self.lengths)
        self.dims = dict(c_z=w.c_z, heads=w.heads, head_dim=w.head_dim)
        self.params = [synth.pair_block_params(w, block=b) for b in range(w.blocks)]
        self.W = [to_device(p, w.dtype, device) for p in self.params]
        C, H = w.c_z, w.heads
        for Wb in self.W:                      # gated attention: [q; k; v; bias] regrouped for one projection
            for key in [t for t in w.steps if t.startswith("att_") and t.endswith("_g")]:
                Wb[key + ".w_qkvb"] = torch.cat([Wb[key + ".w"][:3 * C], Wb[key + ".w"][4 * C:4 * C + H]]).contiguous()
                Wb[key + ".b_qkvb"] = torch.cat([Wb[key + ".b"][:3 * C], Wb[key + ".b"][4 * C:4 * C + H]]).contiguous()
        self.s_init = synth.normal(w.seed, "s", (sum(self.lengths), w.c_s), w.s_scale, w.dtype)
        td = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.s0 = torch.from_numpy(self.s_init).to(device=device, dtype=td)
        self.s = self.s0.clone()
        self.ws = PairWorkspace(self.layout, w.c_s, w.c_z, w.heads, w.dtype, device,
                                gated=any(t.endswith("_g") for t in w.steps))
        self.z = None

    def step(self, tap=None):
        """One pass of all blocks; tap(block, op, **outputs) sees every op's outputs."""
        self.s.copy_(self.s0)
        z = None
        for b in range(self.w.blocks):
            steps = self.w.steps if b == 0 else tuple(t for t in self.w.steps if t != "lin")
            btap = None if tap is None else (lambda op, _b=b, **t: tap(_b, op, **t))
            z = pair_block(self.layout, self.s, self.W[b], self.dims, steps, self.ws, z=z, tap=btap)
        self.z = z
        return self.s, z


class TokenRun:
    """The token-path workload prepared on the device; step() runs one encoder
    layer and the per-sample mean pool."""

    def __init__(self, w, lengths=None, device="cuda"):
        from . import synth
        self.w = w
        self.lengths = [int(n) for n in (synth.lengths_for(w) if lengths is None else lengths)]
        self.layout = B.NestedLayout(self.lengths)
        self.params = synth.encoder_layer_params(w)
        self.W = to_device(self.params, w.dtype, device)
        self.x_init = synth.normal(w.seed, "x", (sum(self.lengths), w.c_s), 0.5, w.dtype)
        td = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.x0 = torch.from_numpy(self.x_init).to(device=device, dtype=td)
        self.x = self.x0.clone()
        self.ws = TokenWorkspace(self.layout, w.c_s, w.hidden, w.dtype, device)

    def step(self):
        self.x.copy_(self.x0)
        pooled = encoder_layer(self.layout, self.x, self.W, self.w.heads, self.w.head_dim, self.ws)
        return self.x, pooled


class MechanismRun:
    """The measured single-pair-single program as one training step on the
    device: forward (Eq. running-block), the joint diagnostic loss, and the
    backward of every parameter and input, one C-ABI call per op.

    Square pairs take both pair operands from x; rectangular pairs take the
    column operand from y (M_i rows per sample).  Weight gradients are
    overwritten every step (fp32); the loss stays on the device as per-sample
    terms.  Every buffer, scratch included, is allocated here: a step
    allocates nothing."""

    def __init__(self, w, lengths=None, cols=None, device="cuda"):
        from . import synth
        td = torch.bfloat16
        self.w = w
        self.lengths = [int(n) for n in (synth.lengths_for(w) if lengths is None else lengths)]
        c = synth.cols_for(w) if cols is None else cols
        self.cols = None if c is None else [int(m) for m in c]
        self.rect = self.cols is not None
        self.layout = B.NestedLayout(self.lengths, cols=self.cols)
        lay = self.layout
        S, Mr, cells = lay.sum_n, lay.sum_m, lay.sum_n2
        Cx, Cp, F = w.c_s, w.c_z, w.hidden
        # non-leading layout: elements (Sx, N_i, C) pack as (N_i, Sx, C), so
        # every packed row holds Sx feature vectors; row-wise ops see Sx times
        # the rows, ragged ops (broadcast, reductions, loss) Sx times the width
        self.Sx = Sx = w.s_axis
        self.sep = self.rect or Sx > 1          # u and v from separate projections
        self.params = synth.mechanism_params(w)
        self.W = to_device(self.params, w.dtype, device)
        if not self.sep:         # one projection computes u and v from the same rows
            self.W["uv.w"] = torch.cat([self.W["u.w"], self.W["v.w"]], 0).contiguous()
            self.W["uv.b"] = torch.cat([self.W["u.b"], self.W["v.b"]], 0).contiguous()
        self.x_init = synth.normal(w.seed, "mech.x", (S, Sx * Cx), 1.0, w.dtype)
        self.y_init = synth.normal(w.seed, "mech.y", (Mr, Cx), 1.0, w.dtype) if self.rect else None
        self.x = torch.from_numpy(self.x_init).to(device=device, dtype=td)
        self.y = torch.from_numpy(self.y_init).to(device=device, dtype=td) if self.rect else None
        Bn = lay.batch
        self.alpha = torch.tensor([1.0 + i / Bn for i in range(Bn)], dtype=torch.float32, device=device)
        self.beta = torch.tensor([1.5 - i / (2.0 * Bn) for i in range(Bn)], dtype=torch.float32, device=device)
        self.scale_s = 1.0 / (Sx * Cx * S)
        self.scale_p = 1.0 / (Sx * Cp * cells)
        e = lambda *shape, dt=td: torch.empty(shape, dtype=dt, device=device)   # noqa: E731
        f32 = torch.float32
        self.uv = e(S, 2 * Cp) if not self.sep else None
        self.u, self.v = (self.uv[:, :Cp], self.uv[:, Cp:]) if not self.sep else (e(S, Sx * Cp), e(Mr, Sx * Cp))
        self.P, self.Pt = e(cells, Sx * Cp), e(cells, Sx * Cp)
        self.m = e(S, Sx * Cp, dt=f32)
        self.xt = e(S, Sx * Cx)
        self.loss_s, self.loss_p, self.loss_tmp = e(Bn, dt=f32), e(Bn, dt=f32), e(Bn, dt=f32)
        self.dxt = e(S, Sx * Cx)
        self.dx = e(S, Sx * Cx, dt=f32)
        self.dy = e(Mr, Cx, dt=f32) if self.rect else None
        self.dpt, self.dP = e(cells, Sx * Cp), e(cells, Sx * Cp)
        self.dm = e(S, Sx * Cp, dt=f32)
        self.duv = e(S, 2 * Cp) if not self.sep else None
        self.du, self.dv = (self.duv[:, :Cp], self.duv[:, Cp:]) if not self.sep else (e(S, Sx * Cp), e(Mr, Sx * Cp))
        self.grads = {k: torch.empty(v.shape, dtype=f32, device=device) for k, v in self.W.items()
                      if k not in ("uv.w", "uv.b")}
        if not self.sep:
            self.grads["uv.w"] = torch.empty((2 * Cp, Cx), dtype=f32, device=device)
            self.grads["uv.b"] = torch.empty((2 * Cp,), dtype=f32, device=device)
        # op scratch, used one op at a time on one stream
        need = [B.layernorm_linear_workspace_bytes(Sx * cells, Cp, Cp, w.dtype, epilogue="swiglu_residual",
                                                   hidden=F),
                B.loss_workspace_bytes(lay)]
        need += [self._bwd_ws(Sx * cells, Cp, Cp, True, "swiglu_residual", F),
                 self._bwd_ws(Sx * S, Cp, Cx, False, "residual", 0),
                 self._bwd_ws(Sx * S, Cx, Cp if self.sep else 2 * Cp, False, "none", 0)]
        if self.rect:
            need.append(self._bwd_ws(Mr, Cx, Cp, False, "none", 0))
        self.scratch = B.workspace_tensor(max(need), device)

    @staticmethod
    def _bwd_ws(rows, K, N, ln, epi, F):
        import ctypes
        a = B.LinearBwdArgs()
        a.rows, a.c_in, a.c_out = int(rows), int(K), int(N)
        a.ldx, a.ld_dy, a.ld_dx = K, N, K
        a.x_dtype = a.dx_dtype = B.NT_BF16
        a.ln_gamma = ctypes.c_void_p(16) if ln else None
        a.epilogue, a.hidden = B.EPILOGUES[epi], int(F)
        n = ctypes.c_uint64()
        B._check(B.load().nt_layernorm_linear_backward_workspace(ctypes.byref(a), ctypes.byref(n)))
        return int(n.value)

    def step(self):
        """Forward, loss and backward; returns (loss terms, xt, pt, grads)."""
        lay, W, G, ws = self.layout, self.W, self.grads, self.scratch
        Cx, Cp, F, Sx = self.w.c_s, self.w.c_z, self.w.hidden, self.Sx
        # row views of the non-leading layout ([rows, Sx * C] as [rows * Sx, C]);
        # the identity for Sx = 1 (row-wise calls then also check the layout)
        rv = (lambda t: t.view(-1, t.shape[1] // Sx)) if Sx > 1 else (lambda t: t)   # noqa: E731
        rl = dict(layout=lay) if Sx == 1 else {}
        # forward
        with _op("mech_proj"):
            if self.rect:
                B.nt_layernorm_linear(self.x, W["u.w"], W["u.b"], self.u, layout=lay, level="singles")
                B.nt_layernorm_linear(self.y, W["v.w"], W["v.b"], self.v)
            elif self.sep:
                B.nt_layernorm_linear(rv(self.x), W["u.w"], W["u.b"], rv(self.u))
                B.nt_layernorm_linear(rv(self.x), W["v.w"], W["v.b"], rv(self.v))
            else:
                B.nt_layernorm_linear(self.x, W["uv.w"], W["uv.b"], self.uv, layout=lay, level="singles")
        with _op("mech_broadcast"):
            B.nt_pair_broadcast(lay, self.u, self.v, self.P)
        with _op("mech_transition"):
            B.nt_layernorm_linear(rv(self.P), W["trans.w"], W["trans.b"], rv(self.Pt),
                                  ln=(W["trans.ln_g"], W["trans.ln_b"]), epilogue="swiglu_residual", w2=W["trans.w2"],
                                  bias2=W["trans.b2"], hidden=F, residual=rv(self.P), level="pairs", workspace=ws, **rl)
        with _op("mech_column_mean"):
            B.nt_segment_reduce(lay, "pairs", "mean", self.Pt, self.m)
        with _op("mech_single_update"):
            B.nt_layernorm_linear(rv(self.m), W["g.w"], W["g.b"], rv(self.xt), epilogue="residual",
                                  residual=rv(self.x), level="singles", **rl)
        # loss (Eq. joint-diagnostic-loss) and its gradient
        with _op("mech_loss"):
            B.nt_weighted_square_loss(lay, "singles", self.xt, self.alpha, self.scale_s, self.loss_s, dx=self.dxt,
                                      workspace=ws)
            B.nt_weighted_square_loss(lay, "singles", self.xt, self.alpha, self.scale_s, self.loss_tmp, dx=self.dx,
                                      workspace=ws)
            B.nt_weighted_square_loss(lay, "pairs", self.Pt, self.beta, self.scale_p, self.loss_p, dx=self.dpt,
                                      workspace=ws)
        # backward
        with _op("mech_single_update_bwd"):
            B.nt_layernorm_linear_backward(rv(self.m), W["g.w"], rv(self.dxt), epilogue="residual", dx=rv(self.dm),
                                           dw=G["g.w"], db=G["g.b"], overwrite_weights=True, workspace=ws)
        with _op("mech_column_mean_bwd"):
            B.nt_segment_reduce_backward(lay, "pairs", "mean", self.dm, self.dpt, accumulate=True)
        with _op("mech_transition_bwd"):
            B.nt_layernorm_linear_backward(rv(self.P), W["trans.w"], rv(self.dpt), ln=(W["trans.ln_g"], W["trans.ln_b"]),
                                           bias=W["trans.b"], epilogue="swiglu_residual", w2=W["trans.w2"], hidden=F,
                                           dx=rv(self.dP), dw=G["trans.w"], db=G["trans.b"], dgamma=G["trans.ln_g"],
                                           dbeta=G["trans.ln_b"], dw2=G["trans.w2"], db2=G["trans.b2"],
                                           overwrite_weights=True, workspace=ws)
        with _op("mech_broadcast_bwd"):
            B.nt_pair_broadcast_backward(lay, self.dP, self.du, self.dv)
        with _op("mech_proj_bwd"):
            if self.rect:
                B.nt_layernorm_linear_backward(self.x, W["u.w"], self.du, dx=self.dx, accumulate_dx=True, dw=G["u.w"],
                                               db=G["u.b"], overwrite_weights=True, workspace=ws)
                B.nt_layernorm_linear_backward(self.y, W["v.w"], self.dv, dx=self.dy, dw=G["v.w"], db=G["v.b"],
                                               overwrite_weights=True, workspace=ws)
            elif self.sep:
                B.nt_layernorm_linear_backward(rv(self.x), W["u.w"], rv(self.du), dx=rv(self.dx), accumulate_dx=True,
                                               dw=G["u.w"], db=G["u.b"], overwrite_weights=True, workspace=ws)
                B.nt_layernorm_linear_backward(rv(self.x), W["v.w"], rv(self.dv), dx=rv(self.dx), accumulate_dx=True,
                                               dw=G["v.w"], db=G["v.b"], overwrite_weights=True, workspace=ws)
            else:
                B.nt_layernorm_linear_backward(self.x, W["uv.w"], self.duv, dx=self.dx, accumulate_dx=True,
                                               dw=G["uv.w"], db=G["uv.b"], overwrite_weights=True, workspace=ws)
        return self.loss_s, self.loss_p, self.xt, self.Pt
