"""Thin ctypes binding of libnt.so (include/nt.h).

Argument marshalling only: every computation runs in the HIP kernels behind
the C ABI.  torch supplies device memory and the current HIP stream.  The
library must have been built (paper_2609_30379_amd.build); nothing here falls
back to any other implementation.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libnt.so")

NT_OK, NT_ERR_INVALID_ARG, NT_ERR_LAYOUT_MISMATCH, NT_ERR_OVERFLOW, NT_ERR_UNSUPPORTED, NT_ERR_HIP, NT_ERR_OOM = \
    0, -1, -2, -3, -4, -5, -6
NT_F32, NT_BF16 = 0, 1
EPILOGUES = {"none": 0, "residual": 1, "swiglu_residual": 2, "gelu": 3, "gated_residual": 4, "sigmoid_glu": 5}
LEVELS = {"singles": 0, "pairs": 1, "pairs_first": 2}
TAILS = {"channel_major": 0, "pair_tiled": 1, "pair_tiled_t": 2}
TRI_OPERANDS = {"packed": 0, "pair_tiled": 1, "pair_tiled_t": 2}
ARRAYS = {"lengths": 0, "cu_seqlens": 1, "cu_pairs": 2, "row_splits2": 3, "row_sample": 4,
          "attn_work": 5, "tri_work": 6, "seq_work": 7, "cu_pad": 8, "cols": 9, "cu_cols": 10,
          "tri_split": 11}
NT_LAYOUT_HOST_ONLY = 1


class NtError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"nt status {status}: {msg}")
        self.status = status


class LayoutInfo(C.Structure):
    _fields_ = [("batch", C.c_int32), ("max_len", C.c_int32), ("sum_n", C.c_int64), ("sum_n2", C.c_int64),
                ("sum_n3", C.c_int64), ("sum_pad", C.c_int64), ("d_cu_seqlens", C.c_void_p),
                ("d_cu_pairs", C.c_void_p), ("d_row_splits2", C.c_void_p), ("sum_m", C.c_int64),
                ("rect", C.c_int32), ("d_cu_cols", C.c_void_p)]


class LinearBwdArgs(C.Structure):
    _fields_ = [("rows", C.c_int64), ("c_in", C.c_int32), ("c_out", C.c_int32),
                ("x", C.c_void_p), ("ldx", C.c_int64), ("x_dtype", C.c_int),
                ("ln_gamma", C.c_void_p), ("ln_beta", C.c_void_p), ("ln_eps", C.c_float),
                ("w", C.c_void_p), ("bias", C.c_void_p), ("epilogue", C.c_int),
                ("hidden", C.c_int32), ("w2", C.c_void_p), ("residual_is_x", C.c_int32),
                ("dy", C.c_void_p), ("ld_dy", C.c_int64),
                ("dx", C.c_void_p), ("ld_dx", C.c_int64), ("dx_dtype", C.c_int), ("accumulate_dx", C.c_int32),
                ("overwrite_weights", C.c_int32),
                ("dw", C.c_void_p), ("db", C.c_void_p), ("dgamma", C.c_void_p), ("dbeta", C.c_void_p),
                ("dw2", C.c_void_p), ("db2", C.c_void_p),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_uint64)]


class LinearArgs(C.Structure):
    _fields_ = [("rows", C.c_int64), ("c_in", C.c_int32), ("c_out", C.c_int32), ("dtype", C.c_int),
                ("x", C.c_void_p), ("ldx", C.c_int64), ("x_dtype", C.c_int),
                ("ln_gamma", C.c_void_p), ("ln_beta", C.c_void_p), ("ln_eps", C.c_float),
                ("w", C.c_void_p), ("bias", C.c_void_p), ("epilogue", C.c_int),
                ("hidden", C.c_int32), ("w2", C.c_void_p), ("bias2", C.c_void_p),
                ("residual", C.c_void_p), ("ld_residual", C.c_int64),
                ("y", C.c_void_p), ("ldy", C.c_int64),
                ("n_tail", C.c_int32), ("y_tail", C.c_void_p), ("ld_tail", C.c_int64), ("tail_layout", C.c_int),
                ("layout", C.c_void_p), ("level", C.c_int), ("residual_layout", C.c_void_p),
                ("bcast_u", C.c_void_p), ("ld_bcast_u", C.c_int64), ("bcast_v", C.c_void_p), ("ld_bcast_v", C.c_int64),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_uint64),
                ("gate", C.c_void_p), ("ld_gate", C.c_int64)]


_lib = None


def load(path: str = LIB_PATH):
    """Loads libnt.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_30379_amd.build`")
    lib = C.CDLL(path)
    vp, i32, i64, u64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float
    sig = {
        "nt_from_lengths": [vp, i32, C.c_uint32, vp, C.POINTER(vp)],
        "nt_from_offsets": [vp, i32, C.c_uint32, vp, C.POINTER(vp)],
        "nt_layout_destroy": [vp],
        "nt_layout_info": [vp, C.POINTER(LayoutInfo)],
        "nt_layout_host_array": [vp, C.c_int, C.POINTER(C.POINTER(i32)), C.POINTER(i64)],
        "nt_layouts_compatible": [vp, vp],
        "nt_pair_broadcast": [vp, i32, vp, i64, vp, i64, vp, i64, i32, C.c_int, vp],
        "nt_layernorm_linear": [C.POINTER(LinearArgs), vp],
        "nt_layernorm_linear_workspace": [C.POINTER(LinearArgs), C.POINTER(u64)],
        "nt_pair_row_attention": [vp, i32, i32, i32, vp, vp, vp, i64, vp, i64, i64, f32, vp, i64, C.c_int, vp, u64, vp],
        "nt_pair_row_attention_workspace": [vp, i32, i32, i32, C.c_int, i32, C.POINTER(u64)],
        "nt_cross_attention": [vp, vp, i32, i32, vp, i64, vp, vp, i64, f32, vp, i64, C.c_int, vp],
        "nt_pair_row_attention_gated": [vp, i32, i32, i32, vp, vp, vp, i64, vp, i64, vp, i64, i64, f32, vp, i64,
                                        C.c_int, vp, u64, vp],
        "nt_pair_row_attention_noalloc": [vp, i32, i32, i32, vp, vp, vp, i64, vp, i64, i64, f32, vp, i64, C.c_int, vp],
        "nt_triangle_mul": [vp, i32, i32, vp, vp, i64, C.c_int, vp, i64, C.c_int, vp, u64, vp],
        "nt_triangle_mul_workspace": [vp, i32, C.c_int, C.c_int, C.POINTER(u64)],
        "nt_triangle_mul_gated": [vp, i32, i32, vp, vp, i64, C.c_int, vp, i64, C.c_int, vp, u64, vp],
        "nt_segment_reduce": [vp, C.c_int, i32, i32, vp, i64, C.c_int, vp, i64, vp],
        "nt_pair_broadcast_backward": [vp, i32, vp, i64, C.c_int, vp, i64, vp, i64, C.c_int, i32, vp],
        "nt_from_rect_lengths": [vp, vp, i32, C.c_uint32, vp, C.POINTER(vp)],
        "nt_weighted_square_loss": [vp, C.c_int, i32, vp, i64, C.c_int, vp, f32, vp, vp, i64, C.c_int, vp, u64, vp],
        "nt_weighted_square_loss_workspace": [vp, C.POINTER(u64)],
        "nt_segment_reduce_backward": [vp, C.c_int, i32, i32, vp, i64, vp, i64, C.c_int, i32, vp],
        "nt_triangle_mul_backward": [vp, i32, i32, vp, vp, i64, vp, i64, vp, vp, i64, C.c_int, vp, u64, vp],
        "nt_layernorm_linear_backward": [C.POINTER(LinearBwdArgs), vp],
        "nt_layernorm_linear_backward_workspace": [C.POINTER(LinearBwdArgs), C.POINTER(u64)],
        "nt_pair_row_attention_backward": [vp, i32, i32, i32, vp, vp, vp, i64, vp, i64, i64, vp, i64, f32,
                                           vp, vp, vp, i64, vp, i64, i64, C.c_int, vp, u64, vp],
        "nt_pair_row_attention_backward_workspace": [vp, i32, i32, i32, C.c_int, C.POINTER(u64)],
        "nt_last_error": [],
        "nt_version": [],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_char_p if name in ("nt_last_error", "nt_version") else C.c_int
    _lib = lib
    return lib


def _check(status: int):
    if status != NT_OK:
        raise NtError(status, load().nt_last_error().decode())


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return NT_BF16
    if t.dtype == torch.float32:
        return NT_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _mat(t, name):
    """(device pointer, row stride in elements) of a 2-D device tensor with unit column stride."""
    if t is None:
        return None, 0
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dim() != 2 or (t.size(1) > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be 2-D with contiguous rows")
    return C.c_void_p(t.data_ptr()), int(t.stride(0)) if t.size(0) > 1 else int(t.size(1))


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def workspace_tensor(nbytes: int, device="cuda"):
    """A device buffer of at least nbytes (16-byte aligned) for an op's
    workspace argument, or None when the op needs none."""
    import torch
    if nbytes <= 0:
        return None
    words = (int(nbytes) + 15) // 16 * 2          # whole 16-byte units, as 8-byte words (16-byte aligned)
    return torch.empty((words,), dtype=torch.int64, device=device).view(torch.uint8)[:int(nbytes)]


def _ws(ws):
    return (C.c_void_p(ws.data_ptr()), int(ws.numel() * ws.element_size())) if ws is not None else (None, 0)


class NestedLayout:
    """Partitions of a batch of pair states: square (nt_from_lengths /
    nt_from_offsets) or, with cols, rectangular N_i x M_i (nt_from_rect_lengths)."""

    def __init__(self, lengths, host_only: bool = False, offsets: bool = False, cols=None):
        lib = load()
        arr = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
        self._arr = arr
        handle = C.c_void_p()
        flags = NT_LAYOUT_HOST_ONLY if host_only else 0
        stream = None if host_only else _stream()
        batch = len(arr) - 1 if offsets else len(arr)
        if cols is not None:
            carr = np.ascontiguousarray(np.asarray(cols, dtype=np.int32))
            if len(carr) != len(arr) or offsets:
                raise ValueError("cols needs one entry per sample (lengths, not offsets)")
            self._carr = carr
            _check(lib.nt_from_rect_lengths(arr.ctypes.data_as(C.c_void_p), carr.ctypes.data_as(C.c_void_p), batch,
                                            flags, stream, C.byref(handle)))
        else:
            fn = lib.nt_from_offsets if offsets else lib.nt_from_lengths
            _check(fn(arr.ctypes.data_as(C.c_void_p), batch, flags, stream, C.byref(handle)))
        self.handle = handle
        info = LayoutInfo()
        _check(lib.nt_layout_info(handle, C.byref(info)))
        self.batch, self.max_len = info.batch, info.max_len
        self.sum_n, self.sum_n2, self.sum_n3, self.sum_pad = info.sum_n, info.sum_n2, info.sum_n3, info.sum_pad
        self.sum_m, self.rect = info.sum_m, bool(info.rect)

    def host_array(self, name: str) -> np.ndarray:
        ptr, count = C.POINTER(C.c_int32)(), C.c_int64()
        _check(load().nt_layout_host_array(self.handle, ARRAYS[name], C.byref(ptr), C.byref(count)))
        return np.ctypeslib.as_array(ptr, shape=(count.value,)).copy() if count.value else np.zeros(0, np.int32)

    def compatible(self, other: "NestedLayout") -> bool:
        return bool(load().nt_layouts_compatible(self.handle, other.handle))

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            _check(load().nt_layout_destroy(self.handle))
            self.handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def nt_pair_broadcast(layout: NestedLayout, u, v, z, accumulate: bool = False):
    pu, ldu = _mat(u, "u")
    pv, ldv = _mat(v, "v")
    pz, ldz = _mat(z, "z")
    _check(load().nt_pair_broadcast(layout.handle, int(z.size(1)), pu, ldu, pv, ldv, pz, ldz,
                                    int(accumulate), _dtype(z), _stream()))
    return z


def nt_layernorm_linear(x, w, bias, y, ln=None, eps: float = 1e-5, epilogue: str = "none", w2=None, bias2=None,
                        hidden: int = 0, residual=None, n_tail: int = 0, y_tail=None,
                        tail_layout: str = "channel_major", layout: NestedLayout | None = None,
                        level: str = "pairs", residual_layout: NestedLayout | None = None, c_out: int | None = None,
                        bcast=None, workspace=None, gate=None):
    """bcast=(u, v) with x=None: the rows are the pair broadcast u[eta_i+a] + v[eta_i+b] over `layout`.
    workspace: a device buffer from workspace_tensor(), or None to allocate one of the queried size.
    gate: gate logits [rows, c_out] of the "gated_residual" epilogue."""
    a = LinearArgs()
    if bcast is not None:
        if x is not None or layout is None:
            raise ValueError("broadcast rows need x=None and a layout")
        u, v = bcast
        a.bcast_u, a.ld_bcast_u = _mat(u, "u")
        a.bcast_v, a.ld_bcast_v = _mat(v, "v")
        a.rows, a.c_in = int(layout.sum_n2), int(u.size(1))
        a.x, a.ldx, a.x_dtype = None, 0, _dtype(u)
    else:
        px, ldx = _mat(x, "x")
        a.rows, a.c_in = int(x.size(0)), int(x.size(1))
        a.x, a.ldx, a.x_dtype = px, ldx, _dtype(x)
    a.c_out = int(c_out if c_out is not None else (w2.size(0) if epilogue == "swiglu_residual" else w.size(0)))
    a.dtype = _dtype(w)
    if ln is not None:
        a.ln_gamma, a.ln_beta = _ptr(ln[0]), _ptr(ln[1])
    a.ln_eps = eps
    a.w, a.bias, a.epilogue = _ptr(w), _ptr(bias), EPILOGUES[epilogue]
    a.hidden, a.w2, a.bias2 = int(hidden), _ptr(w2), _ptr(bias2)
    a.residual, a.ld_residual = _mat(residual, "residual")
    a.y, a.ldy = _mat(y, "y")
    a.n_tail = int(n_tail)
    a.y_tail, a.ld_tail = (_ptr(y_tail), int(y_tail.stride(0))) if y_tail is not None else (None, 0)
    a.tail_layout = TAILS[tail_layout]
    a.layout = layout.handle if layout is not None else None
    a.level = LEVELS[level]
    a.residual_layout = residual_layout.handle if residual_layout is not None else None
    a.gate, a.ld_gate = _mat(gate, "gate")
    if workspace is None:
        workspace = workspace_tensor(_linear_ws_bytes(a))
    a.workspace, a.workspace_bytes = _ws(workspace)
    _check(load().nt_layernorm_linear(C.byref(a), _stream()))
    return y


def _linear_ws_bytes(a) -> int:
    n = C.c_uint64()
    _check(load().nt_layernorm_linear_workspace(C.byref(a), C.byref(n)))
    return int(n.value)


def layernorm_linear_workspace_bytes(x_rows: int, c_in: int, c_out: int, dtype: str = "bf16", ln: bool = True,
                                     epilogue: str = "none", hidden: int = 0, residual_is_x: bool = True,
                                     n_tail: int = 0) -> int:
    """Workspace bytes of an nt_layernorm_linear call with these sizes and flags
    (row-major operands with their natural strides)."""
    a = LinearArgs()
    a.rows, a.c_in, a.c_out = int(x_rows), int(c_in), int(c_out)
    a.dtype = a.x_dtype = NT_BF16 if dtype == "bf16" else NT_F32
    a.ldx, a.ldy = int(c_in), int(c_out - n_tail)
    a.ld_residual = int(c_out - n_tail)
    a.ln_gamma = C.c_void_p(16) if ln else None
    a.epilogue, a.hidden, a.n_tail = EPILOGUES[epilogue], int(hidden), int(n_tail)
    if epilogue == "swiglu_residual" and not residual_is_x:
        a.residual = C.c_void_p(32)
    return _linear_ws_bytes(a)


def nt_pair_row_attention_noalloc(layout: NestedLayout, axis: int, heads: int, head_dim: int, q, k, v, o,
                                  bias=None, scale: float | None = None, bias_layout: str = "cells"):
    """nt_pair_row_attention without a workspace: the library's per-device
    scratch array holds the bias image (at most 16 MiB)."""
    pq, ld = _mat(q, "q")
    pk, ldk = _mat(k, "k")
    pv, ldv = _mat(v, "v")
    if not (ld == ldk == ldv):
        raise ValueError("q, k and v must share one row stride")
    po, ldo = _mat(o, "o")
    if bias is None:
        pb, ldb, ldbh = None, 0, 0
    elif bias_layout == "cells":
        pb, ldb, ldbh = _ptr(bias), int(bias.stride(0)), 1
    else:
        pb, ldb, ldbh = _ptr(bias), 1, int(bias.stride(0))
    scale = 1.0 / float(np.sqrt(head_dim)) if scale is None else float(scale)
    _check(load().nt_pair_row_attention_noalloc(layout.handle, int(axis), int(heads), int(head_dim), pq, pk, pv, ld,
                                                pb, ldb, ldbh, scale, po, ldo, _dtype(q), _stream()))
    return o


def attention_workspace_bytes(layout: NestedLayout, axis: int, heads: int, head_dim: int, dtype: str = "bf16",
                              has_bias: bool = True) -> int:
    n = C.c_uint64()
    _check(load().nt_pair_row_attention_workspace(layout.handle, int(axis), int(heads), int(head_dim),
                                                  NT_BF16 if dtype == "bf16" else NT_F32, int(bool(has_bias)),
                                                  C.byref(n)))
    return int(n.value)


def nt_pair_row_attention(layout: NestedLayout, axis: int, heads: int, head_dim: int, q, k, v, o,
                          bias=None, scale: float | None = None, bias_layout: str = "cells", workspace=None,
                          gate=None):
    """bias: [sum N^2, H] with a row stride (bias_layout "cells"), or head-major
    [H, >= sum N^2] (bias_layout "heads").  gate: [sum N^2, H*d] logits of the
    output gate (nt_pair_row_attention_gated), or None."""
    pq, ld = _mat(q, "q")
    pk, ldk = _mat(k, "k")
    pv, ldv = _mat(v, "v")
    if not (ld == ldk == ldv):
        raise ValueError("q, k and v must share one row stride")
    po, ldo = _mat(o, "o")
    if bias is None:
        pb, ldb, ldbh = None, 0, 0
    elif bias_layout == "cells":
        if bias.dim() != 2 or bias.stride(1) != 1:
            raise ValueError("bias must be [sum N^2, H] with unit head stride")
        pb, ldb, ldbh = _ptr(bias), int(bias.stride(0)), 1
    elif bias_layout == "heads":
        if bias.dim() != 2 or bias.stride(1) != 1:
            raise ValueError("head-major bias must be [H, ld] with contiguous rows")
        pb, ldb, ldbh = _ptr(bias), 1, int(bias.stride(0))
    else:
        raise ValueError(bias_layout)
    scale = 1.0 / float(np.sqrt(head_dim)) if scale is None else float(scale)
    dt = _dtype(q)
    if workspace is None:
        workspace = workspace_tensor(attention_workspace_bytes(layout, axis, heads, head_dim,
                                                               "bf16" if dt == NT_BF16 else "f32", bias is not None))
    pw, nw = _ws(workspace)
    if gate is not None:
        pg, ldg = _mat(gate, "gate")
        _check(load().nt_pair_row_attention_gated(layout.handle, int(axis), int(heads), int(head_dim), pq, pk, pv, ld,
                                                  pg, ldg, pb, ldb, ldbh, scale, po, ldo, dt, pw, nw, _stream()))
        return o
    _check(load().nt_pair_row_attention(layout.handle, int(axis), int(heads), int(head_dim), pq, pk, pv, ld,
                                        pb, ldb, ldbh, scale, po, ldo, dt, pw, nw, _stream()))
    return o


def nt_cross_attention(q_layout: NestedLayout, kv_layout: NestedLayout, heads: int, head_dim: int, q, k, v, o,
                       scale: float | None = None):
    """q, o: [sum N, H*d] by q_layout; k, v: [sum M, H*d] by kv_layout (one row stride)."""
    pq, ldq = _mat(q, "q")
    pk, ldk = _mat(k, "k")
    pv, ldv = _mat(v, "v")
    if ldk != ldv:
        raise ValueError("k and v must share one row stride")
    po, ldo = _mat(o, "o")
    scale = 1.0 / float(np.sqrt(head_dim)) if scale is None else float(scale)
    _check(load().nt_cross_attention(q_layout.handle, kv_layout.handle, int(heads), int(head_dim), pq, ldq, pk, pv,
                                     ldk, scale, po, ldo, _dtype(q), _stream()))
    return o


def triangle_workspace_bytes(layout: NestedLayout, C_: int, operands: str = "packed", dtype: str = "bf16") -> int:
    n = C.c_uint64()
    _check(load().nt_triangle_mul_workspace(layout.handle, int(C_), TRI_OPERANDS[operands],
                                            NT_BF16 if dtype == "bf16" else NT_F32, C.byref(n)))
    return int(n.value)


def nt_triangle_mul(layout: NestedLayout, direction: int, a, b, z, operands: str = "packed", workspace=None):
    """operands "packed": a, b are [sum N^2, C] pair tensors (row stride shared);
    "pair_tiled" / "pair_tiled_t": pair-tiled channel-major planes [C, >= sum_pad]."""
    pz, ldz = _mat(z, "z")
    Cz = int(z.size(1))
    if operands == "packed":
        pa, lda = _mat(a, "a")
        pb, ldb = _mat(b, "b")
        if lda != ldb:
            raise ValueError("a and b must share one row stride")
    else:
        pa, lda = _ptr(a), int(a.stride(0))
        pb = _ptr(b)
    if workspace is None:
        workspace = workspace_tensor(triangle_workspace_bytes(layout, Cz, operands, "bf16" if _dtype(z) == NT_BF16 else "f32"))
    pw, nw = _ws(workspace)
    _check(load().nt_triangle_mul(layout.handle, int(direction), Cz, pa, pb, lda, TRI_OPERANDS[operands], pz, ldz,
                                  _dtype(z), pw, nw, _stream()))
    return z


def nt_triangle_mul_gated(layout: NestedLayout, direction: int, a, b, t, operands: str = "packed", workspace=None):
    """operands "packed": a, b are [sum N^2, >= 2C] rows of [projection | gate
    logits] (one row stride); "pair_tiled" / "pair_tiled_t": gated operands in
    pair-tiled planes [C, >= sum_pad].  t: [sum N^2, C], overwritten with the
    contraction of the gated operands."""
    pt, ldt = _mat(t, "t")
    Ct = int(t.size(1))
    if operands == "packed":
        pa, lda = _mat(a, "a")
        pb, ldb = _mat(b, "b")
        if lda != ldb:
            raise ValueError("a and b must share one row stride")
    else:
        pa, lda = _ptr(a), int(a.stride(0))
        pb = _ptr(b)
    if workspace is None:
        workspace = workspace_tensor(triangle_workspace_bytes(layout, Ct, operands, "bf16" if _dtype(t) == NT_BF16 else "f32"))
    pw, nw = _ws(workspace)
    _check(load().nt_triangle_mul_gated(layout.handle, int(direction), Ct, pa, pb, lda, TRI_OPERANDS[operands], pt,
                                        ldt, _dtype(t), pw, nw, _stream()))
    return t


def nt_segment_reduce(layout: NestedLayout, level: str, op: str, x, y):
    px, ldx = _mat(x, "x")
    py, ldy = _mat(y, "y")
    _check(load().nt_segment_reduce(layout.handle, LEVELS[level], {"sum": 0, "mean": 1}[op], int(x.size(1)),
                                    px, ldx, _dtype(x), py, ldy, _stream()))
    return y


# ---------------------------------------------------------------- backward
def nt_pair_broadcast_backward(layout: NestedLayout, dz, du=None, dv=None, accumulate: bool = False):
    """du[eta_i + a] = sum_b dz[a, b], dv[kappa_i + b] = sum_a dz[a, b]; du and
    dv share one dtype (fp32 or bf16)."""
    pz, ldz = _mat(dz, "dz")
    pu, ldu = _mat(du, "du") if du is not None else (None, int(dz.size(1)))
    pv, ldv = _mat(dv, "dv") if dv is not None else (None, int(dz.size(1)))
    outs = [t for t in (du, dv) if t is not None]
    if len(outs) == 2 and du.dtype != dv.dtype:
        raise ValueError("du and dv must share one dtype")
    out_dt = _dtype(outs[0]) if outs else NT_F32
    _check(load().nt_pair_broadcast_backward(layout.handle, int(dz.size(1)), pz, ldz, _dtype(dz), pu, ldu, pv, ldv,
                                             out_dt, int(accumulate), _stream()))
    return du, dv


def loss_workspace_bytes(layout: NestedLayout) -> int:
    n = C.c_uint64()
    _check(load().nt_weighted_square_loss_workspace(layout.handle, C.byref(n)))
    return int(n.value)


def nt_weighted_square_loss(layout: NestedLayout, level: str, x, weights, scale: float, loss, dx=None,
                            workspace=None):
    """loss[i] = scale * weights[i] * ||x_i||^2 (device fp32 [B]); dx = 2 scale w_i x."""
    px, ldx = _mat(x, "x")
    pdx, lddx = _mat(dx, "dx") if dx is not None else (None, int(x.size(1)))
    if workspace is None:
        workspace = workspace_tensor(loss_workspace_bytes(layout))
    pw, nw = _ws(workspace)
    _check(load().nt_weighted_square_loss(layout.handle, LEVELS[level], int(x.size(1)), px, ldx, _dtype(x),
                                          _ptr(weights), float(scale), _ptr(loss), pdx, lddx,
                                          _dtype(dx) if dx is not None else NT_F32, pw, nw, _stream()))
    return loss


def nt_segment_reduce_backward(layout: NestedLayout, level: str, op: str, dy, dx, accumulate: bool = False):
    py, ldy = _mat(dy, "dy")
    px, ldx = _mat(dx, "dx")
    _check(load().nt_segment_reduce_backward(layout.handle, LEVELS[level], {"sum": 0, "mean": 1}[op], int(dx.size(1)),
                                             py, ldy, px, ldx, _dtype(dx), int(accumulate), _stream()))
    return dx


def nt_triangle_mul_backward(layout: NestedLayout, direction: int, a, b, dt, da=None, db=None, workspace=None):
    """Packed operands [sum N^2, C]; da, db accumulate (either may be None)."""
    pa, lda = _mat(a, "a")
    pb, ldb = _mat(b, "b")
    if lda != ldb:
        raise ValueError("a and b must share one row stride")
    pt, ldt = _mat(dt, "dt")
    pda, ldda = _mat(da, "da") if da is not None else (None, 0)
    pdb, lddb = _mat(db, "db") if db is not None else (None, 0)
    if da is not None and db is not None and ldda != lddb:
        raise ValueError("da and db must share one row stride")
    ld_dab = ldda if da is not None else (lddb if db is not None else int(dt.size(1)))
    Cz = int(dt.size(1))
    dt_ = "bf16" if _dtype(dt) == NT_BF16 else "f32"
    if workspace is None:
        workspace = workspace_tensor(triangle_workspace_bytes(layout, Cz, "packed", dt_))
    pw, nw = _ws(workspace)
    _check(load().nt_triangle_mul_backward(layout.handle, int(direction), Cz, pa, pb, lda, pt, ldt, pda, pdb, ld_dab,
                                           _dtype(dt), pw, nw, _stream()))
    return da, db


def nt_layernorm_linear_backward(x, w, dy, ln=None, eps: float = 1e-5, bias=None, epilogue: str = "none",
                                 w2=None, hidden: int = 0, residual_is_x: bool = True, dx=None,
                                 accumulate_dx: bool = False, dw=None, db=None, dgamma=None, dbeta=None, dw2=None,
                                 db2=None, workspace=None, overwrite_weights: bool = False):
    """Gradients of y = epilogue(LN(x) W^T + b) given dy; weight gradients (fp32)
    accumulate, dx is overwritten unless accumulate_dx."""
    a = LinearBwdArgs()
    px, ldx = _mat(x, "x")
    a.rows, a.c_in = int(x.size(0)), int(x.size(1))
    a.c_out = int(dy.size(1))
    a.x, a.ldx, a.x_dtype = px, ldx, _dtype(x)
    if ln is not None:
        a.ln_gamma, a.ln_beta = _ptr(ln[0]), _ptr(ln[1])
    a.ln_eps = eps
    a.w, a.bias, a.epilogue = _ptr(w), _ptr(bias), EPILOGUES[epilogue]
    a.hidden, a.w2, a.residual_is_x = int(hidden), _ptr(w2), int(bool(residual_is_x))
    a.dy, a.ld_dy = _mat(dy, "dy")
    if dx is not None:
        a.dx, a.ld_dx = _mat(dx, "dx")
        a.dx_dtype = _dtype(dx)
    else:
        a.dx, a.ld_dx, a.dx_dtype = None, a.c_in, NT_BF16
    a.accumulate_dx = int(bool(accumulate_dx))
    a.overwrite_weights = int(bool(overwrite_weights))
    a.dw, a.db, a.dgamma, a.dbeta = _ptr(dw), _ptr(db), _ptr(dgamma), _ptr(dbeta)
    a.dw2, a.db2 = _ptr(dw2), _ptr(db2)
    if workspace is None:
        n = C.c_uint64()
        _check(load().nt_layernorm_linear_backward_workspace(C.byref(a), C.byref(n)))
        workspace = workspace_tensor(int(n.value))
    a.workspace, a.workspace_bytes = _ws(workspace)
    _check(load().nt_layernorm_linear_backward(C.byref(a), _stream()))
    return dx


def attention_backward_workspace_bytes(layout: NestedLayout, axis: int, heads: int, head_dim: int,
                                       dtype: str = "bf16") -> int:
    n = C.c_uint64()
    _check(load().nt_pair_row_attention_backward_workspace(layout.handle, int(axis), int(heads), int(head_dim),
                                                           NT_BF16 if dtype == "bf16" else NT_F32, C.byref(n)))
    return int(n.value)


def nt_pair_row_attention_backward(layout: NestedLayout, axis: int, heads: int, head_dim: int, q, k, v, dout,
                                   dq, dk, dv, bias=None, dbias=None, scale: float | None = None,
                                   bias_layout: str = "cells", workspace=None):
    """dq, dk, dv (bf16, one row stride) overwritten; dbias fp32 [sum N^2, H]
    (bias_layout "cells") or [H, ld] ("heads"), overwritten."""
    pq, ld = _mat(q, "q")
    pk, ldk = _mat(k, "k")
    pv, ldv = _mat(v, "v")
    if not (ld == ldk == ldv):
        raise ValueError("q, k and v must share one row stride")
    pg, ldg = _mat(dout, "dout")
    pdq, ldd = _mat(dq, "dq")
    pdk, ldk2 = _mat(dk, "dk")
    pdv, ldv2 = _mat(dv, "dv")
    if not (ldd == ldk2 == ldv2):
        raise ValueError("dq, dk and dv must share one row stride")

    def strides(t):
        if t is None:
            return None, 0, 0
        if bias_layout == "cells":
            return _ptr(t), int(t.stride(0)), 1
        return _ptr(t), 1, int(t.stride(0))

    pb, ldb, ldbh = strides(bias)
    pdb, lddb, lddbh = strides(dbias)
    scale = 1.0 / float(np.sqrt(head_dim)) if scale is None else float(scale)
    if workspace is None:
        workspace = workspace_tensor(attention_backward_workspace_bytes(layout, axis, heads, head_dim))
    pw, nw = _ws(workspace)
    _check(load().nt_pair_row_attention_backward(layout.handle, int(axis), int(heads), int(head_dim), pq, pk, pv, ld,
                                                 pb, ldb, ldbh, pg, ldg, scale, pdq, pdk, pdv, ldd,
                                                 pdb, lddb, lddbh, _dtype(q), pw, nw, _stream()))
    return dq, dk, dv, dbias


def version() -> str:
    return load().nt_version().decode()
