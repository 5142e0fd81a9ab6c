"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every declared symbol, host-only layouts match the oracle's offsets bit
for bit, the work maps cover every item exactly once with balanced XCD loads,
and argument errors are reported before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import layout as OL
from paper_2609_30379_amd import binding as B
from paper_2609_30379_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return B.load()


def test_exports_every_declared_symbol(lib):
    hdr = open(os.path.join(ROOT, "include", "nt.h")).read()
    names = set(re.findall(r"^\s*(?:nt_status|int32_t|const char\*)\s+(nt_\w+)\s*\(", hdr, re.M))
    assert len(names) >= 12
    for n in sorted(names):
        assert hasattr(lib, n), f"libnt.so does not export {n}"
    assert B.version().startswith("nt-mi355x")


LENGTH_CASES = [[2, 3], [15, 12, 10, 7], [5, 0, 1, 37, 64, 3, 70], [0], [1], [0, 0, 4]]


@pytest.mark.parametrize("L", LENGTH_CASES + [synth.lengths_for(w).tolist() for w in synth.WORKLOADS.values()])
def test_host_layout_matches_oracle(L):
    lay = B.NestedLayout(L, host_only=True)
    assert lay.host_array("lengths").tolist() == list(L)
    assert lay.host_array("cu_seqlens").tolist() == OL.single_offsets(L).tolist()
    assert lay.host_array("cu_pairs").tolist() == OL.pair_offsets(L).tolist()
    assert lay.host_array("row_splits2").tolist() == OL.pair_row_splits(L)[1].tolist()
    plane = [(-(-n // 16) * 16) * (-(-n // 32) * 32) for n in L]     # pair-tiled plane extents
    assert lay.host_array("cu_pad").tolist() == OL.offsets(plane).tolist()
    rs = lay.host_array("row_sample")
    assert rs.tolist() == [i for i, n in enumerate(L) for _ in range(n)]
    assert (lay.sum_n, lay.sum_n2, lay.sum_n3) == (sum(L), sum(n * n for n in L), sum(n ** 3 for n in L))
    assert lay.max_len == max(L)


def _xcd_loads(items, cost):
    loads = np.zeros(8)
    for p, it in enumerate(items):
        if it[0] >= 0:
            loads[p % 8] += cost(it)
    return loads


@pytest.mark.parametrize("L", [[15, 12, 10, 7], [259, 278, 395, 489, 48, 101, 427, 488], [5, 0, 1, 37, 64, 3, 70],
                               synth.lengths_for(synth.WORKLOADS["pairformer4_b16_lognormal192_bf16"]).tolist()])
def test_work_maps_cover_each_item_once(L):
    lay = B.NestedLayout(L, host_only=True)
    att = lay.host_array("attn_work").reshape(-1, 2)
    assert len(att) % 8 == 0
    got = sorted(map(tuple, att[att[:, 0] >= 0].tolist()))
    assert got == sorted((i, r) for i, n in enumerate(L) for r in range(n))
    tri = lay.host_array("tri_work").reshape(-1, 4)
    assert len(tri) % 8 == 0
    got = sorted(map(tuple, tri[tri[:, 0] >= 0, :3].tolist()))
    T = 64
    assert got == sorted((i, x, y) for i, n in enumerate(L) for x in range(-(-n // T)) for y in range(-(-n // T)))
    # a sample's tiles are contiguous, in bands of two tile rows walked column
    # by column, and carry the index of its first tile
    for j, (i, x, y, first) in enumerate(tri.tolist()):
        if i < 0:
            continue
        nt = -(-L[i] // T)
        xb = x - x % 2
        pos = xb * nt + y * min(2, nt - xb) + (x - xb)
        assert first == j - pos and tri[first, 0] == i and tri[first, 1] == 0 and tri[first, 2] == 0
    seq = lay.host_array("seq_work").reshape(-1, 2)
    got = sorted(map(tuple, seq[seq[:, 0] >= 0].tolist()))
    assert got == sorted((i, q) for i, n in enumerate(L) for q in range(-(-n // 64)))
    # balanced XCD loads: no XCD above the mean by more than one sample's largest item
    loads = _xcd_loads(att.tolist(), lambda it: L[it[0]] ** 2)
    assert loads.max() - loads.mean() <= max(L) ** 2 + 1e-9
    # the triangle tile map is cut into 8 contiguous XCD ranges whose costs
    # (32-wide k-steps + 2 per tile) are within one tile of the mean
    split = lay.host_array("tri_split")
    assert len(split) == 9 and split[0] == 0 and split[-1] == len(tri) and np.all(np.diff(split) >= 0)
    cost = np.array([0 if i < 0 else -(-L[i] // 32) + 2 for i in tri[:, 0].tolist()], float)
    pre = np.concatenate([[0.0], np.cumsum(cost)])
    per = np.diff(pre[split])
    assert np.all(np.abs(per - pre[-1] / 8) <= cost.max() + 1e-9)


def test_uniform_batch_puts_each_sample_on_its_own_xcd():
    L = synth.lengths_for(synth.WORKLOADS["pair_b8_n208_224_bf16"]).tolist()
    att = B.NestedLayout(L, host_only=True).host_array("attn_work").reshape(-1, 2)
    xcd_samples = [set(att[p::8, 0].tolist()) - {-1} for p in range(8)]
    assert all(len(s) <= 2 for s in xcd_samples)


def test_layout_errors():
    with pytest.raises(B.NtError) as e:
        B.NestedLayout([3, -1], host_only=True)
    assert e.value.status == B.NT_ERR_INVALID_ARG
    with pytest.raises(B.NtError) as e:
        B.NestedLayout([46341], host_only=True)            # 46341^2 > INT32_MAX
    assert e.value.status == B.NT_ERR_OVERFLOW
    with pytest.raises(B.NtError) as e:
        B.NestedLayout([], host_only=True)
    assert e.value.status == B.NT_ERR_INVALID_ARG
    with pytest.raises(B.NtError) as e:
        B.NestedLayout([0, 3, 2], host_only=True, offsets=True)   # decreasing offsets
    assert e.value.status == B.NT_ERR_INVALID_ARG
    with pytest.raises(B.NtError):
        B.NestedLayout([1, 3, 5], host_only=True, offsets=True)   # o_0 != 0
    lay = B.NestedLayout([0, 2, 5], host_only=True, offsets=True)
    assert lay.host_array("lengths").tolist() == [2, 3]


def test_compatibility_distinguishes_equal_totals():
    # (3,4) and (4,3) hold the same 7 singles and 25 pair cells but differ per sample
    a = B.NestedLayout([3, 4], host_only=True)
    b = B.NestedLayout([4, 3], host_only=True)
    c = B.NestedLayout([3, 4], host_only=True)
    assert (a.sum_n, a.sum_n2) == (b.sum_n, b.sum_n2)
    assert not a.compatible(b)
    assert a.compatible(c)


def _linear_args(**kw):
    a = B.LinearArgs()
    a.rows, a.c_in, a.c_out, a.dtype, a.x_dtype = 16, 16, 16, B.NT_BF16, B.NT_BF16
    a.x, a.w, a.y = C.c_void_p(0x1000), C.c_void_p(0x2000), C.c_void_p(0x3000)
    a.ldx, a.ldy = 16, 16
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def test_op_argument_errors_need_no_device(lib):
    host = B.NestedLayout([3, 4], host_only=True)
    other = B.NestedLayout([4, 3], host_only=True)
    # op calls reject host-only layouts before touching the device
    st = lib.nt_pair_broadcast(host.handle, 8, C.c_void_p(16), 8, C.c_void_p(16), 8, C.c_void_p(16), 8, 0, B.NT_BF16, None)
    assert st == B.NT_ERR_INVALID_ARG and b"host-only" in lib.nt_last_error()
    st = lib.nt_triangle_mul(host.handle, 0, 32, None, None, 0, 1, None, 32, B.NT_BF16, None, 0, None)
    assert st == B.NT_ERR_INVALID_ARG
    st = lib.nt_segment_reduce(None, 1, 0, 8, None, 8, B.NT_BF16, None, 8, None)
    assert st == B.NT_ERR_INVALID_ARG
    # LayerNorm+Linear validation
    cases = [
        (dict(c_in=12), B.NT_ERR_INVALID_ARG),                            # K not a multiple of 8
        (dict(epilogue=7), B.NT_ERR_INVALID_ARG),
        (dict(x=C.c_void_p(0x1002)), B.NT_ERR_INVALID_ARG),               # misaligned
        (dict(epilogue=1), B.NT_ERR_INVALID_ARG),                         # residual missing
        (dict(epilogue=2, hidden=64, w2=C.c_void_p(0x4000), c_in=96, c_out=96, ldx=96, ldy=96), B.NT_ERR_UNSUPPORTED),
        (dict(n_tail=4, y_tail=C.c_void_p(0x5000), ld_tail=16, tail_layout=1), B.NT_ERR_UNSUPPORTED),
        (dict(rows=25, layout=host.handle, level=1, residual_layout=other.handle,
              residual=C.c_void_p(0x6000), ld_residual=16, epilogue=1), B.NT_ERR_LAYOUT_MISMATCH),
        (dict(rows=24, layout=host.handle, level=1), B.NT_ERR_LAYOUT_MISMATCH),
        (dict(dtype=B.NT_F32, x_dtype=B.NT_BF16), B.NT_ERR_INVALID_ARG),
        (dict(ldy=4), B.NT_ERR_INVALID_ARG),
        # broadcast rows: both sources, x NULL, a pair layout with device mirrors
        (dict(bcast_u=C.c_void_p(0x7000), ld_bcast_u=16), B.NT_ERR_INVALID_ARG),
        (dict(bcast_u=C.c_void_p(0x7000), bcast_v=C.c_void_p(0x8000), ld_bcast_u=16, ld_bcast_v=16),
         B.NT_ERR_INVALID_ARG),                                          # x set
        (dict(x=None, bcast_u=C.c_void_p(0x7000), bcast_v=C.c_void_p(0x8000), ld_bcast_u=16, ld_bcast_v=16,
              rows=25, layout=host.handle, level=1), B.NT_ERR_INVALID_ARG),   # host-only layout
        # gated residual: needs residual and gate, no tail; a gate needs that epilogue
        (dict(epilogue=4, residual=C.c_void_p(0x6000), ld_residual=16), B.NT_ERR_INVALID_ARG),
        (dict(epilogue=4, gate=C.c_void_p(0x6000), ld_gate=16), B.NT_ERR_INVALID_ARG),
        (dict(epilogue=4, residual=C.c_void_p(0x6000), ld_residual=16, gate=C.c_void_p(0x9000), ld_gate=12),
         B.NT_ERR_INVALID_ARG),                                          # ld_gate not a multiple of 8
        (dict(epilogue=4, residual=C.c_void_p(0x6000), ld_residual=16, gate=C.c_void_p(0x9000), ld_gate=16,
              n_tail=4, y_tail=C.c_void_p(0x5000), ld_tail=16), B.NT_ERR_UNSUPPORTED),
        (dict(gate=C.c_void_p(0x9000), ld_gate=16), B.NT_ERR_INVALID_ARG),
        (dict(epilogue=5), B.NT_ERR_UNSUPPORTED),                        # sigmoid GLU outside its one shape
        (dict(epilogue=6), B.NT_ERR_INVALID_ARG),
    ]
    for kw, want in cases:
        a = _linear_args(**kw)
        assert lib.nt_layernorm_linear(C.byref(a), None) == want, (kw, lib.nt_last_error())
    # attention validation
    dev = B.NestedLayout([2, 3], host_only=True)
    assert lib.nt_pair_row_attention(dev.handle, 0, 4, 32, None, None, None, 384, None, 0, 0, 1.0, None, 128,
                                     B.NT_BF16, None, 0, None) == B.NT_ERR_INVALID_ARG    # host-only layout
    # cross-attention validation: batch mismatch, head_dim, key length, host-only layouts
    lq, lk = B.NestedLayout([2, 3], host_only=True), B.NestedLayout([4, 0, 1], host_only=True)
    lk2 = B.NestedLayout([4, 600], host_only=True)
    ca = lambda a, b, H, D, dt: lib.nt_cross_attention(a.handle, b.handle, H, D, C.c_void_p(16), 64, C.c_void_p(16),  # noqa: E731
                                                        C.c_void_p(16), 64, 1.0, C.c_void_p(16), 64, dt, None)
    assert ca(lq, lk, 2, 32, B.NT_BF16) == B.NT_ERR_LAYOUT_MISMATCH
    assert ca(lq, lk2, 2, 32, B.NT_BF16) == B.NT_ERR_UNSUPPORTED          # more than 512 keys in bf16
    assert ca(lq, lq, 2, 16, B.NT_BF16) == B.NT_ERR_UNSUPPORTED           # head_dim 16 in bf16
    assert ca(lq, lq, 4, 32, B.NT_BF16) == B.NT_ERR_INVALID_ARG           # H*d beyond the row strides
    assert ca(lq, lk2, 2, 32, B.NT_F32) == B.NT_ERR_INVALID_ARG           # fp32 allows it; host-only layout


def _q(fn, *args):
    n = C.c_uint64()
    assert fn(*args, C.byref(n)) == B.NT_OK
    return int(n.value)


def test_workspace_queries_and_missing_workspace_is_an_error(lib):
    """Ops take scratch memory only from the caller: the queries return its
    size from sizes alone, and a call that needs scratch but is given none (or
    too little) returns NT_ERR_INVALID_ARG instead of allocating."""
    L = [222, 208, 33, 0, 1]
    lay = B.NestedLayout(L, host_only=True)
    tiles = sum(-(-n // 16) * (-(-n // 64) * 4) for n in L)
    # pair attention, bf16, d = 32, N <= 512, with a bias: the bias image
    assert _q(lib.nt_pair_row_attention_workspace, lay.handle, 0, 4, 32, B.NT_BF16, 1) == 4 * tiles * 512
    assert _q(lib.nt_pair_row_attention_workspace, lay.handle, 1, 3, 32, B.NT_BF16, 1) == 3 * tiles * 512
    assert _q(lib.nt_pair_row_attention_workspace, lay.handle, 0, 4, 32, B.NT_BF16, 0) == 0
    assert _q(lib.nt_pair_row_attention_workspace, lay.handle, 2, 12, 64, B.NT_BF16, 0) == 0
    assert _q(lib.nt_pair_row_attention_workspace, lay.handle, 0, 2, 8, B.NT_F32, 1) == 0
    long = B.NestedLayout([600, 3], host_only=True)           # past 512: the per-row kernel reads the bias directly
    assert _q(lib.nt_pair_row_attention_workspace, long.handle, 0, 4, 32, B.NT_BF16, 1) == 0
    # triangle: packed operands are re-tiled into the workspace, tiled ones need none
    ldp = -(-lay.sum_pad // 8) * 8
    assert _q(lib.nt_triangle_mul_workspace, lay.handle, 128, 0, B.NT_BF16) == 2 * 128 * ldp * 2
    assert _q(lib.nt_triangle_mul_workspace, lay.handle, 16, 0, B.NT_F32) == 2 * 16 * ldp * 4
    assert _q(lib.nt_triangle_mul_workspace, lay.handle, 128, 1, B.NT_BF16) == 0
    # LayerNorm+Linear: large-K rows with a LayerNorm, and the SwiGLU transition
    a = _linear_args(rows=600, c_in=768, c_out=2304, ldx=768, ldy=2304, ln_gamma=C.c_void_p(0x9000))
    assert _q(lib.nt_layernorm_linear_workspace, C.byref(a)) == 600 * 768 * 2
    a = _linear_args(rows=600, c_in=768, c_out=2304, ldx=768, ldy=2304)           # no LayerNorm: none
    assert _q(lib.nt_layernorm_linear_workspace, C.byref(a)) == 0
    a = _linear_args(rows=1000, c_in=128, c_out=128, ldx=128, ldy=128, epilogue=2, hidden=512,
                     w2=C.c_void_p(0xa000), ln_gamma=C.c_void_p(0x9000))
    assert _q(lib.nt_layernorm_linear_workspace, C.byref(a)) == 3 * 512 * 128 * 2
    a = _linear_args(rows=1000, c_in=128, c_out=128, ldx=128, ldy=128, ln_gamma=C.c_void_p(0x9000))
    assert _q(lib.nt_layernorm_linear_workspace, C.byref(a)) == 0
    # calls that need scratch and get none, or too little: an error, nothing enqueued
    a = _linear_args(rows=600, c_in=768, c_out=2304, ldx=768, ldy=2304, ln_gamma=C.c_void_p(0x9000))
    assert lib.nt_layernorm_linear(C.byref(a), None) == B.NT_ERR_INVALID_ARG
    assert b"workspace" in lib.nt_last_error()
    a.workspace, a.workspace_bytes = C.c_void_p(0xb000), 600 * 768 * 2 - 1
    assert lib.nt_layernorm_linear(C.byref(a), None) == B.NT_ERR_INVALID_ARG
    assert b"workspace" in lib.nt_last_error()
    st = lib.nt_pair_row_attention(lay.handle, 0, 4, 32, C.c_void_p(16), C.c_void_p(16), C.c_void_p(16), 384,
                                   C.c_void_p(16), 1, lay.sum_n2, 0.17, C.c_void_p(16), 128, B.NT_BF16, None, 0, None)
    assert st == B.NT_ERR_INVALID_ARG and b"workspace" in lib.nt_last_error()
    st = lib.nt_triangle_mul(lay.handle, 1, 128, C.c_void_p(16), C.c_void_p(16), 256, 0, C.c_void_p(16), 128,
                             B.NT_BF16, None, 0, None)
    assert st == B.NT_ERR_INVALID_ARG and b"workspace" in lib.nt_last_error()
    # with enough workspace the same calls get past the workspace check (and stop
    # at the host-only layout, still before any device work)
    st = lib.nt_triangle_mul(lay.handle, 1, 128, C.c_void_p(16), C.c_void_p(16), 256, 0, C.c_void_p(16), 128,
                             B.NT_BF16, C.c_void_p(0x10000), 2 * 128 * ldp * 2, None)
    assert st == B.NT_ERR_INVALID_ARG and b"host-only" in lib.nt_last_error()
    # a pair-tiled variant that does not match the direction
    st = lib.nt_triangle_mul(lay.handle, 1, 128, C.c_void_p(16), C.c_void_p(16), ldp, 1, C.c_void_p(16), 128,
                             B.NT_BF16, None, 0, None)
    assert st == B.NT_ERR_INVALID_ARG and b"transposed" in lib.nt_last_error()


@pytest.mark.parametrize("n", [1, 15, 16, 17, 33, 216])
def test_pair_tiled_plane_is_a_fragment_order_bijection(n):
    """The pair-tiled plane of an N x N matrix places every cell once inside the
    round_up(N,16) x round_up(N,32) extent, and the 8 consecutive k of (row r,
    k-group g) of a 16 x 32 tile form the 16-byte piece of lane g*16 + r%16."""
    from tests.gpu_util import _tiled_plane_index, pair_tiled, untile_pair
    idx = _tiled_plane_index(n, False)
    ext = (-(-n // 16) * 16) * (-(-n // 32) * 32)
    assert len(set(idx.tolist())) == n * n and idx.min() >= 0 and idx.max() < ext
    a, b = np.divmod(np.arange(n * n), n)
    tile_base = ((a // 16) * (-(-n // 32)) + b // 32) * 512
    lane = ((b % 32) // 8) * 16 + a % 16
    assert np.array_equal(idx, tile_base + lane * 8 + b % 8)
    t = _tiled_plane_index(n, True)
    assert np.array_equal(t.reshape(n, n).T, idx.reshape(n, n))
    x = np.random.default_rng(n).standard_normal((n * n + 9, 3))
    L = [n, 3]
    for tr in (False, True):
        assert np.array_equal(untile_pair(pair_tiled(x, L, tr, fill=np.nan), L, tr), x)


@pytest.mark.parametrize("n", [1, 15, 16, 17, 401408, 393216 + 3])
def test_workspace_tensor_holds_the_requested_bytes(n):
    t = B.workspace_tensor(n, device="cpu")
    assert t.numel() * t.element_size() == n and t.data_ptr() % 16 == 0
    assert B.workspace_tensor(0, device="cpu") is None


def test_linear_backward_rejects_misaligned_parameters(lib):
    """The backward reads the LayerNorm affine and the bias in 16-byte pieces:
    misaligned pointers are rejected before any device work."""
    base = dict(rows=64, c_in=128, c_out=128, x=C.c_void_p(0x1000), ldx=128, x_dtype=B.NT_BF16,
                w=C.c_void_p(0x2000), dy=C.c_void_p(0x3000), ld_dy=128, dx=C.c_void_p(0x4000), ld_dx=128,
                dx_dtype=B.NT_BF16, ln_gamma=C.c_void_p(0x5000), ln_beta=C.c_void_p(0x6000), ln_eps=1e-5,
                workspace=C.c_void_p(0x10000), workspace_bytes=1 << 30)
    for field in ("ln_gamma", "ln_beta", "bias"):
        a = B.LinearBwdArgs()
        for k, v in base.items():
            setattr(a, k, v)
        setattr(a, field, C.c_void_p(0x7004))
        st = lib.nt_layernorm_linear_backward(C.byref(a), None)
        assert st == B.NT_ERR_INVALID_ARG and b"aligned" in lib.nt_last_error(), field
