"""The allocation-free attention entry point against the workspace entry
point, through the C ABI: two calls in a row (the second on a smaller input)
must give the bits the workspace call gives, and a request beyond the scratch
array is rejected before any work."""
import numpy as np
import pytest

from oracle import ops as O
from paper_2609_30379_amd import synth
from tests.gpu_util import check, dev, host

pytestmark = pytest.mark.gpu


def _inputs(L, H, D, seed):
    R = sum(n * n for n in L)
    qkv = synth.normal(seed, "noalloc_qkv", (R, 3 * H * D), 1.0, "bf16")
    bias = synth.normal(seed, "noalloc_bias", (R, H), 1.0, "bf16")
    return qkv, bias


@pytest.fixture(scope="module")
def B():
    from paper_2609_30379_amd import binding
    binding.load()
    return binding


def test_noalloc_matches_workspace_entry_point_twice(B):
    import torch
    cases = [([259, 278, 395, 489, 48, 101, 427, 488], 0, 4, "cells"),   # bias image 8.2 MiB
             ([37, 5, 64, 1, 0, 120], 1, 2, "heads")]                      # then a smaller input
    for L, axis, H, bias_layout in cases:
        D = 32
        lay = B.NestedLayout(L)
        qkv, bias = _inputs(L, H, D, 50 + axis)
        c = H * D
        qd = dev(qkv, "bf16")
        bd = dev(bias, "bf16") if bias_layout == "cells" else dev(np.ascontiguousarray(bias.T), "bf16")
        R = qkv.shape[0]
        o_ws = torch.full((R, c), float("nan"), dtype=torch.bfloat16, device="cuda")
        o_na = torch.full((R, c), float("nan"), dtype=torch.bfloat16, device="cuda")
        B.nt_pair_row_attention(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o_ws, bias=bd,
                                bias_layout=bias_layout)
        B.nt_pair_row_attention_noalloc(lay, axis, H, D, qd[:, :c], qd[:, c:2 * c], qd[:, 2 * c:], o_na, bias=bd,
                                        bias_layout=bias_layout)
        torch.cuda.synchronize()
        print(f"noalloc lengths={L} axis={axis} H={H}", flush=True)
        assert torch.equal(o_na, o_ws), "allocation-free call differs from the workspace call"
        # and the oracle on the shortest nonempty sample of the batch
        i = min((j for j, n in enumerate(L) if n), key=lambda j: L[j])
        cu = np.concatenate([[0], np.cumsum([n * n for n in L])])
        sl = slice(int(cu[i]), int(cu[i + 1]))
        ref = O.pair_row_attention(qkv[sl, :c], qkv[sl, c:2 * c], qkv[sl, 2 * c:], bias[sl], [L[i]], H, D, axis=axis)
        check(host(o_na)[sl], ref, "bf16", f"allocation-free attention sample N={L[i]} axis {axis}")


def test_noalloc_rejects_requests_beyond_its_scratch(B):
    import torch
    L = synth.lengths_for(synth.WORKLOADS["tokens_b64_lognormal230_bf16"]).tolist()   # bias image 44 MiB at 4 heads
    lay = B.NestedLayout(L)
    small = torch.zeros((8, 3 * 128), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((8, 128), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros((8, 4), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.NtError) as e:
        B.nt_pair_row_attention_noalloc(lay, 0, 4, 32, small[:, :128], small[:, 128:256], small[:, 256:], o, bias=b)
    assert e.value.status == B.NT_ERR_UNSUPPORTED and "scratch" in str(e.value)
