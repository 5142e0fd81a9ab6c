"""The single-pair-single training step (forward, joint diagnostic loss,
backward) on the GPU against the oracle's mechanism_step, for the square,
rectangular and non-leading (S = 3) workloads at full size.

Forward outputs are chained bf16 values (held to 2e-2 or two bf16 ulps, as
the other chained checks); the loss to a relative 1e-3; every gradient to the
normwise 1e-2 of the backward tests (bf16 operands, fp32 accumulation, the
oracle mirroring the GPU's bf16 storage points)."""
import numpy as np
import pytest

from oracle import blocks as OB
from paper_2609_30379_amd import synth
from tests.gpu_util import PARITY_LOG, check_chained, host
from tests.test_gpu_backward import check_grad

pytestmark = pytest.mark.gpu

MECH = ["mechanism_square_b8_n66_317_bf16", "mechanism_rect_b8_n66_307_m66_309_bf16",
        "mechanism_nonleading_s3_b8_n40_182_bf16"]


@pytest.mark.parametrize("wname", MECH)
def test_mechanism_training_step(wname):
    from paper_2609_30379_amd.blocks import MechanismRun
    w = synth.WORKLOADS[wname]
    run = MechanismRun(w)
    print(f"{wname}: rows {run.lengths} cols {run.cols}", flush=True)
    ls, lp, xt, pt = run.step()
    first = [host(t) for t in (ls, lp, xt, pt)] + [host(g) for g in run.grads.values()] + [host(run.dx)]
    ls, lp, xt, pt = run.step()                     # a second step must give the same bits
    again = [host(t) for t in (ls, lp, xt, pt)] + [host(g) for g in run.grads.values()] + [host(run.dx)]
    assert all(np.array_equal(a, b) for a, b in zip(first, again)), "the training step is not deterministic"
    if w.s_axis > 1:
        ref = OB.mechanism_step_nonleading(run.x_init, run.lengths, run.params, w.s_axis, dtype="bf16")
    else:
        ref = OB.mechanism_step(run.x_init, run.lengths, run.params, dtype="bf16", y=run.y_init, cols=run.cols)
    check_chained(host(xt), ref["xt"], f"{wname} xt")
    check_chained(host(pt), ref["pt"], f"{wname} pt")
    loss = float(host(ls).sum() + host(lp).sum())
    rel = abs(loss - ref["loss"]) / abs(ref["loss"])
    PARITY_LOG.append((f"{wname} loss {loss:.6g} vs {ref['loss']:.6g} (relative)", rel, 1e-3, ref["loss"]))
    assert rel <= 1e-3, (loss, ref["loss"])
    G = {k: host(v) for k, v in run.grads.items()}
    if not run.sep:
        Cp = w.c_z
        G["u.w"], G["v.w"] = G["uv.w"][:Cp], G["uv.w"][Cp:]
        G["u.b"], G["v.b"] = G["uv.b"][:Cp], G["uv.b"][Cp:]
    for name in run.params:
        check_grad(G[name], ref["d_" + name], f"{wname} d{name}")
    check_grad(host(run.dx), ref["dx"], f"{wname} dx")
    if run.rect:
        check_grad(host(run.dy), ref["dy"], f"{wname} dy")
