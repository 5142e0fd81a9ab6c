import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large CPU oracle runs")


@pytest.fixture(scope="session")
def torch_cpu():
    import torch
    torch.set_default_dtype(torch.float64)
    return torch


def pytest_collection_modifyitems(config, items):
    """GPU tests are skipped only when no GPU is present; on a GPU machine a missing
    HIP library makes them fail, never fall back."""
    if not any("gpu" in it.keywords for it in items):
        return
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU in this environment")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Prints every recorded parity comparison with its margin (error / bar)."""
    try:
        from tests.gpu_util import PARITY_LOG
    except Exception:
        return
    if not PARITY_LOG:
        return
    tr = terminalreporter
    tr.section(f"parity margins ({len(PARITY_LOG)} comparisons, error / bar)")
    for what, err, bar, amax in sorted(PARITY_LOG, key=lambda r: -r[1] / r[2]):
        tr.write_line(f"{err / bar:6.3f}  err {err:.3e}  bar {bar:.0e}  max|ref| {amax:.3g}  {what}")
    path = os.environ.get("NT_PARITY_LOG")
    if path:
        import json
        with open(path, "w") as f:
            json.dump([{"case": w, "error": e, "bar": b, "max_abs_ref": a} for w, e, b, a in PARITY_LOG], f, indent=0)
