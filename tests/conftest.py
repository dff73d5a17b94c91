import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: larger CPU case")


def pytest_collection_modifyitems(config, items):
    # GPU tests run only where a GPU is visible; everything else runs anywhere.
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter):
    """Totals of the int4 code comparisons made in this run (tests/parity.py)."""
    parity = sys.modules.get("tests.parity")
    if parity is None or not parity.STATS["elements"]:
        return
    s = parity.STATS
    terminalreporter.write_line(
        "int4 code parity: {elements} elements, {mismatches} mismatches ({frac:.2e}), "
        "{mismatches_beyond_1ulp} of them beyond 1 fp32 ulp of the boundary; {within_1ulp} elements within "
        "1 ulp of a boundary; max |r_gpu - r_exact| = {max_ratio_err_ulp:.1f} ulp over {ratio_elements} "
        "ratios".format(frac=s["mismatches"] / s["elements"], **s))
