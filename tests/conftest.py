import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
for _p in (ROOT, os.path.dirname(os.path.abspath(__file__))):
    if _p not in sys.path:
        sys.path.insert(0, _p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_collection_modifyitems(config, items):
    # GPU tests cannot run without a device; keep the CPU suite green anywhere.
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter):
    # how many W elements the parity tests let through on the update-size bar
    mod = sys.modules.get("parity_checks")
    if mod is None:
        return
    for kind, (calls, checked, through) in mod.cancel_tally.items():
        if not calls:
            continue
        cap = f"; cap {mod.CANCEL_CAP:.0e} per call" if kind == "bf16" else ""
        terminalreporter.write_line(
            f"W {kind}: {through} of {checked} checked elements passed through the update-size bar "
            f"({through / max(checked, 1):.2e}{cap}) over {calls} comparisons")
