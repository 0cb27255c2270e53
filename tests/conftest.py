import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Under tests/run_sanitized.py: load the ASan + UBSan builds of the library and
# of the oracle instead of the ordinary ones (before any test loads either).
if os.environ.get("MDGEMM_SANITIZED") == "1":
    from oracle import build_oracle
    from paper_2607_06881_amd import build as _build
    from paper_2607_06881_amd import mdgemm as _md

    _md.LIB_PATH = _build.SAN_LIB
    build_oracle.OUT = build_oracle.SAN_OUT


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def pytest_collection_modifyitems(config, items):
    # GPU tests are skipped (not failed) when no GPU is visible, e.g. in the build container.
    try:
        import torch

        have_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
