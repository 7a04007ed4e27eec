import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    # DMS_TEST_LIBRARY: run the tests against another build of libdms (the
    # host-sanitizer build of tests/test_abi_sanitized.py)
    alt = os.environ.get("DMS_TEST_LIBRARY")
    if alt:
        from paper_2506_05345_amd import dms
        dms.LIB_PATH = alt
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_collection_modifyitems(config, items):
    # GPU tests cannot run without a device; keep them collected but skipped
    # so that "-m gpu" on a GPU machine runs them and CPU runs stay green.
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU in this environment")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
