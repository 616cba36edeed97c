import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _gpu_present() -> bool:
    try:
        import torch
        return torch.cuda.is_available() and torch.cuda.device_count() > 0
    except Exception:
        return False


def pytest_collection_modifyitems(config, items):
    if any("gpu" in item.keywords for item in items) and not _gpu_present():
        skip = pytest.mark.skip(reason="no GPU device visible in this process")
        for item in items:
            if "gpu" in item.keywords:
                item.add_marker(skip)


def pytest_sessionfinish(session, exitstatus):
    """With PG_MARGINS_OUT set, writes the largest error-to-bar ratios that
    the step parity tests reached (per case and tensor) as JSON lines."""
    path = os.environ.get("PG_MARGINS_OUT")
    mod = sys.modules.get("test_gpu_parity") or sys.modules.get("tests.test_gpu_parity")
    if not path or mod is None or not getattr(mod, "MARGINS", None):
        return
    import json
    with open(path, "w") as f:
        for case, k, pr, dr in mod.MARGINS:
            f.write(json.dumps({"case": case, "tensor": k, "param_ratio": round(pr, 4),
                                "delta_ratio": round(dr, 4)}) + "\n")
