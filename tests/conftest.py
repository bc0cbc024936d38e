import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def rocrand_philox(tmp_path_factory):
    """Path to a host executable running rocRAND's Philox4x32-10 (library pin)."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("rocrand") / "rocrand_philox"
    src = os.path.join(ROOT, "tests", "helpers", "rocrand_philox.cpp")
    subprocess.run([hipcc, "-O1", "-x", "hip", "--offload-host-only", "-o", str(out), src],
                   check=True, capture_output=True)
    return str(out)
