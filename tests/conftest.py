import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# PyTorch ships its own HIP runtime.  Loading it before the library makes both use
# that one runtime (the library's libamdhip64.so.7 resolves to the copy already
# loaded); loaded the other way round, the process would hold two runtimes and
# PyTorch, used by some GPU tests for device memory, would find no device.
try:
    import torch  # noqa: F401
except Exception:  # CPU-only environments without PyTorch still run the CPU tests
    pass


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")
