import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _keep_freed_memory_mapped():
    """The fp64 oracle allocates many large temporaries; keep freed blocks in
    the process heap instead of returning them to the OS (first-touch page
    faults dominate its run time on some hosts).  Test infrastructure only."""
    try:
        import ctypes
        libc = ctypes.CDLL("libc.so.6")
        libc.mallopt(-3, 1 << 30)   # M_MMAP_THRESHOLD
        libc.mallopt(-1, 1 << 36)   # M_TRIM_THRESHOLD
    except Exception:
        pass


_keep_freed_memory_mapped()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def lib():
    """The HIP C-ABI library through its Python binding (loads the built .so)."""
    from paper_2609_35139_amd import binding
    return binding.load()
