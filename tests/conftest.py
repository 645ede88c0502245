import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")


def _stale(lib, sources):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    return any(os.path.getmtime(s) > t for s in sources)


@pytest.fixture(scope="session")
def oracle_lib():
    """The fp64 oracle, compiled with gcc if missing or older than its source."""
    import oracle
    from oracle import build as obuild
    if _stale(obuild.LIB, [obuild.SRC]):
        obuild.build()
    return oracle


@pytest.fixture(scope="session")
def mocap_lib():
    """libmocap_attn; built for gfx950 here if it is missing (a CPU-side build step)."""
    from paper_2606_22968_amd import binding, build
    sources = [os.path.join(build.CSRC, f) for f in os.listdir(build.CSRC)]
    sources.append(os.path.join(build.INCLUDE, "mocap_attn.h"))
    if _stale(build.LIB, sources):
        build.build()
    return binding


@pytest.fixture(scope="session")
def gpu(mocap_lib):
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X; run them with -m gpu on the GPU machine")
    name = torch.cuda.get_device_properties(0).gcnArchName
    print(f"[gpu] device 0: {torch.cuda.get_device_name(0)} ({name})", flush=True)
    return torch.device("cuda:0")
