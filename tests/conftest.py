import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_sessionstart(session):
    """Build libkvio.so (hipcc cross-compiles for gfx950 without a GPU) if the
    tree has none yet; the package itself never builds and refuses to load
    without it."""
    lib = os.path.join(ROOT, "paper_2508_18572_amd", "libkvio.so")
    if not os.path.exists(lib):
        import importlib.util
        spec = importlib.util.spec_from_file_location(
            "kvio_build", os.path.join(ROOT, "paper_2508_18572_amd", "_build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD Instinct GPU (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def io_stream():
    """One transfer stream with a hardware queue of its own (a CU mask over all
    CUs), shared by every GPU test: ordinary streams share a few hardware queues
    round-robin and can serialise, and the runtime allows few masked streams
    per process.  Falls back to a torch stream if the runtime refuses."""
    import torch
    import paper_2508_18572_amd as kv
    try:
        n = torch.cuda.get_device_properties(0).multi_processor_count
        st = kv.Stream(list(range(n)))
    except kv.KvioError:
        yield torch.cuda.Stream()
        return
    yield st.torch
    st.close()
