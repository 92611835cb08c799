import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _gpu_run(config) -> bool:
    """Does this run select GPU tests?  (-m gpu, or no mark filter at all.)"""
    expr = (config.getoption("markexpr", default="") or "").replace(" ", "")
    return "notgpu" not in expr


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP library")
    # the oracle's column energies of the full-size inputs run on worker
    # processes; they are started here, before this process touches the GPU
    if _gpu_run(config) and os.environ.get("RMM_ORACLE_WORKERS", "1") != "0":
        from tests import oracle_pool
        oracle_pool.start()


def pytest_unconfigure(config):
    mod = sys.modules.get("tests.oracle_pool")
    if mod is not None:
        mod.stop()
