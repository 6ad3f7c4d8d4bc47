import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    # GPU parity tests hand the oracle's per-unit work to CPU workers, forked
    # here while nothing has touched the GPU yet
    if "not gpu" not in (config.option.markexpr or "") and not config.option.collectonly:
        from tests import oracle_pool
        oracle_pool.start()


def pytest_unconfigure(config):
    from tests import oracle_pool
    oracle_pool.shutdown()
