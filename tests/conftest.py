import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def pytest_collection_modifyitems(config, items):
    # GPU tests fail loudly when there is no GPU rather than silently passing:
    # they are deselected with -m "not gpu" on CPU-only machines.
    pass


@pytest.fixture(scope="session")
def gpu_lib():
    """The built HIP library on a GPU; fails (not skips) when either is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    import paper_2407_16847_amd as splat
    splat.load()  # raises if libsplat.so is not built
    return splat


# largest parity errors per workload, printed at the end of the run (also
# under -q) so that every GPU run reports the margins it passed with
_ERRORS = {}


@pytest.fixture(scope="session")
def record_errors():
    def record(name, values):
        _ERRORS[name] = dict(values)
    return record


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    if not _ERRORS:
        return
    terminalreporter.section("largest errors against the oracle")
    for name in sorted(_ERRORS):
        terminalreporter.write_line(
            f"{name}: " + ", ".join(f"{k} {v:.3e}" for k, v in _ERRORS[name].items()))
