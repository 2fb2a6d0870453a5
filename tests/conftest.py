import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads (minutes of host work)")


@pytest.fixture(scope="session")
def rng():
    import numpy as np
    return np.random.Generator(np.random.PCG64(12345))


@pytest.fixture(scope="session")
def flowmoe_lib():
    """The built libflowmoe (built in-tree first if it is missing)."""
    from paper_2510_00207_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2510_00207_amd import build
        build.build(verbose=False)
    return _lib.load()


def pytest_sessionfinish(session, exitstatus):
    """Write the error measures of every parity comparison of the session
    (max-normalised and element-wise) to parity_report.tsv in the output
    folder (FLOWMOE_REPORT_DIR, default: the folder that a remote run copies
    back)."""
    mod = sys.modules.get("gpu_helpers")
    rep = getattr(mod, "REPORT", None) if mod is not None else None
    if not rep:
        return
    out = os.environ.get("FLOWMOE_REPORT_DIR") or os.path.join(ROOT, "gpurun_out")
    os.makedirs(out, exist_ok=True)
    with open(os.path.join(out, "parity_report.tsv"), "w") as f:
        f.write("test\tquantity\tdtype\tmax_rel_err\telem_rel_err\n")
        for test, what, dt, e1, e2 in rep:
            f.write(f"{test}\t{what}\t{dt}\t{e1:.3e}\t{e2:.3e}\n")
