import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size case (seconds to minutes of oracle time)")


@pytest.fixture(scope="session")
def lib():
    """The HIP library through its ctypes binding; GPU tests only."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU")
    from paper_2404_14712_amd import load
    return load()


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """One line per test with the worst per-tensor relative error it checked
    (max|gpu - oracle| / max|oracle|) against its bound, then the overall worst."""
    try:
        from helpers import RESULTS
    except ImportError:
        return
    if not RESULTS:
        return
    worst = {}
    for test, name, err, tol in RESULTS:
        key = test.split("[")[0]
        cur = worst.get(key)
        if cur is None or err / tol > cur[1] / cur[2]:
            worst[key] = (f"{test.split('::')[-1]} {name}", err, tol)
    tr = terminalreporter
    tr.write_sep("-", f"parity: worst tensor per test function ({len(RESULTS)} tensors checked)")
    for key in sorted(worst):
        what, err, tol = worst[key]
        tr.write_line(f"{key.split('::')[0].split('/')[-1]}: {what} {err:.2e} (bound {tol:.0e})")
    t, n, e, tol = max(RESULTS, key=lambda r: r[2] / r[3])
    tr.write_line(f"parity overall worst: {t.split('::')[-1]} {n} {e:.2e} (bound {tol:.0e}, ratio {e / tol:.2f})")
