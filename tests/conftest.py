import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    return oracle.load()


def pytest_collection_modifyitems(config, items):
    """GPU tests skip (with a reason) where no GPU is visible."""
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)


def pytest_terminal_summary(terminalreporter):
    """Worst parity margin of each GPU test family against the oracle (the
    tolerances are max-abs / rel-L2; a share of 1.0 would be at the bound)."""
    try:
        from tests import _gpu
    except Exception:
        return
    if not _gpu.MARGINS:
        return
    fam = {}
    for test, kv, ma, rl, what in _gpu.MARGINS:
        name = test.split("::")[-1].split("[")[0]
        tol_abs, tol_rel = _gpu.TOL[kv]
        f = fam.setdefault((name, kv), [0, 0.0, 0.0, "", 0.0, ""])
        f[0] += 1
        if ma / tol_abs > f[1]:
            f[1], f[3] = ma / tol_abs, what
        if rl / tol_rel > f[2]:
            f[2], f[5] = rl / tol_rel, what
            f[4] = rl
    tr = terminalreporter
    tr.write_sep("-", "parity margins vs the oracle (worst case per test; share of the bound)")
    for (name, kv), (n, fa, fr, wa, rl, wr) in sorted(fam.items()):
        tr.write_line(f"{name:<44s} {kv:<4s} n={n:<4d} max-abs {fa:5.3f}  rel-L2 {fr:5.3f} ({rl:.2e})  [{wr[:60]}]")
