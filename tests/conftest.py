import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: longer CPU oracle runs")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.build()
    return oracle


def pytest_terminal_summary(terminalreporter):
    """Flip counts of every MoE-layer check of the run: Q8_0(h) blocks that
    differ from the oracle's own choice (each within the valid set)."""
    try:
        from tests import moe_check
    except Exception:
        return
    if not moe_check.STATS:
        return
    # (the GDN and stack lines below are printed with the MoE checks)
    tr = terminalreporter
    tr.write_sep("-", "MoE-layer checks: Q8_0(h) flips / blocks, max |out - ref| / sum|terms|")
    for name, st in moe_check.STATS:
        tr.write_line(f"{st['flips']:4d} / {st['blocks']:6d}  {st['max_rel_err']:.2e}  {name}")
    import sys
    for name, mod in list(sys.modules.items()):
        if name.endswith("test_gpu_stack"):
            for T, nl, rel in getattr(mod, "DRIFT", []):
                tr.write_line(f"stack drift, {nl} layers, T = {T}: max over tokens of "
                              f"|x_gpu - x_oracle|_2 / |x_oracle|_2 = {rel:.3g}")
        if name.endswith("test_gpu_gdn"):
            for case, eo, es in getattr(mod, "REL", []):
                tr.write_line(f"gdn {case}: max error / bound: output {eo:.3g}, state {es:.3g}")
