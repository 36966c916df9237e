import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="session")
def golden_dir():
    return GOLDEN


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Report the staged parity bookkeeping of the GPU tests (near-tie swaps
    and the recall of the GPU's tokens against the oracle's independent
    selection), when any GPU comparison ran."""
    harness = sys.modules.get("gpu_harness")
    stats = getattr(harness, "PARITY_STATS", None) if harness else None
    if not stats:
        return
    tr = terminalreporter
    tr.section("staged parity: near-tie swaps and token recall vs the independent oracle selection")
    for label, st in sorted(stats.items()):
        mean = st["recall_sum"] / st["units"] if st["units"] else 1.0
        tr.write_line(f"{label}: {st['units']} units, {st['block_swap_units']} with a block near-tie swap, "
                      f"{st['token_swap_units']} with a token near-tie swap, recall mean {mean:.5f} "
                      f"min {st['recall_min']:.5f}")
