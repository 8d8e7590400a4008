import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line(
        "markers", "slow: long statistical checks (run with -m slow)")


def pytest_collection_modifyitems(config, items):
    # Statistical checks are opt-in: skip them unless "slow" is selected.
    markexpr = config.getoption("-m") or ""
    if "slow" in markexpr:
        return
    skip = pytest.mark.skip(reason="slow statistical check; select with -m slow")
    for item in items:
        if "slow" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """The parity margins of the session: the largest score, summary and
    output errors the oracle checks saw, the band swaps, and the tolerances
    they were held to. Also written as JSON to $RADAR_MARGINS_OUT when set."""
    import json
    h = sys.modules.get("_harness")
    if h is None or not h.MARGINS["episodes"]:
        return
    M = h.MARGINS
    terminalreporter.write_line(
        "parity margins: " + ", ".join(
            f"{k}={v:.3g}" if isinstance(v, float) else f"{k}={v}"
            for k, v in M.items() if k != "tolerances")
        + " | tolerances: " + json.dumps(M["tolerances"]))
    path = os.environ.get("RADAR_MARGINS_OUT")
    if path:
        with open(path, "w") as f:
            json.dump(M, f, indent=1)
