import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    import oracle
    if not os.path.exists(oracle._LIB):
        oracle.build()
    yield


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """The measured parity figures of the GPU tests, at the end of the run:
    the worst error of every state over all comparisons (fp32 states: the
    floored relative error; bf16 x: bf16 ulps; the outer momentum: relative
    to the outer parameters) and one line per full-size comparison."""
    gh = sys.modules.get("gpu_harness")
    if gh is None or not getattr(gh, "REPORT", None):
        return
    tr = terminalreporter
    tr.write_sep("-", f"parity figures ({len(gh.REPORT)} comparisons against the oracle)")
    worst = {}
    for label, d in gh.REPORT:
        for k, v in d.items():
            if v >= worst.get(k, (-1.0, ""))[0]:
                worst[k] = (v, label)
        if "full" in label:
            tr.write_line(label + ": " + " ".join(f"{k}={v:.2e}" for k, v in d.items()))
    tr.write_line("worst: " + " ".join(f"{k}={v:.2e}({lab})" for k, (v, lab) in sorted(worst.items())))
    out = os.path.join(ROOT, "gpurun_out")
    # only GPU comparisons are written (the CPU suite compares the harness with itself)
    if os.path.isdir(out) and any(not label.startswith("self") for label, _ in gh.REPORT) \
            and "torch" in sys.modules and sys.modules["torch"].cuda.is_available():
        import json
        with open(os.path.join(out, "parity_report.jsonl"), "w") as f:
            for label, d in gh.REPORT:
                f.write(json.dumps({"label": label, **d}) + "\n")
