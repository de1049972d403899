import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the C-ABI on the GPU)")


def pytest_sessionfinish(session, exitstatus):
    """Keep the parity runs' largest attention errors (and their fraction of
    the tolerance) as JSON when any ran: at BATON_MARGINS_OUT, else as
    parity_margins.json in the results folder the GPU runs hand back."""
    parity = sys.modules.get("tests.parity")
    if parity is not None:
        parity.write_margins(os.environ.get("BATON_MARGINS_OUT",
                                            os.path.join(ROOT, "gpurun_out", "parity_margins.json")))
