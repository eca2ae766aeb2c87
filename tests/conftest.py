import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built libbnn.so")


def pytest_runtest_teardown(item, nextitem):
    """Kernel-selection options are per thread and outlive a test: put the
    library defaults back after every test that may have changed them."""
    from paper_1808_00209_amd import bnn
    if bnn._lib is not None:
        bnn.bnn_set_options()
