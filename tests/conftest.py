import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950); runs the HIP library through its C ABI")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle.so")):
        oracle.build()
    return oracle


@pytest.fixture(scope="session")
def hcms():
    """The HIP binding on cuda:0; a missing library is an error, not a skip."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("gpu test collected without a visible GPU")
    import paper_2607_01817_amd as hcms_pkg
    hcms_pkg.load()          # raises if libhcms.so is missing
    return hcms_pkg
