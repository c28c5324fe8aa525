import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session")
def c5_oracle():
    """The 31x31 workload (B=16, 128->128, 56x56, pad 15): its seeded inputs and
    the fp64 direct oracle's whole output y[16][128][56][56], computed once per
    session (a few seconds of BLAS on the host)."""
    from oracle.direct import direct_conv2d
    from paper_2102_13272_amd.workloads import WORKLOADS, make_workload
    L = WORKLOADS["c5_r31"].layers[0]
    x, (w,) = make_workload("c5_r31")
    return L, x, w, direct_conv2d(x, w, L.pad)
