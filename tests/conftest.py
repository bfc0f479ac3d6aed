import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.build()
    return oracle


@pytest.fixture(scope="session")
def medium_bundle(orc):
    """The 1.2M-node pin-board workload with the oracle's neighbourhood table."""
    import synth
    wl = synth.WORKLOADS["medium"]
    data = synth.make_workload(wl)
    idx, cnt, wts, steps = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                                   wl.seed, wl.walks, wl.hops, wl.T)
    return {"wl": wl, "data": data, "idx": idx, "cnt": cnt, "wts": wts, "steps": steps}
