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
    # the tests' torch CPU work is small convolutions: one thread each keeps parallel test
    # workers from oversubscribing the cores
    import torch
    torch.set_num_threads(1)


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    stale = (not os.path.exists(oracle.LIB) or
             os.path.getmtime(oracle.LIB) < max(os.path.getmtime(oracle.SRC),
                                                os.path.getmtime(os.path.join(oracle.HERE,
                                                                              "avo.h"))))
    if stale:
        oracle.build()
    return oracle
