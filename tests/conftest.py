import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running parity case")


@pytest.fixture(scope="session")
def tiny_fit():
    """Tiny workload fitted by the oracle (float64) and rounded once to the
    float32 arrays the GPU receives."""
    import numpy as np
    import oracle as O
    from paper_2609_37842_amd import synth as S
    raw = S.tiny_raw()
    f = O.fit(raw["a"], raw["ds"], raw["mask"], S.TINY.damping, S.TINY.m, S.TINY.k)
    art = dict(Q_A=f["Q_A"].astype(np.float32), Q_S=f["Q_S"].astype(np.float32),
               eigvals=f["eigvals"].astype(np.float32), P=f["P"].astype(np.float32),
               damping=float(S.TINY.damping))
    return dict(raw=raw, fit=f, art=art)
