import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def tbn():
    """The product binding; fails loudly when the HIP library is missing."""
    if not gpu_available():
        pytest.skip("no GPU visible")
    import paper_1701_00485_amd as tbn_mod
    tbn_mod.load()  # raises if libtbn.so is absent or does not load
    return tbn_mod


@pytest.fixture
def knobs(tbn):
    """Setter of the library's test and tuning knobs (include/tbn_tuning.h) for one test;
    every knob is restored to its previous value afterwards."""
    saved = {k: tbn.tuning_get(k) for k in tbn.KNOBS}

    def set_knobs(**kw):
        for k, v in kw.items():
            tbn.tuning_set(k, v)

    yield set_knobs
    for k, v in saved.items():
        tbn.tuning_set(k, v)
