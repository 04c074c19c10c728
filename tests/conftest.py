import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    # Many cases use shapes the matrix-core kernels do not take on purpose
    # (odd K, few channels, fp32 attention); they check uses_mfma /
    # tuned_limit themselves, so the binding's warning is noise here.
    config.addinivalue_line("filterwarnings",
                            "ignore::paper_2607_20501_amd.mk.TunedLimitWarning")


@pytest.fixture(scope="session")
def has_gpu():
    import torch
    return torch.cuda.is_available()
