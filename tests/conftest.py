import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size checks that take tens of seconds")


def relerr(got, ref):
    """max|got - ref| / max|ref| (complex moduli for complex input); if ref
    is all zeros, max|got - ref|. Real and complex arguments may not be
    mixed: a spectrum compared with a real array (or the other way round)
    would hide the imaginary part."""
    import numpy as np
    got = np.asarray(got)
    ref = np.asarray(ref)
    if np.iscomplexobj(got) != np.iscomplexobj(ref):
        raise AssertionError(f"real/complex mismatch: {got.dtype} against {ref.dtype}")
    dt = np.complex128 if np.iscomplexobj(ref) else np.float64
    got = got.astype(dt)
    ref = ref.astype(dt)
    if got.shape != ref.shape:
        raise AssertionError(f"shape {got.shape} != {ref.shape}")
    err = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    return err / scale if scale > 0 else err


@pytest.fixture(scope="session")
def gpu_lib():
    """The loaded HIP library; GPU tests fail loudly when it is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    from paper_1601_06815_amd import binding
    return binding.load()
