import functools
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size cases (minutes on CPU)")


@functools.lru_cache(maxsize=None)
def latent_maps(name: str, B: int = None):
    """Latent-resolution position maps of a workload, computed with the
    oracle's downsample (the sphere workload is ray-cast at latent res)."""
    import oracle
    import synth
    w = synth.CONFIGS[name]
    if B is not None:
        w = synth.shrink(w, B=B)
    hi = synth.render_position_maps(w)
    if w.factor == 1:
        return hi
    return oracle.downsample(hi, w.factor)


@pytest.fixture(scope="session")
def maps():
    return latent_maps


def ulp_diff(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """|a - b| in float32 ulps (same-sign finite values)."""
    ia = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    ib = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(ia - ib)


def visible_weights(corr, wts):
    """The builder writes the weights of (token, anchor) pairs with a non-zero
    word only; this zeroes the others (whatever the buffer held), which is what
    the oracle stores there."""
    import numpy as np
    corr = corr.cpu().numpy() if hasattr(corr, "cpu") else corr
    wts = wts.cpu().numpy() if hasattr(wts, "cpu") else wts
    return np.where((corr != 0)[..., None], wts, np.float32(0))
