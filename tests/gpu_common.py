"""Shared helpers of the GPU parity tests."""
import numpy as np
import pytest

FP32_TOL = 1e-3     # max relative error, fp32 mode
BF16_TOL = 2e-2     # max relative error, bf16-MFMA mode


def rel_err(a, r) -> float:
    """max_i |a_i - r_i| / max(|r_i|, 1e-2 * max_j |r_j|): the relative error with
    a floor at 1% of the tensor's largest magnitude, so entries near zero are
    judged against the tensor's scale."""
    a = np.asarray(a, np.float64).reshape(-1)
    r = np.asarray(r, np.float64).reshape(-1)
    assert a.shape == r.shape, (a.shape, r.shape)
    if r.size == 0:
        return 0.0
    assert np.all(np.isfinite(a)), "non-finite values in the GPU result"
    scale = np.max(np.abs(r))
    if scale == 0:
        return float(np.max(np.abs(a)))
    den = np.maximum(np.abs(r), 1e-2 * scale)
    return float(np.max(np.abs(a - r) / den))


def assert_close(a, r, tol, what=""):
    e = rel_err(a, r)
    assert e <= tol, f"{what}: max relative error {e:.3e} > {tol:.1e}"
    return e


@pytest.fixture(scope="session")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X; none is visible"
    from paper_2005_14038_amd import hetpipe
    hetpipe.lib()            # raises if libhetpipe.so is missing
    return torch.device("cuda:0")


def to_dev(a, dev, dtype=None):
    import torch
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(dev)
