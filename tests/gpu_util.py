"""Shared helpers of the GPU parity tests."""
import numpy as np
import pytest

# Tolerance for float32 results against the oracle: relative L2 error <= 1e-5
# and max |got - ref| <= 1e-4 * (1 + |ref|) element-wise.
REL_L2 = 1e-5
ABS_REL = 1e-4


def rel_l2(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref.ravel())
    return np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0)


def assert_close(got, ref, what="", rel_l2_tol=REL_L2, abs_rel_tol=ABS_REL):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), what + ": non-finite output"
    e = rel_l2(got, ref)
    bound = abs_rel_tol * (1.0 + np.abs(ref.astype(np.float64)))
    viol = np.abs(got.astype(np.float64) - ref) > bound
    assert e <= rel_l2_tol, f"{what}: rel L2 {e:.3e} > {rel_l2_tol}"
    assert not viol.any(), (f"{what}: {int(viol.sum())} elements beyond 1e-4*(1+|ref|); "
                            f"max abs err {np.abs(got - ref).max():.3e}")
    return e


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()
