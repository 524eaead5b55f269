"""Helpers shared by the GPU parity tests: host<->device transfers of the seeded
inputs and the error metrics (max-abs and relative L2 against the fp64 oracle)."""
from __future__ import annotations

import sys

import numpy as np

# tolerances: bf16 storage / MFMA against the fp64 oracle, and the fp32 path
BF16_MAX_ABS, BF16_REL_L2 = 2e-2, 1e-2
F32_MAX_ABS, F32_REL_L2 = 1e-5, 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray, dtype: str):
    """float32 numpy array (bf16-representable for bf16) -> device tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.cuda()


def host(t) -> np.ndarray:
    import torch
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits16(t) -> np.ndarray:
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy()


def errors(got: np.ndarray, want: np.ndarray):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.isfinite(got).all(), "non-finite values in the GPU result"
    d = got - want
    max_abs = float(np.abs(d).max()) if d.size else 0.0
    nrm = float(np.linalg.norm(want))
    rel = float(np.linalg.norm(d) / nrm) if nrm > 0 else float(np.linalg.norm(d))
    return max_abs, rel


def assert_close(got, want, dtype: str, what: str = ""):
    max_abs, rel = errors(got, want)
    tol_a, tol_r = (BF16_MAX_ABS, BF16_REL_L2) if dtype == "bf16" else (F32_MAX_ABS, F32_REL_L2)
    say(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} (tol {tol_a:g}/{tol_r:g})")
    assert max_abs <= tol_a and rel <= tol_r, f"{what}: max_abs={max_abs:.3e} rel_l2={rel:.3e}"
