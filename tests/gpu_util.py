"""Helpers shared by the GPU parity tests: tensor upload, tolerance checks."""
from __future__ import annotations

import numpy as np
import pytest

# Acceptance bounds.  max-abs and LSE bounds are the stated bars; the RMS bound
# is a tighter statistical check derived from bf16 rounding of P and of the
# output (each a relative 2^-9 per term, averaging down over thousands of
# keys), so that a dropped tile or a mis-scaled row cannot hide under the
# loose max-abs bar.
TOL = {
    "bf16": {"max_abs": 2e-2, "rms": 2e-3, "lse_rel": 1e-3},
    "f32": {"max_abs": 1e-5, "rms": 1e-6, "lse_rel": 1e-5},
}


def torch_mod():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def tdtype(dtype: str):
    torch = torch_mod()
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def to_gpu(x: np.ndarray, dtype: str):
    """Upload float32 values that are exact in `dtype`."""
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to("cuda").to(tdtype(dtype))


def to_np(t) -> np.ndarray:
    return t.float().cpu().numpy()


def check_out(gpu, ref, dtype: str, what: str, scale: float = 1.0):
    """Element-wise check against the stated bars; `scale` (>= 1) widens
    both for inputs whose conditioning the caller has bounded."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite GPU output"
    if gpu.size == 0:
        return
    err = np.abs(gpu - ref)
    t = {k: v * max(1.0, scale) for k, v in TOL[dtype].items()}
    rms = float(np.sqrt(np.mean(err ** 2)))
    assert err.max() <= t["max_abs"], f"{what}: max abs err {err.max():.3e} > {t['max_abs']:.3e}"
    assert rms <= t["rms"], f"{what}: rms err {rms:.3e} > {t['rms']:.3e}"


def check_lse(gpu, ref, dtype: str, what: str):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    if gpu.size == 0:
        return
    inf_ref = np.isinf(ref)
    assert np.array_equal(np.isinf(gpu), inf_ref), f"{what}: -inf pattern differs"
    if inf_ref.all():
        return
    g, r = gpu[~inf_ref], ref[~inf_ref]
    rel = np.abs(g - r) / np.maximum(np.abs(r), 1.0)
    assert rel.max() <= TOL[dtype]["lse_rel"], f"{what}: LSE rel err {rel.max():.3e}"
