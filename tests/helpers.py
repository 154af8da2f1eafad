"""Shared helpers for the test suite (no method arithmetic here)."""
import numpy as np


def rel_rms(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.sqrt(np.sum((got - ref) ** 2)) / np.sqrt(np.sum(ref ** 2)))


def max_abs(got, ref):
    return float(np.max(np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))))


def dev(a, dtype="bf16", device="cuda"):
    """Device tensor holding exactly the values of a bf16/fp32-exact array."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.to(device)


def host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


# Tolerances (fp32 / bf16 outputs against the fp64 oracle).
TOL_F32_MAXABS = 1e-4
TOL_BF16_MAXABS = 2e-2
TOL_BF16_RELRMS = 5e-3


def assert_close_bf16(got, ref, what=""):
    ma, rr = max_abs(got, ref), rel_rms(got, ref)
    assert ma <= TOL_BF16_MAXABS and rr <= TOL_BF16_RELRMS, f"{what}: max-abs {ma:.3e}, rel-RMS {rr:.3e}"
    return ma, rr


def assert_close_f32(got, ref, what=""):
    ma = max_abs(got, ref)
    assert ma <= TOL_F32_MAXABS, f"{what}: max-abs {ma:.3e}"
    return ma
