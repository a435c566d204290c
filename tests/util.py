"""Helpers shared by the GPU tests: host<->device moves of bf16 bit patterns
and the output tolerance check."""
import numpy as np
import torch

OUT_RTOL = 2e-2   # max|gpu - ref| <= 2e-2 * max|ref|
W_ATOL = 1e-6     # gate weights


def dev_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host_bf16(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_f64(a: np.ndarray) -> np.ndarray:
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_close_rel(got: np.ndarray, ref: np.ndarray, rtol: float = OUT_RTOL, what: str = ""):
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    err = float(np.abs(got - ref).max()) if ref.size else 0.0
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert err <= rtol * scale + 1e-30, f"{what}: max|err|={err:.3e} > {rtol}*max|ref|={rtol * scale:.3e}"
    return err, scale
