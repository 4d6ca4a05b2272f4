"""Test-side plumbing: moving seeded numpy inputs to the device and comparing.

Holds no arithmetic of the DP-SGD method.
"""
import numpy as np

# Parity bars: relative error 1e-4 for fp32 inputs, 2e-2 for bf16 inputs with
# fp32 accumulation. Squared norms are compared per example (|x-y|/|y|);
# gradient tensors by ||x-y||_F / ||y||_F; cross terms (which can be near 0
# or negative) by |x-y| <= tol * ||g_in|| ||g_out||.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def dev(arr: np.ndarray, dtype: str = None):
    """numpy -> torch device tensor. bf16 inputs are uint16 bit patterns."""
    import torch
    a = np.ascontiguousarray(arr)
    if dtype == "bf16" or a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def rel(x, y):
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    return np.abs(x - y) / np.maximum(np.abs(y), 1e-300)


def fro_rel(x, y) -> float:
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    return float(np.linalg.norm(x - y) / max(np.linalg.norm(y), 1e-300))
