"""Test-side plumbing: moving seeded numpy inputs to the device and comparing.

Holds no arithmetic of the DP-SGD method.
"""
import numpy as np

# Parity bars: relative error 1e-4 for fp32 inputs, 2e-2 for bf16 inputs with
# fp32 accumulation. Squared norms are compared per example (|x-y|/|y|);
# cross terms (which can be near 0 or negative) by |x-y| <= tol * ||g_in||
# ||g_out||; gradient tensors both as a whole (||x-y||_F / ||y||_F) and
# element by element (elem_rel below), so that a wrong tile or a dropped row,
# which moves the Frobenius ratio by less than the bar, still fails.
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


def elem_rel(x, y) -> float:
    """Largest element-wise error max |x - y| / s, with s = max(|y|, rms of
    y's row) per element (rows = the last axis; a 1-D array is one row).

    The row rms keeps elements near zero (cancellations) from demanding more
    than the row's scale allows; a row of y that is zero throughout is held to
    the rms of the whole of y. Exact arithmetic on either side gives 0; fp32
    accumulation order gives ~1e-6; a zeroed output tile or a token missing
    from an embedding row gives ~1."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    if x.shape != y.shape:
        raise ValueError(f"shapes differ: {x.shape} vs {y.shape}")
    if y.size == 0:
        return 0.0
    y2 = y.reshape(-1, y.shape[-1]) if y.ndim else y.reshape(1, 1)
    x2 = x.reshape(y2.shape)
    row_rms = np.sqrt(np.mean(y2 * y2, axis=1, keepdims=True))
    all_rms = float(np.sqrt(np.mean(y2 * y2)))
    s = np.maximum(np.abs(y2), np.where(row_rms > 0, row_rms, all_rms))
    d = np.abs(x2 - y2)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(s > 0, d / np.where(s > 0, s, 1.0), np.where(d > 0, np.inf, 0.0))
    r = np.where(np.isnan(d), np.inf, r)
    return float(r.max())


def assert_close(x, y, tol: float, what: str = "") -> tuple:
    """Both bars at once: ||x-y||_F / ||y||_F <= tol and elem_rel(x, y) <= tol.
    Returns (fro, elem) for logging."""
    f, e = fro_rel(x, y), elem_rel(x, y)
    assert f <= tol and e <= tol, f"{what}: fro rel {f:.3e}, element rel {e:.3e} (bar {tol:g})"
    return f, e
