"""Shared test helpers: dtype handling and the tolerance checks of the parity bar.

Tolerances: bf16 inputs with fp32 accumulation -> max abs error 2e-2 and mean
abs error 2e-3; fp32 inputs -> max abs error 1e-5.  Index and cache work is
compared bit for bit.
"""
import numpy as np
import torch

BF16_MAX_ABS, BF16_MEAN_ABS, F32_MAX_ABS = 2e-2, 2e-3, 1e-5


def to_dtype(x, dtype):
    """Seeded float32 numpy array -> torch tensor of `dtype` (bf16 by RNE)."""
    return torch.from_numpy(np.ascontiguousarray(x)).to(dtype)


def f64(t):
    """Exact float64 copy of a torch tensor (bf16 values upcast exactly)."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits(t):
    """Bit pattern of a tensor as a numpy integer array (for bit-exact checks)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.numpy()


def err_stats(got, want):
    d = np.abs(np.asarray(got, dtype=np.float64) - np.asarray(want, dtype=np.float64))
    return float(d.max()), float(d.mean())


def assert_parity(got, want, dtype, what=""):
    """got: torch tensor (any device); want: float64 numpy oracle result."""
    g = f64(got)
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    mx, mean = err_stats(g, want)
    if dtype == torch.float32:
        assert mx <= F32_MAX_ABS, f"{what}: max abs err {mx:.3e} > {F32_MAX_ABS}"
    else:
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS, \
            f"{what}: max abs err {mx:.3e} (<= {BF16_MAX_ABS}), mean {mean:.3e} (<= {BF16_MEAN_ABS})"
    return mx, mean
