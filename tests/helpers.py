"""Shared helpers for the GPU parity tests: seeded inputs, oracle calls and
the error metric."""
import numpy as np

from paper_2510_27258_amd import inputs as I


def gen(B, H, n, d, dv, dist, seed):
    return I.draw_qkv(B, H, n, d, dv, dist, seed)


def dev(x, code):
    return I.to_torch(x, code, "cuda")


def rowwise_err(got, ref):
    """max over rows t of ||got_t - ref_t||_inf / ||ref_t||_inf (rows on the last axis)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.abs(got - ref).max(-1)
    den = np.abs(ref).max(-1)
    return float((num / np.maximum(den, 1e-300)).max())


def tol_for(code):
    """Parity bars: 1e-5 for fp32 inputs, 2e-3 for bf16 inputs with fp32 accumulation."""
    return 1e-5 if code == I.HLA_FP32 else 2e-3
