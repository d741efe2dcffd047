"""Seeded synthetic inputs and the named workloads.

This module holds no HLA arithmetic: it only draws random q/k/v, shapes them
and rounds them to the storage dtype.  Both the GPU path and the CPU checks
consume exactly these values.

Recipe: numpy PCG64 `default_rng(seed)`, float32 standard normals drawn in the
order q [B,H,n,d], k [B,H,n,d], v [B,H,n,dv].
  dist "scaled": q, k, v divided by sqrt(d) in float32, kept float32.
  dist "unit":   q and k L2-normalised per token (last axis) in float32, v kept
                 N(0,1); all three rounded to bfloat16 (round-to-nearest-even).
"""
import math

import numpy as np
import torch

HLA_FP32 = 0
HLA_BF16 = 1


def draw_qkv(B, H, n, d, dv, dist, seed):
    """Returns (q, k, v) as float32 numpy arrays holding the exact input values
    and the storage dtype code (HLA_FP32 or HLA_BF16)."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, n, d), dtype=np.float32)
    k = rng.standard_normal((B, H, n, d), dtype=np.float32)
    v = rng.standard_normal((B, H, n, dv), dtype=np.float32)
    if dist == "scaled":
        s = np.float32(1.0 / math.sqrt(d))
        return q * s, k * s, v * s, HLA_FP32
    if dist == "unit":
        q = q / np.linalg.norm(q, axis=-1, keepdims=True).astype(np.float32)
        k = k / np.linalg.norm(k, axis=-1, keepdims=True).astype(np.float32)
        q, k, v = (round_bf16(x) for x in (q, k, v))
        return q, k, v, HLA_BF16
    raise ValueError(f"unknown dist {dist!r}")


def draw_grad(B, H, n, dv, seed):
    """Upstream gradient dL/dout for the backward: float32 standard normals
    [B,H,n,dv] from default_rng(seed), kept float32."""
    return np.random.default_rng(seed).standard_normal((B, H, n, dv), dtype=np.float32)


def round_bf16(x):
    """float32 -> nearest bfloat16 (ties to even), returned as float32."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy()


def to_torch(x, dtype_code, device="cpu"):
    """float32 numpy array -> torch tensor in the storage dtype on `device`."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype_code == HLA_BF16:
        t = t.to(torch.bfloat16)
    return t.to(device)


# Named workloads.  Keys say what each one is; sizes are in the record.
WORKLOADS = {
    "hla2-masked-fp32-B1H2-n256-d32-C64": dict(
        kind="forward", B=1, H=2, n=256, d=32, dv=32, chunk=64, dist="scaled",
        masked=1, normalized=0, eps=1e-6, seed=0),
    "hla2-masked-bf16-B4H16-n4096-d64-C64": dict(
        kind="forward", B=4, H=16, n=4096, d=64, dv=64, chunk=64, dist="unit",
        masked=1, normalized=0, eps=1e-6, seed=0),
    "hla2-masked-normalized-bf16-B2H32-n16384-d128-C128": dict(
        kind="forward", B=2, H=32, n=16384, d=128, dv=128, chunk=128, dist="unit",
        masked=1, normalized=1, eps=1e-6, seed=0),
    "hla2-decode-bf16-B64H32-d128-prefix2048-steps1024": dict(
        kind="decode", B=64, H=32, n=2048, steps=1024, d=128, dv=128, chunk=128,
        dist="unit", masked=1, normalized=0, eps=1e-6, seed=0, step_seed=1),
    "hla3-masked-fp32-B1H8-n2048-d16-C32": dict(
        kind="hla3", B=1, H=8, n=2048, d=16, dv=16, chunk=32, dist="scaled",
        masked=1, normalized=0, eps=1e-6, seed=0),
    # the B4H16 d=64 shape with decay gamma = 0.99 (the paper gives no decayed configuration)
    "hla2-decay-bf16-B4H16-n4096-d64-C64": dict(
        kind="decay", B=4, H=16, n=4096, d=64, dv=64, chunk=64, dist="unit",
        masked=1, normalized=0, eps=1e-6, seed=0, gamma=0.99),
    # AHLA (Sec. 6) on the B4H16 d=64 shape of the second-order workload
    "ahla-bf16-B4H16-n4096-d64-C64": dict(
        kind="ahla", B=4, H=16, n=4096, d=64, dv=64, chunk=64, dist="unit",
        masked=1, normalized=0, eps=1e-6, seed=0),
}
