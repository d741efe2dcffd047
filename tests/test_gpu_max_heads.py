"""The largest head count the ABI accepts, B*H = 65535, through the entry points
that place heads on a grid dimension (one workgroup, or one row of segment
workgroups, per head).  The GPU computes every head; the oracle checks 64
sampled heads, the first and last among them."""
import sys

import numpy as np
import pytest
import torch

import paper_2510_27258_amd as hla
from paper_2510_27258_amd import capi
from oracle import hla2_backward as OB
from oracle import native
from tests.helpers import dev, gen, rowwise_err, tol_for

pytestmark = pytest.mark.gpu

B, H = 5, 13107          # 65535 heads
_SEL = sorted(set([0, 1, B * H // 2, B * H - 1] + np.random.default_rng(7).choice(B * H, 60, replace=False).tolist()))
BS, HS = np.array(_SEL) // H, np.array(_SEL) % H


def _pick(x):
    """Sampled heads of a [B, H, ...] array (numpy or torch) as [len, ...]."""
    if isinstance(x, torch.Tensor):
        return x[torch.as_tensor(BS, device=x.device), torch.as_tensor(HS, device=x.device)].cpu().numpy()
    return x[BS, HS]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("algo", [capi.HLA_ALGO_FUSED, capi.HLA_ALGO_CHUNKED])
def test_forward_max_heads(algo):
    q, k, v, code = gen(B, H, 70, 64, 64, "unit", 1)
    _say(f"case max heads forward B={B} H={H} n=70 d=64 algo={algo}")
    num_ref, _, _, _ = native.hla2_serial_c(_pick(q), _pick(k), _pick(v), masked=True, threads=16)
    got = _pick(hla.forward(dev(q, code), dev(k, code), dev(v, code), 64, algo=algo))
    assert rowwise_err(got, num_ref) <= tol_for(code)


def test_decode_max_heads():
    q, k, v, code = gen(B, H, 6, 16, 16, "scaled", 2)
    _say(f"case max heads prefill + steps B={B} H={H} d=16")
    num_ref, _, _, _ = native.hla2_serial_c(_pick(q), _pick(k), _pick(v), masked=True, threads=16)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    state = hla.State(B, H, 16, 16, dtype=qd.dtype)
    hla.prefill(state, qd[:, :, :4].contiguous(), kd[:, :, :4].contiguous(), vd[:, :, :4].contiguous(), 16,
                want_out=False)
    got = torch.stack([hla.step(state, qd[:, :, t].contiguous(), kd[:, :, t].contiguous(), vd[:, :, t].contiguous())
                       for t in (4, 5)], dim=2)
    assert rowwise_err(_pick(got), num_ref[:, 4:]) <= tol_for(code)


def test_hla3_max_heads():
    q, k, v, code = gen(B, H, 40, 16, 16, "scaled", 3)
    _say(f"case max heads hla3 B={B} H={H} n=40 d=16")
    for masked in (True, False):
        num_ref, _, _ = native.hla3_serial_c(_pick(q), _pick(k), _pick(v), masked=masked, threads=16)
        got = _pick(hla.hla3_forward(dev(q, code), dev(k, code), dev(v, code), 32, masked=masked))
        assert rowwise_err(got, num_ref) <= tol_for(code)


def test_ahla_max_heads():
    q, k, v, code = gen(B, H, 70, 64, 64, "unit", 4)
    _say(f"case max heads ahla B={B} H={H} n=70 d=64")
    num_ref, _, _ = native.ahla_serial_c(_pick(q), _pick(k), _pick(v), threads=16)
    got = _pick(hla.ahla_forward(dev(q, code), dev(k, code), dev(v, code), 64))
    assert rowwise_err(got, num_ref) <= tol_for(code)


def test_backward_max_heads():
    q, k, v, code = gen(B, H, 70, 64, 64, "unit", 5)
    g = np.random.default_rng(6).standard_normal((B, H, 70, 64), dtype=np.float32)
    _say(f"case max heads backward B={B} H={H} n=70 d=64")
    got = hla.backward(dev(q, code), dev(k, code), dev(v, code), torch.from_numpy(g).cuda(), 64)
    for name, x, r in zip(("dq", "dk", "dv"), got, OB.hla2_vjp_serial(_pick(q), _pick(k), _pick(v), _pick(g))):
        err = rowwise_err(_pick(x), r)
        assert err <= tol_for(code), f"{name} row-wise error {err:.3e}"
