"""GPU parity of the masked second-order HLA backward (hla2_backward)
against the fp64 oracle's written-out VJP (pinned against torch autograd,
finite differences and a hand-worked example).

Bar: 2e-3 on the row-wise relative error (bf16 inputs, fp32 accumulation)
of each of dq, dk, dv."""
import sys

import numpy as np
import pytest
import torch

import paper_2510_27258_amd as hla
from paper_2510_27258_amd import capi
from paper_2510_27258_amd import inputs as I
from oracle import hla2_backward as OB
from tests.helpers import dev, gen, rowwise_err, tol_for

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _check(B, H, n, d, seed=0, heads=None, chunk=64):
    q, k, v, code = gen(B, H, n, d, d, "unit", seed)
    g = I.draw_grad(B, H, n, d, seed + 100)
    _say(f"case backward B={B} H={H} n={n} d={d} seed={seed}")
    dq, dk, dv = (x.cpu().numpy() for x in hla.backward(dev(q, code), dev(k, code), dev(v, code),
                                                        torch.from_numpy(g).cuda(), chunk))
    sel = (slice(None),) if heads is None else (0, slice(0, heads))
    ref = OB.hla2_vjp_serial(q[sel], k[sel], v[sel], g[sel])
    tol = tol_for(code)
    errs = {}
    for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        errs[name] = rowwise_err(got[sel], r)
        assert errs[name] <= tol, f"{name} row-wise error {errs[name]:.3e} > {tol}"
    return errs


@pytest.mark.parametrize("d", [64, 128])
def test_backward_shapes(d):
    for n in (1, 7, 64, 65, 190, 513):
        _check(1, 2, n, d, seed=n + d)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("segments", [1, 2, 3, 7])
def test_backward_segment_counts(d, segments, monkeypatch):
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    _check(2, 1, 64 * 9 + 5, d, seed=segments)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("segments", [17, 34])
def test_backward_many_segments(d, segments, monkeypatch):
    """More segments than the moment scan's sixteen thread groups: runs of
    two or three segments, the last ones partial or empty."""
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    n = 64 * 33 + 17
    P, _ = _plan(n, segments)
    assert P == segments
    _check(1, 1, n, d, seed=segments + d)


def _plan(n, p):
    """Segments and tiles per segment of the walks for a requested count p."""
    M = (n + 63) // 64
    p = max(1, min(p, M))
    cps = (M + p - 1) // p
    return (M + cps - 1) // cps, cps


def test_backward_matches_autograd_of_definition_small():
    q, k, v, code = gen(1, 1, 70, 64, 64, "unit", 3)
    g = I.draw_grad(1, 1, 70, 64, 4)
    got = hla.backward(dev(q, code), dev(k, code), dev(v, code), torch.from_numpy(g).cuda())
    for a, b in zip(got, OB.hla2_vjp_autograd(q, k, v, g)):
        assert rowwise_err(a.cpu().numpy(), b) <= tol_for(code)


def test_autograd_function():
    """hla2_attention's backward is hla2_backward; its forward is hla2_forward."""
    q, k, v, code = gen(1, 2, 200, 64, 64, "unit", 5)
    g = torch.from_numpy(I.draw_grad(1, 2, 200, 64, 6)).cuda()
    qd, kd, vd = (dev(x, code).requires_grad_(True) for x in (q, k, v))
    out = hla.hla2_attention(qd, kd, vd, 64)
    assert torch.equal(out.detach(), hla.forward(qd.detach(), kd.detach(), vd.detach(), 64))
    out.backward(g)
    dq, dk, dv = hla.backward(qd.detach(), kd.detach(), vd.detach(), g)
    for a, b in ((qd.grad, dq), (kd.grad, dk), (vd.grad, dv)):
        assert a.dtype == torch.bfloat16
        assert torch.equal(a, b.to(torch.bfloat16))


def test_backward_deterministic():
    q, k, v, code = gen(2, 2, 700, 64, 64, "unit", 7)
    g = torch.from_numpy(I.draw_grad(2, 2, 700, 64, 8)).cuda()
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    a = hla.backward(qd, kd, vd, g)
    b = hla.backward(qd, kd, vd, g)
    assert all(torch.equal(x, y) for x, y in zip(a, b))


def test_backward_workload_b4h16_d64_sampled_heads():
    """B4 H16 n4096 d=dv=64 bf16: all heads on the GPU, heads 0-3 against the oracle."""
    errs = _check(4, 16, 4096, 64, seed=0, heads=4)
    _say(f"backward workload row-wise errors {errs}")


def test_backward_errors():
    q = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16, device="cuda")
    g = torch.zeros(1, 1, 64, 64, device="cuda")
    outs = [torch.full((1, 1, 64, 64), 7.0, device="cuda") for _ in range(3)]
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    p = q.data_ptr()

    def call(d=64, dv=64, dtype=I.HLA_BF16, wsb=ws.numel(), gp=g.data_ptr()):
        capi.hla2_backward(p, p, p, gp, *(o.data_ptr() for o in outs), 1, 1, 64, d, dv, 64, dtype, ws.data_ptr(),
                           wsb, None)

    for kw, code in ((dict(d=32, dv=32), capi.HLA_ERR_UNSUPPORTED), (dict(dv=32), capi.HLA_ERR_UNSUPPORTED),
                     (dict(dtype=I.HLA_FP32), capi.HLA_ERR_UNSUPPORTED), (dict(d=96, dv=96), capi.HLA_ERR_UNSUPPORTED),
                     (dict(gp=None), capi.HLA_ERR_INVALID), (dict(wsb=16), capi.HLA_ERR_WORKSPACE)):
        with pytest.raises(capi.HLAError) as ei:
            call(**kw)
        assert ei.value.code == code, (kw, ei.value.code)
    torch.cuda.synchronize()
    assert all(bool((o == 7.0).all()) for o in outs), "a rejected call wrote an output"
