"""GPU parity of the AHLA forward (ahla_forward, Sec. 6) against the fp64
AHLA oracle (the C streaming recurrence of Thm. AHLA, itself pinned against
the double sum, the hand example and closed forms).

Bar: 2e-3 on the row-wise relative error for bf16 inputs (the only dtype the
AHLA path takes); the normalised output on rows whose denominator is well
away from zero (|den + eps| >= 0.05 D_t, D_t = sum_j |(A A)_tj|), num and den
separately everywhere."""
import sys

import numpy as np
import pytest
import torch

import paper_2510_27258_amd as hla
from paper_2510_27258_amd import capi
from paper_2510_27258_amd import inputs as I
from oracle import ahla as OA
from oracle import native
from tests.helpers import dev, gen, rowwise_err, tol_for

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _check(B, H, n, d, chunk, normalized=False, seed=0, eps=1e-6, dist="unit"):
    q, k, v, code = gen(B, H, n, d, d, dist, seed)
    _say(f"case ahla B={B} H={H} n={n} d={d} chunk={chunk} normalized={normalized} seed={seed}")
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    num_ref, den_ref, _ = native.ahla_serial_c(q, k, v, threads=16)
    tol = tol_for(code)
    num = hla.ahla_forward(qd, kd, vd, chunk).cpu().numpy()
    err = rowwise_err(num, num_ref)
    assert err <= tol, f"num row-wise error {err:.3e} > {tol}"
    if normalized:
        out = hla.ahla_forward(qd, kd, vd, chunk, normalized=True, eps=eps).cpu().numpy()
        ones = torch.ones_like(vd)
        den = hla.ahla_forward(qd, kd, ones, chunk)[..., 0].cpu().numpy()
        D = OA.ahla_den_scale(q, k)
        e_den = float((np.abs(den - den_ref) / D).max())
        assert e_den <= tol, f"den error {e_den:.3e} > {tol}"
        good = np.abs(den_ref + eps) >= 0.05 * D
        assert good.mean() > 0.3
        e_out = rowwise_err(out[good], (num_ref / (den_ref + eps)[..., None])[good])
        assert e_out <= tol, f"normalised output error {e_out:.3e} > {tol}"
    return err


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("chunk", [64, 128])
def test_ahla_shapes(d, chunk):
    for n in (1, 7, 64, 65, 190, 513):
        _check(1, 2, n, d, chunk, seed=n + d)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("segments", [1, 2, 3, 7, 10])
def test_ahla_segment_counts(d, segments, monkeypatch):
    """Segments of several tiles: the P prefix (summed by the walks up to 8
    segments, a prefix launch above), the brackets and the fix-up."""
    monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    _check(2, 1, 64 * 9 + 5, d, 64, seed=segments)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("segments", [1, 4, 0])
def test_ahla_normalized(d, segments, monkeypatch):
    if segments:
        monkeypatch.setenv("HLA_FUSED_SEGMENTS", str(segments))
    _check(1, 2, 400, d, 64, normalized=True, seed=d + segments)


def test_ahla_matches_oracle_definition_small():
    """A tiny case against the dense definition ((A A) (.) L) V as well."""
    q, k, v, code = gen(1, 1, 70, 64, 64, "unit", 5)
    ref = OA.ahla_definition(q, k, v)
    got = hla.ahla_forward(dev(q, code), dev(k, code), dev(v, code), 64).cpu().numpy()
    assert rowwise_err(got, ref) <= tol_for(code)


def test_ahla_chunk128_equals_chunk64():
    """chunk 128 is walked in 64-token tiles: the same kernels, bit for bit."""
    q, k, v, code = gen(2, 2, 300, 64, 64, "unit", 6)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    assert torch.equal(hla.ahla_forward(qd, kd, vd, 64), hla.ahla_forward(qd, kd, vd, 128))


def test_ahla_deterministic():
    q, k, v, code = gen(2, 4, 1000, 64, 64, "unit", 7)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    a = hla.ahla_forward(qd, kd, vd, 64, normalized=True)
    b = hla.ahla_forward(qd, kd, vd, 64, normalized=True)
    assert torch.equal(a, b)


def test_ahla_workload_b4h16_d64():
    """B4 H16 n4096 d=dv=64 bf16 unit, chunk 64: every head."""
    w = I.WORKLOADS["ahla-bf16-B4H16-n4096-d64-C64"]
    err = _check(w["B"], w["H"], w["n"], w["d"], w["chunk"], seed=w["seed"], dist=w["dist"])
    _say(f"ahla workload row-wise error {err:.3e}")


def test_ahla_errors():
    q = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16, device="cuda")
    out = torch.full((1, 1, 64, 64), 7.0, device="cuda")
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    p = q.data_ptr()

    def call(d=64, dv=64, chunk=64, dtype=I.HLA_BF16, wsb=ws.numel(), normalized=0, eps=1e-6):
        capi.ahla_forward(p, p, p, out.data_ptr(), 1, 1, 64, d, dv, chunk, normalized, eps, dtype, ws.data_ptr(),
                          wsb, None)

    for kw, code in ((dict(d=32, dv=32), capi.HLA_ERR_UNSUPPORTED), (dict(dv=32), capi.HLA_ERR_UNSUPPORTED),
                     (dict(chunk=32), capi.HLA_ERR_UNSUPPORTED), (dict(dtype=I.HLA_FP32), capi.HLA_ERR_UNSUPPORTED),
                     (dict(d=96, dv=96), capi.HLA_ERR_UNSUPPORTED), (dict(normalized=2), capi.HLA_ERR_INVALID),
                     (dict(eps=-1.0), capi.HLA_ERR_INVALID), (dict(wsb=16), capi.HLA_ERR_WORKSPACE)):
        with pytest.raises(capi.HLAError) as ei:
            call(**kw)
        assert ei.value.code == code, (kw, ei.value.code)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all()), "a rejected call wrote its output"
    assert capi.ahla_workspace_bytes(1, 1, 64, 32, 32, 64, I.HLA_BF16) == 0
