"""hla2_forward_noalloc (the entry point for callers that cannot allocate)
against hla2_forward through the C ABI: the same kernels on a library-held
workspace, so the outputs must agree bit for bit (and with the oracle within
the bf16 bar).  Two calls in a row on one GPU, the second smaller, so the
second runs on scratch the first left behind; then sizes above the scratch
are rejected before anything is enqueued."""
import sys

import numpy as np
import pytest
import torch

from paper_2510_27258_amd import capi
from paper_2510_27258_amd import inputs as I
from oracle import native
from tests.helpers import dev, gen, rowwise_err

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _pair(B, H, n, d, dv, chunk, normalized, seed):
    q, k, v, code = gen(B, H, n, d, dv, "unit", seed)
    qd, kd, vd = dev(q, code), dev(k, code), dev(v, code)
    s = torch.cuda.current_stream().cuda_stream
    a = torch.full((B, H, n, dv), float("nan"), device="cuda")
    b = torch.full((B, H, n, dv), float("nan"), device="cuda")
    capi.hla2_forward_noalloc(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(), a.data_ptr(), B, H, n, d, dv, chunk, 1,
                              normalized, 1e-6, code, s)
    wsb = capi.hla2_workspace_bytes(B, H, n, d, dv, chunk, code)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    capi.hla2_forward(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(), b.data_ptr(), B, H, n, d, dv, chunk, 1,
                      normalized, 1e-6, code, ws.data_ptr(), wsb, s)
    torch.cuda.synchronize()
    return q, k, v, a.cpu().numpy(), b.cpu().numpy()


@pytest.mark.parametrize("normalized", [0, 1])
def test_noalloc_matches_forward_twice(normalized):
    for (B, H, n, d, chunk, seed) in ((2, 8, 1500, 64, 64, 3), (1, 3, 333, 128, 128, 4)):
        _say(f"case noalloc B={B} H={H} n={n} d={d} chunk={chunk} normalized={normalized}")
        q, k, v, a, b = _pair(B, H, n, d, d, chunk, normalized, seed)
        assert np.array_equal(a, b, equal_nan=False), "no-alloc output differs from hla2_forward"
        num, den, _, _ = native.hla2_serial_c(q, k, v, masked=True, threads=16, return_state=False)
        if not normalized:
            assert rowwise_err(a, num) <= 2e-3


def test_noalloc_full_size_workload():
    """The d = 64 workload (B4 H16 n4096) fits the scratch; bit-identical to hla2_forward."""
    w = I.WORKLOADS["hla2-masked-bf16-B4H16-n4096-d64-C64"]
    _say("case noalloc B4H16 n4096 d64")
    _, _, _, a, b = _pair(w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"], 0, 0)
    assert np.array_equal(a, b)


def test_noalloc_rejects_sizes_above_scratch():
    q = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    out = torch.full((4,), 7.0, device="cuda")
    L = capi.lib()
    B, H, n = 64, 64, 65536     # workspace far above 128 MiB; nothing is read or written
    rc = L.hla2_forward_noalloc(q.data_ptr(), q.data_ptr(), q.data_ptr(), out.data_ptr(), B, H, n, 64, 64, 64, 1, 0,
                                1e-6, capi.HLA_BF16, torch.cuda.current_stream().cuda_stream)
    assert rc == capi.HLA_ERR_WORKSPACE and "scratch" in capi.hla_last_error()
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
