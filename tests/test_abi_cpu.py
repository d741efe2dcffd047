"""Host-side checks of the C ABI: the library loads without a GPU, exports
every function include/hla.h declares, and the Python binding's argument
lists match the header.  No compute call is made."""
import ctypes
import os
import re

import pytest
import torch

from paper_2510_27258_amd import capi
from paper_2510_27258_amd import hla

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "hla.h")


def _declarations():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    decls = {}
    for m in re.finditer(r"^\s*(?:const\s+)?[a-z_]+\s*\*?\s*(a?hla[0-9a-z_]*)\s*\(([^)]*)\)\s*;", text, flags=re.M):
        name, args = m.group(1), m.group(2).strip()
        decls[name] = 0 if args in ("", "void") else len(args.split(","))
    return decls


def test_header_parses():
    decls = _declarations()
    for name in ("hla2_forward", "hla2_step", "hla2_scan", "hla2_chunk_summaries", "hla2_prefill", "hla2_forward_decay",
                 "hla3_forward", "ahla_forward", "ahla_workspace_bytes", "hla2_backward",
                 "hla2_backward_workspace_bytes"):
        assert name in decls


def test_library_exports_every_declared_symbol():
    lib = capi.lib()
    missing = [n for n in _declarations() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_arity_matches_header():
    decls = _declarations()
    for name, (_, args) in capi._SIGS.items():
        if name in decls:
            assert len(args) == decls[name], (name, len(args), decls[name])
    for name in decls:
        assert name in capi._SIGS, f"{name} has no binding"


def test_state_floats():
    assert capi.hla2_state_floats(128, 128) == 128 * 128 + 2 * 128 * 128 + 2 * 128
    assert capi.hla2_state_floats(16, 64) == 16 * 16 + 2 * 16 * 64 + 32


def test_workspace_queries_reject_bad_sizes():
    assert capi.hla2_workspace_bytes(1, 1, 100, 24, 16, 16, 0) == 0
    assert capi.hla2_workspace_bytes(1, 1, 100, 16, 16, 16, 0) > 0


# ----------------------------------------------------------------------------
# Argument checks.  Every entry point validates sizes, flags and pointers on the
# host and returns before any device call, so these run without a GPU.  Device
# pointers are never dereferenced: NULL and misaligned values are rejected first.
FP32, BF16 = 0, 1
INVALID, UNSUP = capi.HLA_ERR_INVALID, capi.HLA_ERR_UNSUPPORTED
P = 256            # a 16-byte aligned non-NULL value, rejected before any use by the cases below


def _fwd(L, **kw):
    a = dict(q=None, k=None, v=None, out=None, B=1, H=1, n=64, d=64, dv=64, chunk=64, masked=1, normalized=0,
             eps=1e-6, dtype=BF16, ws=None, wsb=0, s=None)
    a.update(kw)
    return L.hla2_forward(a["q"], a["k"], a["v"], a["out"], a["B"], a["H"], a["n"], a["d"], a["dv"], a["chunk"],
                          a["masked"], a["normalized"], a["eps"], a["dtype"], a["ws"], a["wsb"], a["s"])


def test_forward_rejects_empty_and_bad_sizes():
    L = capi.lib()
    for kw, code, text in ((dict(n=0), INVALID, "n must be"), (dict(n=-5), INVALID, "n must be"),
                           (dict(B=0), INVALID, "B and H"), (dict(H=-1), INVALID, "B and H"),
                           (dict(B=256, H=256), UNSUP, "exceeds"), (dict(d=24), UNSUP, "d and dv"),
                           (dict(n=1 << 23), UNSUP, "too long"), (dict(n=2**31 - 1), UNSUP, "too long"),
                           (dict(n=(1 << 22), d=128, dv=128), UNSUP, "too long"),
                           (dict(dv=256), UNSUP, "d and dv"), (dict(d=8), UNSUP, "d and dv"),
                           (dict(chunk=48), UNSUP, "chunk"), (dict(chunk=0), INVALID, "chunk must be set"),
                           (dict(dtype=2), INVALID, "dtype"), (dict(masked=2), INVALID, "masked"),
                           (dict(normalized=-1), INVALID, "normalized"), (dict(eps=float("inf")), INVALID, "eps"),
                           (dict(eps=-1.0), INVALID, "eps")):
        assert _fwd(L, **kw) == code, kw
        assert text in capi.hla_last_error(), (kw, capi.hla_last_error())


def test_longest_sequence_passes_the_size_checks():
    """n = 2^22 - 1 at d = dv = 128 is the longest accepted sequence: it gets past
    every size check to the pointer checks (NULL q)."""
    L = capi.lib()
    assert _fwd(L, n=(1 << 22) - 1, d=128, dv=128) == INVALID and "q is NULL" in capi.hla_last_error()
    assert _fwd(L, n=(1 << 23) - 1, d=64, dv=64) == INVALID and "q is NULL" in capi.hla_last_error()


def test_forward_rejects_null_and_misaligned_pointers():
    L = capi.lib()
    assert _fwd(L) == INVALID and "q is NULL" in capi.hla_last_error()
    assert _fwd(L, q=P, k=P, v=P) == INVALID and "out is NULL" in capi.hla_last_error()
    assert _fwd(L, q=P + 4, k=P, v=P, out=P) == INVALID and "aligned" in capi.hla_last_error()
    assert _fwd(L, q=P, k=P, v=P + 2, out=P) == INVALID and "v is not 16-byte aligned" in capi.hla_last_error()


def test_other_entry_points_reject_bad_arguments():
    L = capi.lib()
    # decay: gamma outside (0, 1], and gamma^(2 chunk) below the normal fp32 range
    for g, code in ((0.0, INVALID), (-0.5, INVALID), (1.5, INVALID), (float("nan"), INVALID), (0.3, UNSUP)):
        rc = L.hla2_forward_decay(P, P, P, P, 1, 1, 64, 64, 64, 64, 1, 0, 1e-6, g, BF16, None, 0, None)
        assert rc == code, g
    assert L.hla2_forward_decay(None, P, P, P, 1, 1, 0, 64, 64, 64, 1, 0, 1e-6, 0.9, BF16, None, 0, None) == INVALID
    # third order: d outside {16, 32}, masked flag, empty input
    assert L.hla3_forward(P, P, P, P, 1, 1, 64, 64, 64, 32, 1, 0, 1e-6, FP32, None, 0, None) == UNSUP
    assert L.hla3_forward(P, P, P, P, 1, 1, 64, 16, 16, 32, 3, 0, 1e-6, FP32, None, 0, None) == INVALID
    assert L.hla3_forward(P, P, P, P, 1, 1, 0, 16, 16, 32, 1, 0, 1e-6, FP32, None, 0, None) == INVALID
    # AHLA: fp32 inputs and d = 32 are not built
    assert L.ahla_forward(P, P, P, P, 1, 1, 64, 64, 64, 64, 0, 1e-6, FP32, None, 0, None) == UNSUP
    assert L.ahla_forward(P, P, P, P, 1, 1, 64, 32, 32, 64, 0, 1e-6, BF16, None, 0, None) == UNSUP
    # backward: d != dv, NULL gradient
    assert L.hla2_backward(P, P, P, P, P, P, P, 1, 1, 64, 64, 128, 64, BF16, None, 0, None) == UNSUP
    assert L.hla2_backward(P, P, P, None, P, P, P, 1, 1, 64, 64, 64, 64, BF16, None, 0, None) == INVALID
    assert "g is NULL" in capi.hla_last_error()
    # scan: no segments, misaligned init
    assert L.hla2_scan(P, None, P, None, 1, 1, 0, 64, 64, None) == INVALID
    assert L.hla2_scan(P, P + 8, P, None, 1, 1, 4, 64, 64, None) == INVALID
    # decode step and prefill: NULL descriptor, one not made by hla2_state_init
    assert L.hla2_step(None, P, P, P, P, None) == INVALID
    assert L.hla2_prefill(None, P, P, P, 64, 64, None, None, 0, None) == INVALID
    forged = capi.HLA2State(B=1, H=1, d=64, dv=64, masked=1, normalized=0, dtype=BF16, eps=1e-6, data=P,
                            head_floats=capi.hla2_state_floats(64, 64), check=12345)
    assert L.hla2_step(ctypes.byref(forged), P, P, P, P, None) == INVALID
    assert "hla2_state_init" in capi.hla_last_error()
    assert L.hla2_prefill(ctypes.byref(forged), P, P, P, 64, 64, None, None, 0, None) == INVALID
    assert L.hla2_prefill_workspace_bytes(ctypes.byref(forged), 64, 64) == 0
    assert L.hla2_state_export(ctypes.byref(forged), P, None) == INVALID
    assert L.hla2_state_export(None, P, None) == INVALID
    # chunk summaries: empty input
    assert L.hla2_chunk_summaries(P, P, P, P, 1, 1, 0, 64, 64, 64, BF16, None) == INVALID


def test_workspace_queries_follow_the_checks():
    """A workspace query returns 0 for arguments the entry point would reject."""
    assert capi.hla2_workspace_bytes(1, 1, 0, 64, 64, 64, BF16) == 0
    assert capi.hla3_workspace_bytes(1, 1, 64, 64, 64, 32, FP32) == 0
    assert capi.ahla_workspace_bytes(1, 1, 64, 64, 64, 64, FP32) == 0
    assert capi.hla2_backward_workspace_bytes(1, 1, 64, 64, 128, 64, BF16) == 0
    assert capi.hla3_workspace_bytes(1, 1, 64, 16, 16, 32, FP32) > 0
    assert capi.ahla_workspace_bytes(1, 1, 64, 64, 64, 64, BF16) > 0
    assert capi.hla2_backward_workspace_bytes(1, 1, 64, 64, 64, 64, BF16) > 0


def test_state_queries_and_init_checks():
    """hla2_state_bytes follows the size rules; hla2_state_init rejects bad
    arguments before it enqueues anything (its zeroing launch needs a GPU)."""
    L = capi.lib()
    # S packed symmetric: d(d+1)/2 floats, then C, m, G, h
    assert capi.hla2_state_bytes(2, 3, 64, 32) == 4 * 6 * (64 * 65 // 2 + 2 * 64 * 32 + 2 * 64)
    assert capi.hla2_state_bytes(64, 32, 128, 128) == 4 * 2048 * (128 * 129 // 2 + 2 * 128 * 128 + 2 * 128)
    assert capi.hla2_state_bytes(1, 1, 24, 64) == 0 and "d and dv" in capi.hla_last_error()
    assert capi.hla2_state_bytes(0, 1, 64, 64) == 0
    st = capi.HLA2State()
    need = capi.hla2_state_bytes(1, 2, 64, 64)
    assert L.hla2_state_init(None, P, need, 1, 2, 64, 64, 1, 0, 1e-6, BF16, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), None, need, 1, 2, 64, 64, 1, 0, 1e-6, BF16, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), P + 4, need, 1, 2, 64, 64, 1, 0, 1e-6, BF16, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), P, need - 16, 1, 2, 64, 64, 1, 0, 1e-6, BF16, None) == INVALID
    assert "state buffer" in capi.hla_last_error()
    assert L.hla2_state_init(ctypes.byref(st), P, need, 1, 2, 64, 64, 2, 0, 1e-6, BF16, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), P, need, 1, 2, 64, 64, 1, 0, -1.0, BF16, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), P, need, 1, 2, 64, 64, 1, 0, 1e-6, 3, None) == INVALID
    assert L.hla2_state_init(ctypes.byref(st), P, need, 1, 2, 96, 64, 1, 0, 1e-6, BF16, None) == UNSUP
    assert st.check == 0      # nothing was written on failure


def test_descriptor_layout_matches_header():
    """The ctypes mirror of hla2_state has the C layout: ints, the float eps,
    then pointer-aligned fields."""
    assert ctypes.sizeof(capi.HLA2State) == 96
    assert capi.HLA2State.data.offset == 32 and capi.HLA2State.check.offset == 88


def test_workspace_query_status():
    nb = ctypes.c_size_t(7)
    L = capi.lib()
    assert L.hla2_workspace_query(1, 1, 0, 64, 64, 64, BF16, 0, ctypes.byref(nb)) == INVALID and nb.value == 0
    assert L.hla2_workspace_query(1, 1, 64, 64, 64, 64, BF16, 0, None) == INVALID
    assert L.hla2_workspace_query(1, 1, 64, 64, 64, 64, FP32, capi.HLA_ALGO_FUSED, ctypes.byref(nb)) == UNSUP
    assert L.hla2_workspace_query(1, 1, 64, 64, 64, 64, BF16, 9, ctypes.byref(nb)) == INVALID
    assert capi.hla2_workspace_query(2, 3, 500, 64, 64, 64, BF16, 0) == capi.hla2_workspace_bytes_ex(
        2, 3, 500, 64, 64, 64, BF16, 0) > 0
    with pytest.raises(capi.HLAError):
        capi.hla2_workspace_query(1, 1, 64, 24, 64, 64, BF16, 0)


def test_fused_plan_query():
    P_, tile = capi.hla2_fused_plan(2, 32, 16384, 128, 128, 128)
    assert tile == 64 and 1 <= P_ <= 256
    P2, tile2 = capi.hla2_fused_plan(4, 16, 4096, 64, 64, 64)
    assert tile2 == 64 and P2 >= 1
    with pytest.raises(capi.HLAError) as ei:
        capi.hla2_fused_plan(1, 1, 64, 16, 16, 16)
    assert ei.value.code == UNSUP
    L = capi.lib()
    seg, tl = ctypes.c_int(0), ctypes.c_int(0)
    assert L.hla2_fused_plan(2, 32, 16384, 128, 128, 128, ctypes.byref(seg), ctypes.byref(tl), None, None) == 0
    assert (seg.value, tl.value) == (P_, tile)


def _segment_tiles(P, first, per, M):
    """Tile counts of the segments: segment 0 holds `first`, the others `per`, the last the rest."""
    if P == 1:
        return [M]
    return [first] + [per] * (P - 2) + [M - first - per * (P - 2)]


@pytest.mark.parametrize("B,H", [(2, 32), (1, 1), (1, 2), (4, 16), (8, 32), (1, 100), (3, 5)])
@pytest.mark.parametrize("n", [1, 64, 130, 596, 4096, 16384])
def test_fused_plan_d128_segments(B, H, n):
    """The d = 128 plan (two launches of one walk per CU each, segment 0
    shorter than the others) covers every tile once with non-empty segments,
    and walks at most 256 workgroups per launch."""
    P, tile, first, per = capi.hla2_fused_plan(B, H, n, 128, 128, 128, tiles=True)
    M = -(-n // tile)
    sizes = _segment_tiles(P, first, per, M)
    assert sum(sizes) == M and min(sizes) >= 1 and len(sizes) == P
    if P > 1:
        assert P >= 3 and (P - 1) * B * H <= 256
        assert first <= per and max(sizes[1:]) == per
    if (B, H, n) == (2, 32, 16384):
        assert (P, first, per) == (5, 36, 56)


def test_forward_den_needs_normalized():
    L = capi.lib()
    rc = L.hla2_forward_ex(P, P, P, P, P, 1, 1, 64, 64, 64, 64, 1, 0, 1e-6, BF16, P, 1 << 30, 0, None)
    assert rc == INVALID and "normalized" in capi.hla_last_error()
    rc = L.hla2_forward_ex(P, P, P, P, P + 4, 1, 1, 64, 64, 64, 64, 1, 1, 1e-6, BF16, P, 1 << 30, 0, None)
    assert rc == INVALID and "den is not 16-byte aligned" in capi.hla_last_error()


# ----------------------------------------------------------------------------
# The torch binding checks shapes, dtypes and devices before any launch (the C
# ABI sees only pointers and sizes taken from q).  CPU tensors: each case must
# fail on its own mismatch, before the device check.
def _t(*shape, dtype=torch.bfloat16):
    return torch.zeros(*shape, dtype=dtype)


@pytest.mark.parametrize("case", ["k_shape", "v_rows", "k_dtype", "v_dtype", "rank"])
def test_binding_rejects_mismatched_inputs(case):
    q = _t(1, 2, 16, 32)
    k, v = _t(1, 2, 16, 32), _t(1, 2, 16, 64)
    if case == "k_shape":
        k = _t(1, 2, 16, 16)
    elif case == "v_rows":
        v = _t(1, 2, 15, 64)
    elif case == "k_dtype":
        k = _t(1, 2, 16, 32, dtype=torch.float32)
    elif case == "v_dtype":
        v = _t(1, 2, 16, 64, dtype=torch.float32)
    else:
        q, k = _t(2, 16, 32), _t(2, 16, 32)
    for fn in (lambda: hla.forward(q, k, v, 16), lambda: hla.forward_decay(q, k, v, 16, 0.9),
               lambda: hla.hla3_forward(q, k, v, 16), lambda: hla.ahla_forward(q, k, v, 64),
               lambda: hla.chunk_summaries(q, k, v, 16)):
        with pytest.raises(ValueError) as ei:
            fn()
        assert "GPU" not in str(ei.value), str(ei.value)


def test_binding_rejects_wrong_out_and_state():
    q = _t(1, 2, 16, 32)
    with pytest.raises(ValueError):
        hla._fp32_out(torch.zeros(1, 2, 16, 31), (1, 2, 16, 32), q.device)
    with pytest.raises(ValueError):
        hla._fp32_out(torch.zeros(1, 2, 16, 32, dtype=torch.float64), (1, 2, 16, 32), q.device)
    with pytest.raises(ValueError):
        hla.scan(torch.zeros(1, 1, 3, 100), 32, 32)
    with pytest.raises(ValueError):
        hla.backward(q, q, q, torch.zeros(1, 2, 15, 32))


def test_decay_underflow_check_uses_the_walked_tile():
    """gamma^(2*64) must stay normal for chunk 64 and 128 alike (both walk
    64-token tiles): 0.6 passes the check at chunk 128 and stops at the NULL
    pointer check; 0.4 fails it."""
    L = capi.lib()
    assert L.hla2_forward_decay(None, P, P, P, 1, 1, 64, 64, 64, 128, 1, 0, 1e-6, 0.6, BF16, None, 0, None) == INVALID
    assert "q is NULL" in capi.hla_last_error()
    assert L.hla2_forward_decay(P, P, P, P, 1, 1, 64, 64, 64, 128, 1, 0, 1e-6, 0.4, BF16, None, 0, None) == UNSUP
