"""Host-side checks of the C ABI: the library loads without a GPU, exports
every function include/hla.h declares, and the Python binding's argument
lists match the header.  No compute call is made."""
import os
import re

from paper_2510_27258_amd import capi

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
    # decode step and prefill: NULL state, bad flags
    assert L.hla2_step(None, P, P, P, P, 1, 1, 64, 64, 1, 0, 1e-6, BF16, None) == INVALID
    assert L.hla2_step(P, P, P, P, P, 1, 1, 64, 64, 1, 2, 1e-6, BF16, None) == INVALID
    assert L.hla2_prefill(None, P, P, P, None, 1, 1, 64, 64, 64, 64, 1, 0, 1e-6, BF16, None, 0, None) == INVALID
    assert L.hla2_prefill(P, P, P, P, P + 4, 1, 1, 64, 64, 64, 64, 1, 0, 1e-6, BF16, None, 0, None) == INVALID
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
