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
