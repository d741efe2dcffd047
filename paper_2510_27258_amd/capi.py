"""ctypes binding of libhla.so: one Python function per C entry point, same
names and argument order as include/hla.h.  Pointers are passed as integers
(device addresses), streams as integers (hipStream_t, 0 = default stream).

The library must have been built (paper_2510_27258_amd/build.py); there is no
fallback: a missing library raises at first use.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhla.so")

HLA_OK, HLA_ERR_INVALID, HLA_ERR_UNSUPPORTED, HLA_ERR_WORKSPACE, HLA_ERR_HIP = range(5)
HLA_FP32, HLA_BF16 = 0, 1
HLA_ALGO_AUTO, HLA_ALGO_CHUNKED, HLA_ALGO_FUSED = 0, 1, 2

_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_Z = ctypes.c_size_t


class HLA2State(ctypes.Structure):
    """The hla2_state descriptor of include/hla.h (a host object)."""
    _fields_ = [("B", _I), ("H", _I), ("d", _I), ("dv", _I), ("masked", _I), ("normalized", _I), ("dtype", _I),
                ("eps", _F), ("data", _P), ("head_floats", _Z), ("S", _P), ("C", _P), ("m", _P), ("G", _P),
                ("h", _P), ("check", ctypes.c_ulonglong)]


_SP = ctypes.POINTER(HLA2State)
_ZP = ctypes.POINTER(_Z)
_IP = ctypes.POINTER(_I)

_SIGS = {
    "hla_last_error": (ctypes.c_char_p, []),
    "hla2_state_floats": (_Z, [_I, _I]),
    "hla2_workspace_bytes": (_Z, [_I] * 7),
    "hla2_workspace_bytes_ex": (_Z, [_I] * 8),
    "hla2_algo_supported": (_I, [_I] * 7),
    "hla2_forward": (_I, [_P, _P, _P, _P] + [_I] * 8 + [_F, _I, _P, _Z, _P]),
    "hla2_forward_ex": (_I, [_P, _P, _P, _P, _P] + [_I] * 8 + [_F, _I, _P, _Z, _I, _P]),
    "hla2_workspace_query": (_I, [_I] * 8 + [_ZP]),
    "hla2_forward_noalloc": (_I, [_P, _P, _P, _P] + [_I] * 8 + [_F, _I, _P]),
    "hla2_fused_plan": (_I, [_I] * 6 + [_IP, _IP, _IP, _IP]),
    "hla2_state_bytes": (_Z, [_I] * 4),
    "hla2_state_init": (_I, [_SP, _P, _Z] + [_I] * 6 + [_F, _I, _P]),
    "hla2_chunk_summaries": (_I, [_P, _P, _P, _P] + [_I] * 7 + [_P]),
    "hla2_scan": (_I, [_P, _P, _P, _P] + [_I] * 5 + [_P]),
    "hla2_prefill_workspace_bytes": (_Z, [_SP, _I, _I]),
    "hla2_prefill": (_I, [_SP, _P, _P, _P, _I, _I, _P, _P, _Z, _P]),
    "hla2_step": (_I, [_SP, _P, _P, _P, _P, _P]),
    "hla2_state_export": (_I, [_SP, _P, _P]),
    "hla_profile_begin": (_I, [_I]),
    "hla_profile_end": (_I, []),
    "hla_profile_summary": (_I, [ctypes.c_char_p, _Z]),
    "hla2_forward_decay_workspace_bytes": (_Z, [_I] * 7),
    "hla2_forward_decay": (_I, [_P, _P, _P, _P] + [_I] * 8 + [_F, _F, _I, _P, _Z, _P]),
    "hla2_backward_workspace_bytes": (_Z, [_I] * 7),
    "hla2_backward": (_I, [_P] * 7 + [_I] * 7 + [_P, _Z, _P]),
    "ahla_workspace_bytes": (_Z, [_I] * 7),
    "ahla_forward": (_I, [_P, _P, _P, _P] + [_I] * 7 + [_F, _I, _P, _Z, _P]),
    "hla3_workspace_bytes": (_Z, [_I] * 7),
    "hla3_forward": (_I, [_P, _P, _P, _P] + [_I] * 8 + [_F, _I, _P, _Z, _P]),
}


class HLAError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"HLA error {code}: {msg}")
        self.code = code


def lib():
    """The loaded library (ctypes.CDLL).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2510_27258_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name, None)
            if fn is None:
                continue
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return [n for n in _SIGS if hasattr(lib(), n)]


def _call(name, *args):
    rc = getattr(lib(), name)(*args)
    if rc != HLA_OK:
        raise HLAError(rc, lib().hla_last_error().decode())
    return rc


def hla_last_error():
    return lib().hla_last_error().decode()


def hla2_state_floats(d, dv):
    return lib().hla2_state_floats(d, dv)


def hla2_workspace_bytes(B, H, n, d, dv, chunk, dtype):
    return lib().hla2_workspace_bytes(B, H, n, d, dv, chunk, dtype)


def hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype, algo):
    return lib().hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype, algo)


def hla2_algo_supported(algo, n, d, dv, chunk, dtype, masked):
    return lib().hla2_algo_supported(algo, n, d, dv, chunk, dtype, masked)


def hla2_forward(q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws, ws_bytes, stream):
    return _call("hla2_forward", q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws,
                 ws_bytes, stream)


def hla2_forward_ex(q, k, v, out, den, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws, ws_bytes, algo,
                    stream):
    return _call("hla2_forward_ex", q, k, v, out, den, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws,
                 ws_bytes, algo, stream)


def hla2_forward_noalloc(q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, stream):
    return _call("hla2_forward_noalloc", q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, stream)


def hla2_workspace_query(B, H, n, d, dv, chunk, dtype, algo):
    """Workspace bytes of hla2_forward_ex; raises HLAError for arguments it would reject."""
    nb = _Z(0)
    _call("hla2_workspace_query", B, H, n, d, dv, chunk, dtype, algo, ctypes.byref(nb))
    return nb.value


def hla2_fused_plan(B, H, n, d, dv, chunk, tiles=False):
    """(segments per head, token tile) of the fused path's plan, and with
    tiles=True also (tiles of segment 0, tiles of each later segment);
    raises HLAError if it does not cover the shape."""
    P, tile, first, per = _I(0), _I(0), _I(0), _I(0)
    _call("hla2_fused_plan", B, H, n, d, dv, chunk, ctypes.byref(P), ctypes.byref(tile), ctypes.byref(first),
          ctypes.byref(per))
    if tiles:
        return P.value, tile.value, first.value, per.value
    return P.value, tile.value


def hla2_state_bytes(B, H, d, dv):
    return lib().hla2_state_bytes(B, H, d, dv)


def hla2_state_init(st, buf, buf_bytes, B, H, d, dv, masked, normalized, eps, dtype, stream):
    return _call("hla2_state_init", ctypes.byref(st), buf, buf_bytes, B, H, d, dv, masked, normalized, eps, dtype,
                 stream)


def hla2_chunk_summaries(q, k, v, states, B, H, n, d, dv, chunk, dtype, stream):
    return _call("hla2_chunk_summaries", q, k, v, states, B, H, n, d, dv, chunk, dtype, stream)


def hla2_scan(states, init, prefix, total, B, H, M, d, dv, stream):
    return _call("hla2_scan", states, init, prefix, total, B, H, M, d, dv, stream)


def hla2_prefill_workspace_bytes(st, n, chunk):
    return lib().hla2_prefill_workspace_bytes(ctypes.byref(st), n, chunk)


def hla2_prefill(st, q, k, v, n, chunk, out, ws, ws_bytes, stream):
    return _call("hla2_prefill", ctypes.byref(st), q, k, v, n, chunk, out, ws, ws_bytes, stream)


def hla2_step(st, q_t, k_t, v_t, out_t, stream):
    return _call("hla2_step", ctypes.byref(st), q_t, k_t, v_t, out_t, stream)


def hla2_state_export(st, full, stream):
    return _call("hla2_state_export", ctypes.byref(st), full, stream)


def hla2_forward_decay_workspace_bytes(B, H, n, d, dv, chunk, dtype):
    return lib().hla2_forward_decay_workspace_bytes(B, H, n, d, dv, chunk, dtype)


def hla2_forward_decay(q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, gamma, dtype, ws, ws_bytes,
                       stream):
    return _call("hla2_forward_decay", q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, gamma, dtype,
                 ws, ws_bytes, stream)


def hla2_backward_workspace_bytes(B, H, n, d, dv, chunk, dtype):
    return lib().hla2_backward_workspace_bytes(B, H, n, d, dv, chunk, dtype)


def hla2_backward(q, k, v, g, dq, dk, dv, B, H, n, d, dv_dim, chunk, dtype, ws, ws_bytes, stream):
    return _call("hla2_backward", q, k, v, g, dq, dk, dv, B, H, n, d, dv_dim, chunk, dtype, ws, ws_bytes, stream)


def ahla_workspace_bytes(B, H, n, d, dv, chunk, dtype):
    return lib().ahla_workspace_bytes(B, H, n, d, dv, chunk, dtype)


def ahla_forward(q, k, v, out, B, H, n, d, dv, chunk, normalized, eps, dtype, ws, ws_bytes, stream):
    return _call("ahla_forward", q, k, v, out, B, H, n, d, dv, chunk, normalized, eps, dtype, ws, ws_bytes, stream)


def hla3_workspace_bytes(B, H, n, d, dv, chunk, dtype):
    return lib().hla3_workspace_bytes(B, H, n, d, dv, chunk, dtype)


def hla3_forward(q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws, ws_bytes, stream):
    return _call("hla3_forward", q, k, v, out, B, H, n, d, dv, chunk, masked, normalized, eps, dtype, ws,
                 ws_bytes, stream)


def hla_profile_begin(max_records):
    return _call("hla_profile_begin", max_records)


def hla_profile_end():
    return _call("hla_profile_end")


def hla_profile_summary():
    """{kernel name: (launches, total_ms)} of the records since the last call."""
    buf = ctypes.create_string_buffer(1 << 16)
    _call("hla_profile_summary", buf, len(buf))
    res = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        res[name] = (int(cnt), float(ms))
    return res
