"""Build and load the C oracle (test infrastructure only).

`build()` compiles oracle/*.c with gcc into oracle/liboracle.so; `load()`
returns the ctypes handle, building first if the library is missing.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(_HERE, "liboracle.so")
SOURCES = ["hla2_ref.c", "hla2_decay_ref.c", "hla3_ref.c", "ahla_ref.c"]
_handle = None


def build(verbose=False):
    srcs = [os.path.join(_HERE, s) for s in SOURCES if os.path.exists(os.path.join(_HERE, s))]
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-o", LIB + ".tmp"] + srcs + ["-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    global _handle
    _handle = None


def load():
    global _handle
    if _handle is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        P = ctypes.POINTER(ctypes.c_double)
        lib.hla2_serial_f64.argtypes = [P, P, P, P, P, ctypes.c_long, ctypes.c_long,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        P, P, P, P, P, ctypes.c_int]
        lib.hla2_serial_f64.restype = ctypes.c_int
        if hasattr(lib, "hla2_decay_serial_f64"):
            lib.hla2_decay_serial_f64.argtypes = [P, P, P, P, P, ctypes.c_long, ctypes.c_long,
                                                  ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                                  P, P, P, P, P, ctypes.c_int]
            lib.hla2_decay_serial_f64.restype = ctypes.c_int
        if hasattr(lib, "ahla_serial_f64"):
            lib.ahla_serial_f64.argtypes = [P, P, P, P, P, ctypes.c_long, ctypes.c_long, ctypes.c_int,
                                            ctypes.c_int, ctypes.c_int]
            lib.ahla_serial_f64.restype = ctypes.c_int
        if hasattr(lib, "hla3_serial_f64"):
            lib.hla3_serial_f64.argtypes = [P, P, P, P, P, ctypes.c_long, ctypes.c_long,
                                            ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
            lib.hla3_serial_f64.restype = ctypes.c_int
        _handle = lib
    return _handle


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def hla2_serial_c(q, k, v, masked=True, state=None, threads=0, return_state=True):
    """Serial second-order recurrence in C over heads [..., n, d].

    Returns (num [..., n, dv], den [..., n], final state tuple or None,
    threads used).  `state` = (S, C, m, G, h) continues from that prefix.
    """
    lib = load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    BH = int(np.prod(batch)) if batch else 1
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    shapes = [(d, d), (d, dv), (d,), (d, dv), (d,)]
    if state is not None:
        st = [np.ascontiguousarray(np.broadcast_to(np.asarray(x, np.float64), batch + s)).copy()
              for x, s in zip(state, shapes)]
    elif return_state:
        st = [np.zeros(batch + s) for s in shapes]
    else:
        st = [None] * 5
    used = lib.hla2_serial_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(num), _ptr(den), BH, n, d, dv,
                               int(bool(masked)), *[_ptr(x) for x in st], int(threads))
    final = tuple(st) if st[0] is not None else None
    return num, den, final, used


def available():
    try:
        load()
        return True
    except Exception:
        return False


def hla3_serial_c(q, k, v, masked=True, threads=0):
    """Serial third-order recurrence (Alg. 3) in C over heads [..., n, d].
    Returns (num [..., n, dv], den [..., n], threads used)."""
    lib = load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    BH = int(np.prod(batch)) if batch else 1
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    used = lib.hla3_serial_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(num), _ptr(den), BH, n, d, dv,
                               int(bool(masked)), int(threads))
    return num, den, used


def hla2_decay_serial_c(q, k, v, gamma, masked=True, state=None, threads=0, return_state=True):
    """Decayed serial recurrence in C over heads [..., n, d] (oracle.hla2_decay
    reading).  Returns (num, den, final state tuple or None, threads used)."""
    lib = load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    BH = int(np.prod(batch)) if batch else 1
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    shapes = [(d, d), (d, dv), (d,), (d, dv), (d,)]
    if state is not None:
        st = [np.ascontiguousarray(np.broadcast_to(np.asarray(x, np.float64), batch + s)).copy()
              for x, s in zip(state, shapes)]
    elif return_state:
        st = [np.zeros(batch + s) for s in shapes]
    else:
        st = [None] * 5
    used = lib.hla2_decay_serial_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(num), _ptr(den), BH, n, d, dv,
                                     int(bool(masked)), float(gamma), *[_ptr(x) for x in st], int(threads))
    final = tuple(st) if st[0] is not None else None
    return num, den, final, used


def ahla_serial_c(q, k, v, threads=0):
    """AHLA streaming recurrence (Sec. 6) in C over heads [..., n, d].
    Returns (num [..., n, dv], den [..., n], threads used)."""
    lib = load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv = v.shape[-1]
    BH = int(np.prod(batch)) if batch else 1
    num = np.empty(batch + (n, dv))
    den = np.empty(batch + (n,))
    used = lib.ahla_serial_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(num), _ptr(den), BH, n, d, dv, int(threads))
    return num, den, used
