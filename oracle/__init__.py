"""CPU oracle for the segment re-prefill path — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the device
library (``paper_2607_00151_amd``) and neither imports the other.

* ``attention_rows`` wraps ``oracle.c``: the plain double-precision definition
  of causal grouped-query attention over contiguous K/V.
* ``pages`` holds the paged-cache definitions (append, assemble).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import pages  # noqa: F401  (re-exported)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# AddressSanitizer + UndefinedBehaviorSanitizer build, loaded instead of the
# plain one when ORACLE_SANITIZED=1 (the process must then preload libasan)
_LIB_SAN = os.path.join(_HERE, "liboracle_san.so")
_lib = None


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile oracle.c with gcc (no fast-math: IEEE double, source order)."""
    out = _LIB_SAN if sanitize else _LIB
    if force or not os.path.exists(out):
        tmp = out + f".tmp{os.getpid()}"
        flags = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                 "-fno-omit-frame-pointer"] if sanitize else ["-O2"]
        subprocess.check_call(["gcc", *flags, "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-Werror", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, out)
    return out


def _load():
    global _lib
    if _lib is None:
        path = _LIB_SAN if os.environ.get("ORACLE_SANITIZED") == "1" else _LIB
        if not os.path.exists(path):
            build(force=True, sanitize=path == _LIB_SAN)
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        lib.oracle_attn_rows.argtypes = [p, p, p, ctypes.c_int, p, p, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_double, ctypes.c_int64, p, p, p, p, p]
        lib.oracle_attn_rows.restype = ctypes.c_int
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def attention_rows(q, k, v, q_indptr, kv_indptr, num_q_heads, num_kv_heads, scale,
                   row_token, row_head):
    """Attention outputs of the listed (token, head) rows.

    q: uint16 bf16 bits [sum q][Hq][D]; k, v: uint16 [sum kv][Hkv][D] (contiguous,
    logical order per sequence); q_indptr / kv_indptr: [B+1].
    Returns (out [n][D] float64, lse [n] float64, n_keys [n] int64).
    """
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    qi = np.ascontiguousarray(q_indptr, dtype=np.int64)
    ki = np.ascontiguousarray(kv_indptr, dtype=np.int64)
    rt = np.ascontiguousarray(row_token, dtype=np.int64)
    rh = np.ascontiguousarray(row_head, dtype=np.int32)
    D = q.shape[-1]
    n = rt.shape[0]
    out = np.zeros((n, D), dtype=np.float64)
    lse = np.zeros(n, dtype=np.float64)
    nk = np.zeros(n, dtype=np.int64)
    rc = _load().oracle_attn_rows(_ptr(q), _ptr(k), _ptr(v), len(qi) - 1, _ptr(qi), _ptr(ki),
                                  int(num_q_heads), int(num_kv_heads), int(D), float(scale),
                                  n, _ptr(rt), _ptr(rh), _ptr(out), _ptr(lse), _ptr(nk))
    if rc != 0:
        raise ValueError("oracle_attn_rows rejected its inputs")
    return out, lse, nk


def attention_all(q, k, v, q_indptr, kv_indptr, num_q_heads, num_kv_heads, scale):
    """Every (token, head) output, shaped [sum q][Hq][D] (and lse [sum q][Hq])."""
    T = int(q_indptr[-1])
    tok = np.repeat(np.arange(T, dtype=np.int64), num_q_heads)
    head = np.tile(np.arange(num_q_heads, dtype=np.int32), T)
    out, lse, nk = attention_rows(q, k, v, q_indptr, kv_indptr, num_q_heads, num_kv_heads,
                                  scale, tok, head)
    D = q.shape[-1]
    return out.reshape(T, num_q_heads, D), lse.reshape(T, num_q_heads), nk.reshape(T, num_q_heads)
