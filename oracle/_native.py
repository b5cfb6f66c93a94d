"""Build and load the oracle's C core (``ckks_oracle.c``) with gcc.

Test infrastructure only (see the package docstring)."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ckks_oracle.c")
_LIB = os.path.join(_HERE, "libckks_oracle.so")

_u64p = ctypes.POINTER(ctypes.c_uint64)
_i64p = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = False) -> str:
    """Compile the C core (gcc -O2 -fopenmp) next to its source."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        u64, i32, lng = ctypes.c_uint64, ctypes.c_int, ctypes.c_long
        sig = {
            "or_mulmod": (u64, [u64, u64, u64]),
            "or_philox4x64": (None, [_u64p, u64, u64, _u64p]),
            "or_seeded_key_a": (None, [_u64p, i32, i32, lng, _u64p, _u64p, u64, u64, u64]),
            "or_powmod": (u64, [u64, u64, u64]),
            "or_invmod": (u64, [u64, u64]),
            "or_is_prime": (i32, [u64]),
            "or_find_primes": (i32, [i32, i32, i32, _u64p]),
            "or_min_psi": (u64, [u64, i32]),
            "or_ntt_fwd_rows": (None, [_u64p, lng, i32, _u64p, _u64p]),
            "or_ntt_inv_rows": (None, [_u64p, lng, i32, _u64p, _u64p]),
            "or_mul_rows": (None, [_u64p, _u64p, _u64p, lng, lng, _u64p]),
            "or_mac_rows": (None, [_u64p, _u64p, _u64p, lng, lng, lng, _u64p]),
            "or_mul_scalar_rows": (None, [_u64p, _u64p, lng, lng, _u64p, _u64p]),
            "or_add_rows": (None, [_u64p, _u64p, _u64p, lng, lng, _u64p]),
            "or_sub_rows": (None, [_u64p, _u64p, _u64p, lng, lng, _u64p]),
            "or_lift_signed_rows": (None, [_i64p, _u64p, lng, lng, _u64p]),
            "or_automorph_coef_rows": (None, [_u64p, _u64p, lng, i32, _u64p, u64]),
            "or_fast_bconv": (None, [_u64p, i32, _u64p, _u64p, i32, _u64p, lng]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def u64p(a: np.ndarray):
    assert a.dtype == np.uint64 and a.flags["C_CONTIGUOUS"], (a.dtype, a.flags)
    return a.ctypes.data_as(_u64p)


def i64p(a: np.ndarray):
    assert a.dtype == np.int64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_i64p)


def moduli(qs) -> np.ndarray:
    return np.ascontiguousarray(np.asarray([int(q) for q in qs], dtype=np.uint64))
