"""ctypes binding of ``libfesc.so`` (declared in ``include/fesc.h``).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Device buffers are torch tensors on the GPU (int64 storage holding
uint64 residues, all below 2^50); torch supplies memory and the current HIP
stream.  There is no fallback path: if the library is missing this module
raises at import.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfesc.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_17442_amd.build`")

_lib = ctypes.CDLL(LIB_PATH)

_u32, _u64, _i32, _sz, _vp = (ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32,
                              ctypes.c_size_t, ctypes.c_void_p)


class _Params(ctypes.Structure):
    _fields_ = [("log_n", _u32), ("num_q", _u32), ("num_p", _u32), ("dnum", _u32),
                ("q", ctypes.POINTER(_u64)), ("p", ctypes.POINTER(_u64))]


_SIGS = {
    "fesc_ctx_create": [ctypes.POINTER(_Params), ctypes.POINTER(_vp)],
    "fesc_ctx_destroy": [_vp],
    "fesc_last_error": [],
    "fesc_find_primes": [_u32, _u32, _u32, ctypes.POINTER(_u64)],
    "fesc_root_of_unity": [_u32, _u64, ctypes.POINTER(_u64)],
    "fesc_get_psi": [_vp, _u32, ctypes.POINTER(_u64)],
    "fesc_ntt_fwd": [_vp, _vp, _u32, _sz, _u32, _sz, _u32, _vp],
    "fesc_ntt_inv": [_vp, _vp, _u32, _sz, _u32, _sz, _u32, _vp],
    "fesc_mac": [_vp, _vp, _vp, _vp, _u32, _sz, _u32, _u32, _vp],
}

for _name, _args in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int
_lib.fesc_ctx_destroy.restype = None
_lib.fesc_last_error.restype = ctypes.c_char_p


class FescError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"fesc error {code}: {msg}")
        self.code = code


def _check(rc: int) -> int:
    if rc < 0:
        raise FescError(rc, _lib.fesc_last_error().decode())
    return rc


def _ptr(t) -> int:
    if t is None:
        return None
    assert isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.int64, \
        "device buffers are CUDA int64 tensors"
    assert t.is_contiguous()
    return t.data_ptr()


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def find_primes(log_n: int, bits: int, count: int) -> list[int]:
    buf = (_u64 * count)()
    got = _check(_lib.fesc_find_primes(log_n, bits, count, buf))
    return [int(buf[i]) for i in range(got)]


def root_of_unity(log_n: int, q: int) -> int:
    v = _u64()
    _check(_lib.fesc_root_of_unity(log_n, q, ctypes.byref(v)))
    return int(v.value)


class Context:
    """A parameter set (ring degree, ciphertext and special primes) on the
    current device."""

    def __init__(self, log_n: int, q: list, p: list):
        self.log_n, self.n = log_n, 1 << log_n
        self.q, self.p = [int(x) for x in q], [int(x) for x in p]
        self.L, self.alpha = len(self.q), len(self.p)
        self.dnum = -(-self.L // self.alpha)
        qa, pa = (_u64 * self.L)(*self.q), (_u64 * self.alpha)(*self.p)
        params = _Params(log_n, self.L, self.alpha, self.dnum, qa, pa)
        h = _vp()
        _check(_lib.fesc_ctx_create(ctypes.byref(params), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            _lib.fesc_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def psi(self, idx: int) -> int:
        v = _u64()
        _check(_lib.fesc_get_psi(self._h, idx, ctypes.byref(v)))
        return int(v.value)

    # -- transforms and Hadamard products --------------------------------

    def ntt_fwd(self, d, batch, batch_stride, limbs, limb_stride, prime0, stream=None):
        _check(_lib.fesc_ntt_fwd(self._h, _ptr(d), batch, batch_stride, limbs, limb_stride,
                                 prime0, _stream(stream)))

    def ntt_inv(self, d, batch, batch_stride, limbs, limb_stride, prime0, stream=None):
        _check(_lib.fesc_ntt_inv(self._h, _ptr(d), batch, batch_stride, limbs, limb_stride,
                                 prime0, _stream(stream)))

    def mac(self, a, b, out, pairs, pair_stride, limbs, prime0, stream=None):
        _check(_lib.fesc_mac(self._h, _ptr(a), _ptr(b), _ptr(out), pairs, pair_stride, limbs,
                             prime0, _stream(stream)))
