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
    "fesc_add": [_vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_sub": [_vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_mul_plain": [_vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_mul_monomial": [_vp, _vp, _vp, _u32, _u32, _vp],
    "fesc_mul_relin": [_vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_rescale": [_vp, _vp, _vp, _u32, _vp],
    "fesc_mul_relin_rescale": [_vp, _u32, ctypes.POINTER(_vp), ctypes.POINTER(_vp),
                               ctypes.POINTER(_vp), _u32, _vp],
    "fesc_galois_element": [_vp, _i32, ctypes.POINTER(_u32)],
    "fesc_rotate": [_vp, _vp, _vp, _u32, _i32, _vp],
    "fesc_rotate_hoisted": [_vp, _vp, _u32, ctypes.POINTER(_i32), ctypes.POINTER(_vp), _u32,
                            _vp],
    "fesc_rotate_batch": [_vp, _u32, ctypes.POINTER(_vp), ctypes.POINTER(_i32),
                          ctypes.POINTER(_vp), _u32, _vp],
    "fesc_rotate_batch_noalloc": [_vp, _u32, ctypes.POINTER(_vp), ctypes.POINTER(_i32),
                                  ctypes.POINTER(_vp), _u32, _vp],
    "fesc_keygen": [_vp, _u32, _vp, _vp, _vp, _vp],
    "fesc_keygen_seeded": [_vp, _u32, _vp, _vp, _vp, _vp],
    "fesc_key_load": [_vp, _u32, _vp, _vp],
    "fesc_key_store": [_vp, _u32, _vp, _vp],
    "fesc_key_upload": [_vp, _u32, _vp, _u32, _vp],
    "fesc_encrypt_sk": [_vp, _vp, _vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_plain_from_coeffs": [_vp, _vp, _vp, _u32, _vp],
    "fesc_encode": [_u32, _vp, _vp, ctypes.c_double, _vp],
    "fesc_scan_contract": [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.POINTER(_vp),
                           _u32, _u32, _u32, ctypes.POINTER(_vp), _u32, _vp],
    "fesc_calib_valu": [_vp, ctypes.c_int, _u32, ctypes.POINTER(ctypes.c_double), _vp],
    "fesc_affine_scan": [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _u32, _u32, _u32, _u32,
                         ctypes.POINTER(_u32), _vp],
    "fesc_affine_scan_info": [_vp, _u32, _u32, _u32, ctypes.POINTER(_u32), ctypes.POINTER(_u64)],
    "fesc_affine_scan_network": [_u32, _u32, ctypes.POINTER(_u32), _sz, ctypes.POINTER(_sz)],
    "fesc_affine_scan_resident_program": [_u32, _u32, ctypes.POINTER(_u64), _sz,
                                          ctypes.POINTER(_sz)],
    "fesc_affine_scan_program": [_u32, _u32, _u32, ctypes.POINTER(_u64), _sz,
                                 ctypes.POINTER(_sz)],
    "fesc_affine_scan_resident_info": [_vp, _u32, _u32, _u32, _u32, ctypes.POINTER(_u32),
                                       ctypes.POINTER(_sz), ctypes.POINTER(_u64)],
    "fesc_heconv": [_vp, _vp, _u32, ctypes.POINTER(_i32), ctypes.POINTER(_vp), _vp, _vp, _u32,
                    _vp],
    "fesc_post_ssm": [_vp, _vp, _vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_add_plain": [_vp, _vp, _vp, _vp, _u32, _vp],
    "fesc_encode_plain": [_vp, _vp, _u32, ctypes.c_double, _vp, _u32, _vp],
    "fesc_encode_plain_ext": [_vp, _vp, _u32, ctypes.c_double, _vp, _u32, _vp],
    "fesc_decode_plain": [_vp, _vp, _u32, _u32, ctypes.c_double, _vp, _vp],
    "fesc_c2m_level": [ctypes.POINTER(_u64), _u32, _u32, _u32, ctypes.c_double, ctypes.c_double,
                       ctypes.POINTER(_u32)],
    "fesc_affine_scan_resident": [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _u32, _u32,
                                  _u32, ctypes.POINTER(_vp), _u32, _vp, _sz, _vp],
}

CONJ = -(2 ** 31)
CALIB_CT, CALIB_GS, CALIB_MAC, CALIB_MODMUL_F64, CALIB_MODMUL_U64, CALIB_PHILOX = 0, 1, 2, 3, 4, 5
CALIB_HBM_READ, CALIB_HBM_COPY = 0, 1
SCAN_STATES_ONLY = 1

for _name, _args in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int
_lib.fesc_calib_hbm.argtypes = [_vp, ctypes.c_int, ctypes.c_size_t, ctypes.POINTER(ctypes.c_double),
                               _vp]
_lib.fesc_calib_hbm.restype = ctypes.c_int
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


def _ptr(t, words: int = 0, what: str = "buffer", dtype=torch.int64):
    """Device address of a contiguous CUDA tensor of `dtype` holding at least
    `words` elements of that type (None -> NULL).  Residues, coefficients and
    keys are int64 (8 bytes per word); only the secret is int8.  The size
    check is in bytes, so no other element type can pass for a shorter
    buffer than the library reads or writes."""
    if t is None:
        return None
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dtype):
        raise TypeError(f"{what}: expected a CUDA {dtype} tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what}: tensor must be contiguous")
    need = words * torch.empty((), dtype=dtype).element_size()
    have = t.numel() * t.element_size()
    if have < need:
        raise ValueError(f"{what}: {have} bytes, the call reads or writes {need}")
    return t.data_ptr()


def _ptrs(ts, count: int, words: int, what: str):
    """ctypes array of `count` device addresses (each buffer >= words)."""
    if len(ts) != count:
        raise ValueError(f"{what}: {len(ts)} buffers, expected {count}")
    return (_vp * max(count, 1))(*[_ptr(t, words, what) for t in ts])


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

    def _rows(self, batch, batch_stride, limbs, limb_stride):
        if batch == 0 or limbs == 0:
            return 0
        return (batch - 1) * batch_stride + (limbs - 1) * limb_stride + self.n

    def ntt_fwd(self, d, batch, batch_stride, limbs, limb_stride, prime0, stream=None):
        _check(_lib.fesc_ntt_fwd(self._h, _ptr(d, self._rows(batch, batch_stride, limbs,
                                                             limb_stride), "d"),
                                 batch, batch_stride, limbs, limb_stride, prime0,
                                 _stream(stream)))

    def ntt_inv(self, d, batch, batch_stride, limbs, limb_stride, prime0, stream=None):
        _check(_lib.fesc_ntt_inv(self._h, _ptr(d, self._rows(batch, batch_stride, limbs,
                                                             limb_stride), "d"),
                                 batch, batch_stride, limbs, limb_stride, prime0,
                                 _stream(stream)))

    def mac(self, a, b, out, pairs, pair_stride, limbs, prime0, stream=None):
        w = self._rows(pairs, pair_stride, limbs, self.n)
        _check(_lib.fesc_mac(self._h, _ptr(a, w, "a"), _ptr(b, w, "b"),
                             _ptr(out, limbs * self.n, "out"), pairs, pair_stride, limbs,
                             prime0, _stream(stream)))

    # -- ciphertext operations -------------------------------------------

    # Buffer sizes of a ciphertext / plaintext at `level`; a level the context
    # does not have is left to the library's own check (FESC_ERR_LEVEL).
    def _ct(self, level):
        return level * 2 * self.n if 1 <= level <= self.L else 0

    def _pt(self, level):
        return level * self.n if 1 <= level <= self.L else 0

    def add(self, a, b, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_add(self._h, _ptr(a, w, "a"), _ptr(b, w, "b"), _ptr(out, w, "out"),
                             level, _stream(stream)))

    def sub(self, a, b, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_sub(self._h, _ptr(a, w, "a"), _ptr(b, w, "b"), _ptr(out, w, "out"),
                             level, _stream(stream)))

    def mul_plain(self, ct, pt, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_mul_plain(self._h, _ptr(ct, w, "ct"), _ptr(pt, self._pt(level), "pt"),
                                   _ptr(out, w, "out"), level, _stream(stream)))

    def mul_monomial(self, ct, out, level, k, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_mul_monomial(self._h, _ptr(ct, w, "ct"), _ptr(out, w, "out"), level, k,
                                      _stream(stream)))

    def mul_relin(self, a, b, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_mul_relin(self._h, _ptr(a, w, "a"), _ptr(b, w, "b"),
                                   _ptr(out, w, "out"), level, _stream(stream)))

    def mul_relin_rescale(self, a, b, outs, level, stream=None):
        """out_i = relin(a_i * b_i) / (P q_{level-1}), batched (level - 1)."""
        m, w = len(a), self._ct(level)
        _check(_lib.fesc_mul_relin_rescale(self._h, m, _ptrs(a, m, w, "a"), _ptrs(b, m, w, "b"),
                                           _ptrs(outs, m, self._ct(level - 1), "outs"), level,
                                           _stream(stream)))

    def rescale(self, ct, out, level, stream=None):
        _check(_lib.fesc_rescale(self._h, _ptr(ct, self._ct(level), "ct"),
                                 _ptr(out, self._ct(level - 1), "out"), level, _stream(stream)))

    def galois_element(self, step: int) -> int:
        v = _u32()
        _check(_lib.fesc_galois_element(self._h, step, ctypes.byref(v)))
        return int(v.value)

    def rotate(self, ct, out, level, step, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_rotate(self._h, _ptr(ct, w, "ct"), _ptr(out, w, "out"), level, step,
                                _stream(stream)))

    def rotate_hoisted(self, ct, steps, outs, level, stream=None):
        m, w = len(steps), self._ct(level)
        _check(_lib.fesc_rotate_hoisted(self._h, _ptr(ct, w, "ct"), m, (_i32 * max(m, 1))(*steps),
                                        _ptrs(outs, m, w, "outs"), level, _stream(stream)))

    def rotate_batch(self, cts, steps, outs, level, stream=None):
        m, w = len(cts), self._ct(level)
        if len(steps) != m:
            raise ValueError(f"steps: {len(steps)} values, expected {m}")
        _check(_lib.fesc_rotate_batch(self._h, m, _ptrs(cts, m, w, "cts"),
                                      (_i32 * max(m, 1))(*steps), _ptrs(outs, m, w, "outs"),
                                      level, _stream(stream)))

    def rotate_batch_noalloc(self, cts, steps, outs, level, stream=None):
        """fesc_rotate_batch_noalloc: the same batch with its temporaries in
        the library's statically allocated device array (no allocation)."""
        m, w = len(cts), self._ct(level)
        if len(steps) != m:
            raise ValueError(f"steps: {len(steps)} values, expected {m}")
        _check(_lib.fesc_rotate_batch_noalloc(self._h, m, _ptrs(cts, m, w, "cts"),
                                              (_i32 * max(m, 1))(*steps),
                                              _ptrs(outs, m, w, "outs"), level,
                                              _stream(stream)))

    def keygen(self, galois_elt, s, a, e, stream=None):
        E = self.L + self.alpha
        _check(_lib.fesc_keygen(self._h, galois_elt, _ptr(s, self.n, "s", torch.int8),
                                _ptr(a, self.dnum * E * self.n, "a"),
                                _ptr(e, self.dnum * self.n, "e"), _stream(stream)))

    def keygen_seeded(self, galois_elt, s, seed_words, e, stream=None):
        """fesc_keygen_seeded: the key's uniform half drawn from two 64-bit
        seed words (host integers); the context keeps the seed and b only."""
        w = [int(v) for v in seed_words]
        if len(w) != 2 or not all(0 <= v < 1 << 64 for v in w):
            raise ValueError("seed_words: two integers in [0, 2^64)")
        seed = (ctypes.c_uint64 * 2)(*w)
        _check(_lib.fesc_keygen_seeded(self._h, galois_elt, _ptr(s, self.n, "s", torch.int8),
                                       ctypes.addressof(seed),
                                       _ptr(e, self.dnum * self.n, "e"), _stream(stream)))

    def key_load(self, galois_elt, key, stream=None):
        _check(_lib.fesc_key_load(self._h, galois_elt, _ptr(key, self.key_words(), "key"),
                                  _stream(stream)))

    def key_upload(self, galois_elt, host_key, key_level, stream=None):
        """Host numpy uint64 key over the chain prefix of key_level primes,
        [ceil(key_level/alpha)][key_level+alpha][2][N]."""
        import numpy as np
        hk = np.ascontiguousarray(host_key, dtype=np.uint64)
        dk = -(-int(key_level) // self.alpha)
        need = dk * (int(key_level) + self.alpha) * 2 * self.n
        if hk.size < need:
            raise ValueError(f"host_key: {hk.size} words, the call reads {need}")
        _check(_lib.fesc_key_upload(self._h, galois_elt, hk.ctypes.data, key_level,
                                    _stream(stream)))

    def key_store(self, galois_elt, key, stream=None):
        _check(_lib.fesc_key_store(self._h, galois_elt, _ptr(key, self.key_words(), "key"),
                                   _stream(stream)))

    def encrypt_sk(self, s, m, a, e, ct, level, stream=None):
        _check(_lib.fesc_encrypt_sk(self._h, _ptr(s, self.n, "s", torch.int8), _ptr(m, self.n, "m"),
                                    _ptr(a, self._pt(level), "a"), _ptr(e, self.n, "e"),
                                    _ptr(ct, self._ct(level), "ct"), level, _stream(stream)))

    def plain_from_coeffs(self, m, pt, level, stream=None):
        _check(_lib.fesc_plain_from_coeffs(self._h, _ptr(m, self.n, "m"),
                                           _ptr(pt, self._pt(level), "pt"), level,
                                           _stream(stream)))

    def scan_contract(self, h, decay, cfac, d_state, outs, level, tokens=1, stream=None):
        """Lists of tokens * chunks ciphertexts, token-major; decay None for
        the contraction alone."""
        m, w = len(h), self._ct(level)
        if tokens < 1 or m % tokens:
            raise ValueError(f"{m} ciphertexts do not split into {tokens} tokens")
        lo = level - (1 if decay is None else 2)
        dec = None if decay is None else _ptrs(decay, m, w, "decay")
        _check(_lib.fesc_scan_contract(self._h, _ptrs(h, m, w, "h"), dec, _ptrs(cfac, m, w, "cfac"),
                                       m // tokens, tokens, d_state,
                                       _ptrs(outs, m, self._ct(max(lo, 0)), "outs"), level,
                                       _stream(stream)))

    def affine_scan(self, a, s, chunks, level, states_only=False, stream=None) -> int:
        """In-place Brent-Kung scan of `chunks` sequences of len(a) // chunks
        token maps (a[c*L + k], s[c*L + k]); returns the output level."""
        n, w = len(a), self._ct(level)
        if chunks < 1 or n % chunks:
            raise ValueError(f"{n} tuples do not split into {chunks} chunks")
        out = _u32()
        _check(_lib.fesc_affine_scan(self._h, _ptrs(a, n, w, "a"), _ptrs(s, n, w, "s"),
                                     n // chunks, chunks, level,
                                     SCAN_STATES_ONLY if states_only else 0, ctypes.byref(out),
                                     _stream(stream)))
        return int(out.value)

    def affine_scan_info(self, L, level, states_only=False):
        """(output level, key switches per chunk) of affine_scan."""
        lo, ks = _u32(), _u64()
        _check(_lib.fesc_affine_scan_info(self._h, L, level, SCAN_STATES_ONLY if states_only else 0,
                                          ctypes.byref(lo), ctypes.byref(ks)))
        return int(lo.value), int(ks.value)

    def affine_scan_resident_info(self, L, chunks, block, level):
        """(output level, workspace bytes, key switches per chunk) of the
        resident schedule."""
        lo, ws, ks = _u32(), _sz(), _u64()
        _check(_lib.fesc_affine_scan_resident_info(self._h, L, chunks, block, level,
                                                   ctypes.byref(lo), ctypes.byref(ws),
                                                   ctypes.byref(ks)))
        return int(lo.value), int(ws.value), int(ks.value)

    def affine_scan_resident(self, a, s, chunks, block, h, level, workspace, stream=None):
        """States of the resident block schedule into h (see the C header)."""
        n, w = len(a), self._ct(level)
        if chunks < 1 or n % chunks:
            raise ValueError(f"{n} tuples do not split into {chunks} chunks")
        lo, _, _ = self.affine_scan_resident_info(n // chunks, chunks, block, level)
        ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
        _check(_lib.fesc_affine_scan_resident(self._h, _ptrs(a, n, w, "a"), _ptrs(s, n, w, "s"),
                                              n // chunks, chunks, block,
                                              _ptrs(h, n, self._ct(lo), "h"), level,
                                              _ptr(workspace) if ws_bytes else None,
                                              ws_bytes, _stream(stream)))

    def heconv(self, q, deltas, masks, bias, out, level, stream=None):
        """out = RS(sum_r masks[r] (.) rho(q; deltas[r])) + bias (see the C header)."""
        t = len(deltas)
        _check(_lib.fesc_heconv(self._h, _ptr(q, self._ct(level), "q"), t,
                                (_i32 * max(t, 1))(*deltas),
                                _ptrs(masks, t, self._pt(level), "masks"),
                                _ptr(bias, self._pt(level), "bias"),
                                _ptr(out, self._ct(level - 1), "out"), level, _stream(stream)))

    def post_ssm(self, m, x_skip, d_skip, g, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_post_ssm(self._h, _ptr(m, w, "m"), _ptr(x_skip, w, "x_skip"),
                                  _ptr(d_skip, self._pt(level), "d_skip"), _ptr(g, w, "g"),
                                  _ptr(out, self._ct(level - 2), "out"), level,
                                  _stream(stream)))

    def add_plain(self, ct, pt, out, level, stream=None):
        w = self._ct(level)
        _check(_lib.fesc_add_plain(self._h, _ptr(ct, w, "ct"), _ptr(pt, self._pt(level), "pt"),
                                   _ptr(out, w, "out"), level, _stream(stream)))

    def encode_plain(self, z, scale, pt, level, stream=None):
        """Device encoding: z a complex128 CUDA tensor [count][N/2] (or [N/2])
        -> evaluation-form plaintexts pt (int64 tensor, [count][level][N])."""
        zr = torch.view_as_real(z.reshape(-1, self.n // 2)).contiguous()
        if not (zr.is_cuda and zr.dtype == torch.float64):
            raise TypeError("z: a complex128 CUDA tensor")
        count = zr.shape[0]
        _check(_lib.fesc_encode_plain(self._h, zr.data_ptr(), count, float(scale),
                                      _ptr(pt, count * self._pt(level), "pt"), level,
                                      _stream(stream)))

    def encode_plain_ext(self, z, scale, pt, level, stream=None):
        """Device encoding over the extended basis of `level` (q_0..q_{level-1},
        p_0..p_{alpha-1}): pt [count][level+alpha][N]."""
        zr = torch.view_as_real(z.reshape(-1, self.n // 2)).contiguous()
        if not (zr.is_cuda and zr.dtype == torch.float64):
            raise TypeError("z: a complex128 CUDA tensor")
        count = zr.shape[0]
        _check(_lib.fesc_encode_plain_ext(self._h, zr.data_ptr(), count, float(scale),
                                          _ptr(pt, count * (level + self.alpha) * self.n, "pt"),
                                          level, _stream(stream)))

    def decode_plain(self, pt, count, level, scale, z, stream=None):
        """Device decoding: evaluation-form plaintexts pt (int64 tensor,
        [count][level][N]) -> slot vectors z (complex128 CUDA tensor,
        [count][N/2])."""
        if not (z.is_cuda and z.dtype == torch.complex128 and z.is_contiguous()):
            raise TypeError("z: a contiguous complex128 CUDA tensor")
        if z.numel() < count * (self.n // 2):
            raise ValueError(f"z: {z.numel()} slots, the call writes {count * (self.n // 2)}")
        _check(_lib.fesc_decode_plain(self._h, _ptr(pt, count * self._pt(level), "pt"), count,
                                      level, float(scale), z.data_ptr(), _stream(stream)))

    def key_words(self) -> int:
        return self.dnum * (self.L + self.alpha) * 2 * self.n

    def calib_hbm(self, kind: int, nbytes: int = 8 << 30, stream=None) -> float:
        """Measured streaming HBM rate (bytes/s): CALIB_HBM_READ or
        CALIB_HBM_COPY (read plus write) over an nbytes buffer."""
        r = ctypes.c_double()
        _check(_lib.fesc_calib_hbm(self._h, kind, ctypes.c_size_t(nbytes), ctypes.byref(r),
                                   _stream(stream)))
        return float(r.value)

    def calib_valu(self, kind: int, iters: int = 4096, stream=None) -> float:
        """Measured register-resident rate (operations/s) of NTT butterflies
        (CALIB_CT, CALIB_GS) or modular multiply-accumulates (CALIB_MAC)."""
        r = ctypes.c_double()
        _check(_lib.fesc_calib_valu(self._h, kind, iters, ctypes.byref(r), _stream(stream)))
        return float(r.value)


def c2m_level(q, level: int, ell: int, sigma: int, delta: float, bmax: float) -> int:
    """Smallest admissible conversion level (0: none); host-only."""
    qs = (_u64 * len(q))(*q)
    out = _u32()
    _check(_lib.fesc_c2m_level(qs, level, ell, sigma, float(delta), float(bmax),
                               ctypes.byref(out)))
    return int(out.value)


def affine_scan_network(L: int, states_only: bool = False):
    """Nodes (stage, dst, src, decay) of the affine scan's network; host-only."""
    flags = SCAN_STATES_ONLY if states_only else 0
    cnt = _sz()
    _check(_lib.fesc_affine_scan_network(L, flags, None, 0, ctypes.byref(cnt)))
    buf = (_u32 * (4 * max(cnt.value, 1)))()
    _check(_lib.fesc_affine_scan_network(L, flags, buf, cnt.value, ctypes.byref(cnt)))
    return [tuple(buf[4 * i:4 * i + 4]) for i in range(cnt.value)]


def affine_scan_program(L: int, chunks: int, states_only: bool = False):
    """Products (group, x, y, add, out) of the in-place scan; host-only."""
    flags = SCAN_STATES_ONLY if states_only else 0
    cnt = _sz()
    _check(_lib.fesc_affine_scan_program(L, chunks, flags, None, 0, ctypes.byref(cnt)))
    buf = (_u64 * (5 * max(cnt.value, 1)))()
    _check(_lib.fesc_affine_scan_program(L, chunks, flags, buf, cnt.value, ctypes.byref(cnt)))
    return [tuple(buf[5 * i:5 * i + 5]) for i in range(cnt.value)]


def affine_scan_resident_program(L: int, block: int):
    """Products (group, x, y, add, out) of the resident schedule; host-only."""
    cnt = _sz()
    _check(_lib.fesc_affine_scan_resident_program(L, block, None, 0, ctypes.byref(cnt)))
    buf = (_u64 * (5 * max(cnt.value, 1)))()
    _check(_lib.fesc_affine_scan_resident_program(L, block, buf, cnt.value, ctypes.byref(cnt)))
    return [tuple(buf[5 * i:5 * i + 5]) for i in range(cnt.value)]


def encode(log_n: int, z, scale: float):
    """Host encoder: complex slot vector (length N/2) -> int64 coefficients."""
    import numpy as np
    z = np.asarray(z, dtype=np.complex128)
    re = np.ascontiguousarray(z.real)
    im = np.ascontiguousarray(z.imag)
    out = np.empty(1 << log_n, dtype=np.int64)
    _check(_lib.fesc_encode(log_n, re.ctypes.data, im.ctypes.data, float(scale),
                            out.ctypes.data))
    return out


class _MatvecDesc(ctypes.Structure):
    _fields_ = [(f, _u32) for f in ("level", "n_in", "n_out", "n1", "n2", "unit",
                                    "real_extract", "rescale", "complex_pair",
                                    "lazy_moddown")]


_lib.fesc_matvec_plan_create.argtypes = [_vp, ctypes.POINTER(_MatvecDesc), ctypes.POINTER(_vp),
                                         ctypes.POINTER(_vp)]
_lib.fesc_matvec_plan_create.restype = ctypes.c_int
_lib.fesc_matvec_plan_destroy.argtypes = [_vp]
_lib.fesc_matvec_plan_destroy.restype = None
_lib.fesc_ptct_matvec.argtypes = [_vp, _vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _vp]
_lib.fesc_ptct_matvec.restype = ctypes.c_int
_lib.fesc_matvec_phase_ms.argtypes = [_vp] + [ctypes.POINTER(ctypes.c_float)] * 3
_lib.fesc_matvec_phase_ms.restype = ctypes.c_int


_lib.fesc_matvec_bank_words.argtypes = [_vp, ctypes.POINTER(_MatvecDesc),
                                        ctypes.POINTER(ctypes.c_size_t)]
_lib.fesc_matvec_bank_words.restype = ctypes.c_int
_lib.fesc_matvec_bank_pack.argtypes = [_vp, ctypes.POINTER(_MatvecDesc), _vp, _u32, _vp, _vp]
_lib.fesc_matvec_bank_pack.restype = ctypes.c_int
_lib.fesc_matvec_bank_pack_many.argtypes = [_vp, ctypes.POINTER(_MatvecDesc), _vp, _u32, _u32,
                                            _vp, _sz, _vp]
_lib.fesc_matvec_bank_pack_many.restype = ctypes.c_int
_lib.fesc_matvec_plan_create_bank.argtypes = [_vp, ctypes.POINTER(_MatvecDesc), _vp,
                                              ctypes.POINTER(_vp)]
_lib.fesc_matvec_plan_create_bank.restype = ctypes.c_int


def matvec_desc(level, n_in, n_out, n1, n2, unit, real_extract, rescale,
                complex_pair=False, lazy_moddown=False) -> _MatvecDesc:
    return _MatvecDesc(level, n_in, n_out, n1, n2, unit, int(real_extract), int(rescale),
                       int(complex_pair), int(lazy_moddown))


def _diag_words(ctx, desc) -> int:
    """Words of one diagonal plaintext (over the extended basis with
    lazy_moddown)."""
    return (desc.level + (ctx.alpha if desc.lazy_moddown else 0)) * ctx.n


_lib.fesc_bsgs_diagonal_slots.argtypes = [_vp, ctypes.POINTER(_MatvecDesc), _vp, _u32, _u32,
                                          _u32, _u32, _u32, _vp, _vp]
_lib.fesc_bsgs_diagonal_slots.restype = ctypes.c_int


def bsgs_diagonal_slots(ctx: Context, desc: _MatvecDesc, W, segs: int, first: int, count: int,
                        z, stream=None):
    """Slot vectors of diagonals first .. first+count-1 (bank order) into the
    device complex128 tensor z [>= count][N/2]; W a device float64
    [d_in][d_out]; segs segments of desc.unit slots per period."""
    if not (isinstance(W, torch.Tensor) and W.is_cuda and W.dtype == torch.float64
            and W.dim() == 2 and W.is_contiguous()):
        raise TypeError("W: expected a contiguous 2-D CUDA float64 tensor")
    if not (isinstance(z, torch.Tensor) and z.is_cuda and z.dtype == torch.complex128
            and z.is_contiguous()):
        raise TypeError("z: expected a contiguous CUDA complex128 tensor")
    if z.numel() < count * (ctx.n // 2):
        raise ValueError(f"z: {z.numel()} slots, the call writes {count * (ctx.n // 2)}")
    _check(_lib.fesc_bsgs_diagonal_slots(ctx._h, ctypes.byref(desc), W.data_ptr(), W.shape[0],
                                         W.shape[1], segs, first, count, z.data_ptr(),
                                         _stream(stream)))


def matvec_bank_words(ctx: Context, desc: _MatvecDesc) -> int:
    w = ctypes.c_size_t()
    _check(_lib.fesc_matvec_bank_words(ctx._h, ctypes.byref(desc), ctypes.byref(w)))
    return int(w.value)


def matvec_bank_pack(ctx: Context, desc: _MatvecDesc, bank, index: int, pt, stream=None):
    _check(_lib.fesc_matvec_bank_pack(ctx._h, ctypes.byref(desc),
                                      _ptr(bank, matvec_bank_words(ctx, desc), "bank"), index,
                                      _ptr(pt, _diag_words(ctx, desc), "pt"), _stream(stream)))


def matvec_bank_pack_many(ctx: Context, desc: _MatvecDesc, bank, first: int, pts, stream=None):
    """Slots first .. first + len(pts) - 1 from the rows of ``pts``, a 2-D
    tensor [count][words >= the plaintext's rows * N], in one launch."""
    count, stride = (pts.shape[0], pts.shape[1]) if pts.dim() == 2 else (0, 0)
    if pts.dim() != 2 or stride < _diag_words(ctx, desc):
        raise ValueError("pts: expected [count][rows * N] plaintexts")
    _check(_lib.fesc_matvec_bank_pack_many(ctx._h, ctypes.byref(desc),
                                           _ptr(bank, matvec_bank_words(ctx, desc), "bank"),
                                           first, count, _ptr(pts, count * stride, "pts"),
                                           stride, _stream(stream)))


class MatvecPlan:
    """BSGS projection plan over pre-encoded diagonals: either ``diags``, a
    flat list of device plaintexts in [b][p][u][q] order, or ``bank``, one
    diagonal bank (see fesc_matvec_bank_pack).  Inputs are kept alive."""

    def __init__(self, ctx: Context, level, n_in, n_out, n1, n2, unit, real_extract, rescale,
                 diags=None, bank=None, complex_pair=False, lazy_moddown=False):
        self.ctx = ctx
        self.desc = matvec_desc(level, n_in, n_out, n1, n2, unit, real_extract, rescale,
                                complex_pair, lazy_moddown)
        h = _vp()
        if bank is not None:
            self._bank = bank
            _check(_lib.fesc_matvec_plan_create_bank(
                ctx._h, ctypes.byref(self.desc),
                _ptr(bank, matvec_bank_words(ctx, self.desc), "bank"), ctypes.byref(h)))
        else:
            self._diags = list(diags)
            arr = _ptrs(self._diags, n_out * n2 * n_in * n1, _diag_words(ctx, self.desc),
                        "diags")
            _check(_lib.fesc_matvec_plan_create(ctx._h, ctypes.byref(self.desc), arr,
                                                ctypes.byref(h)))
        self._h = h

    def __call__(self, ins, outs, stream=None):
        d, c = self.desc, self.ctx
        a = _ptrs(ins, d.n_in, c._ct(d.level), "ins")
        n_res = d.n_out // 2 if d.complex_pair else d.n_out
        b = _ptrs(outs, n_res, c._ct(d.level - (1 if d.rescale else 0)), "outs")
        _check(_lib.fesc_ptct_matvec(self.ctx._h, self._h, a, b, _stream(stream)))

    def phase_ms(self):
        """(baby steps, pt-MAC, tail) durations of the last completed run."""
        v = [ctypes.c_float() for _ in range(3)]
        _check(_lib.fesc_matvec_phase_ms(self._h, *[ctypes.byref(x) for x in v]))
        return tuple(float(x.value) for x in v)

    def close(self):
        if getattr(self, "_h", None):
            _lib.fesc_matvec_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------- slot maps and broadcasts

BR_A, BR_X, BR_B, BR_C = 0, 1, 2, 3
_BR_KIND = {"a": BR_A, "x": BR_X, "B": BR_B, "C": BR_C}


class SlotMapDesc(ctypes.Structure):
    _fields_ = [("level", _u32), ("offset", _i32), ("stride", _i32), ("giant_stride", _i32),
                ("terms", _u32), ("n1", _u32), ("dst0", _u32), ("dst_stride", _u32),
                ("dst_giant", _u32), ("width", _u32), ("rep_stride", _i32), ("rep_count", _u32)]

    @property
    def n2(self) -> int:
        return -(-self.terms // self.n1)


class _BrShape(ctypes.Structure):
    _fields_ = [(f, _u32) for f in ("H", "P", "G", "d_s", "c_state")]


_lib.fesc_br_desc.argtypes = [_u32, ctypes.POINTER(_BrShape), _u32, _u32, _u32, _u32,
                              ctypes.POINTER(SlotMapDesc)]
_lib.fesc_br_desc.restype = ctypes.c_int
_lib.fesc_slot_map_mask_slots.argtypes = [_vp, ctypes.POINTER(SlotMapDesc), _u32, _u32, _vp,
                                          _vp]
_lib.fesc_slot_map_mask_slots.restype = ctypes.c_int
_lib.fesc_slot_map_plan_create.argtypes = [_vp, ctypes.POINTER(SlotMapDesc),
                                           ctypes.POINTER(_vp), ctypes.POINTER(_vp)]
_lib.fesc_slot_map_plan_create.restype = ctypes.c_int
_lib.fesc_slot_map_plan_destroy.argtypes = [_vp]
_lib.fesc_slot_map_plan_destroy.restype = None
_lib.fesc_slot_map.argtypes = [_vp, _vp, _vp, _vp, _vp]
_lib.fesc_slot_map.restype = ctypes.c_int
_lib.fesc_slot_map_batch.argtypes = [_vp, _vp, _u32, ctypes.POINTER(_vp), ctypes.POINTER(_i32),
                                     ctypes.POINTER(_vp), _vp]
_lib.fesc_slot_map_batch.restype = ctypes.c_int


def br_desc(log_n: int, H: int, P: int, G: int, d_s: int, c_state: int, kind: str, k: int,
            kappa: int, level: int) -> SlotMapDesc:
    """Slot map of br^(kappa) for token k's factor `kind` ("a", "x", "B" or
    "C"); host only."""
    d = SlotMapDesc()
    _check(_lib.fesc_br_desc(log_n, ctypes.byref(_BrShape(H, P, G, d_s, c_state)),
                             _BR_KIND[kind], k, kappa, level, ctypes.byref(d)))
    return d


def slot_map_mask_slots(ctx: Context, desc: SlotMapDesc, first: int, count: int, z,
                        stream=None):
    """Mask slot vectors first .. first+count-1 into the device complex128
    tensor z [>= count][N/2] (encode them at the scale of q_{level-1})."""
    if not (isinstance(z, torch.Tensor) and z.is_cuda and z.dtype == torch.complex128
            and z.is_contiguous()):
        raise TypeError("z: expected a contiguous CUDA complex128 tensor")
    if z.numel() < count * (ctx.n // 2):
        raise ValueError(f"z: {z.numel()} slots, the call writes {count * (ctx.n // 2)}")
    _check(_lib.fesc_slot_map_mask_slots(ctx._h, ctypes.byref(desc), first, count,
                                         z.data_ptr(), _stream(stream)))


class SlotMapPlan:
    """Homomorphic slot map over encoded masks (device plaintexts, one per
    term, [level][N]); inputs are kept alive."""

    def __init__(self, ctx: Context, desc: SlotMapDesc, masks):
        self.ctx, self.desc = ctx, desc
        self._masks = list(masks)
        h = _vp()
        _check(_lib.fesc_slot_map_plan_create(
            ctx._h, ctypes.byref(desc), _ptrs(self._masks, desc.terms, ctx._pt(desc.level),
                                               "masks"), ctypes.byref(h)))
        self._h = h

    def __call__(self, ct, out, stream=None):
        c, d = self.ctx, self.desc
        _check(_lib.fesc_slot_map(c._h, self._h, _ptr(ct, c._ct(d.level), "ct"),
                                  _ptr(out, c._ct(d.level - 1), "out"), _stream(stream)))

    def batch(self, cts, offsets, outs, stream=None):
        """fesc_slot_map_batch: the map over several inputs, item i rotated
        first by offsets[i]."""
        c, d, m = self.ctx, self.desc, len(cts)
        if len(offsets) != m:
            raise ValueError(f"offsets: {len(offsets)} values, expected {m}")
        _check(_lib.fesc_slot_map_batch(c._h, self._h, m, _ptrs(cts, m, c._ct(d.level), "cts"),
                                        (_i32 * max(m, 1))(*offsets),
                                        _ptrs(outs, m, c._ct(d.level - 1), "outs"),
                                        _stream(stream)))

    def close(self):
        if getattr(self, "_h", None):
            _lib.fesc_slot_map_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
