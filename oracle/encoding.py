"""CKKS slot encoding and decoding for the oracle (test infrastructure only).

The paper packs n = N/2 complex slots into R = Z[X]/(X^N + 1) (Sec. 2.1) and
rotates them cyclically, rho(v; r)_j = v_{(j + r) mod n} (Sec. 4.1).  Neither
the slot ordering nor the rounding is printed; this module fixes them:

* slot j is the evaluation of the plaintext polynomial at zeta^(5^j mod 2N),
  zeta = exp(i pi / N), j < n, so the automorphism X -> X^(5^r) rotates the
  slots left by r and X -> X^(2N-1) conjugates them;
* encode(z, Delta) is the real polynomial m with m(zeta^(5^j)) = Delta z_j and
  m(zeta^(-5^j)) = Delta conj(z_j), i.e.
      m_k = (2/N) Re( sum_j Delta z_j zeta^(-5^j k) ),
  rounded half away from zero.  It is evaluated with one length-N FFT over the
  odd exponents t = 2u + 1:  m_k = (1/N) zeta^-k sum_u Z[2u+1] w^(-uk),
  w = zeta^2;
* decode is the plain evaluation z_j = m(zeta^(5^j)) / Delta, again by one FFT,
  after an exact CRT lift of the residues (centred in (-Q/2, Q/2]).
"""
from __future__ import annotations

import numpy as np


def slot_exponents(n_slots: int, two_n: int) -> np.ndarray:
    """e_j = 5^j mod 2N for j < n_slots."""
    e = np.empty(n_slots, dtype=np.int64)
    x = 1
    for j in range(n_slots):
        e[j] = x
        x = (x * 5) % two_n
    return e


def _round_half_away(x: np.ndarray) -> np.ndarray:
    return np.where(x >= 0, np.floor(x + 0.5), -np.floor(-x + 0.5))


def encode_real_coeffs(z: np.ndarray, scale: float, n: int) -> np.ndarray:
    """Unrounded real coefficients Delta * m_k (float64, length n)."""
    n_slots = n // 2
    z = np.asarray(z, dtype=np.complex128)
    assert z.shape == (n_slots,), (z.shape, n_slots)
    e = slot_exponents(n_slots, 2 * n)
    y = np.zeros(n, dtype=np.complex128)
    y[(e - 1) // 2] = z
    y[(2 * n - e - 1) // 2] = np.conj(z)
    k = np.arange(n)
    w = np.fft.fft(y) * np.exp(-1j * np.pi * k / n) / n
    return w.real * scale


def encode(z: np.ndarray, scale: float, n: int) -> np.ndarray:
    """int64 coefficients of the encoding of slot vector z at scale Delta."""
    c = _round_half_away(encode_real_coeffs(z, scale, n))
    assert np.all(np.abs(c) < 2.0 ** 63), "encoded coefficient exceeds int64"
    return c.astype(np.int64)


def decode_coeffs(m, scale: float, n: int) -> np.ndarray:
    """Slots of a real coefficient vector m (any numeric / object dtype)."""
    mf = np.asarray([float(v) for v in m], dtype=np.float64) if np.asarray(m).dtype == object \
        else np.asarray(m, dtype=np.float64)
    n_slots = n // 2
    e = slot_exponents(n_slots, 2 * n)
    k = np.arange(n)
    v = np.fft.ifft(mf * np.exp(1j * np.pi * k / n)) * n
    return v[(e - 1) // 2] / scale


def crt_centered(res: np.ndarray, qs) -> np.ndarray:
    """Exact CRT lift of ``u64[l][N]`` residues to Python ints in (-Q/2, Q/2]."""
    qs = [int(q) for q in qs]
    Q = 1
    for q in qs:
        Q *= q
    acc = np.zeros(res.shape[1], dtype=object)
    for i, q in enumerate(qs):
        Qi = Q // q
        Mi = pow(Qi % q, -1, q)
        acc = acc + ((res[i].astype(object) * Mi) % q) * Qi
    acc = acc % Q
    half = Q // 2
    return np.where(acc > half, acc - Q, acc)
