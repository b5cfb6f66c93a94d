"""Seeded synthetic input draws shared by the tests, the benchmark and the CPU
reference.

This module holds random draws only: no ring arithmetic, no modular products,
no transforms.  Everything the CKKS computation needs from randomness (the
secret, the uniform masks, the error polynomials, the workload values) is drawn
here and handed to either side as plain arrays, so the GPU library and the CPU
reference see identical randomness by construction.

Generator: numpy's Philox (a counter-based generator, Salmon et al., SC 2011)
keyed through ``numpy.random.SeedSequence([seed, *tag_words])``.  A *tag* is a
short string naming the role of the draw (e.g. ``"secret"``, ``"ksk-a/g=5"``)
plus integer indices, so that independent roles never share a stream.
"""
from __future__ import annotations

import hashlib

import numpy as np

__all__ = [
    "rng",
    "uniform_residues",
    "ternary_secret",
    "rounded_gaussian",
    "uniform_pm1",
    "normal",
    "moduli_tag",
    "switch_key_seed_draws",
]


def _tag_words(tag: str, *idx: int) -> list[int]:
    h = hashlib.sha256(tag.encode("utf-8")).digest()
    words = [int.from_bytes(h[i:i + 4], "little") for i in range(0, 16, 4)]
    return words + [int(i) & 0xFFFFFFFF for i in idx]


def rng(seed: int, tag: str, *idx: int) -> np.random.Generator:
    """Independent generator for (seed, tag, idx...)."""
    ss = np.random.SeedSequence([int(seed) & 0xFFFFFFFF] + _tag_words(tag, *idx))
    return np.random.Generator(np.random.Philox(ss))


def uniform_residues(seed: int, tag: str, moduli, n: int, *idx: int) -> np.ndarray:
    """Array ``u64[len(moduli)][n]``; row i uniform in [0, moduli[i])."""
    g = rng(seed, tag, *idx)
    out = np.empty((len(moduli), n), dtype=np.uint64)
    for i, q in enumerate(moduli):
        out[i] = g.integers(0, int(q), size=n, dtype=np.uint64)
    return out


def ternary_secret(seed: int, n: int, h: int, tag: str = "secret") -> np.ndarray:
    """``int8[n]`` with exactly ``h`` entries in {-1, +1}, the rest 0.

    Positions: the first ``h`` entries of a uniform random permutation of
    range(n); signs: one fair coin each.
    """
    g = rng(seed, tag)
    s = np.zeros(n, dtype=np.int8)
    pos = g.permutation(n)[:h]
    sign = g.integers(0, 2, size=h, dtype=np.int64) * 2 - 1
    s[pos] = sign.astype(np.int8)
    return s


def rounded_gaussian(seed: int, tag: str, shape, sigma: float = 3.2, bound: int = 19,
                     *idx: int) -> np.ndarray:
    """``int64`` array: round-half-away-from-zero of sigma*z, z ~ N(0,1),
    entries with |e| > bound redrawn."""
    g = rng(seed, tag, *idx)
    shape = tuple(np.atleast_1d(shape))
    e = g.standard_normal(size=shape) * sigma
    e = np.where(e >= 0, np.floor(e + 0.5), -np.floor(-e + 0.5))
    bad = np.abs(e) > bound
    while bad.any():
        r = g.standard_normal(size=int(bad.sum())) * sigma
        e[bad] = np.where(r >= 0, np.floor(r + 0.5), -np.floor(-r + 0.5))
        bad = np.abs(e) > bound
    return e.astype(np.int64)


def uniform_pm1(seed: int, tag: str, shape, *idx: int) -> np.ndarray:
    """fp64 array, U[-1, 1]."""
    g = rng(seed, tag, *idx)
    return g.random(size=shape) * 2.0 - 1.0


def normal(seed: int, tag: str, shape, std: float = 1.0, *idx: int) -> np.ndarray:
    """fp64 array, N(0, std^2)."""
    g = rng(seed, tag, *idx)
    return g.standard_normal(size=shape) * std


# --------------------------------------------------------------------------
# Draw recipes.  Each returns the raw random arrays one CKKS object needs; the
# arithmetic that turns them into keys or ciphertexts lives on each side.

SECRET_HAMMING_WEIGHT = 64
ERROR_SIGMA = 3.2
ERROR_BOUND = 19


def secret(seed: int, n: int, h: int = SECRET_HAMMING_WEIGHT) -> np.ndarray:
    """Ternary secret coefficients, ``int8[n]``, Hamming weight h."""
    return ternary_secret(seed, n, h, tag="secret")


def moduli_tag(moduli) -> str:
    """Short digest of an ordered list of moduli.

    Draws that belong to one modulus chain carry it in their tag: two key
    sets (or encryptions) over chains that share a prefix then use
    independent randomness.  Shared uniform rows and errors would let anyone
    holding both sets subtract them and recover the secret (for two switching
    keys of one Galois element, b - b' = (P - P') s' on the digit's rows)."""
    h = hashlib.sha256(b"".join(int(m).to_bytes(8, "little") for m in moduli)).hexdigest()
    return h[:16]


def switch_key_draws(seed: int, ext_moduli, n: int, dnum: int, elt: int):
    """Raw draws of one switching key: ``a`` is ``u64[dnum][len(ext_moduli)][n]``
    uniform per modulus (already in evaluation form), ``e`` is
    ``int64[dnum][n]`` rounded-Gaussian coefficients.  ``elt`` names the key
    (Galois element; 0 for the relinearisation key).  The tags include the
    extended modulus chain, so keys of one element in two contexts (e.g. a
    context over a chain prefix with fewer special primes) are independent."""
    mt = moduli_tag(ext_moduli)
    a = np.stack([uniform_residues(seed, "ksk-a/" + mt, ext_moduli, n, elt, j)
                  for j in range(dnum)])
    e = np.stack([rounded_gaussian(seed, "ksk-e/" + mt, n, ERROR_SIGMA, ERROR_BOUND, elt, j)
                  for j in range(dnum)])
    return np.ascontiguousarray(a), np.ascontiguousarray(e)


def switch_key_seed_draws(seed: int, ext_moduli, n: int, dnum: int, elt: int):
    """Raw draws of one seed-expanded switching key: two 64-bit seed words
    (the uniform half is regenerated from them by the counter-based generator
    on either side) and ``int64[dnum][n]`` rounded-Gaussian errors.  Tags
    differ from switch_key_draws' (a seeded and a stored key of one element
    must not share errors) and include the extended modulus chain."""
    mt = moduli_tag(ext_moduli)
    words = rng(seed, "ksk-seed/" + mt, elt).integers(0, 2 ** 64, size=2, dtype=np.uint64)
    e = np.stack([rounded_gaussian(seed, "ksk-se/" + mt, n, ERROR_SIGMA, ERROR_BOUND, elt, j)
                  for j in range(dnum)])
    return words, np.ascontiguousarray(e)


def encrypt_draws(seed: int, moduli, n: int, tag: str, *idx: int):
    """Raw draws of one secret-key encryption: ``a`` uniform ``u64[l][n]``
    (evaluation form), ``e`` rounded-Gaussian ``int64[n]``.  The tags include
    the moduli, as for switching keys."""
    mt = moduli_tag(moduli)
    a = uniform_residues(seed, "enc-a/" + tag + "/" + mt, moduli, n, *idx)
    e = rounded_gaussian(seed, "enc-e/" + tag + "/" + mt, n, ERROR_SIGMA, ERROR_BOUND, *idx)
    return a, e
