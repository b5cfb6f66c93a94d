"""Plain RNS-CKKS reference for the linear hot path (test infrastructure only).

Scope follows the paper's primitive table (Sec. 4.1, Table "CKKS primitives":
add, ptmul, ctmul, rot, conj), its description of key switching with special
primes and of rescaling (Sec. 2.1), the BSGS projection kernel (Appendix
"Projection Kernel Breakdown") and the complex-packed reduction (Appendix
"Complex-Packed Reduction Accounting").  The paper fixes none of the ring
internals, so the textbook ones are written out here:

* layouts: plaintext ``u64[l][N]``; ciphertext ``u64[l][2][N]`` (limb-major,
  c0 and c1 per limb); switching key ``u64[dnum][L+alpha][2][N]`` with rows
  q_0..q_{L-1}, p_0..p_{alpha-1} and (b, a) per row; all in evaluation form;
* secret-key encryption: c1 = a, c0 = -a*s + m + e;
* hybrid key switching (Han-Ki, CT-RSA 2020): digits of alpha consecutive
  primes, ModUp by fast basis conversion, inner product with the key, ModDown
  by fast basis conversion of the P part and multiplication by P^-1 (floor
  variant);
* rescale: c' = round(c / q_last), computed as (c - [c mod q_last]_centred) *
  q_last^-1 limb by limb;
* automorphism X -> X^g applied on coefficients (the plain definition).

Every function works on numpy ``uint64`` arrays; the C core does the modular
products.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

import synth
from . import _native as nat
from . import encoding as enc

# --------------------------------------------------------------- parameters


def find_primes(log_n: int, bits: int, count: int) -> list[int]:
    out = np.zeros(count, dtype=np.uint64)
    got = nat.lib().or_find_primes(log_n, bits, count, nat.u64p(out))
    assert got == count, (got, count)
    return [int(x) for x in out]


def min_psi(q: int, log_n: int) -> int:
    return int(nat.lib().or_min_psi(q, log_n))


@dataclass
class Params:
    log_n: int
    q: list          # ciphertext primes q_0..q_{L-1}
    p: list          # special primes p_0..p_{alpha-1}
    psi: dict = field(default_factory=dict)

    def __post_init__(self):
        self.n = 1 << self.log_n
        self.L = len(self.q)
        self.alpha = len(self.p)
        self.dnum = -(-self.L // self.alpha)
        for m in list(self.q) + list(self.p):
            if m not in self.psi:
                self.psi[m] = min_psi(m, self.log_n)
        self.P = math.prod(self.p)

    def qs(self, level: int) -> list:
        return list(self.q[:level])

    def ext(self, level: int) -> list:
        """Moduli of the extended basis Q_level u P, in row order."""
        return list(self.q[:level]) + list(self.p)

    def key_rows(self, level: int) -> list:
        """Row indices into a switching key for the basis ext(level)."""
        return list(range(level)) + [self.L + k for k in range(self.alpha)]

    def digits(self, level: int) -> list:
        """Digit j covers q_{j*alpha} .. q_{min((j+1)*alpha, level)-1}."""
        return [(lo, min(lo + self.alpha, level)) for lo in range(0, level, self.alpha)]

    def galois_elt(self, r: int) -> int:
        """Galois element of the left rotation by r slots (5^r mod 2N)."""
        return pow(5, r % (self.n // 2), 2 * self.n)

    @property
    def conj_elt(self) -> int:
        return 2 * self.n - 1


def params_p12() -> Params:
    """N = 2^12; the four largest 36-bit primes = 1 mod 2N: the largest is the
    special prime, the next three (descending) are q_0, q_1, q_2."""
    pr = find_primes(12, 36, 4)
    return Params(12, pr[1:4], pr[0:1])


def params_p16(L: int = 24) -> Params:
    """N = 2^16; the 32 largest 50-bit primes = 1 mod 2N: the 8 largest are
    the special primes p_0..p_7, the next 24 (descending) q_0..q_23."""
    pr = find_primes(16, 50, 8 + L)
    return Params(16, pr[8:8 + L], pr[0:8])


def params_small(log_n: int, bits: int, L: int, alpha: int) -> Params:
    pr = find_primes(log_n, bits, L + alpha)
    return Params(log_n, pr[alpha:alpha + L], pr[0:alpha])


# ------------------------------------------------------------ poly helpers


def _c(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def ntt(P: Params, a: np.ndarray, mods) -> np.ndarray:
    """Forward negacyclic NTT of each row (row i modulo mods[i])."""
    out = _c(a).copy()
    rows = out.shape[0]
    assert rows == len(mods)
    nat.lib().or_ntt_fwd_rows(nat.u64p(out), rows, P.log_n, nat.u64p(nat.moduli(mods)),
                              nat.u64p(nat.moduli([P.psi[m] for m in mods])))
    return out


def intt(P: Params, a: np.ndarray, mods) -> np.ndarray:
    out = _c(a).copy()
    rows = out.shape[0]
    assert rows == len(mods)
    nat.lib().or_ntt_inv_rows(nat.u64p(out), rows, P.log_n, nat.u64p(nat.moduli(mods)),
                              nat.u64p(nat.moduli([P.psi[m] for m in mods])))
    return out


def pmul(a, b, mods):
    a, b = _c(a), _c(b)
    out = np.empty_like(a)
    nat.lib().or_mul_rows(nat.u64p(a), nat.u64p(b), nat.u64p(out), a.shape[0], a.shape[1],
                          nat.u64p(nat.moduli(mods)))
    return out


def padd(a, b, mods):
    a, b = _c(a), _c(b)
    out = np.empty_like(a)
    nat.lib().or_add_rows(nat.u64p(a), nat.u64p(b), nat.u64p(out), a.shape[0], a.shape[1],
                          nat.u64p(nat.moduli(mods)))
    return out


def psub(a, b, mods):
    a, b = _c(a), _c(b)
    out = np.empty_like(a)
    nat.lib().or_sub_rows(nat.u64p(a), nat.u64p(b), nat.u64p(out), a.shape[0], a.shape[1],
                          nat.u64p(nat.moduli(mods)))
    return out


def pscalar(a, consts, mods):
    a = _c(a)
    out = np.empty_like(a)
    nat.lib().or_mul_scalar_rows(nat.u64p(a), nat.u64p(out), a.shape[0], a.shape[1],
                                 nat.u64p(nat.moduli(mods)), nat.u64p(nat.moduli(consts)))
    return out


def lift(x: np.ndarray, mods) -> np.ndarray:
    """Signed integer coefficients -> residues, one row per modulus."""
    x = np.ascontiguousarray(x, dtype=np.int64)
    out = np.empty((len(mods), x.shape[0]), dtype=np.uint64)
    nat.lib().or_lift_signed_rows(nat.i64p(x), nat.u64p(out), len(mods), x.shape[0],
                                  nat.u64p(nat.moduli(mods)))
    return out


def automorph_coef(P: Params, a: np.ndarray, mods, g: int) -> np.ndarray:
    """X -> X^g on coefficient-form rows."""
    a = _c(a)
    out = np.empty_like(a)
    nat.lib().or_automorph_coef_rows(nat.u64p(a), nat.u64p(out), a.shape[0], P.log_n,
                                     nat.u64p(nat.moduli(mods)), g)
    return out


def automorph(P: Params, a: np.ndarray, mods, g: int) -> np.ndarray:
    """X -> X^g on evaluation-form rows (through the coefficient form)."""
    return ntt(P, automorph_coef(P, intt(P, a, mods), mods, g), mods)


def fast_bconv(x: np.ndarray, src_mods, dst_mods) -> np.ndarray:
    """Fast basis conversion of coefficient-form rows (see the C core)."""
    x = _c(x)
    out = np.empty((len(dst_mods), x.shape[1]), dtype=np.uint64)
    nat.lib().or_fast_bconv(nat.u64p(x), len(src_mods), nat.u64p(nat.moduli(src_mods)),
                            nat.u64p(out), len(dst_mods), nat.u64p(nat.moduli(dst_mods)),
                            x.shape[1])
    return out


# -------------------------------------------------------- keys and ciphers


@dataclass
class SecretKey:
    coeffs: np.ndarray            # int8[N], ternary
    ntt_ext: np.ndarray           # u64[L+alpha][N], evaluation form over Q_L u P


def secret_key(P: Params, s: np.ndarray) -> SecretKey:
    return SecretKey(np.asarray(s, dtype=np.int8),
                     ntt(P, lift(s.astype(np.int64), P.ext(P.L)), P.ext(P.L)))


def switch_key(P: Params, sk: SecretKey, s_from_ext: np.ndarray, a: np.ndarray,
               e: np.ndarray) -> np.ndarray:
    """Hybrid switching key from s_from to sk (evaluation form, full level L).

    For digit j and row i (modulus m_i of Q_L u P):
        b_j = -a_j * s + e_j + [P]_{q_i} * s_from     (q_i in digit j)
        b_j = -a_j * s + e_j                           (every other row)
    Output ``u64[dnum][L+alpha][2][N]`` with (b, a) per row.
    """
    mods = P.ext(P.L)
    key = np.empty((P.dnum, P.L + P.alpha, 2, P.n), dtype=np.uint64)
    for j, (lo, hi) in enumerate(P.digits(P.L)):
        e_ntt = ntt(P, lift(e[j], mods), mods)
        b = psub(e_ntt, pmul(a[j], sk.ntt_ext, mods), mods)
        gadget = np.zeros((len(mods), P.n), dtype=np.uint64)
        for i in range(lo, hi):
            gadget[i] = pscalar(s_from_ext[i:i + 1], [P.P % mods[i]], [mods[i]])[0]
        b = padd(b, gadget, mods)
        key[j, :, 0] = b
        key[j, :, 1] = a[j]
    return key


def galois_key(P: Params, sk: SecretKey, g: int, a, e) -> np.ndarray:
    """Key from sigma_g(s) to s."""
    mods = P.ext(P.L)
    s_g = ntt(P, automorph_coef(P, lift(sk.coeffs.astype(np.int64), mods), mods, g), mods)
    return switch_key(P, sk, s_g, a, e)


def relin_key(P: Params, sk: SecretKey, a, e) -> np.ndarray:
    """Key from s^2 to s."""
    mods = P.ext(P.L)
    return switch_key(P, sk, pmul(sk.ntt_ext, sk.ntt_ext, mods), a, e)


def philox4x64(ctr, k0: int, k1: int) -> list:
    """Philox4x64-10 block of a 4-word counter under a 2-word key."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    out = np.empty(4, dtype=np.uint64)
    nat.lib().or_philox4x64(nat.u64p(c), int(k0), int(k1), nat.u64p(out))
    return [int(v) for v in out]


def seeded_key_a(P: Params, seed_words, elt: int) -> np.ndarray:
    """Uniform half of a seed-expanded switching key, ``u64[dnum][L+alpha][N]``
    (evaluation form), regenerated from two 64-bit seed words (see the C core
    or_seeded_key_a for the counter layout and the residue rule)."""
    mods = P.ext(P.L)
    out = np.empty((P.dnum, len(mods), P.n), dtype=np.uint64)
    row_ids = np.arange(len(mods), dtype=np.uint64)
    nat.lib().or_seeded_key_a(nat.u64p(out), P.dnum, len(mods), P.n,
                              nat.u64p(nat.moduli(mods)), nat.u64p(row_ids),
                              int(seed_words[0]), int(seed_words[1]), int(elt))
    return out


def keygen_seeded(P: Params, sk: SecretKey, seed_words, e, elt: int) -> np.ndarray:
    """Switching key for ``elt`` (0: relinearisation) whose uniform half is
    regenerated from ``seed_words``; returned in the full layout."""
    a = seeded_key_a(P, seed_words, elt)
    return relin_key(P, sk, a, e) if elt == 0 else galois_key(P, sk, elt, a, e)


def keygen_from_seed(P: Params, sk: SecretKey, seed: int, elt: int) -> np.ndarray:
    """Key for Galois element ``elt`` (0: relinearisation), randomness drawn
    by the shared recipe."""
    a, e = synth.switch_key_draws(seed, P.ext(P.L), P.n, P.dnum, elt)
    return relin_key(P, sk, a, e) if elt == 0 else galois_key(P, sk, elt, a, e)


def encode_plain(P: Params, z, scale: float, level: int) -> np.ndarray:
    """Encoded slot vector as an evaluation-form plaintext ``u64[level][N]``."""
    m = enc.encode(np.asarray(z, dtype=np.complex128), scale, P.n)
    return ntt(P, lift(m, P.qs(level)), P.qs(level))


def decode_plain(P: Params, pt: np.ndarray, scale: float) -> np.ndarray:
    """Slots of an evaluation-form plaintext ``u64[level][N]``: its centred
    integer coefficients (exact CRT) evaluated at zeta^(5^j), over scale."""
    mods = P.qs(pt.shape[0])
    return enc.decode_coeffs(enc.crt_centered(intt(P, pt, mods), mods), scale, P.n)


def encrypt(P: Params, sk: SecretKey, pt: np.ndarray, level: int, a, e) -> np.ndarray:
    """Secret-key encryption: c1 = a, c0 = -a*s + m + e.  ``u64[level][2][N]``."""
    mods = P.qs(level)
    s = sk.ntt_ext[:level]
    e_ntt = ntt(P, lift(e, mods), mods)
    c0 = padd(psub(e_ntt, pmul(a, s, mods), mods), pt[:level], mods)
    ct = np.empty((level, 2, P.n), dtype=np.uint64)
    ct[:, 0] = c0
    ct[:, 1] = a
    return ct


def decrypt_coeffs(P: Params, sk: SecretKey, ct: np.ndarray) -> np.ndarray:
    """Centred integer coefficients of c0 + c1*s (object array of ints)."""
    level = ct.shape[0]
    mods = P.qs(level)
    m = padd(ct[:, 0], pmul(ct[:, 1], sk.ntt_ext[:level], mods), mods)
    return enc.crt_centered(intt(P, m, mods), mods)


def decrypt(P: Params, sk: SecretKey, ct: np.ndarray, scale: float) -> np.ndarray:
    return enc.decode_coeffs(decrypt_coeffs(P, sk, ct), scale, P.n)


# ------------------------------------------------------------- operations


def ct_add(P, a, b):
    level = a.shape[0]
    out = np.empty_like(a)
    for t in range(2):
        out[:, t] = padd(a[:, t], b[:, t], P.qs(level))
    return out


def ct_sub(P, a, b):
    level = a.shape[0]
    out = np.empty_like(a)
    for t in range(2):
        out[:, t] = psub(a[:, t], b[:, t], P.qs(level))
    return out


def add_plain(P: Params, ct: np.ndarray, pt: np.ndarray) -> np.ndarray:
    """(c0 + p, c1): adds the plaintext p to the message."""
    level = ct.shape[0]
    out = ct.copy()
    out[:, 0] = padd(ct[:, 0], pt[:level], P.qs(level))
    return out


def mul_plain(P: Params, ct: np.ndarray, pt: np.ndarray) -> np.ndarray:
    """ptmul: (c0 * p, c1 * p) limb-wise."""
    level = ct.shape[0]
    out = np.empty_like(ct)
    for t in range(2):
        out[:, t] = pmul(ct[:, t], pt[:level], P.qs(level))
    return out


def mul_monomial(P: Params, ct: np.ndarray, k: int) -> np.ndarray:
    """Multiply by X^k (negacyclic shift of the coefficients)."""
    level = ct.shape[0]
    mods = P.qs(level)
    k %= 2 * P.n
    out = np.empty_like(ct)
    for t in range(2):
        c = intt(P, ct[:, t], mods)
        r = np.zeros_like(c)
        for i, q in enumerate(mods):
            shifted = np.roll(c[i], k % P.n)
            # coefficients that wrapped past X^N pick up a sign (X^N = -1)
            wrapped = np.zeros(P.n, dtype=bool)
            wrapped[: k % P.n] = True
            if k >= P.n:
                wrapped = ~wrapped
            neg = np.where(shifted == 0, np.uint64(0), np.uint64(q) - shifted)
            r[i] = np.where(wrapped, neg, shifted)
        out[:, t] = ntt(P, r, mods)
    return out


def tensor(P: Params, a: np.ndarray, b: np.ndarray):
    """(a0 b0, a0 b1 + a1 b0, a1 b1)."""
    level = a.shape[0]
    mods = P.qs(level)
    d0 = pmul(a[:, 0], b[:, 0], mods)
    d1 = padd(pmul(a[:, 0], b[:, 1], mods), pmul(a[:, 1], b[:, 0], mods), mods)
    d2 = pmul(a[:, 1], b[:, 1], mods)
    return d0, d1, d2


def modup(P: Params, c_coef: np.ndarray, level: int) -> list:
    """Per digit: the coefficient-form extension of digit j to every row of
    ext(level).  Own-digit rows are the input rows; the others come from fast
    basis conversion of the digit's rows."""
    ext = P.ext(level)
    out = []
    for lo, hi in P.digits(level):
        others = [i for i in range(len(ext)) if not (lo <= i < hi)]
        conv = fast_bconv(c_coef[lo:hi], ext[lo:hi], [ext[i] for i in others])
        d = np.empty((len(ext), P.n), dtype=np.uint64)
        d[lo:hi] = c_coef[lo:hi]
        d[others] = conv
        out.append(d)
    return out


def key_inner_product(P: Params, digits_ntt: list, key: np.ndarray, level: int):
    """acc_t = sum_j d_j * key_j[t] over ext(level), t in (b, a)."""
    ext = P.ext(level)
    rows = P.key_rows(level)
    acc = [np.zeros((len(ext), P.n), dtype=np.uint64) for _ in range(2)]
    for j, d in enumerate(digits_ntt):
        for t in range(2):
            acc[t] = padd(acc[t], pmul(d, key[j, rows, t], ext), ext)
    return acc


def moddown(P: Params, acc: np.ndarray, level: int) -> np.ndarray:
    """(acc - FastBConv_{P->Q}([acc]_P)) * P^-1 on the Q rows (floor variant)."""
    qs = P.qs(level)
    pc = intt(P, acc[level:], P.p)
    y = ntt(P, fast_bconv(pc, P.p, qs), qs)
    pinv = [pow(P.P % q, -1, q) for q in qs]
    return pscalar(psub(acc[:level], y, qs), pinv, qs)


def moddown_rescale(P: Params, x: np.ndarray, level: int) -> np.ndarray:
    """ModDown and rescale as one division by M = P q_{level-1}: x over
    ext(level) (evaluation form) -> (x - FastBConv_{M->Q}([x]_M)) * M^-1 on
    q_0..q_{level-2}, the conversion digits coming from the q_{level-1} row and
    the special-prime rows (the floor variant of ModDown with q_{level-1}
    joined to the special primes)."""
    assert level >= 2
    ql = P.q[level - 1]
    src = [ql] + list(P.p)
    coef = intt(P, np.concatenate([x[level - 1:level], x[level:]]), src)
    qs = P.qs(level - 1)
    y = ntt(P, fast_bconv(coef, src, qs), qs)
    M = P.P * ql
    return pscalar(psub(x[:level - 1], y, qs), [pow(M % q, -1, q) for q in qs], qs)


def mul_relin_rescale(P: Params, a, b, rlk):
    """Relinearised product divided by P q_{level-1} in one step: acc = key
    product of d2 over ext(level); x_t = acc_t + P d_t on the Q rows (P d_t
    vanishes modulo every special prime); out_t = moddown_rescale(x_t).  The
    result is at level - 1; it differs from rescale(mul_relin(a, b)) only in
    the rounding (one conversion error of at most (alpha + 1) / 2 units)."""
    level = a.shape[0]
    d0, d1, d2 = tensor(P, a, b)
    qs, ext = P.qs(level), P.ext(level)
    digits = [ntt(P, d, ext) for d in modup(P, intt(P, d2, qs), level)]
    acc = key_inner_product(P, digits, rlk, level)
    pm = [P.P % q for q in qs]
    out = np.empty((level - 1, 2, P.n), dtype=np.uint64)
    for t, d in enumerate((d0, d1)):
        x = acc[t].copy()
        x[:level] = padd(acc[t][:level], pscalar(d, pm, qs), qs)
        out[:, t] = moddown_rescale(P, x, level)
    return out


def key_switch(P: Params, c: np.ndarray, key: np.ndarray, level: int):
    """Hybrid key switch of one evaluation-form polynomial ``u64[level][N]``;
    returns (out_b, out_a), each ``u64[level][N]``."""
    qs = P.qs(level)
    ext = P.ext(level)
    c_coef = intt(P, c, qs)
    digits = [ntt(P, d, ext) for d in modup(P, c_coef, level)]
    acc = key_inner_product(P, digits, key, level)
    return moddown(P, acc[0], level), moddown(P, acc[1], level)


def relinearize(P: Params, d0, d1, d2, rlk, level):
    kb, ka = key_switch(P, d2, rlk, level)
    qs = P.qs(level)
    out = np.empty((level, 2, P.n), dtype=np.uint64)
    out[:, 0] = padd(d0, kb, qs)
    out[:, 1] = padd(d1, ka, qs)
    return out


def mul_relin(P: Params, a, b, rlk):
    """ctmul followed by relinearisation; no rescale."""
    level = a.shape[0]
    return relinearize(P, *tensor(P, a, b), rlk, level)


def apply_galois(P: Params, ct: np.ndarray, g: int, key: np.ndarray) -> np.ndarray:
    """sigma_g on both parts, then key switch of the c1 part (sigma_g(s) -> s)."""
    level = ct.shape[0]
    qs = P.qs(level)
    c0 = automorph(P, ct[:, 0], qs, g)
    c1 = automorph(P, ct[:, 1], qs, g)
    kb, ka = key_switch(P, c1, key, level)
    out = np.empty_like(ct)
    out[:, 0] = padd(c0, kb, qs)
    out[:, 1] = ka
    return out


def rotate(P: Params, ct: np.ndarray, r: int, keys: dict) -> np.ndarray:
    """rho(ct; r): left rotation by r slots; r = 0 mod N/2 is an exact copy."""
    if r % (P.n // 2) == 0:
        return ct.copy()
    g = P.galois_elt(r)
    return apply_galois(P, ct, g, keys[g])


def conjugate(P: Params, ct: np.ndarray, keys: dict) -> np.ndarray:
    return apply_galois(P, ct, P.conj_elt, keys[P.conj_elt])


def rotate_hoisted(P: Params, ct: np.ndarray, rs, keys: dict) -> list:
    """Rotations of one ciphertext sharing one ModUp of c1: the automorphism
    is applied to the extended digits (after ModUp), then inner product and
    ModDown per rotation.  r = 0 mod N/2 gives an exact copy."""
    level = ct.shape[0]
    qs = P.qs(level)
    ext = P.ext(level)
    ext_coef = modup(P, intt(P, ct[:, 1], qs), level)
    outs = []
    for r in rs:
        if r % (P.n // 2) == 0:
            outs.append(ct.copy())
            continue
        g = P.galois_elt(r)
        digits = [ntt(P, automorph_coef(P, d, ext, g), ext) for d in ext_coef]
        acc = key_inner_product(P, digits, keys[g], level)
        kb, ka = moddown(P, acc[0], level), moddown(P, acc[1], level)
        out = np.empty_like(ct)
        out[:, 0] = padd(automorph(P, ct[:, 0], qs, g), kb, qs)
        out[:, 1] = ka
        outs.append(out)
    return outs


def rotate_hoisted_ext(P: Params, ct: np.ndarray, rs, keys: dict) -> list:
    """Hoisted rotations left in the extended basis Q u P: one ModUp of c1,
    then per rotation the key product acc (as in rotate_hoisted) plus the
    rotated c0 multiplied by the special modulus P, with no ModDown
    (Bossuat et al., Eurocrypt 2021, double hoisting).  Each result is
    ``u64[2][level+alpha][N]`` (component, extended row, coefficient) and
    moddown_ct of it is the ordinary rotation.  r = 0 mod N/2 gives
    (P c0, P c1), zero on the special-prime rows."""
    level = ct.shape[0]
    qs, ext = P.qs(level), P.ext(level)
    pm = [P.P % q for q in qs]
    ext_coef = modup(P, intt(P, ct[:, 1], qs), level)
    outs = []
    for r in rs:
        x = np.zeros((2, len(ext), P.n), dtype=np.uint64)
        if r % (P.n // 2) == 0:
            x[0, :level] = pscalar(ct[:, 0], pm, qs)
            x[1, :level] = pscalar(ct[:, 1], pm, qs)
            outs.append(x)
            continue
        g = P.galois_elt(r)
        digits = [ntt(P, automorph_coef(P, d, ext, g), ext) for d in ext_coef]
        acc = key_inner_product(P, digits, keys[g], level)
        x[0] = acc[0]
        x[0, :level] = padd(acc[0][:level], pscalar(automorph(P, ct[:, 0], qs, g), pm, qs), qs)
        x[1] = acc[1]
        outs.append(x)
    return outs


def moddown_ct(P: Params, x: np.ndarray, level: int) -> np.ndarray:
    """ModDown of both components of an extended-basis ciphertext
    ``u64[2][level+alpha][N]`` into ``u64[level][2][N]``."""
    out = np.empty((level, 2, P.n), dtype=np.uint64)
    for t in range(2):
        out[:, t] = moddown(P, x[t], level)
    return out


def encode_plain_ext(P: Params, z, scale: float, level: int) -> np.ndarray:
    """Encoded slot vector over the extended basis Q_level u P (evaluation
    form), ``u64[level+alpha][N]``."""
    ext = P.ext(level)
    m = enc.encode(np.asarray(z, dtype=np.complex128), scale, P.n)
    return ntt(P, lift(m, ext), ext)


def mul_plain_ext(P: Params, x: np.ndarray, pt: np.ndarray) -> np.ndarray:
    """Extended-basis ciphertext times an extended-basis plaintext."""
    ext = P.ext(x.shape[1] - P.alpha)
    return np.stack([pmul(x[t], pt, ext) for t in range(2)])


def ext_add(P: Params, x: np.ndarray, y: np.ndarray) -> np.ndarray:
    ext = P.ext(x.shape[1] - P.alpha)
    return np.stack([padd(x[t], y[t], ext) for t in range(2)])


def rescale(P: Params, ct: np.ndarray) -> np.ndarray:
    """Divide by the last prime with rounding: c' = (c - v) * q_last^-1 where
    v is the centred residue of c modulo q_last."""
    level = ct.shape[0]
    assert level >= 2
    ql = P.q[level - 1]
    qs = P.qs(level - 1)
    out = np.empty((level - 1, 2, P.n), dtype=np.uint64)
    for t in range(2):
        v = intt(P, ct[level - 1:level, t], [ql])[0].astype(object)
        v = np.where(v > ql // 2, v - ql, v).astype(np.int64)
        vt = ntt(P, lift(v, qs), qs)
        qinv = [pow(ql % q, -1, q) for q in qs]
        out[:, t] = pscalar(psub(ct[:level - 1, t], vt, qs), qinv, qs)
    return out
