"""Pins of the oracle's number theory and transforms against independent
definitions: brute force, Python big integers and schoolbook products."""
import random

import numpy as np
import pytest

from oracle import ckks as C
from oracle import encoding as E


def _mr(n: int, rounds: int = 24) -> bool:
    """Independent probabilistic Miller-Rabin in pure Python (random bases)."""
    if n < 2:
        return False
    for p in (2, 3, 5, 7, 11, 13):
        if n % p == 0:
            return n == p
    d, s = n - 1, 0
    while d % 2 == 0:
        d //= 2
        s += 1
    rnd = random.Random(n)
    for _ in range(rounds):
        a = rnd.randrange(2, n - 1)
        x = pow(a, d, n)
        if x in (1, n - 1):
            continue
        for _ in range(s - 1):
            x = x * x % n
            if x == n - 1:
                break
        else:
            return False
    return True


@pytest.mark.parametrize("log_n,bits,count", [(12, 36, 4), (16, 50, 32), (5, 20, 6)])
def test_primes_are_the_largest_ntt_friendly(log_n, bits, count):
    ps = C.find_primes(log_n, bits, count)
    m = 2 << log_n
    assert ps == sorted(ps, reverse=True)
    for q in ps:
        assert q < 2 ** bits and q % m == 1 and _mr(q)
    # nothing skipped: every candidate between 2^bits and the last prime
    # (same residue class) other than the listed ones is composite
    c = ((2 ** bits - 1) // m) * m + 1
    listed = set(ps)
    while c >= ps[-1]:
        assert (c in listed) == _mr(c), c
        c -= m


def test_brute_force_smallest_psi():
    for log_n, bits in [(3, 12), (4, 14), (5, 16)]:
        n = 1 << log_n
        for q in C.find_primes(log_n, bits, 3):
            roots = [x for x in range(1, q) if pow(x, n, q) == q - 1]
            assert C.min_psi(q, log_n) == min(roots)


def test_p16_psi_is_primitive():
    P = C.params_p16()
    for q in P.q + P.p:
        psi = P.psi[q]
        assert pow(psi, P.n, q) == q - 1 and pow(psi, 2 * P.n, q) == 1


def _brv(x, bits):
    return int(format(x, f"0{bits}b")[::-1], 2)


@pytest.mark.parametrize("log_n", [1, 2, 3, 5, 8])
def test_ntt_is_evaluation_at_odd_powers(log_n):
    """A[j] = a(psi^(2 brv(j) + 1)) by direct evaluation with big ints."""
    n = 1 << log_n
    P = C.params_small(log_n, 40, 2, 1)
    rnd = np.random.default_rng(log_n)
    for q in P.q:
        a = rnd.integers(0, q, size=n, dtype=np.uint64)
        got = C.ntt(P, a[None, :], [q])[0]
        psi = P.psi[q]
        for j in range(n):
            x = pow(psi, 2 * _brv(j, log_n) + 1, q)
            want = sum(int(a[k]) * pow(x, k, q) for k in range(n)) % q
            assert int(got[j]) == want


def _schoolbook_negacyclic(a, b, q):
    n = len(a)
    out = [0] * n
    for i in range(n):
        ai = int(a[i])
        if ai == 0:
            continue
        for j in range(n):
            k = i + j
            if k < n:
                out[k] += ai * int(b[j])
            else:
                out[k - n] -= ai * int(b[j])
    return np.array([x % q for x in out], dtype=np.uint64)


@pytest.mark.parametrize("log_n", [4, 7, 10])
def test_ntt_product_is_negacyclic_convolution(log_n):
    n = 1 << log_n
    P = C.params_small(log_n, 50, 3, 1)
    rnd = np.random.default_rng(100 + log_n)
    for q in P.q + P.p:
        a = rnd.integers(0, q, size=n, dtype=np.uint64)
        b = rnd.integers(0, q, size=n, dtype=np.uint64)
        prod = C.intt(P, C.pmul(C.ntt(P, a[None], [q]), C.ntt(P, b[None], [q]), [q]), [q])[0]
        np.testing.assert_array_equal(prod, _schoolbook_negacyclic(a, b, q))


def test_intt_inverts_ntt_full_size():
    P = C.params_p16()
    rnd = np.random.default_rng(7)
    mods = [P.q[0], P.q[23], P.p[7]]
    a = np.stack([rnd.integers(0, q, size=P.n, dtype=np.uint64) for q in mods])
    b = C.ntt(P, a, mods)
    assert not np.array_equal(a, b)
    np.testing.assert_array_equal(C.intt(P, b, mods), a)


def test_elementwise_against_bigint():
    P = C.params_p16()
    rnd = np.random.default_rng(8)
    mods = P.q[:3]
    a = np.stack([rnd.integers(0, q, size=512, dtype=np.uint64) for q in mods])
    b = np.stack([rnd.integers(0, q, size=512, dtype=np.uint64) for q in mods])
    for i, q in enumerate(mods):
        A, B = a[i].astype(object), b[i].astype(object)
        np.testing.assert_array_equal(C.pmul(a, b, mods)[i].astype(object), A * B % q)
        np.testing.assert_array_equal(C.padd(a, b, mods)[i].astype(object), (A + B) % q)
        np.testing.assert_array_equal(C.psub(a, b, mods)[i].astype(object), (A - B) % q)
    x = rnd.integers(-(2 ** 62), 2 ** 62, size=512, dtype=np.int64)
    x[:3] = [-(2 ** 63), 2 ** 63 - 1, 0]
    got = C.lift(x, mods)
    for i, q in enumerate(mods):
        np.testing.assert_array_equal(got[i].astype(object), x.astype(object) % q)


def test_crt_against_bigint():
    P = C.params_p16()
    rnd = np.random.default_rng(9)
    mods = P.q[:5]
    Q = 1
    for q in mods:
        Q *= q
    vals = [int(rnd.integers(-(2 ** 62), 2 ** 62)) * (2 ** 180) + int(rnd.integers(0, 2 ** 60))
            for _ in range(64)]
    vals += [0, 1, -1, Q // 2, -(Q // 2) + 1]
    res = np.array([[v % q for v in vals] for q in mods], dtype=np.uint64)
    got = E.crt_centered(res, mods)
    assert [int(x) for x in got] == vals


def test_fast_bconv_against_bigint():
    """y mod m = sum_i x_i (Q/q_i) mod m with x_i = [src_i (Q/q_i)^-1]_{q_i}
    centred in (-q_i/2, q_i/2); the integer it represents is congruent to the
    input modulo Q and below ns*Q/2 in absolute value."""
    P = C.params_p16()
    rnd = np.random.default_rng(10)
    src = P.q[:8]
    dst = P.q[8:11] + P.p[:2]
    Q = 1
    for q in src:
        Q *= q
    x = np.stack([rnd.integers(0, q, size=64, dtype=np.uint64) for q in src])
    x[:, 0] = 0
    got = C.fast_bconv(x, src, dst)
    xint = [int(v) for v in E.crt_centered(x, src)]
    for k in range(64):
        s = 0
        for i, q in enumerate(src):
            qh = Q // q
            xi = int(x[i, k]) * pow(qh, -1, q) % q
            if xi > q // 2:
                xi -= q
            s += xi * qh
        assert (s - xint[k]) % Q == 0
        assert abs(s) < len(src) * Q // 2
        for m_i, m in enumerate(dst):
            assert int(got[m_i, k]) == s % m
    # odd map: converting -x gives -y exactly
    negx = np.stack([(np.uint64(q) - x[i]) % np.uint64(q) for i, q in enumerate(src)])
    gotn = C.fast_bconv(negx, src, dst)
    for m_i, m in enumerate(dst):
        np.testing.assert_array_equal((got[m_i] + gotn[m_i]) % np.uint64(m), 0)


def test_automorphism_coefficient_definition():
    """sigma_g(a)(X) = a(X^g) checked by evaluating both sides at the odd
    powers of psi with big ints, for several g including conjugation."""
    log_n = 5
    n = 1 << log_n
    P = C.params_small(log_n, 40, 1, 1)
    q = P.q[0]
    psi = P.psi[q]
    rnd = np.random.default_rng(11)
    a = rnd.integers(0, q, size=n, dtype=np.uint64)
    for g in [5, 25, 2 * n - 1, pow(5, 7, 2 * n)]:
        b = C.automorph_coef(P, a[None], [q], g)[0]
        for t in range(1, 2 * n, 2):
            x = pow(psi, t, q)
            lhs = sum(int(b[k]) * pow(x, k, q) for k in range(n)) % q
            rhs = sum(int(a[k]) * pow(x, g * k, q) for k in range(n)) % q
            assert lhs == rhs
