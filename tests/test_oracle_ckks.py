"""Pins of the oracle's CKKS layer: encoding against the O(N^2) definition
and the ring homomorphism; rescale and ModDown against big-integer division;
every operation against the plaintext result after decryption."""
import numpy as np
import pytest

import synth
from oracle import ckks as C
from oracle import encoding as E

# small ring with multi-prime digits: N = 2^10, L = 5, alpha = 2 (dnum = 3)
SMALL = dict(log_n=10, bits=50, L=5, alpha=2)


@pytest.fixture(scope="module")
def small():
    P = C.params_small(**SMALL)
    sk = C.secret_key(P, synth.secret(5, P.n))
    return P, sk


def _z(seed, n_slots, complex_=True):
    re = synth.uniform_pm1(seed, "z-re", n_slots)
    im = synth.uniform_pm1(seed, "z-im", n_slots) if complex_ else 0.0
    return re + 1j * im


def _enc(P, sk, z, scale, level, tag, idx=0):
    a, e = synth.encrypt_draws(77, P.qs(level), P.n, tag, idx)
    return C.encrypt(P, sk, C.encode_plain(P, z, scale, level), level, a, e)


def _negacyclic_int(a, b):
    n = len(a)
    full = np.convolve(np.asarray(a, dtype=object), np.asarray(b, dtype=object))
    out = full[:n].copy()
    out[: n - 1] -= full[n:]
    return out


# ------------------------------------------------------------ encoding


@pytest.mark.parametrize("log_n", [3, 4, 6])
def test_encode_matches_direct_definition(log_n):
    n = 1 << log_n
    z = _z(log_n, n // 2)
    zeta = np.exp(1j * np.pi / n)
    e = [pow(5, j, 2 * n) for j in range(n // 2)]
    direct = np.array([(2.0 / n) * sum(z[j] * zeta ** (-e[j] * k) for j in range(n // 2)).real
                       for k in range(n)])
    np.testing.assert_allclose(E.encode_real_coeffs(z, 1.0, n), direct, atol=1e-12)
    # decode is evaluation at zeta^(5^j)
    m = direct
    ev = np.array([sum(m[k] * zeta ** (e[j] * k) for k in range(n)) for j in range(n // 2)])
    np.testing.assert_allclose(E.decode_coeffs(m, 1.0, n), ev, atol=1e-12)
    np.testing.assert_allclose(ev, z, atol=1e-12)


def test_decode_plain_inverts_encode_plain_across_primes():
    """decode_plain of an evaluation-form encoding returns the slots; the
    limb-wise product of two encodings (coefficients near 2^60, beyond one
    36-bit prime) decodes to the slot product at the squared scale, which
    needs the CRT over several primes (a single limb's centred residue is
    far off)."""
    P = C.params_small(10, 36, 4, 1)
    z1, z2 = _z(61, P.n // 2), _z(62, P.n // 2)
    d = 2.0 ** 30
    p1, p2 = C.encode_plain(P, z1, d, 4), C.encode_plain(P, z2, d, 4)
    np.testing.assert_allclose(C.decode_plain(P, p1, d), z1, atol=2.0 ** -20)
    prod = C.pmul(p1, p2, P.qs(4))
    np.testing.assert_allclose(C.decode_plain(P, prod, d * d), z1 * z2, atol=2.0 ** -18)
    assert np.max(np.abs(C.decode_plain(P, prod[:1], d * d) - z1 * z2)) > 1.0


def test_encode_rounding_half_away_from_zero():
    n = 8
    x = np.array([0.5, -0.5, 1.5, -1.5, 2.4999, -2.5001, 0.0, 3.0])
    np.testing.assert_array_equal(E._round_half_away(x), [1, -1, 2, -2, 2, -3, 0, 3])
    assert E.encode(np.zeros(n // 2), 2.0 ** 30, n).dtype == np.int64


@pytest.mark.parametrize("log_n,scale", [(12, 2.0 ** 30), (14, 2.0 ** 40)])
def test_encode_fft_error_within_estimate(log_n, scale):
    """The encoder's fp64 FFT error on Delta m_k stays below
    est = Delta 2^-53 log2(N) rms|z| / sqrt(N) (checked against a direct
    long-double sum over the definition on a sample of coefficients); the
    device encoder's parity band is a multiple of this estimate."""
    n = 1 << log_n
    z = _z(80 + log_n, n // 2)
    raw = E.encode_real_coeffs(z, scale, n)
    e = E.slot_exponents(n // 2, 2 * n).astype(np.longdouble)
    pi = np.longdouble("3.14159265358979323846264338327950288")
    zl = z.astype(np.clongdouble)
    ks = np.arange(0, n, n // 256)
    exact = np.array([2 * np.sum(zl * np.exp(-1j * pi * ((e * k) % (2 * n)) / n)).real / n
                      for k in ks], dtype=np.longdouble) * np.longdouble(scale)
    err = np.abs(raw[ks].astype(np.longdouble) - exact).astype(float)
    est = scale * 2.0 ** -53 * log_n * np.sqrt(np.mean(np.abs(z) ** 2)) / np.sqrt(n)
    assert err.max() < est, (err.max(), est)


def test_encoding_is_a_ring_homomorphism():
    """encode(z1) * encode(z2) (negacyclic) decodes to z1 * z2;
    X -> X^(5^r) rotates left by r; X -> X^(2N-1) conjugates;
    X^(N/2) multiplies every slot by i."""
    n = 256
    z1, z2 = _z(1, n // 2), _z(2, n // 2)
    d = 2.0 ** 20
    m1, m2 = E.encode(z1, d, n), E.encode(z2, d, n)
    prod = _negacyclic_int(m1, m2)
    np.testing.assert_allclose(E.decode_coeffs(prod, d * d, n), z1 * z2, atol=1e-4)
    for r in [1, 5, 17, n // 2 - 1]:
        g = pow(5, r, 2 * n)
        mg = np.zeros(n, dtype=object)
        for k in range(n):
            t = k * g % (2 * n)
            if t < n:
                mg[t] += int(m1[k])
            else:
                mg[t - n] -= int(m1[k])
        np.testing.assert_allclose(E.decode_coeffs(mg, d, n), np.roll(z1, -r), atol=1e-5)
    mc = np.zeros(n, dtype=object)
    for k in range(n):
        t = k * (2 * n - 1) % (2 * n)
        if t < n:
            mc[t] += int(m1[k])
        else:
            mc[t - n] -= int(m1[k])
    np.testing.assert_allclose(E.decode_coeffs(mc, d, n), np.conj(z1), atol=1e-5)
    mono = np.zeros(n, dtype=object)
    mono[n // 2] = 1
    np.testing.assert_allclose(E.decode_coeffs(_negacyclic_int(m1, mono), d, n), 1j * z1,
                               atol=1e-5)


# ------------------------------------------------------- exact RNS steps


def _bigint_rows(res, mods):
    return [int(v) for v in E.crt_centered(res, mods)]


def test_rescale_is_rounded_division(small):
    P, sk = small
    level = 4
    rnd = np.random.default_rng(3)
    ct = np.stack([np.stack([rnd.integers(0, q, size=P.n, dtype=np.uint64) for _ in range(2)])
                   for q in P.qs(level)])
    out = C.rescale(P, ct)
    assert out.shape == (level - 1, 2, P.n)
    Q = 1
    for q in P.qs(level):
        Q *= q
    ql = P.q[level - 1]
    for t in range(2):
        c = C.intt(P, ct[:, t], P.qs(level))
        big = [int(v) % Q for v in E.crt_centered(c, P.qs(level))]
        want = [(2 * v + ql) // (2 * ql) for v in big]  # round(v / ql), ties impossible (ql odd)
        got = C.intt(P, out[:, t], P.qs(level - 1))
        Qp = Q // ql
        gotb = [int(v) % Qp for v in E.crt_centered(got, P.qs(level - 1))]
        assert gotb == [w % Qp for w in want]


def test_moddown_is_exact_division_of_acc_minus_bconv(small):
    P, sk = small
    level = 3
    ext = P.ext(level)
    rnd = np.random.default_rng(4)
    acc = np.stack([rnd.integers(0, m, size=P.n, dtype=np.uint64) for m in ext])
    out = C.moddown(P, C.ntt(P, acc, ext), level)
    # integer semantics: (A - y) / P with y = centred FastBConv(A mod P), A the
    # lift over Q*P of the coefficient form
    QP = 1
    for m in ext:
        QP *= m
    Q = QP // P.P
    A = [int(v) % QP for v in E.crt_centered(acc, ext)]
    got = [int(v) % Q for v in E.crt_centered(C.intt(P, out, P.qs(level)), P.qs(level))]
    for k in range(P.n):
        y = 0
        for i, p in enumerate(P.p):
            ph = P.P // p
            xi = A[k] % p * pow(ph, -1, p) % p
            if xi > p // 2:
                xi -= p
            y += xi * ph
        assert (A[k] - y) % P.P == 0
        assert got[k] == ((A[k] - y) // P.P) % Q
        assert abs(y) < P.alpha * P.P // 2


def test_moddown_rescale_is_exact_division(small):
    """(X - y) / M with M = P q_{l-1} and y the centred conversion of X mod M
    from the digits of q_{l-1} and the special primes, big-integer arithmetic."""
    P, sk = small
    level = 4
    ext = P.ext(level)
    rnd = np.random.default_rng(6)
    x = np.stack([rnd.integers(0, m, size=P.n, dtype=np.uint64) for m in ext])
    out = C.moddown_rescale(P, C.ntt(P, x, ext), level)
    assert out.shape == (level - 1, P.n)
    QP = 1
    for m in ext:
        QP *= m
    ql = P.q[level - 1]
    M = P.P * ql
    Qo = QP // M
    A = [int(v) % QP for v in E.crt_centered(x, ext)]
    got = [int(v) % Qo for v in E.crt_centered(C.intt(P, out, P.qs(level - 1)),
                                                P.qs(level - 1))]
    for k in range(P.n):
        y = 0
        for m in [ql] + list(P.p):
            mh = M // m
            xi = A[k] % m * pow(mh, -1, m) % m
            if xi > m // 2:
                xi -= m
            y += xi * mh
        assert (A[k] - y) % M == 0
        assert got[k] == ((A[k] - y) // M) % Qo
        assert abs(y) < (P.alpha + 1) * M // 2


def test_mul_relin_rescale_decrypts_like_the_two_steps(small):
    P, sk = small
    rlk = C.keygen_from_seed(P, sk, 3, 0)
    level = 5
    z1, z2 = _z(50, P.n // 2), _z(51, P.n // 2)
    ql = P.q[level - 1]
    c1 = _enc(P, sk, z1, 2.0 ** 40, level, "mrr1")
    c2 = _enc(P, sk, z2, float(ql), level, "mrr2")
    fused = C.mul_relin_rescale(P, c1, c2, rlk)
    seq = C.rescale(P, C.mul_relin(P, c1, c2, rlk))
    assert fused.shape == seq.shape == (level - 1, 2, P.n)
    df = C.decrypt(P, sk, fused, 2.0 ** 40)
    np.testing.assert_allclose(df, z1 * z2, atol=2.0 ** -15)
    np.testing.assert_allclose(df, C.decrypt(P, sk, seq, 2.0 ** 40), atol=2.0 ** -28)


# --------------------------------------------- decrypt-based operation pins


def test_encrypt_decrypt(small):
    P, sk = small
    z = _z(20, P.n // 2)
    for level in [1, 3, P.L]:
        ct = _enc(P, sk, z, 2.0 ** 40, level, "encdec", level)
        assert ct.shape == (level, 2, P.n)
        np.testing.assert_allclose(C.decrypt(P, sk, ct, 2.0 ** 40), z, atol=2.0 ** -25)


def test_mul_plain_add_sub_monomial(small):
    P, sk = small
    z1, z2, w = _z(21, P.n // 2), _z(22, P.n // 2), _z(23, P.n // 2)
    level = 4
    c1 = _enc(P, sk, z1, 2.0 ** 40, level, "ops", 1)
    c2 = _enc(P, sk, z2, 2.0 ** 40, level, "ops", 2)
    pt = C.encode_plain(P, w, 2.0 ** 30, level)
    dec = lambda ct, s: C.decrypt(P, sk, ct, s)
    np.testing.assert_allclose(dec(C.mul_plain(P, c1, pt), 2.0 ** 70), z1 * w, atol=2.0 ** -20)
    np.testing.assert_allclose(dec(C.ct_add(P, c1, c2), 2.0 ** 40), z1 + z2, atol=2.0 ** -25)
    np.testing.assert_allclose(dec(C.ct_sub(P, c1, c2), 2.0 ** 40), z1 - z2, atol=2.0 ** -25)
    np.testing.assert_allclose(dec(C.mul_monomial(P, c1, P.n // 2), 2.0 ** 40), 1j * z1,
                               atol=2.0 ** -25)
    np.testing.assert_allclose(dec(C.mul_monomial(P, c1, 3 * P.n // 2), 2.0 ** 40), -1j * z1,
                               atol=2.0 ** -25)
    # X^k on the decrypted coefficients is the exact negacyclic shift
    m = C.decrypt_coeffs(P, sk, c1)
    m3 = C.decrypt_coeffs(P, sk, C.mul_monomial(P, c1, 3))
    want = np.concatenate([-m[-3:], m[:-3]])
    assert [int(v) for v in m3] == [int(v) for v in want]


def test_rescale_decrypts(small):
    P, sk = small
    z, w = _z(24, P.n // 2), _z(25, P.n // 2)
    level = 4
    ct = _enc(P, sk, z, 2.0 ** 40, level, "rs")
    ql = P.q[level - 1]
    prod = C.mul_plain(P, ct, C.encode_plain(P, w, float(ql), level))
    rs = C.rescale(P, prod)
    np.testing.assert_allclose(C.decrypt(P, sk, rs, 2.0 ** 40), z * w, atol=2.0 ** -25)


def test_key_switch_decrypts_to_c_times_s_from(small):
    """dec_s(KS(c)) = c * s' + small, checked on the integer coefficients."""
    P, sk = small
    level = 5
    g = P.galois_elt(3)
    a, e = synth.switch_key_draws(9, P.ext(P.L), P.n, P.dnum, g)
    key = C.galois_key(P, sk, g, a, e)
    rnd = np.random.default_rng(5)
    c = np.stack([rnd.integers(0, q, size=P.n, dtype=np.uint64) for q in P.qs(level)])
    kb, ka = C.key_switch(P, c, key, level)
    qs = P.qs(level)
    s = sk.ntt_ext[:level]
    mods_all = P.ext(P.L)
    s_g = C.ntt(P, C.automorph_coef(P, C.lift(sk.coeffs.astype(np.int64), mods_all), mods_all,
                                     g), mods_all)[:level]
    lhs = C.padd(kb, C.pmul(ka, s, qs), qs)
    rhs = C.pmul(c, s_g, qs)
    diff = E.crt_centered(C.intt(P, C.psub(lhs, rhs, qs), qs), qs)
    assert max(abs(int(v)) for v in diff) < 2 ** 30


def test_key_switch_at_every_level(small):
    P, sk = small
    rlk = C.keygen_from_seed(P, sk, 3, 0)
    for level in range(1, P.L + 1):
        z1, z2 = _z(30 + level, P.n // 2), _z(40 + level, P.n // 2)
        # product scale 2^44 stays below q_0 / 2 ~ 2^49 at level 1
        c1 = _enc(P, sk, z1, 2.0 ** 22, level, "lv1", level)
        c2 = _enc(P, sk, z2, 2.0 ** 22, level, "lv2", level)
        out = C.mul_relin(P, c1, c2, rlk)
        np.testing.assert_allclose(C.decrypt(P, sk, out, 2.0 ** 44), z1 * z2, atol=2.0 ** -12)


def test_rotate_conjugate_hoisted(small):
    P, sk = small
    level = 5
    z = _z(50, P.n // 2)
    ct = _enc(P, sk, z, 2.0 ** 40, level, "rot")
    rs = [1, 2, 7, P.n // 2 - 1, P.n // 2, 0]
    keys = {g: C.keygen_from_seed(P, sk, 3, g)
            for g in {P.galois_elt(r) for r in rs if r % (P.n // 2)} | {P.conj_elt}}
    hoisted = C.rotate_hoisted(P, ct, rs, keys)
    for r, h in zip(rs, hoisted):
        plain = C.rotate(P, ct, r, keys)
        # key-switch noise ~ N sigma dnum (Q_j / P) per coefficient: 2^-22 here
        np.testing.assert_allclose(C.decrypt(P, sk, plain, 2.0 ** 40), np.roll(z, -r),
                                   atol=2.0 ** -20)
        np.testing.assert_allclose(C.decrypt(P, sk, h, 2.0 ** 40), np.roll(z, -r),
                                   atol=2.0 ** -20)
        # centred basis conversion is an odd map, so it commutes with the
        # signed coefficient permutation: both routes give the same residues
        np.testing.assert_array_equal(plain, h)
        if r % (P.n // 2) == 0:
            np.testing.assert_array_equal(h, ct)
    cj = C.conjugate(P, ct, keys)
    np.testing.assert_allclose(C.decrypt(P, sk, cj, 2.0 ** 40), np.conj(z), atol=2.0 ** -20)
    # rot_a o rot_b = rot_{a+b} in value
    r12 = C.rotate(P, C.rotate(P, ct, 1, keys), 2, keys)
    k3 = {P.galois_elt(3): C.keygen_from_seed(P, sk, 3, P.galois_elt(3))}
    np.testing.assert_allclose(C.decrypt(P, sk, r12, 2.0 ** 40),
                               C.decrypt(P, sk, C.rotate(P, ct, 3, k3), 2.0 ** 40),
                               atol=2.0 ** -20)


def test_extended_basis_rotation_takes_one_moddown_to_the_rotation(small):
    """A hoisted rotation left in Q u P (P sigma(c0) + acc, acc') is the
    ordinary rotation after ModDown, residue for residue (ModDown divides by
    P exactly on the P sigma(c0) term, which vanishes modulo every special
    prime); the identity step gives (P c0, P c1)."""
    P, sk = small
    level = 5
    ct = _enc(P, sk, _z(76, P.n // 2), 2.0 ** 30, level, "rot-ext")
    rs = [0, 1, 3, P.n // 2]
    keys = {P.galois_elt(r): C.keygen_from_seed(P, sk, 3, P.galois_elt(r)) for r in (1, 3)}
    exts = C.rotate_hoisted_ext(P, ct, rs, keys)
    for r, x in zip(rs, exts):
        assert x.shape == (2, level + P.alpha, P.n)
        np.testing.assert_array_equal(C.moddown_ct(P, x, level), C.rotate(P, ct, r, keys))
    assert not np.any(exts[0][:, level:])
    # one plaintext factor taken before the ModDown: the product decodes to
    # the rotated slots times the plaintext's
    w = _z(77, P.n // 2)
    pt = C.encode_plain_ext(P, w, float(P.q[level - 1]), level)
    y = C.rescale(P, C.moddown_ct(P, C.mul_plain_ext(P, exts[2], pt), level))
    z = C.decrypt(P, sk, ct, 2.0 ** 30)
    np.testing.assert_allclose(C.decrypt(P, sk, y, 2.0 ** 30), np.roll(z, -3) * w, atol=2.0 ** -12)


def test_p12_parameters_roundtrip():
    """The N = 2^12 ring: alpha = 1, three single-prime digits."""
    P = C.params_p12()
    assert (P.L, P.alpha, P.dnum) == (3, 1, 3)
    sk = C.secret_key(P, synth.secret(0, P.n))
    z = _z(60, P.n // 2, complex_=False)
    ct = _enc(P, sk, z, float(P.q[2]), 3, "p12")
    keys = {P.galois_elt(1): C.keygen_from_seed(P, sk, 0, P.galois_elt(1))}
    out = C.rotate_hoisted(P, ct, [1], keys)[0]
    np.testing.assert_allclose(C.decrypt(P, sk, out, float(P.q[2])), np.roll(z, -1),
                               atol=2.0 ** -20)


def test_key_sets_over_a_shared_chain_prefix_are_independent():
    """A second key set over the chain prefix q_0..q_3 with fewer special
    primes (the contraction's context) must not reuse the first set's
    randomness: with shared uniform rows and errors, two keys of one Galois
    element differ on a digit row only by (P - P') s', which gives the secret
    away.  The draws are tagged with the modulus chain, so the attack fails;
    planting shared draws shows that it would succeed."""
    Pf = C.params_small(10, 50, 8, 4)
    Pc = C.Params(Pf.log_n, Pf.q[:4], Pf.p[:2], dict(Pf.psi))
    s = synth.secret(9, Pf.n)
    skf, skc = C.secret_key(Pf, s), C.secret_key(Pc, s)
    g = Pf.galois_elt(1)
    af, ef = synth.switch_key_draws(9, Pf.ext(Pf.L), Pf.n, Pf.dnum, g)
    ac, ec = synth.switch_key_draws(9, Pc.ext(Pc.L), Pc.n, Pc.dnum, g)
    assert not np.array_equal(af[0, :4], ac[0, :4])
    assert not np.array_equal(ef[0], ec[0])
    # encryptions over one chain at two lengths are independent as well
    e1 = synth.encrypt_draws(9, Pf.qs(8), Pf.n, "t", 0)
    e2 = synth.encrypt_draws(9, Pf.qs(4), Pf.n, "t", 0)
    assert not np.array_equal(e1[0][:4], e2[0]) and not np.array_equal(e1[1], e2[1])

    q0 = Pf.q[0]
    s_g = C.ntt(Pf, C.automorph_coef(Pf, C.lift(s.astype(np.int64), [q0]), [q0], g), [q0])[0]
    inv = pow((Pf.P - Pc.P) % q0, -1, q0)

    def recovered(kc):
        kf = C.galois_key(Pf, skf, g, af, ef)
        d = (kf[0, 0, 0].astype(object) - kc[0, 0, 0].astype(object)) % q0
        return np.array([(int(v) * inv) % q0 for v in d], dtype=np.uint64)

    assert not np.array_equal(recovered(C.galois_key(Pc, skc, g, ac, ec)), s_g)
    # the planted mistake: the prefix context's rows taken from the first set
    rows = list(range(4)) + [Pf.L + k for k in range(Pc.alpha)]
    a_shared = np.ascontiguousarray(af[:Pc.dnum][:, rows])
    e_shared = np.ascontiguousarray(ef[:Pc.dnum])
    np.testing.assert_array_equal(
        recovered(C.galois_key(Pc, skc, g, a_shared, e_shared)), s_g)


# ------------------------------------------------- seed-expanded key halves


def test_philox4x64_matches_numpy():
    """The oracle's Philox4x64-10 block function equals numpy's Philox bit
    generator (which advances its counter before each block)."""
    for key, ctr in [((1, 2), (6, 0, 0, 0)), ((0xDEADBEEF, 7), (1, 2, 3, 4)),
                     ((2 ** 64 - 1, 2 ** 63), (2 ** 64 - 1, 5, 0, 2 ** 40))]:
        prev = list(ctr)
        i = 0
        while prev[i] == 0:          # counter - 1 with borrow
            prev[i] = 2 ** 64 - 1
            i += 1
        prev[i] -= 1
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.array(prev, dtype=np.uint64))
        assert [int(v) for v in bg.random_raw(4)] == C.philox4x64(ctr, *key)


def test_seeded_key_halves_are_uniform_residues():
    """Regenerated key halves: every value below its prime, deterministic,
    different for another seed, element or row, and close to uniform; with a
    modulus just above a power of two (half of the masked words rejected) the
    spare word and the fallback keep every value in range and uniform."""
    P = C.params_small(10, 50, 5, 2)
    a = C.seeded_key_a(P, (11, 22), 5)
    b = C.seeded_key_a(P, (11, 22), 5)
    assert np.array_equal(a, b)
    mods = np.array(P.ext(P.L), dtype=np.uint64)[None, :, None]
    assert np.all(a < mods)
    assert not np.array_equal(a, C.seeded_key_a(P, (11, 23), 5))
    assert not np.array_equal(a, C.seeded_key_a(P, (11, 22), 7))
    assert not np.array_equal(a[0, 0], a[0, 1]) and not np.array_equal(a[0, 0], a[1, 0])
    u = (a / mods).ravel()
    assert abs(u.mean() - 0.5) < 0.01 and abs(u.var() - 1 / 12) < 0.01
    # a contrived modulus 2^49 + 1 (not a ring prime: the expansion rule alone)
    q = (1 << 49) + 1
    out = np.empty((3, 1, 4096), dtype=np.uint64)
    C.nat.lib().or_seeded_key_a(C.nat.u64p(out), 3, 1, 4096,
                                C.nat.u64p(np.array([q], dtype=np.uint64)),
                                C.nat.u64p(np.array([0], dtype=np.uint64)), 5, 6, 0)
    assert np.all(out < q)
    v = out.ravel() / q
    assert abs(v.mean() - 0.5) < 0.02
    hist = np.histogram(v, bins=8, range=(0, 1))[0]
    assert hist.min() > 0.8 * len(v) / 8


def _numpy_philox_block(ctr, key):
    prev = list(ctr)
    i = 0
    while prev[i] == 0:          # counter - 1 with borrow
        prev[i] = 2 ** 64 - 1
        i += 1
    prev[i] -= 1
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(prev, dtype=np.uint64))
    return [int(v) for v in bg.random_raw(4)]


def test_seeded_key_counter_layout_and_rule_from_numpy_philox():
    """Brute force of the key-half expansion on a tiny case with words from
    numpy's Philox (not the oracle's block function): counter (k, row id,
    digit block, element), digit 3c + t from word t masked, the spare word 3
    for the first rejected digit of a block, the remainder after that.  Four
    digits span two blocks; one modulus sits just above a power of two."""
    mods = [C.find_primes(12, 50, 1)[0], (1 << 45) + 1, (1 << 47) + 5]
    row_ids, n, dnum, key, elt = [3, 9, 30], 64, 4, (0x1234, 0xFEDC), 7
    got = np.empty((dnum, len(mods), n), dtype=np.uint64)
    C.nat.lib().or_seeded_key_a(C.nat.u64p(got), dnum, len(mods), n,
                                C.nat.u64p(np.array(mods, dtype=np.uint64)),
                                C.nat.u64p(np.array(row_ids, dtype=np.uint64)), key[0], key[1],
                                elt)
    branches = {"masked": 0, "spare": 0, "rem": 0}
    for r, (q, rid) in enumerate(zip(mods, row_ids)):
        mask = (1 << q.bit_length()) - 1
        for k in range(n):
            for c in range((dnum + 2) // 3):
                w = _numpy_philox_block((k, rid, c, elt), key)
                spare_free = True
                for t in range(3):
                    d = 3 * c + t
                    if d >= dnum:
                        break
                    v = w[t] & mask
                    if v < q:
                        branches["masked"] += 1
                    elif spare_free and (w[3] & mask) < q:
                        v, spare_free = w[3] & mask, False
                        branches["spare"] += 1
                    else:
                        v = w[t] % q
                        branches["rem"] += 1
                    assert int(got[d, r, k]) == v, (d, r, k)
    assert min(branches.values()) > 0, branches


def test_seeded_keys_switch_keys():
    """A rotation and a relinearisation with seed-expanded keys decrypt to
    the rotated / multiplied message."""
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(8, P.n))
    g = P.galois_elt(3)
    w, e = synth.switch_key_seed_draws(8, P.ext(P.L), P.n, P.dnum, g)
    keys = {g: C.keygen_seeded(P, sk, w, e, g)}
    w0, e0 = synth.switch_key_seed_draws(8, P.ext(P.L), P.n, P.dnum, 0)
    rlk = C.keygen_seeded(P, sk, w0, e0, 0)
    z1, z2 = _z(90, P.n // 2), _z(91, P.n // 2)
    c1 = _enc(P, sk, z1, 2.0 ** 40, P.L, "seeded", 0)
    c2 = _enc(P, sk, z2, 2.0 ** 40, P.L, "seeded", 1)
    np.testing.assert_allclose(C.decrypt(P, sk, C.rotate(P, c1, 3, keys), 2.0 ** 40),
                               np.roll(z1, -3), atol=2.0 ** -20)
    np.testing.assert_allclose(C.decrypt(P, sk, C.mul_relin(P, c1, c2, rlk), 2.0 ** 80),
                               z1 * z2, atol=2.0 ** -20)
