"""GPU parity of the device encoder (fesc_encode_plain) against the oracle's
encoding.  The integer coefficients are recovered from the first limb and must
equal the oracle's except where Delta m_k lies within the FFTs' rounding error
of a half-integer (+-1 there, as for the host encoder; the band is derived from
the fp64 FFT error); every limb must then equal
the oracle's lift and NTT of those coefficients exactly.  N = 2^12 (one pass),
2^13 (a 2-point column pass) and 2^16 (16-point columns), and more plaintexts
than one scratch round holds."""
import numpy as np
import pytest
import torch

import synth
from oracle import ckks as C
from oracle import encoding as E
from paper_2608_17442_amd import fesc as F
from tests.gpu_helpers import need_gpu, step, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


@pytest.mark.parametrize("log_n,L,level,count,kind",
                         [(12, 3, 3, 5, "pm1"), (12, 3, 2, 40, "normal"), (13, 4, 4, 3, "pm1"),
                          (16, 24, 16, 3, "pm1"), (16, 24, 24, 2, "normal")])
def test_encode_plain_matches_oracle(log_n, L, level, count, kind):
    P = C.params_p16(L) if log_n == 16 else C.params_small(log_n, 50 if log_n > 12 else 36, L, 1)
    ctx = F.Context(log_n, P.q, P.p)
    n, scale = P.n, 2.0 ** 40 if log_n > 12 else 2.0 ** 30
    zs = []
    for b in range(count):
        if kind == "pm1":
            z = synth.uniform_pm1(70 + b, "genc-re", n // 2) \
                + 1j * synth.uniform_pm1(70 + b, "genc-im", n // 2)
        else:
            z = synth.normal(70 + b, "genc-n", n // 2, 0.02).astype(complex)
        zs.append(z)
    zd = torch.from_numpy(np.stack(zs)).cuda()
    pt = torch.zeros(count * level * n, dtype=torch.int64, device="cuda")
    step(f"encode_plain N=2^{log_n} level={level} count={count}")
    ctx.encode_plain(zd, scale, pt, level)
    got = to_host(pt).reshape(count, level, n)
    qs = P.qs(level)
    for b in range(count):
        c0 = C.intt(P, got[b, :1], qs[:1])[0].astype(object)
        m = np.array([int(v) - qs[0] if int(v) > qs[0] // 2 else int(v) for v in c0], dtype=np.int64)
        want = E.encode(zs[b], scale, n)
        raw = E.encode_real_coeffs(zs[b], scale, n)
        diff = m - want
        # Each fp64 FFT (the device's and the oracle's) leaves an error on
        # Delta m_k of order est = Delta 2^-53 log2(N) rms|z| / sqrt(N) (the
        # oracle's stays below est against a long-double direct sum, a CPU
        # test); only a coefficient within 8 est of a half-integer may round
        # differently on the two sides.
        band = 8 * scale * 2.0 ** -53 * log_n * np.sqrt(np.mean(np.abs(zs[b]) ** 2)) / np.sqrt(n)
        near_tie = np.abs(np.abs(raw - np.trunc(raw)) - 0.5) < band
        assert np.all(np.abs(diff) <= 1), b
        assert not np.any(diff[~near_tie]), (b, np.flatnonzero(diff[~near_tie])[:8])
        # every limb is the exact lift and transform of those coefficients
        full = C.ntt(P, C.lift(m, qs), qs)
        assert np.array_equal(got[b], full), b


def test_encode_plain_empty_and_errors():
    P = C.params_small(12, 36, 3, 1)
    ctx = F.Context(12, P.q, P.p)
    pt = torch.zeros(3 * P.n, dtype=torch.int64, device="cuda")
    z = torch.zeros((0, P.n // 2), dtype=torch.complex128, device="cuda")
    ctx.encode_plain(z, 2.0 ** 30, pt, 3)                  # count 0: nothing to do
    z1 = torch.zeros((1, P.n // 2), dtype=torch.complex128, device="cuda")
    with pytest.raises(F.FescError):
        ctx.encode_plain(z1, 2.0 ** 30, pt, 4)             # level above the chain
    with pytest.raises(F.FescError):
        ctx.encode_plain(z1, float("inf"), pt, 3)


# ------------------------------------------------------------------ decoding


def _slots(seed, n_slots):
    return synth.uniform_pm1(seed, "gdec-re", n_slots) + 1j * synth.uniform_pm1(seed, "gdec-im",
                                                                                 n_slots)


@pytest.mark.parametrize("log_n,L,level,count", [(12, 5, 5, 3), (12, 5, 1, 2), (13, 4, 3, 2),
                                                 (16, 24, 24, 2)])
def test_decode_plain_matches_oracle(log_n, L, level, count):
    """fesc_decode_plain against the oracle's decoding (exact CRT of the
    centred coefficients, numpy FFT) of the same plaintexts: device-encoded
    slot vectors (decoded back within the encoding's rounding), and their
    products limb by limb (coefficients up to 2^80 spanning two or more
    primes, decoded at scale 2^80 to z1 z2).  N = 2^13 has an odd number of
    FFT stages; level 1 is a single prime."""
    P = C.params_p16(L) if log_n == 16 else C.params_small(log_n, 50, L, 2)
    ctx = F.Context(log_n, P.q, P.p)
    n, scale = P.n, 2.0 ** 40
    zs = np.stack([_slots(90 + b, n // 2) for b in range(count)])
    pt = torch.zeros(count * level * n, dtype=torch.int64, device="cuda")
    step(f"decode: encode_plain N=2^{log_n} level={level} count={count}")
    ctx.encode_plain(torch.from_numpy(zs).cuda(), scale, pt, level)
    out = torch.zeros(count, n // 2, dtype=torch.complex128, device="cuda")
    step("decode_plain")
    ctx.decode_plain(pt, count, level, scale, out)
    got = out.cpu().numpy()
    pth = to_host(pt).reshape(count, level, n)
    for b in range(count):
        want = C.decode_plain(P, pth[b], scale)
        np.testing.assert_allclose(got[b], want, rtol=0, atol=1e-9)
        np.testing.assert_allclose(got[b], zs[b], rtol=0, atol=2.0 ** -30)
    if level < 2:
        return
    # products: coefficients near 2^80 need the CRT over several primes
    qs = P.qs(level)
    prod = np.stack([C.pmul(pth[b], pth[(b + 1) % count], qs) for b in range(count)])
    dprod = torch.from_numpy(prod.view(np.int64).reshape(-1)).cuda()
    step("decode_plain of products at scale 2^80")
    ctx.decode_plain(dprod, count, level, scale * scale, out)
    got = out.cpu().numpy()
    for b in range(count):
        want = C.decode_plain(P, prod[b], scale * scale)
        np.testing.assert_allclose(got[b], want, rtol=0, atol=1e-9)
        np.testing.assert_allclose(got[b], zs[b] * zs[(b + 1) % count], rtol=0, atol=2.0 ** -25)


def test_decode_plain_of_a_decrypted_ciphertext():
    """A client-side decode: the oracle decrypts a rotated ciphertext (c0 + c1
    s, evaluation form, noise included) and the device decodes the result
    exactly as the oracle does."""
    P = C.params_small(12, 50, 5, 2)
    ctx = F.Context(P.log_n, P.q, P.p)
    sk = C.secret_key(P, synth.secret(5, P.n))
    z = _slots(99, P.n // 2)
    a, e = synth.encrypt_draws(5, P.qs(P.L), P.n, "gdec", 0)
    ct = C.encrypt(P, sk, C.encode_plain(P, z, 2.0 ** 30, P.L), P.L, a, e)
    keys = {P.galois_elt(3): C.keygen_from_seed(P, sk, 5, P.galois_elt(3))}
    rot = C.rotate(P, ct, 3, keys)
    qs = P.qs(P.L)
    m = C.padd(rot[:, 0], C.pmul(rot[:, 1], sk.ntt_ext[:P.L], qs), qs)
    out = torch.zeros(1, P.n // 2, dtype=torch.complex128, device="cuda")
    step("decode_plain of a decrypted rotation")
    ctx.decode_plain(torch.from_numpy(m.view(np.int64).reshape(-1)).cuda(), 1, P.L, 2.0 ** 30, out)
    got = out.cpu().numpy()[0]
    np.testing.assert_allclose(got, C.decode_plain(P, m, 2.0 ** 30), rtol=0, atol=1e-9)
    np.testing.assert_allclose(got, np.roll(z, -3), rtol=0, atol=2.0 ** -12)


def test_decode_plain_errors():
    P = C.params_small(12, 50, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    pt = torch.zeros(3 * P.n, dtype=torch.int64, device="cuda")
    out = torch.zeros(1, P.n // 2, dtype=torch.complex128, device="cuda")
    for scale in (0.0, float("inf"), float("nan")):
        with pytest.raises(F.FescError):
            ctx.decode_plain(pt, 1, 3, scale, out)
    with pytest.raises(F.FescError):
        ctx.decode_plain(pt, 1, 4, 1.0, out)
    with pytest.raises(ValueError):
        ctx.decode_plain(pt, 2, 1, 1.0, out)       # z holds one vector
    ctx.decode_plain(pt, 0, 3, 1.0, out)           # nothing to do
    ctx.decode_plain(pt, 1, 3, 1.0, out)
    assert torch.count_nonzero(out).item() == 0    # the zero plaintext decodes to zeros
