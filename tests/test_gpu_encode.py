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
