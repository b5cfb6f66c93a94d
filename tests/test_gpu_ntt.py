"""GPU parity of the transforms and the Hadamard multiply-accumulate against
the oracle: bit-exact residues, every row."""
import numpy as np
import pytest
import torch

import synth
import synth.workloads as WL
from oracle import ckks as C
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _ctx(P):
    from paper_2608_17442_amd import fesc as F
    return F.Context(P.log_n, P.q, P.p)


def test_context_psi_matches_oracle():
    for P in [C.params_p12(), C.params_p16()]:
        step(f"ctx psi log_n={P.log_n}")
        ctx = _ctx(P)
        for i, m in enumerate(P.q + P.p):
            assert ctx.psi(i) == P.psi[m]


@pytest.mark.parametrize("log_n", [12, 13, 14, 15, 16])
def test_ntt_roundtrip_all_sizes(log_n):
    P = C.params_small(log_n, 50, 3, 2)
    ctx = _ctx(P)
    mods = P.ext(P.L)            # q0 q1 q2 p0 p1
    batch, limbs, prime0 = 3, 4, 1
    rows = mods[prime0:prime0 + limbs]
    a = np.stack([synth.uniform_residues(10 + log_n, "ntt", rows, P.n, b) for b in range(batch)])
    a[0, 0, :5] = [0, 1, rows[0] - 1, 2, rows[0] - 2]
    want = np.stack([C.ntt(P, a[b], rows) for b in range(batch)])
    d = to_dev(a)
    step(f"ntt_fwd log_n={log_n}")
    ctx.ntt_fwd(d, batch, limbs * P.n, limbs, P.n, prime0)
    got = to_host(d)
    assert np.array_equal(got, want), first_mismatch(got, want)
    step(f"ntt_inv log_n={log_n}")
    ctx.ntt_inv(d, batch, limbs * P.n, limbs, P.n, prime0)
    got = to_host(d)
    assert np.array_equal(got, a), first_mismatch(got, a)
    # inverse of arbitrary residues against the oracle's inverse
    wantinv = np.stack([C.intt(P, a[b], rows) for b in range(batch)])
    d = to_dev(a)
    ctx.ntt_inv(d, batch, limbs * P.n, limbs, P.n, prime0)
    got = to_host(d)
    assert np.array_equal(got, wantinv), first_mismatch(got, wantinv)


def test_ntt_strided_rows_leave_gaps_untouched():
    P = C.params_small(14, 50, 4, 1)
    ctx = _ctx(P)
    n = P.n
    limbs, batch = 2, 2
    limb_stride, batch_stride = n + 512, 3 * (n + 512)
    buf = np.full(batch * batch_stride, 7, dtype=np.uint64)
    rows = P.q[1:3]
    data = {}
    for b in range(batch):
        for i in range(limbs):
            r = synth.uniform_residues(3, "gap", [rows[i]], n, b, i)[0]
            o = b * batch_stride + i * limb_stride
            buf[o:o + n] = r
            data[(b, i)] = r
    d = to_dev(buf)
    step("ntt_fwd strided")
    ctx.ntt_fwd(d, batch, batch_stride, limbs, limb_stride, 1)
    got = to_host(d)
    mask = np.ones_like(buf, dtype=bool)
    for (b, i), r in data.items():
        o = b * batch_stride + i * limb_stride
        mask[o:o + n] = False
        want = C.ntt(P, r[None], [rows[i]])[0]
        assert np.array_equal(got[o:o + n], want)
    assert np.all(got[mask] == 7)


@pytest.mark.parametrize("batch,limbs,gap", [(26, 5, 256), (128, 1, 0), (43, 3, 64)])
def test_ntt_large_strided_batches(batch, limbs, gap):
    """N = 2^16 launches of 128 to 130 rows: a row count that is not a
    multiple of 8, one long batch of single limbs, strided rows with gaps that
    must stay untouched; forward, round trip and inverse of arbitrary
    residues against the oracle."""
    P = C.params_small(16, 50, 6, 2)
    ctx = _ctx(P)
    n = P.n
    mods = P.ext(P.L)
    prime0 = 1
    rows_p = [mods[prime0 + i] for i in range(limbs)]
    ls, bs = n + gap, limbs * (n + gap) + gap
    buf = np.full(batch * bs, 7, dtype=np.uint64)
    data = {}
    for b in range(batch):
        for i in range(limbs):
            r = synth.uniform_residues(90 + b, "sp", [rows_p[i]], n, i)[0]
            if b == 0 and i == 0:
                r[:4] = [0, 1, rows_p[0] - 1, rows_p[0] - 2]
            data[(b, i)] = r
            buf[b * bs + i * ls:b * bs + i * ls + n] = r
    mask = np.ones_like(buf, dtype=bool)
    for (b, i) in data:
        mask[b * bs + i * ls:b * bs + i * ls + n] = False
    d = to_dev(buf)
    step(f"ntt_fwd batch={batch} limbs={limbs} gap={gap}")
    ctx.ntt_fwd(d, batch, bs, limbs, ls, prime0)
    got = to_host(d)
    assert np.all(got[mask] == 7)
    for (b, i), r in data.items():
        o = b * bs + i * ls
        want = C.ntt(P, r[None], [rows_p[i]])[0]
        assert np.array_equal(got[o:o + n], want), (b, i, first_mismatch(got[o:o + n], want))
    step("ntt_inv (round trip)")
    ctx.ntt_inv(d, batch, bs, limbs, ls, prime0)
    got = to_host(d)
    assert np.array_equal(got, buf), first_mismatch(got, buf)
    step("ntt_inv of arbitrary residues")
    ctx.ntt_inv(d, batch, bs, limbs, ls, prime0)
    got = to_host(d)
    assert np.all(got[mask] == 7)
    for (b, i), r in data.items():
        o = b * bs + i * ls
        want = C.intt(P, r[None], [rows_p[i]])[0]
        assert np.array_equal(got[o:o + n], want), (b, i, first_mismatch(got[o:o + n], want))


def test_ntt_maximum_launch_sizes():
    """The largest launches the entry points take: N = 2^12 with the maximum
    batch of 65,535 single-limb rows (2.1 GB; rows 0, 32,767 and 65,534
    against the oracle, the whole batch by its round trip), N = 2^16 with every
    prime of the extended basis in one batch element (32 limbs, against the
    oracle row by row), and one row past the batch limit refused before any
    launch."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 3, 1)
    ctx = _ctx(P)
    n, batch, q = P.n, 65535, P.q[0]
    gen = torch.Generator(device="cuda").manual_seed(11)
    d = torch.randint(0, q, (batch * n,), generator=gen, device="cuda", dtype=torch.int64)
    orig = d.clone()
    step(f"ntt_fwd batch={batch} x 2^12")
    ctx.ntt_fwd(d, batch, n, 1, n, 0)
    for b in (0, 32767, batch - 1):
        a = orig[b * n:(b + 1) * n].cpu().numpy().view(np.uint64)
        g = d[b * n:(b + 1) * n].cpu().numpy().view(np.uint64)
        want = C.ntt(P, a[None], [q])[0]
        assert np.array_equal(g, want), (b, first_mismatch(g, want))
    step("ntt_inv (round trip)")
    ctx.ntt_inv(d, batch, n, 1, n, 0)
    assert torch.equal(d, orig)
    with pytest.raises(F.FescError) as e:
        ctx.ntt_fwd(d, batch + 1, 0, 1, n, 0)
    assert e.value.code == -1
    del d, orig
    P = C.params_p16()
    ctx = _ctx(P)
    mods = P.ext(P.L)
    a = np.stack([synth.uniform_residues(12, "ntt-max", mods, P.n)])
    dv = to_dev(a)
    step(f"ntt_fwd 2^16 x {len(mods)} limbs (the whole extended basis)")
    ctx.ntt_fwd(dv, 1, 0, len(mods), P.n, 0)
    got = to_host(dv).reshape(len(mods), P.n)
    want = C.ntt(P, a[0], mods)
    assert np.array_equal(got, want), first_mismatch(got, want)
    ctx.ntt_inv(dv, 1, 0, len(mods), P.n, 0)
    assert np.array_equal(to_host(dv).reshape(len(mods), P.n), a[0])


def test_bad_prime_range_is_rejected_before_launch():
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 2, 1)
    ctx = _ctx(P)
    d = to_dev(np.zeros(4 * P.n, dtype=np.uint64))
    with pytest.raises(F.FescError) as e:
        ctx.ntt_fwd(d, 1, 0, 4, P.n, 0)   # only 3 primes
    assert e.value.code == -1
    assert np.all(to_host(d) == 0)


@pytest.mark.parametrize("pairs", [1, 3, 8])
def test_mac_small(pairs):
    P = C.params_small(12, 50, 3, 1)
    ctx = _ctx(P)
    mods = P.q
    a = np.stack([synth.uniform_residues(5, "macA", mods, P.n, j) for j in range(pairs)])
    b = np.stack([synth.uniform_residues(5, "macB", mods, P.n, j) for j in range(pairs)])
    a[0, :, :3] = np.array(mods, dtype=np.uint64)[:, None] - 1
    b[0, :, :3] = np.array(mods, dtype=np.uint64)[:, None] - 1
    want = np.zeros((len(mods), P.n), dtype=np.uint64)
    for j in range(pairs):
        want = C.padd(want, C.pmul(a[j], b[j], mods), mods)
    out = torch.zeros(len(mods) * P.n, dtype=torch.int64, device="cuda")
    step(f"mac pairs={pairs}")
    ctx.mac(to_dev(a), to_dev(b), out, pairs, len(mods) * P.n, len(mods), 0)
    got = to_host(out).reshape(len(mods), P.n)
    assert np.array_equal(got, want), first_mismatch(got, want)


def test_cfg2_full_size():
    """64 polynomials x 24 limbs x 2^16: forward transform, inverse, and the
    64-pair multiply-accumulate, compared on every residue."""
    P = C.params_p16()
    ctx = _ctx(P)
    mods = P.q
    B, Lm, n = WL.CFG2["batch"], WL.CFG2["limbs"], P.n
    A = WL.cfg2_polys("A", mods, n, B)
    Bm = WL.cfg2_polys("B", mods, n, B)
    d = to_dev(A)
    step("cfg2 ntt_fwd 64x24x2^16")
    ctx.ntt_fwd(d, B, Lm * n, Lm, n, 0)
    got = to_host(d)
    want = C.ntt(P, A.reshape(B * Lm, n), mods * B).reshape(B, Lm, n)
    assert np.array_equal(got, want), first_mismatch(got, want)
    del want
    step("cfg2 mac 64 pairs")
    out = torch.zeros(Lm * n, dtype=torch.int64, device="cuda")
    db = to_dev(Bm)
    ctx.mac(d, db, out, B, Lm * n, Lm, 0)
    gotm = to_host(out).reshape(Lm, n)
    wantm = np.zeros((Lm, n), dtype=np.uint64)
    from oracle import _native as nat
    nat.lib().or_mac_rows(nat.u64p(np.ascontiguousarray(got)), nat.u64p(Bm),
                          nat.u64p(wantm), B, Lm, n, nat.u64p(nat.moduli(mods)))
    assert np.array_equal(gotm, wantm), first_mismatch(gotm, wantm)
    step("cfg2 ntt_inv 64x24x2^16")
    ctx.ntt_inv(d, B, Lm * n, Lm, n, 0)
    back = to_host(d)
    assert np.array_equal(back, A), first_mismatch(back, A)


def test_calib_valu_rates_are_positive_and_ordered():
    """The VALU calibration helper runs all three kernels and reports finite
    rates; a radix-2 butterfly (one modular product, lazily reduced sum and
    difference) cannot be cheaper than about a third of a multiply-accumulate
    and both stay below the device's fp64 instruction rate."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 36, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    step("calib valu")
    r = {k: ctx.calib_valu(k, 256) for k in (F.CALIB_CT, F.CALIB_GS, F.CALIB_MAC,
                                              F.CALIB_MODMUL_F64, F.CALIB_MODMUL_U64,
                                              F.CALIB_PHILOX)}
    print({k: f"{v / 1e12:.3f} T/s" for k, v in r.items()})
    for v in r.values():
        assert np.isfinite(v) and 1e9 < v < 1e14
    # a generator block is ten rounds of two 64 x 64 -> 128-bit products:
    # far dearer than one modular product
    assert r[F.CALIB_PHILOX] < r[F.CALIB_MODMUL_F64] / 4
    with pytest.raises(F.FescError):
        ctx.calib_valu(7, 16)
    # streaming HBM ceilings: below the 8 TB/s peak, well above a slow path
    for kind in (F.CALIB_HBM_READ, F.CALIB_HBM_COPY):
        v = ctx.calib_hbm(kind, 1 << 30)
        assert 1e12 < v < 8.1e12, (kind, v)
    with pytest.raises(F.FescError):
        ctx.calib_hbm(2, 1 << 30)
    with pytest.raises(F.FescError):
        ctx.calib_hbm(F.CALIB_HBM_READ, (1 << 30) + 8)
