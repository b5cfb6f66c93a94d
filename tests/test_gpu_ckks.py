"""GPU parity of the ciphertext operations against the oracle: key
generation, encryption, add / sub / ptmul / monomial, rescale, rotation
(plain, hoisted, conjugation, identity, in place) and ctmul + relinearisation.
Every comparison is on raw residues (bit-exact); a decrypt check confirms the
values as well."""
import numpy as np
import pytest
import torch

import synth
from oracle import ckks as C
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


class Setup:
    """One parameter set on both sides, with keys generated from the same
    draws on the GPU and in the oracle."""

    def __init__(self, P, seed, rot_steps=(), relin=False, conj=False):
        from paper_2608_17442_amd import fesc as F
        self.P, self.seed = P, seed
        self.ctx = F.Context(P.log_n, P.q, P.p)
        s = synth.secret(seed, P.n)
        self.s_dev = torch.from_numpy(s).cuda()
        self.sk = C.secret_key(P, s)
        elts = {P.galois_elt(r) for r in rot_steps if r % (P.n // 2)}
        if conj:
            elts.add(P.conj_elt)
        if relin:
            elts.add(0)
        self.keys = {}
        for g in sorted(elts):
            a, e = synth.switch_key_draws(seed, P.ext(P.L), P.n, P.dnum, g)
            step(f"keygen g={g} log_n={P.log_n}")
            self.ctx.keygen(g, self.s_dev, to_dev(a), torch.from_numpy(e).cuda())
            self.keys[g] = C.relin_key(P, self.sk, a, e) if g == 0 else \
                C.galois_key(P, self.sk, g, a, e)

    def encrypt(self, z, scale, level, idx, oracle=True):
        """Encrypt on both sides from the same draws; returns (oracle, device)
        (oracle None when not asked for)."""
        P = self.P
        m = C.enc.encode(np.asarray(z, dtype=np.complex128), scale, P.n)
        a, e = synth.encrypt_draws(self.seed, P.qs(level), P.n, "gpu", idx)
        ct_o = None
        if oracle:
            ct_o = C.encrypt(P, self.sk, C.ntt(P, C.lift(m, P.qs(level)), P.qs(level)), level,
                             a, e)
        ct_d = torch.zeros(level * 2 * P.n, dtype=torch.int64, device="cuda")
        step(f"encrypt level={level} idx={idx}")
        self.ctx.encrypt_sk(self.s_dev, torch.from_numpy(m).cuda(), to_dev(a),
                            torch.from_numpy(e).cuda(), ct_d, level)
        return ct_o, ct_d


def _z(seed, n_slots):
    return synth.uniform_pm1(seed, "zr", n_slots) + 1j * synth.uniform_pm1(seed, "zi", n_slots)


def _eq(dev, want, what):
    got = to_host(dev).reshape(want.shape)
    assert np.array_equal(got, want), f"{what}: {first_mismatch(got, want)}"


SMALL = [(12, 50, 5, 2), (13, 45, 4, 3)]


@pytest.mark.parametrize("log_n,bits,L,alpha", SMALL)
def test_keygen_encrypt_elementwise_rescale(log_n, bits, L, alpha):
    P = C.params_small(log_n, bits, L, alpha)
    S = Setup(P, 11, rot_steps=[3], relin=True)
    for g, kw in S.keys.items():
        d = torch.zeros(S.ctx.key_words(), dtype=torch.int64, device="cuda")
        S.ctx.key_store(g, d)
        _eq(d, kw, f"switching key g={g}")
    level = L
    z1, z2, w = _z(1, P.n // 2), _z(2, P.n // 2), _z(3, P.n // 2)
    c1o, c1d = S.encrypt(z1, 2.0 ** 30, level, 1)
    _eq(c1d, c1o, "encrypt")
    c2o, c2d = S.encrypt(z2, 2.0 ** 30, level, 2)
    out = torch.zeros_like(c1d)
    step("add/sub")
    S.ctx.add(c1d, c2d, out, level)
    _eq(out, C.ct_add(P, c1o, c2o), "add")
    S.ctx.sub(c1d, c2d, out, level)
    _eq(out, C.ct_sub(P, c1o, c2o), "sub")
    # plaintext from coefficients and ptmul (in place)
    m = C.enc.encode(w, float(P.q[level - 1]), P.n)
    pt = torch.zeros(level * P.n, dtype=torch.int64, device="cuda")
    S.ctx.plain_from_coeffs(torch.from_numpy(m).cuda(), pt, level)
    pto = C.ntt(P, C.lift(m, P.qs(level)), P.qs(level))
    _eq(pt, pto, "plaintext")
    prod = c1d.clone()
    step("mul_plain in place")
    S.ctx.mul_plain(prod, pt, prod, level)
    prod_o = C.mul_plain(P, c1o, pto)
    _eq(prod, prod_o, "mul_plain")
    for k in [0, 1, 7, P.n // 2, 3 * P.n // 2, 2 * P.n - 1]:
        S.ctx.mul_monomial(c1d, out, level, k)
        _eq(out, C.mul_monomial(P, c1o, k), f"monomial k={k}")
    step("rescale in place")
    rs = prod.clone()
    S.ctx.rescale(rs, rs, level)
    rs_o = C.rescale(P, prod_o)
    _eq(rs[: (level - 1) * 2 * P.n], rs_o, "rescale")
    np.testing.assert_allclose(C.decrypt(P, S.sk, rs_o, 2.0 ** 30), z1 * w, atol=2.0 ** -12)


@pytest.mark.parametrize("log_n,bits,L,alpha", SMALL)
def test_rotations_conjugation_hoisted(log_n, bits, L, alpha):
    P = C.params_small(log_n, bits, L, alpha)
    steps = [1, 5, -3, P.n // 2 - 1]
    S = Setup(P, 12, rot_steps=steps, conj=True)
    F = S.ctx
    for level in [L, 2, 1]:
        z = _z(10 + level, P.n // 2)
        co, cd = S.encrypt(z, 2.0 ** 30, level, 100 + level)
        out = torch.zeros_like(cd)
        for r in steps + [0, P.n // 2]:
            step(f"rotate level={level} step={r}")
            F.rotate(cd, out, level, r)
            want = C.rotate(P, co, r, S.keys)
            _eq(out, want, f"rotate level={level} step={r}")
        from paper_2608_17442_amd.fesc import CONJ
        F.rotate(cd, out, level, CONJ)
        want_c = C.conjugate(P, co, S.keys)
        _eq(out, want_c, f"conjugate level={level}")
        # value check only (scale 2^30 with key-switch noise ~2^16)
        np.testing.assert_allclose(C.decrypt(P, S.sk, want_c, 2.0 ** 30), np.conj(z),
                                   atol=2.0 ** -11)
        # hoisted: all steps from one ModUp, equal to the plain rotations
        outs = [torch.zeros_like(cd) for _ in steps + [0]]
        step(f"hoisted level={level}")
        F.rotate_hoisted(cd, steps + [0], outs, level)
        wants = C.rotate_hoisted(P, co, steps + [0], S.keys)
        for r, o, w in zip(steps + [0], outs, wants):
            _eq(o, w, f"hoisted level={level} step={r}")
        # in place
        inplace = cd.clone()
        F.rotate(inplace, inplace, level, steps[0])
        _eq(inplace, C.rotate(P, co, steps[0], S.keys), "rotate in place")


@pytest.mark.parametrize("log_n,bits,L,alpha", SMALL)
def test_mul_relin(log_n, bits, L, alpha):
    P = C.params_small(log_n, bits, L, alpha)
    S = Setup(P, 13, relin=True)
    # the top level, full-digit levels (every digit alpha primes), level 2, level 1
    levels = sorted({L, alpha * (L // alpha), alpha, 2, 1} & set(range(1, L + 1)), reverse=True)
    for level in levels:
        z1, z2 = _z(20 + level, P.n // 2), _z(30 + level, P.n // 2)
        ao, ad = S.encrypt(z1, 2.0 ** 20, level, 200 + level)
        bo, bd = S.encrypt(z2, 2.0 ** 20, level, 300 + level)
        out = torch.zeros_like(ad)
        step(f"mul_relin level={level}")
        S.ctx.mul_relin(ad, bd, out, level)
        want = C.mul_relin(P, ao, bo, S.keys[0])
        _eq(out, want, f"mul_relin level={level}")
        # aliasing the first operand
        S.ctx.mul_relin(ad, bd, ad, level)
        _eq(ad, want, "mul_relin in place")
        # value check only.  A fresh ciphertext at scale 2^20 carries slot noise
        # of about sigma sqrt(N) / 2^20 <= 3.2 * 2^6.5 / 2^20 ~ 2^-11.8 (N <= 2^13);
        # the product's error is about |z1| e2 + |z2| e1 (|z| <= sqrt 2), ~2^-10.3
        # typical and a few times that at the worst slot: 2^-7 leaves a margin
        np.testing.assert_allclose(C.decrypt(P, S.sk, want, 2.0 ** 40), z1 * z2, atol=2.0 ** -7)


@pytest.mark.parametrize("log_n,bits,L,alpha", SMALL)
def test_rotate_batch(log_n, bits, L, alpha):
    """Independent ciphertexts rotated in one batch (more than one launch
    group of 32, identity and conjugation steps mixed in) equal the oracle's
    single rotations."""
    from paper_2608_17442_amd.fesc import CONJ
    P = C.params_small(log_n, bits, L, alpha)
    base = [1, 2, 3, -1, 7, 0]
    S = Setup(P, 14, rot_steps=base, conj=True)
    level = L - 1
    count = 37
    steps = [base[i % len(base)] if i % 9 else CONJ for i in range(count)]
    cts = [S.encrypt(_z(400 + i, P.n // 2), 2.0 ** 30, level, 400 + i) for i in range(count)]
    outs = [torch.zeros_like(cts[0][1]) for _ in range(count)]
    step(f"rotate_batch count={count}")
    S.ctx.rotate_batch([d for _, d in cts], steps, outs, level)
    for i, ((co, _), st, o) in enumerate(zip(cts, steps, outs)):
        want = C.conjugate(P, co, S.keys) if st == CONJ else C.rotate(P, co, st, S.keys)
        _eq(o, want, f"batch item {i} step {st}")


def test_error_codes():
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    ct = torch.zeros(3 * 2 * P.n, dtype=torch.int64, device="cuda")
    with pytest.raises(F.FescError) as e:
        ctx.rotate(ct, ct, 3, 1)
    assert e.value.code == -3          # no key
    with pytest.raises(F.FescError) as e:
        ctx.rescale(ct, ct, 1)
    assert e.value.code == -2          # level
    with pytest.raises(F.FescError) as e:
        ctx.mul_plain(ct, ct, ct, 4)
    assert e.value.code == -2
    with pytest.raises(F.FescError) as e:
        ctx.mul_relin(ct, ct, ct, 2)
    assert e.value.code == -3
    assert torch.count_nonzero(ct).item() == 0


def test_cfg3_full_size_rotations():
    """N = 2^16, 24 limbs, dnum 3 with 8 special primes: fresh ciphertexts
    rotated by powers of two (and the identity step 2^15), every residue
    compared with the oracle."""
    import synth.workloads as WL
    P = C.params_p16()
    idx = [0, 5, 15]                            # steps 1, 32, 2^15 (identity)
    steps = [WL.cfg3_steps()[i] for i in idx]
    S = Setup(P, WL.CFG3["seed"], rot_steps=steps)
    for i, r in zip(idx, steps):
        z = WL.cfg3_slots(i, P.n // 2)
        co, cd = S.encrypt(z, 2.0 ** 40, 24, i)
        out = torch.zeros_like(cd)
        step(f"cfg3 rotate ct {i} by {r}")
        S.ctx.rotate(cd, out, 24, r)
        want = C.rotate(P, co, r, S.keys)
        _eq(out, want, f"cfg3 rotate {r}")
        got = C.decrypt(P, S.sk, want, 2.0 ** 40)
        assert np.max(np.abs(got - np.roll(z, -r))) < 2.0 ** -15


def test_cfg3_rotation_set_as_benched():
    """The rotation set in the launch configuration the benchmark times: all
    32 fresh ciphertexts (N = 2^16, 24 limbs, dnum 3, 8 special primes) in ONE
    fesc_rotate_batch call, ciphertext i by 2^(i mod 16): 30 key switches
    under 15 keys (two jobs per key group of the key-stationary inner
    product) and two identity copies.  Every output is compared residue by
    residue with the oracle's single rotation and decoded within 2^-15."""
    import synth.workloads as WL
    P = C.params_p16()
    steps = WL.cfg3_steps()
    S = Setup(P, WL.CFG3["seed"], rot_steps=steps)
    assert len(S.keys) == 15
    cts = []
    for i in range(len(steps)):
        cts.append(S.encrypt(WL.cfg3_slots(i, P.n // 2), 2.0 ** 40, 24, 1000 + i))
    outs = [torch.zeros_like(cts[0][1]) for _ in steps]
    step("cfg3 rotate_batch of 32 ciphertexts")
    S.ctx.rotate_batch([d for _, d in cts], steps, outs, 24)
    torch.cuda.synchronize()
    for i, ((co, _), r, o) in enumerate(zip(cts, steps, outs)):
        want = C.rotate(P, co, r, S.keys)
        _eq(o, want, f"cfg3 batch item {i} step {r}")
        got = C.decrypt(P, S.sk, want, 2.0 ** 40)
        err = np.max(np.abs(got - np.roll(WL.cfg3_slots(i, P.n // 2), -r)))
        assert err < 2.0 ** -15, f"item {i}: decoded error {err:.3e}"


def test_mul_relin_full_size_and_square():
    """Relinearised product at N = 2^16 with the 24-limb chain (dnum 3,
    8 special primes): a * b at levels 24 and 20 (a partial last digit), and
    the square a * a with a, b and out the same buffer (the NeRMS square),
    bit-exact against the oracle and decoded within 2^-15 at scale 2^80."""
    P = C.params_p16()
    S = Setup(P, 15, relin=True)
    for level in (24, 20):
        z1, z2 = _z(60 + level, P.n // 2), _z(70 + level, P.n // 2)
        ao, ad = S.encrypt(z1, 2.0 ** 40, level, 600 + level)
        bo, bd = S.encrypt(z2, 2.0 ** 40, level, 700 + level)
        out = torch.zeros_like(ad)
        step(f"mul_relin full size level={level}")
        S.ctx.mul_relin(ad, bd, out, level)
        want = C.mul_relin(P, ao, bo, S.keys[0])
        _eq(out, want, f"mul_relin full size level={level}")
        err = np.max(np.abs(C.decrypt(P, S.sk, want, 2.0 ** 80) - z1 * z2))
        assert err < 2.0 ** -15, f"product level {level}: {err:.3e}"
        step(f"square in place level={level}")
        S.ctx.mul_relin(ad, ad, ad, level)
        want_sq = C.mul_relin(P, ao, ao, S.keys[0])
        _eq(ad, want_sq, f"square in place level={level}")
        err = np.max(np.abs(C.decrypt(P, S.sk, want_sq, 2.0 ** 80) - z1 * z1))
        assert err < 2.0 ** -15, f"square level {level}: {err:.3e}"


def test_key_upload_from_host_over_a_chain_prefix():
    """fesc_key_upload: a key made by the oracle (the client's side) over the
    chain prefix of key_level = 3 primes ([2 digits][3 + 2 rows][2][N]) and
    uploaded from host memory serves rotations at levels 3, 2 and 1
    bit-exactly and is refused at level 4; a full-chain upload equals the
    oracle's key word for word; Galois elements that name no automorphism are
    refused by upload and load alike."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 5, 2)
    S = Setup(P, 16)
    g = P.galois_elt(3)
    a, e = synth.switch_key_draws(16, P.ext(P.L), P.n, P.dnum, g)
    kfull = C.galois_key(P, S.sk, g, a, e)
    key_level = 3
    dk = -(-key_level // P.alpha)
    host = np.ascontiguousarray(np.concatenate([kfull[:dk, :key_level], kfull[:dk, P.L:]],
                                               axis=1))
    step("key_upload prefix key")
    S.ctx.key_upload(g, host, key_level)
    for level in (3, 2, 1):
        co, cd = S.encrypt(_z(90 + level, P.n // 2), 2.0 ** 30, level, 900 + level)
        out = torch.zeros_like(cd)
        step(f"rotate with uploaded prefix key, level {level}")
        S.ctx.rotate(cd, out, level, 3)
        _eq(out, C.rotate(P, co, 3, {g: kfull}), f"uploaded key level {level}")
    _, c4 = S.encrypt(_z(94, P.n // 2), 2.0 ** 30, 4, 904)
    with pytest.raises(F.FescError) as err:
        S.ctx.rotate(c4, torch.zeros_like(c4), 4, 3)
    assert err.value.code == -2
    step("key_upload full chain")
    S.ctx.key_upload(g, kfull, P.L)
    back = torch.zeros(S.ctx.key_words(), dtype=torch.int64, device="cuda")
    S.ctx.key_store(g, back)
    _eq(back, kfull, "full-chain upload")
    co, cd = S.encrypt(_z(95, P.n // 2), 2.0 ** 30, P.L, 905)
    out = torch.zeros_like(cd)
    S.ctx.rotate(cd, out, P.L, 3)
    _eq(out, C.rotate(P, co, 3, {g: kfull}), "uploaded key at the top level")
    for bad in (1, 2, 2 * P.n + 1):
        with pytest.raises(F.FescError) as err:
            S.ctx.key_upload(bad, kfull, P.L)
        assert err.value.code == -1
        with pytest.raises(F.FescError) as err:
            S.ctx.key_load(bad, back)
        assert err.value.code == -1


def test_empty_batches_are_rejected():
    """A zero batch is an argument error (nothing launched), for the NTT and
    for batched rotations."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    d = torch.zeros(3 * P.n, dtype=torch.int64, device="cuda")
    for fn in (ctx.ntt_fwd, ctx.ntt_inv):
        with pytest.raises(F.FescError) as e:
            fn(d, 0, 3 * P.n, 3, P.n, 0)
        assert e.value.code == -1
    with pytest.raises(F.FescError) as e:
        ctx.rotate_batch([], [], [], 3)
    assert e.value.code == -1


def test_binding_rejects_short_buffers():
    """The binding checks every buffer against the words the call touches
    (and list lengths) before calling the library, so a short tensor is an
    exception, never an out-of-bounds kernel access."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    ct = torch.zeros(3 * 2 * P.n, dtype=torch.int64, device="cuda")
    short = torch.zeros(2 * 2 * P.n - 1, dtype=torch.int64, device="cuda")
    with pytest.raises(ValueError, match="out"):
        ctx.rescale(ct, short, 3)                    # needs 2 limbs x 2 x N
    with pytest.raises(ValueError, match="^a: "):
        ctx.add(short, ct, ct, 3)
    with pytest.raises(ValueError, match="outs"):
        ctx.rotate_hoisted(ct, [1, 2], [ct], 3)      # two steps, one output
    with pytest.raises(ValueError, match="steps"):
        ctx.rotate_batch([ct, ct], [1], [ct, ct], 3)
    with pytest.raises(TypeError):
        ctx.add(ct.cpu(), ct, ct, 3)
    # a tensor of another element type holding as many elements as the call
    # needs words is 1/8 (int8) of the bytes, or no residues at all (fp64):
    # rejected by type, whatever its length
    for dt in (torch.int8, torch.int32, torch.float64):
        other = torch.zeros(3 * 2 * P.n, dtype=dt, device="cuda")
        with pytest.raises(TypeError, match="out"):
            ctx.rescale(ct, other, 3)
        with pytest.raises(TypeError, match="^a: "):
            ctx.add(other, ct, ct, 3)
    # the secret is the one int8 argument, and it must be int8
    with pytest.raises(TypeError, match="^s: "):
        ctx.encrypt_sk(ct[:P.n], ct[:P.n], ct, ct[:P.n], ct, 1)
    assert torch.count_nonzero(ct).item() == 0
