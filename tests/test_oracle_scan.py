"""Pins of the oracle's affine prefix scan (Sec. "Parallel Prefix Scans",
Eq. "compact_affine_compose", Eq. "resident-block-schedule", Appendix
"Prefix-Network Selection").

The network is generic over its operator, so its wiring is checked with
operators whose results expose any misplaced, missing or reordered operand:
string concatenation (associative, not commutative) and exact affine maps over
a prime field.  The closed-form counts and the paper's Table
"real-phantom-scan" pin the node and stage counts.  The encrypted composition
is pinned by decoding: the states must follow the plain recurrence
h_k = a_k h_{k-1} + s_k."""
import math
import pathlib

import numpy as np
import pytest

import synth
from oracle import ckks as C
from oracle import scan as S

GOLDEN = pathlib.Path(__file__).parent / "golden" / "scan_topology_ksw.txt"


def _concat(l, r):
    return l + r


def _tokens(L):
    return [f"<{i}>" for i in range(L)]


@pytest.mark.parametrize("L", list(range(1, 70)) + [127, 128, 129, 255, 256])
def test_bk_prefixes_equal_sequential_concatenation(L):
    pre, _, _ = S.brent_kung(_tokens(L), _concat)
    want, acc = [], ""
    for t in _tokens(L):
        acc += t
        want.append(acc)
    assert pre == want


@pytest.mark.parametrize("m", range(1, 12))
def test_bk_counts_match_closed_forms(m):
    Lp = 1 << m
    _, nodes, stages = S.brent_kung(_tokens(Lp), _concat)
    # up-sweep L' - 1, down-sweep L' - 1 - log2 L'
    assert nodes == (Lp - 1) + (Lp - 1 - m) == S.bk_count(Lp)
    assert stages == 2 * m - 1 == S.bk_stages(Lp)


def test_bk_counts_reproduce_the_paper_table():
    K_s = 128 * 1536 // 16384       # state chunks of Mamba-base
    rows = [l.split() for l in GOLDEN.read_text().splitlines() if l and not l.startswith("#")]
    assert len(rows) == 5
    for L, bk_k, bk_dep, seq_k in rows:
        L = int(L)
        _, nodes, stages = S.brent_kung(_tokens(L), _concat)
        assert round(2 * K_s * nodes / 1000, 1) == float(bk_k)   # two products per node
        assert stages == int(bk_dep)
        assert round(2 * K_s * (L - 1) / 1000, 1) == float(seq_k)


def test_bk_affine_maps_exact():
    p = (1 << 61) - 1
    rng = np.random.default_rng(7)
    maps = [(int(rng.integers(1, p)), int(rng.integers(0, p))) for _ in range(37)]

    def comp(left, right):            # right after left
        aL, sL = left
        aR, sR = right
        return (aR * aL % p, (aR * sL + sR) % p)

    pre, _, _ = S.brent_kung(maps, comp)
    h = 0
    A = 1
    for k, (a, s) in enumerate(maps):
        h = (a * h + s) % p
        A = A * a % p
        assert pre[k] == (A, h)


@pytest.mark.parametrize("L", [1, 2, 3, 5, 8, 13, 16, 33])
@pytest.mark.parametrize("block", [1, 2, 3, 4, 8, 64])
def test_resident_schedule_equals_inclusive_scan(L, block):
    want, _, _ = S.brent_kung(_tokens(L), _concat)
    got = S.resident_schedule(_tokens(L), block, _concat, lambda p: p, lambda p, g: g + p)
    assert got == want


def _depth_of(L):
    pre, _, _ = S.brent_kung([0] * L, lambda l, r: max(l, r) + 1)
    return max(pre)


def test_bk_multiplicative_depth():
    assert _depth_of(1) == 0 and _depth_of(2) == 1
    for m in range(2, 12):
        assert _depth_of(1 << m) == 2 * m - 2
    # a ragged length never needs more than its padded length
    for L in range(3, 200):
        Lp = 1 << math.ceil(math.log2(L))
        assert _depth_of(L) <= _depth_of(Lp)


# ------------------------------------------------------ encrypted composition

DELTA_S = 2.0 ** 40


class _Enc:
    def __init__(self, P, seed):
        self.P, self.seed = P, seed
        self.sk = C.secret_key(P, synth.secret(seed, P.n))
        a, e = synth.switch_key_draws(seed, P.ext(P.L), P.n, P.dnum, 0)
        self.rlk = C.relin_key(P, self.sk, a, e)

    def enc(self, z, scale, level, idx):
        P = self.P
        m = C.enc.encode(np.asarray(z, dtype=np.complex128), scale, P.n)
        a, e = synth.encrypt_draws(self.seed, P.qs(level), P.n, "oracle-scan", idx)
        return C.encrypt(P, self.sk, C.ntt(P, C.lift(m, P.qs(level)), P.qs(level)), level, a, e)


def _inputs(E, L, level, tag):
    P = E.P
    n_slots = P.n // 2
    dec = [0.5 + 0.5 * synth.uniform_pm1(E.seed, tag + "a", n_slots, k) ** 2 for k in range(L)]
    upd = [synth.normal(E.seed, tag + "s", n_slots, 1.0, k) for k in range(L)]
    # decay at the scale of the prime its product is rescaled by: the state
    # scale then stays DELTA_S (up to the ratio of neighbouring primes)
    a = [E.enc(dec[k], float(P.q[level - 1]), level, 2 * k) for k in range(L)]
    s = [E.enc(upd[k], DELTA_S, level, 2 * k + 1) for k in range(L)]
    return dec, upd, a, s


@pytest.fixture(scope="module")
def enc():
    return _Enc(C.params_small(12, 50, 8, 2), 41)


def test_encrypted_affine_scan_follows_the_recurrence(enc):
    P, level, L = enc.P, 8, 8
    dec, upd, a, s = _inputs(enc, L, level, "bk")
    A, H = S.affine_scan(P, a, s, enc.rlk)
    assert all(x.shape[0] == level - (2 * 3 - 2) for x in A + H)
    h = np.zeros(P.n // 2)
    prod = np.ones(P.n // 2)
    for k in range(L):
        h = dec[k] * h + upd[k]
        prod = prod * dec[k]
        got = C.decrypt(enc.P, enc.sk, H[k], DELTA_S).real
        assert np.max(np.abs(got - h)) <= 2.0 ** -15, k
        got_a = C.decrypt(enc.P, enc.sk, A[k], float(P.q[level - 1])).real
        assert np.max(np.abs(got_a - prod)) <= 2.0 ** -15, k


def test_encrypted_resident_scan_follows_the_recurrence(enc):
    P, level, L, block = enc.P, 8, 7, 3
    dec, upd, a, s = _inputs(enc, L, level, "res")
    H = S.resident_scan(P, a, s, block, enc.rlk)
    h = np.zeros(P.n // 2)
    for k in range(L):
        h = dec[k] * h + upd[k]
        got = C.decrypt(enc.P, enc.sk, H[k], DELTA_S).real
        assert np.max(np.abs(got - h)) <= 2.0 ** -15, k
