"""GPU parity of the HEScan layer pieces against the oracle, residue by
residue: the batched relinearised product with merged rescale (update
construction), the contraction-only scan-contract slice, and the whole layer
(construction, Brent-Kung or resident scan, contraction of every token)
composed from library calls.  Small rings (N = 2^12)."""
import numpy as np
import pytest
import torch

import synth
from oracle import ckks as C
from oracle import scan as OS
from oracle import workloads as OW
from paper_2608_17442_amd import fesc as F
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_host
from tests.test_gpu_ckks import Setup
from tests.test_oracle_workloads import hescan_packets, hescan_reference

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _eq(dev, want, what):
    got = to_host(dev)[: want.size].reshape(want.shape)
    assert np.array_equal(got, want), f"{what}: {first_mismatch(got, want)}"


@pytest.fixture(scope="module")
def small():
    return Setup(C.params_small(12, 50, 8, 2), 61, rot_steps=[1, 2, 4], relin=True, conj=True)


@pytest.mark.parametrize("level,count", [(6, 35), (2, 3)])
def test_mul_relin_rescale_batch(small, level, count):
    """Two groups of products (35 > 32) with separate, in-place (out = a)
    and in-place (out = b) outputs; and the lowest level (output level 1)."""
    S, P = small, small.P
    n_slots = P.n // 2
    ao, ad, bo, bd = [], [], [], []
    for i in range(count):
        x, y = S.encrypt(synth.normal(61, "pa", n_slots, 1.0, i), 2.0 ** 40, level, 100 + 2 * i)
        ao.append(x)
        ad.append(y)
        x, y = S.encrypt(synth.normal(61, "pb", n_slots, 1.0, i), float(P.q[level - 1]), level,
                         101 + 2 * i)
        bo.append(x)
        bd.append(y)
    outs = []
    for i in range(count):
        if i % 3 == 1:
            outs.append(ad[i])
        elif i % 3 == 2:
            outs.append(bd[i])
        else:
            outs.append(torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda"))
    step(f"mul_relin_rescale level={level} count={count}")
    S.ctx.mul_relin_rescale(ad, bd, outs, level)
    for i in range(count):
        want = C.mul_relin_rescale(P, ao[i], bo[i], S.keys[0])
        assert want.shape[0] == level - 1
        _eq(outs[i], want, f"product {i}")


def test_mul_relin_rescale_errors(small):
    S, P = small, small.P
    level = 4
    cts = [S.encrypt(synth.normal(61, "pe", P.n // 2, 1.0, i), 2.0 ** 40, level, 300 + i)[1]
           for i in range(4)]
    out = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda") for _ in range(2)]
    with pytest.raises(F.FescError, match="aliases"):
        S.ctx.mul_relin_rescale(cts[:2], cts[2:], [cts[1], out[1]], level)
    with pytest.raises(F.FescError, match="distinct"):
        S.ctx.mul_relin_rescale(cts[:2], cts[2:], [out[0], out[0]], level)
    with pytest.raises(F.FescError):
        S.ctx.mul_relin_rescale(cts[:2], cts[2:], out, 1)
    S.ctx.mul_relin_rescale([], [], [], level)          # empty batch: no-op


@pytest.mark.parametrize("K,T,level", [(3, 2, 2), (4, 3, 5)])
def test_scan_contract_contraction_only(small, K, T, level):
    """decay = None: t = RS(relin(h C)) then the reduction; level 2 puts the
    rotations and the conjugation at level 1."""
    S, P = small, small.P
    d_s, n_slots = 8, P.n // 2
    j = np.arange(n_slots)
    hs_o, cs_o, hs_d, cs_d = [], [], [], []
    for u in range(T):
        for k in range(K):
            i = u * K + k
            hv = synth.normal(62, "ch", n_slots, 1.0, i)
            cv = synth.normal(62, "cc", d_s, 1.0, i)[j % d_s]
            x, y = S.encrypt(hv, 2.0 ** 40, level, 400 + 2 * i)
            hs_o.append(x)
            hs_d.append(y)
            x, y = S.encrypt(cv, float(P.q[level - 1]), level, 401 + 2 * i)
            cs_o.append(x)
            cs_d.append(y)
    outs = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
            for _ in range(K * T)]
    step(f"scan_contract contraction only K={K} T={T} level={level}")
    S.ctx.scan_contract(hs_d, None, cs_d, d_s, outs, level, tokens=T)
    for u in range(T):
        sl = slice(u * K, (u + 1) * K)
        want = OW.scan_contract_token(P, hs_o[sl], None, cs_o[sl], S.keys[0], S.keys, d_s)
        for k, (od, oo) in enumerate(zip(outs[sl], want)):
            _eq(od, oo, f"token {u} output {k}")


@pytest.fixture(scope="module")
def prefix16():
    """The bench's contraction context: N = 2^16, chain prefix q_0..q_3 of
    the 24-prime chain, the two largest special primes, d_state 128 keys."""
    P = C.params_p16(24)
    return Setup(C.Params(P.log_n, P.q[:4], P.p[:2]), 65,
                 rot_steps=[128 >> k for k in range(1, 8)], relin=True, conj=True)


@pytest.mark.parametrize("level", [2, 3])
def test_contraction_in_prefix_context_full_ring(prefix16, level):
    """The bench's contraction levels (2 -> 1 full length, 3 -> 2 two-pass) in
    the prefix context: one digit at level 2, two at level 3; one token of a
    chunk pair, bit-exact against the oracle under the same parameter set and
    within 2^-15 of the fp64 contraction."""
    S, P = prefix16, prefix16.P
    d_s, K, n_slots = 128, 2, P.n // 2
    j = np.arange(n_slots)
    ho, hd, co, cd, want = [], [], [], [], []
    for k in range(K):
        hv = synth.normal(65, "ph", n_slots, 1.0, k)
        cv = synth.normal(65, "pc", d_s, 1.0, k)
        want.append((hv * cv[j % d_s]).reshape(-1, d_s).sum(axis=1))
        x, y = S.encrypt(hv, 2.0 ** 40, level, 900 + 2 * k)
        ho.append(x)
        hd.append(y)
        x, y = S.encrypt(cv[j % d_s], float(P.q[level - 1]), level, 901 + 2 * k)
        co.append(x)
        cd.append(y)
    outs = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
            for _ in range(K)]
    step(f"prefix-context contraction N=2^16 level={level}")
    S.ctx.scan_contract(hd, None, cd, d_s, outs, level, tokens=1)
    got = OW.scan_contract_token(P, ho, None, co, S.keys[0], S.keys, d_s)
    for k in range(K):
        _eq(outs[k], got[k], f"chunk {k}")
        dec = C.decrypt(P, S.sk, got[k], 2.0 * 2.0 ** 40).real[::d_s]
        assert np.max(np.abs(dec - want[k])) <= 2.0 ** -15


def hescan_gpu(ctx, X, Bc, A, Cc, K, L, d_s, level, block, cctx=None):
    """The layer from library calls (x, B at `level`, a at level - 1; chunk-
    major lists [k * L + t]): construction in place over x, the scan, the
    contraction of every token (in context cctx when given: a context over a
    prefix of the chain, which takes the states' buffers as they are).
    Returns token-major outputs and their level."""
    ctx.mul_relin_rescale(X, Bc, X, level)
    if block is None:
        lo = ctx.affine_scan(A, X, K, level - 1, states_only=True)
        H = X
    else:
        lo, ws_bytes, _ = ctx.affine_scan_resident_info(L, K, block, level - 1)
        n = X[0].numel() // (2 * level)
        H = [torch.zeros(lo * 2 * n, dtype=torch.int64, device="cuda") for _ in range(K * L)]
        ws = torch.empty(max(ws_bytes // 8, 1), dtype=torch.int64, device="cuda")
        ctx.affine_scan_resident(A, X, K, block, H, level - 1, ws)
    tm = lambda v: [v[k * L + t] for t in range(L) for k in range(K)]
    n = X[0].numel() // (2 * level)
    outs = [torch.zeros((lo - 1) * 2 * n, dtype=torch.int64, device="cuda") for _ in range(K * L)]
    (cctx or ctx).scan_contract(tm(H), None, tm(Cc), d_s, outs, lo, tokens=L)
    return outs, lo - 1


@pytest.mark.parametrize("L,K,block", [(4, 2, None), (5, 3, None), (6, 2, 4)])
def test_hescan_layer(small, L, K, block):
    S, P = small, small.P
    d_s, head_dim, level = 8, 16, 8
    vals, br = hescan_packets(P, 63, L, K, d_s, head_dim)
    lo = {(4, None): 5, (5, None): 4, (6, 4): 4}[(L, block)]   # states: 7 - depth
    Xo, Bo, Ao, Co = ([[] for _ in range(K)] for _ in range(4))
    Xd, Bd, Ad, Cd = [], [], [], []
    for k in range(K):
        for t in range(L):
            xv, av, bv, cv = br(k, t)
            i = 4 * (k * L + t)
            for v, sc, lvl, o, d, r in [(xv, 2.0 ** 40, level, Xo, Xd, 0),
                                        (bv, float(P.q[level - 1]), level, Bo, Bd, 1),
                                        (av, float(P.q[level - 2]), level - 1, Ao, Ad, 2),
                                        (cv, float(P.q[lo - 1]), lo, Co, Cd, 3)]:
                co, cd = S.encrypt(v, sc, lvl, 600 + i + r)
                o[k].append(co)
                d.append(cd)
    step(f"hescan layer L={L} K={K} block={block}")
    outs, lo_out = hescan_gpu(S.ctx, Xd, Bd, Ad, Cd, K, L, d_s, level, block)
    assert lo_out == lo - 1
    want = OS.hescan(P, Xo, Bo, Ao, Co, S.keys[0], S.keys, d_s, block)
    ref = hescan_reference(vals, head_dim)
    c_state = P.n // 2 // d_s
    for t in range(L):
        for k in range(K):
            _eq(outs[t * K + k], want[t][k], f"token {t} chunk {k}")
            factor = 1.0 if (K % 2 and k == K - 1) else 2.0
            dec = C.decrypt(P, S.sk, want[t][k], factor * 2.0 ** 40).real[::d_s]
            assert np.max(np.abs(dec - ref[t, k * c_state:(k + 1) * c_state])) <= 2.0 ** -15


@pytest.mark.parametrize("L,block,low", [(4, None, False), (5, 2, False), (4, None, True)])
def test_hescan_layer_full_size(L, block, low):
    """The layer at the bench's ring and chain (N = 2^16, x and B at 23
    limbs, d_state 128, contraction of every token in one call), one chunk
    pair: four tokens through the Brent-Kung scan in place, five through the
    resident schedule with blocks of 2 (summaries, carries, replay): bit-exact
    against the oracle and within 2^-15 of the fp64 recurrence.  With `low`
    the inputs start at 7 limbs so that the states reach level 4, and the
    contraction runs in the bench's low-level context (chain prefix
    q_0..q_3, two special primes instead of eight: two digits at level 4) on
    the states' buffers as they are."""
    P = C.params_p16(24)
    d_s, head_dim, level, K = 128, 64, 7 if low else 23, 2
    rots = [d_s >> k for k in range(1, 8)]
    S = Setup(P, 64, rot_steps=rots, relin=True, conj=True)
    Sc = Setup(C.Params(P.log_n, P.q[:4], P.p[:2]), 64, rot_steps=rots, relin=True,
               conj=True) if low else S
    vals, br = hescan_packets(P, 64, L, K, d_s, head_dim)
    lo = level - 1 - {None: 2, 2: 3}[block]             # scan depth: 2 (BK of 4), 3 (resident)
    Xo, Bo, Ao, Co = ([[] for _ in range(K)] for _ in range(4))
    Xd, Bd, Ad, Cd = [], [], [], []
    for k in range(K):
        for t in range(L):
            xv, av, bv, cv = br(k, t)
            i = 4 * (k * L + t)
            for v, sc, lvl, o, d, r in [(xv, 2.0 ** 40, level, Xo, Xd, 0),
                                        (bv, float(P.q[level - 1]), level, Bo, Bd, 1),
                                        (av, float(P.q[level - 2]), level - 1, Ao, Ad, 2),
                                        (cv, float(P.q[lo - 1]), lo, Co, Cd, 3)]:
                co, cd = S.encrypt(v, sc, lvl, 700 + i + r)
                o[k].append(co)
                d.append(cd)
    step(f"hescan layer full size L={L} K={K} block={block} level={level} low={low}")
    outs, lo_out = hescan_gpu(S.ctx, Xd, Bd, Ad, Cd, K, L, d_s, level, block, Sc.ctx)
    assert lo_out == lo - 1
    want = OS.hescan(P, Xo, Bo, Ao, Co, S.keys[0], S.keys, d_s, block,
                     (Sc.P, Sc.keys[0], Sc.keys) if low else None)
    ref = hescan_reference(vals, head_dim)
    c_state = P.n // 2 // d_s
    for t in range(L):
        for k in range(K):
            _eq(outs[t * K + k], want[t][k], f"token {t} chunk {k}")
            dec = C.decrypt(P, S.sk, want[t][k], 2.0 * 2.0 ** 40).real[::d_s]
            err = np.max(np.abs(dec - ref[t, k * c_state:(k + 1) * c_state]))
            print(f"full-size layer token {t} chunk {k}: max |decoded - fp64| = {err:.3e}")
            assert err <= 2.0 ** -15


def test_scan_contract_errors(small):
    """Argument errors, all rejected before any launch."""
    S, P = small, small.P
    z = lambda lvl, k=1: [torch.zeros(lvl * 2 * P.n, dtype=torch.int64, device="cuda")
                          for _ in range(k)]
    h, c, o = z(4, 2), z(4, 2), z(3, 2)
    with pytest.raises(F.FescError, match="distinct"):
        S.ctx.scan_contract(h, None, c, 8, [o[0], o[0]], 4)
    with pytest.raises(F.FescError, match="alias"):
        S.ctx.scan_contract(h, None, c, 8, [o[0], h[1]], 4)
    with pytest.raises(F.FescError, match="32 tokens"):      # odd chunk count, 33 tokens
        S.ctx.scan_contract(z(4, 33), None, z(4, 33), 8, z(3, 33), 4, tokens=33)
    with pytest.raises(F.FescError):                         # decay product needs level >= 3
        S.ctx.scan_contract(z(2, 2), z(2, 2), z(2, 2), 8, z(1, 2), 2)
    with pytest.raises(F.FescError):                         # contraction needs level >= 2
        S.ctx.scan_contract(z(1, 2), None, z(1, 2), 8, z(1, 2), 1)
    with pytest.raises(F.FescError, match="rotation 8"):     # d_state 16: no key for step 8
        S.ctx.scan_contract(h, None, c, 16, o, 4)
    with pytest.raises(F.FescError, match="bad scan-contract"):
        S.ctx.scan_contract(h, None, c, 6, o, 4)
