"""GPU parity of the encrypted affine prefix scan (Brent-Kung, in place) and of
the resident two-pass block schedule against the oracle: every residue of the
outputs' leading out_level limbs must match.  Small ring (N = 2^12, 8 levels)
with ragged lengths, several chunks and a partial last block; one full-size
case (N = 2^16, level 24); and the argument errors."""
import numpy as np
import pytest
import torch

import synth
from oracle import ckks as C
from oracle import scan as OS
from paper_2608_17442_amd import fesc as F
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_host
from tests.test_gpu_ckks import Setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _inputs(S, L, chunks, level, tag):
    """Per chunk and token: decay in (0.5, 1] at the scale of q_{level-1},
    update ~ N(0, 1) at 2^40; encrypted on both sides from the same draws."""
    P = S.P
    n_slots = P.n // 2
    ao, so, ad, sd = [], [], [], []
    for c in range(chunks):
        for k in range(L):
            i = c * L + k
            dec = 0.5 + 0.5 * synth.uniform_pm1(S.seed, tag + "a", n_slots, i) ** 2
            upd = synth.normal(S.seed, tag + "s", n_slots, 1.0, i)
            x, y = S.encrypt(dec, float(P.q[level - 1]), level, 1000 + 2 * i)
            ao.append(x)
            ad.append(y)
            x, y = S.encrypt(upd, 2.0 ** 40, level, 1001 + 2 * i)
            so.append(x)
            sd.append(y)
    return ao, so, ad, sd


def _eq_prefix(dev, want, what):
    lvl = want.shape[0]
    got = to_host(dev)[: want.size].reshape(want.shape)
    assert np.array_equal(got, want), f"{what} (level {lvl}): {first_mismatch(got, want)}"


@pytest.fixture(scope="module")
def small():
    return Setup(C.params_small(12, 50, 8, 2), 51, relin=True)


@pytest.mark.parametrize("L,chunks", [(7, 2), (8, 1), (2, 1), (1, 2), (13, 1)])
def test_affine_scan_small(small, L, chunks):
    S, level = small, 8
    ao, so, ad, sd = _inputs(S, L, chunks, level, f"bk{L}")
    step(f"affine_scan L={L} chunks={chunks} level={level}")
    lo = S.ctx.affine_scan(ad, sd, chunks, level)
    depth = {1: 0, 2: 1, 7: 4, 8: 4, 13: 5}[L]
    assert lo == level - depth
    lo_i, ks = S.ctx.affine_scan_info(L, level)
    assert lo_i == lo and ks == 2 * OS.brent_kung(list(range(L)), lambda x, y: x)[1]
    for c in range(chunks):
        A, H = OS.affine_scan(S.P, ao[c * L:(c + 1) * L], so[c * L:(c + 1) * L], S.keys[0])
        for k in range(L):
            _eq_prefix(ad[c * L + k], A[k], f"chunk {c} a-prefix {k}")
            _eq_prefix(sd[c * L + k], H[k], f"chunk {c} state {k}")


@pytest.mark.parametrize("L,chunks", [(7, 2), (16, 1)])
def test_affine_scan_states_only(small, L, chunks):
    """Dead decay products skipped: the states are unchanged, with
    2 (2(L-1) - log2 L) - (dead decay products) key switches."""
    S, level = small, 8
    ao, so, ad, sd = _inputs(S, L, chunks, level, f"so{L}")
    lo_i, ks = S.ctx.affine_scan_info(L, level, states_only=True)
    step(f"affine_scan states-only L={L} chunks={chunks} level={level}")
    lo = S.ctx.affine_scan(ad, sd, chunks, level, states_only=True)
    assert lo == lo_i
    if L == 16:
        assert ks == 37          # 26 state products + 11 live decay products
    for c in range(chunks):
        _, H = OS.affine_scan(S.P, ao[c * L:(c + 1) * L], so[c * L:(c + 1) * L], S.keys[0])
        for k in range(L):
            _eq_prefix(sd[c * L + k], H[k], f"chunk {c} state {k}")


@pytest.mark.parametrize("L,chunks,block", [(11, 2, 4), (9, 1, 3), (5, 1, 8), (6, 2, 1)])
def test_affine_scan_resident_small(small, L, chunks, block):
    S, level = small, 8
    ao, so, ad, sd = _inputs(S, L, chunks, level, f"res{L}-{block}")
    lo, ws_bytes, _ = S.ctx.affine_scan_resident_info(L, chunks, block, level)
    h = [torch.zeros(lo * 2 * S.P.n, dtype=torch.int64, device="cuda") for _ in range(L * chunks)]
    ws = torch.empty(max(ws_bytes // 8, 1), dtype=torch.int64, device="cuda")
    keep = [x.clone() for x in ad + sd]
    step(f"affine_scan_resident L={L} chunks={chunks} block={block} level={level}")
    S.ctx.affine_scan_resident(ad, sd, chunks, block, h, level, ws)
    for c in range(chunks):
        H = OS.resident_scan(S.P, ao[c * L:(c + 1) * L], so[c * L:(c + 1) * L], block, S.keys[0])
        assert H[0].shape[0] == lo
        for k in range(L):
            _eq_prefix(h[c * L + k], H[k], f"chunk {c} state {k}")
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(keep, ad + sd)), "inputs modified"


def test_affine_scan_errors(small):
    S, level = small, 8
    _, _, ad, sd = _inputs(S, 4, 1, level, "err")
    with pytest.raises(F.FescError, match="distinct"):
        S.ctx.affine_scan([ad[0], ad[1], ad[0], ad[3]], sd, 1, level)
    # 16 tokens need 6 levels below the input: level 4 cannot hold them
    _, _, ad16, sd16 = _inputs(S, 16, 1, 4, "deep")
    with pytest.raises(F.FescError, match="levels"):
        S.ctx.affine_scan(ad16, sd16, 1, 4)
    lo, ws_bytes, _ = S.ctx.affine_scan_resident_info(4, 1, 2, level)
    h = [torch.zeros(lo * 2 * S.P.n, dtype=torch.int64, device="cuda") for _ in range(4)]
    short = torch.empty(ws_bytes // 8 - 1, dtype=torch.int64, device="cuda")
    with pytest.raises(F.FescError, match="workspace"):
        S.ctx.affine_scan_resident(ad, sd, 1, 2, h, level, short)
    bare = Setup(small.P, 52)
    with pytest.raises(F.FescError, match="relinearisation"):
        bare.ctx.affine_scan(ad, sd, 1, level)


def test_affine_scan_full_size():
    """N = 2^16, 24 levels (Mamba-base ring), four tokens of one chunk."""
    S = Setup(C.params_p16(24), 53, relin=True)
    L, level = 4, 24
    ao, so, ad, sd = _inputs(S, L, 1, level, "p16")
    step(f"affine_scan full size L={L} level={level}")
    lo = S.ctx.affine_scan(ad, sd, 1, level)
    assert lo == level - 2
    A, H = OS.affine_scan(S.P, ao, so, S.keys[0])
    for k in range(L):
        _eq_prefix(ad[k], A[k], f"a-prefix {k}")
        _eq_prefix(sd[k], H[k], f"state {k}")


@pytest.mark.parametrize("L,level,states_only", [(2, 2, False), (4, 3, False), (4, 3, True),
                                                 (3, 4, True)])
def test_affine_scan_down_to_level_one(small, L, level, states_only):
    """The last compositions at level 2 (one q prime left with the special
    primes in the merged division): outputs at level 1."""
    S = small
    ao, so, ad, sd = _inputs(S, L, 1, level, f"low{L}-{level}")
    step(f"affine_scan low L={L} level={level} states_only={states_only}")
    lo = S.ctx.affine_scan(ad, sd, 1, level, states_only=states_only)
    assert lo == {(2, 2): 1, (4, 3): 1, (3, 4): 2}[(L, level)]
    A, H = OS.affine_scan(S.P, ao, so, S.keys[0])
    for k in range(L):
        _eq_prefix(sd[k], H[k], f"state {k}")
        if not states_only:
            _eq_prefix(ad[k], A[k], f"a-prefix {k}")


def test_affine_scan_bench_configuration():
    """The benchmark's launch: 128 tokens x 12 chunks at 16 limbs (N = 2^16),
    states only, in place.  Chunk 0 holds 128 real tokens and is compared
    whole against the oracle's 128-token network (every up- and down-sweep
    position, down to the deepest); chunk 11 holds 8 real tokens, compared
    through prefix 8 (prefix k depends only on tokens 0..k and the network
    forms positions below 2^m exactly as a 2^m-token network does); every
    other tuple is uniform residues.  Compared on the leading limbs of the
    common output level."""
    P = C.params_p16(24)
    S = Setup(P, 54, relin=True)
    L, chunks, level = 128, 12, 16
    real = {0: L, chunks - 1: 8}
    words = level * 2 * P.n
    ad, sd, ao, so = [], [], {}, {}
    for c in range(chunks):
        for k in range(L):
            if k < real.get(c, 0):
                i = c * L + k
                dec = 0.5 + 0.5 * synth.uniform_pm1(S.seed, "bench-a", P.n // 2, i) ** 2
                upd = synth.normal(S.seed, "bench-s", P.n // 2, 1.0, i)
                x, y = S.encrypt(dec, float(P.q[level - 1]), level, 3000 + 2 * i)
                ao.setdefault(c, []).append(x)
                ad.append(y)
                x, y = S.encrypt(upd, 2.0 ** 40, level, 3001 + 2 * i)
                so.setdefault(c, []).append(x)
                sd.append(y)
            else:
                ad.append(torch.randint(0, 1 << 49, (words,), dtype=torch.int64, device="cuda"))
                sd.append(torch.randint(0, 1 << 49, (words,), dtype=torch.int64, device="cuda"))
    lo_i, _ = S.ctx.affine_scan_info(L, level, states_only=True)
    step(f"affine_scan bench configuration L={L} chunks={chunks} level={level}")
    lo = S.ctx.affine_scan(ad, sd, chunks, level, states_only=True)
    assert lo == lo_i == level - 12
    for c, m in real.items():
        _, H = OS.affine_scan(S.P, ao[c], so[c], S.keys[0])
        for k in range(m):
            want = H[k][:lo]
            _eq_prefix(sd[c * L + k], want, f"chunk {c} state {k}")
