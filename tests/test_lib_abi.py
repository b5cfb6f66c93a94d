"""CPU checks of the C ABI: the library loads, exports every symbol that
include/fesc.h declares, and its host-side parameter helpers agree with the
oracle's (no compute call needs a GPU here)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fesc.h")
LIB = os.path.join(ROOT, "paper_2608_17442_amd", "libfesc.so")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fesc_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2608_17442_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for name in ["fesc_ntt_fwd", "fesc_ntt_inv", "fesc_mac"]:
        assert name in syms


def test_every_declared_symbol_is_exported(lib):
    missing = [s for s in declared_symbols() if not hasattr(lib, s)]
    assert not missing, missing


def test_prime_search_and_roots_match_oracle():
    from oracle import ckks as C
    from paper_2608_17442_amd import fesc as F
    for log_n, bits, count in [(12, 36, 4), (16, 50, 32), (13, 45, 6)]:
        ps = F.find_primes(log_n, bits, count)
        assert ps == C.find_primes(log_n, bits, count)
        for q in ps:
            assert F.root_of_unity(log_n, q) == C.min_psi(q, log_n)


def test_host_helpers_reject_bad_input():
    from paper_2608_17442_amd import fesc as F
    with pytest.raises(F.FescError) as e:
        F.root_of_unity(12, 1000003)   # prime, but not 1 mod 2N
    assert e.value.code == -1


@pytest.mark.parametrize("log_n,scale_bits,kind", [(12, 30, "pm1"), (16, 40, "pm1"),
                                                   (16, 49, "normal")])
def test_host_encoder_matches_oracle_encoding(log_n, scale_bits, kind):
    """fesc_encode (host slot encoder, Sec. 2.1 packing) against the oracle's
    encoding.  Both round Delta * m_k half away from zero after an FFT of their
    own, so the integers agree except where Delta * m_k lies within the two
    FFTs' rounding error of a half-integer; there they may differ by one."""
    import numpy as np

    import synth
    from oracle import encoding as E
    from paper_2608_17442_amd import fesc as F
    n = 1 << log_n
    if kind == "pm1":
        z = synth.uniform_pm1(50 + log_n, "enc-re", n // 2) \
            + 1j * synth.uniform_pm1(50 + log_n, "enc-im", n // 2)
    else:
        z = synth.normal(51, "enc-n", n // 2, 0.02).astype(complex)
    scale = 2.0 ** scale_bits
    got = F.encode(log_n, z, scale)
    raw = E.encode_real_coeffs(z, scale, n)
    want = E.encode(z, scale, n)
    diff = got - want
    near_tie = np.abs(np.abs(raw - np.trunc(raw)) - 0.5) < 1e-2
    assert np.all(np.abs(diff) <= 1)
    assert not np.any(diff[~near_tie]), np.flatnonzero(diff[~near_tie])[:8]
    assert np.count_nonzero(diff) <= np.count_nonzero(near_tie)


def test_c2m_level_matches_oracle():
    """Host modulus trimming (exact big-integer comparisons) against the
    oracle's, over boundary-adjacent and out-of-range bounds."""
    from oracle import ckks as C
    from oracle import workloads as W
    from paper_2608_17442_amd import fesc as F
    P = C.params_p16(24)
    cases = [(64, 40, 2.0 ** 40, 2.0 ** 10), (16, 40, 2.0 ** 40, 2.0 ** 120), (64, 40, 2.0 ** 40, 1.0),
             (0, 0, 0.0, 0.0), (200, 40, 1.0, 1.0), (1100, 40, 1.0, 1.0), (20, 20, 2.0 ** 40, 2.0 ** 900),
             (20, 20, 2.0 ** 40, 1e300), (32, 40, 3.5, 7.25)]
    # bounds placed exactly at the product of the first primes
    for lp in (1, 2, 3, 5):
        Q = 1
        for i in range(lp):
            Q *= P.q[i]
        cases += [(8, 8, float(Q) / 2, 0.5), (8, 8, float(Q) / 2, 0.5 * (1 + 2.0 ** -52)),
                  (Q.bit_length() - 10, 9, 1.0, 1.0), (Q.bit_length() - 10, 8, 1.0, 1.0)]
    for level in (1, 2, 5, 24):
        for ell, sig, d, b in cases:
            want = W.c2m_level(P, level, ell, sig, d, b)
            assert F.c2m_level(P.q, level, ell, sig, d, b) == (want or 0), (level, ell, sig, d, b)


SCAN_LENGTHS = list(range(1, 70)) + [127, 128, 129, 255, 256, 1000, 1024, 2047, 2048, 4096]


@pytest.mark.parametrize("states_only", [False, True])
def test_affine_scan_network_matches_oracle(states_only):
    """The library's scan network (host export) against the oracle's
    Brent-Kung network: the same compositions (dst <- src o dst), independent
    nodes within a stage, adjacent intervals composed so that every position
    ends with its full prefix, the same composition depth; every decay product
    formed without states_only, and with it the pruned network still gives the
    recurrence's states (affine maps mod a prime, skipped decay products left
    stale)."""
    from oracle import scan as OS
    from paper_2608_17442_amd import fesc as F
    prime = (1 << 61) - 1
    for L in SCAN_LENGTHS:
        nodes = F.affine_scan_network(L, states_only)
        ops = []
        OS.brent_kung([(k, k) for k in range(L)],
                      lambda l, r: ops.append((r[1], l[1])) or (l[0], r[1]))
        assert sorted((d, s) for _, d, s, _ in nodes) == sorted(ops), L
        # stages: non-decreasing; within a stage no node reads another's destination
        stages = {}
        for st, d, s, _ in nodes:
            stages.setdefault(st, []).append((d, s))
        assert [n[0] for n in nodes] == sorted(n[0] for n in nodes)
        for st, v in stages.items():
            dsts = {d for d, _ in v}
            assert len(dsts) == len(v) and not any(s in dsts for _, s in v), (L, st)
        # interval semantics and depth
        iv = [(k, k) for k in range(L)]
        depth = [0] * L
        for _, d, s, _ in nodes:
            assert iv[s][1] + 1 == iv[d][0], (L, d, s)
            iv[d] = (iv[s][0], iv[d][1])
            depth[d] = max(depth[d], depth[s]) + 1
        assert iv == [(0, k) for k in range(L)]
        want_depth = OS.brent_kung([0] * L, lambda l, r: max(l, r) + 1)[0] if L > 1 else [0]
        assert max(depth) == max(want_depth), L
        if not states_only:
            assert all(n[3] == 1 for n in nodes)
            continue
        # pruned network: states equal the sequential recurrence
        rng = np.random.default_rng(L)
        a0 = [int(x) for x in rng.integers(1, prime, L)]
        s0 = [int(x) for x in rng.integers(0, prime, L)]
        a, s = list(a0), list(s0)
        for _, d, src, live in nodes:
            s[d] = (a[d] * s[src] + s[d]) % prime
            if live:
                a[d] = a[d] * a[src] % prime
            else:
                a[d] = None                      # a product nothing may read
        h = 0
        for k in range(L):
            h = (a0[k] * h + s0[k]) % prime
            assert s[k] == h, (L, k)


@pytest.mark.parametrize("L,block", [(2048, 1024), (2048, 256), (2048, 64), (1000, 128),
                                     (11, 4), (9, 3), (5, 5), (6, 1), (1, 1)])
def test_resident_schedule_program_gives_the_recurrence(L, block):
    """The library's resident two-pass driver, recorded on the host
    (fesc_affine_scan_resident_program), replayed over GF(2^61 - 1): every
    product out = x y (+ add) in issue order, in launches of 32 products whose
    operands are all read before any output is written (a batched key
    switch), a skipped decay never read.  Every state equals the sequential
    recurrence h_k = a_k h_(k-1) + s_k, at the benchmark's L = 2048 with
    blocks of 1024 and at ragged and degenerate shapes."""
    from paper_2608_17442_amd import fesc as F
    prime = (1 << 61) - 1
    A0, S0, H0 = 1 << 24, 2 << 24, 3 << 24
    prog = F.affine_scan_resident_program(L, block)
    rng = np.random.default_rng(L * 7919 + block)
    a = [int(v) for v in rng.integers(1, prime, L)]
    s = [int(v) for v in rng.integers(0, prime, L)]
    mem = {A0 + k: a[k] for k in range(L)}
    mem.update({S0 + k: s[k] for k in range(L)})
    _replay(prog, mem, prime)
    h = 0
    for k in range(L):
        h = (a[k] * h + s[k]) % prime
        assert mem[H0 + k] == h, (L, block, k)


def _replay(prog, mem, prime):
    """Products out = x y (+ add) / copies, in launches of 32 whose operands are
    all read before any output is written."""
    import itertools
    for _, group in itertools.groupby(prog, key=lambda e: e[0]):
        group = list(group)
        for i in range(0, len(group), 32):
            vals = []
            for _, x, y, add, out in group[i:i + 32]:
                vals.append((out, mem[x] if y == 0 else
                             (mem[x] * mem[y] + (mem[add] if add else 0)) % prime))
            for out, v in vals:
                mem[out] = v


@pytest.mark.parametrize("L,chunks,states_only", [(2048, 2, True), (2048, 1, False),
                                                  (128, 12, True), (13, 3, False), (1, 2, True)])
def test_in_place_scan_program_gives_the_recurrence(L, chunks, states_only):
    """The library's in-place Brent-Kung driver, recorded on the host
    (fesc_affine_scan_program) with chunks batched together as on the GPU,
    replayed over GF(2^61 - 1): every state (and without states_only every
    decay prefix) equals the sequential recurrence, at the benchmark's shapes
    (2048 tokens, two chunks per launch; 128 tokens x 12 chunks)."""
    from paper_2608_17442_amd import fesc as F
    prime = (1 << 61) - 1
    A0, S0 = 1 << 24, 2 << 24
    prog = F.affine_scan_program(L, chunks, states_only)
    rng = np.random.default_rng(L * 31 + chunks)
    a = [int(v) for v in rng.integers(1, prime, L * chunks)]
    s = [int(v) for v in rng.integers(0, prime, L * chunks)]
    mem = {A0 + i: a[i] for i in range(L * chunks)}
    mem.update({S0 + i: s[i] for i in range(L * chunks)})
    _replay(prog, mem, prime)
    for c in range(chunks):
        h, pa = 0, 1
        for k in range(L):
            i = c * L + k
            h, pa = (a[i] * h + s[i]) % prime, pa * a[i] % prime
            assert mem[S0 + i] == h, (c, k)
            if not states_only:
                assert mem[A0 + i] == pa, (c, k)


def _br_shapes():
    from oracle import broadcast as BR
    return [(BR.Dims(2, 4, 1, 2, 4, 64), 7), (BR.Dims(4, 2, 2, 4, 4, 128), 8),
            (BR.Dims(8, 2, 4, 2, 8, 128), 8), (BR.Dims(8, 2, 2, 4, 4, 256), 9),
            (BR.Dims(4, 4, 2, 8, 8, 512), 10), (BR.Dims(24, 64, 1, 128, 128, 32768), 16)]


@pytest.mark.parametrize("i", range(6))
def test_broadcast_slot_maps_match_the_appendix_maps(i):
    """fesc_br_desc (host only): the library's decomposition of br^(kappa),
    applied on plain slot vectors by the oracle's slot-map definition, gives
    exactly the appendix's broadcast of the oracle; and its fields equal the
    oracle's decomposition of the same reading."""
    from oracle import broadcast as BR
    from paper_2608_17442_amd import fesc as F
    D, log_n = _br_shapes()[i]
    assert D.n_slots == 1 << (log_n - 1)
    rng = np.random.default_rng(i)
    v = rng.standard_normal(D.n_slots) + 1j * rng.standard_normal(D.n_slots)
    L = D.n_slots // max(D.E, D.H, D.G * D.d_s)
    for kind in BR.KINDS:
        for k in sorted({0, L // 2, L - 1}):
            for kappa in sorted({0, D.K_s // 2, D.K_s - 1}):
                d = F.br_desc(log_n, D.H, D.P, D.G, D.d_s, D.c_state, kind, k, kappa, 5)
                M = BR.SlotMap(d.level, d.offset, d.stride, d.terms, d.n1, d.giant_stride,
                               d.dst0, d.dst_stride, d.dst_giant, d.width, d.rep_count,
                               d.rep_stride)
                assert np.array_equal(BR.slot_map_plain(M, v), BR.br(D, kind, v, k, kappa))
                O = BR.br_slot_map(D, kind, k, kappa, 5)
                assert (M.r0 - O.r0) % D.n_slots == 0 and M.n == O.n and M.n1 == O.n1
                assert (M.j0, M.w, M.R, M.S) == (O.j0, O.w, O.R, O.S)
                if M.n1 > 1:
                    assert (M.d, M.J) == (O.d, O.J)
                if M.n2 > 1:
                    assert (M.g, M.Jg) == (O.g, O.Jg)


def test_broadcast_slot_map_rejects_uncovered_shapes():
    from paper_2608_17442_amd import fesc as F
    with pytest.raises(F.FescError, match="a broadcast"):    # 6 channels: not whole heads of 4
        F.br_desc(7, 3, 4, 1, 2, 6, "a", 0, 0, 3)
    with pytest.raises(F.FescError, match="x broadcast"):    # d_s = 3
        F.br_desc(7, 2, 4, 1, 3, 4, "x", 0, 0, 3)
    with pytest.raises(F.FescError, match="x broadcast"):    # token 8 leaves 64 slots
        F.br_desc(7, 2, 4, 1, 2, 4, "x", 8, 0, 3)
    with pytest.raises(F.FescError, match="chunks"):         # kappa past the last chunk
        F.br_desc(7, 2, 4, 1, 2, 4, "B", 0, 2, 3)
    with pytest.raises(F.FescError, match="groups"):         # 12-channel groups, 16-channel chunks
        F.br_desc(12, 24, 2, 4, 2, 16, "B", 0, 1, 3)
