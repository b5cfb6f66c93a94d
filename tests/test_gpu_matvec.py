"""GPU parity of the plaintext-matrix x ciphertext projection (BSGS) against
the oracle, on the N = 2^12 diagonal-method workload (64 x 64 matrix, 63
hoisted rotations, rescale), on a complex-paired BSGS instance with several
inputs, outputs and giant steps, with complex-paired outputs (small ring and
the full cfg4 shape), and the device generator of the diagonals' slot
vectors against the oracle's."""
import numpy as np
import pytest
import torch

import synth
import synth.workloads as WL
from oracle import ckks as C
from oracle import workloads as OW
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_dev, to_host
from tests.test_gpu_ckks import Setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _run(P, S, desc, X_slots, scale_x, diag_slots, scale_d, seed_tag):
    """Encrypt inputs, encode diagonals, run both sides; returns (oracle outs,
    device outs)."""
    from paper_2608_17442_amd import fesc as F
    level = desc.level
    ins_o, ins_d = [], []
    for u, z in enumerate(X_slots):
        co, cd = S.encrypt(z, scale_x, level, 1000 + u)
        ins_o.append(co)
        ins_d.append(cd)
    keys_needed = OW.required_rotations(desc, P.n // 2)
    lazy = desc.lazy_moddown
    encode = C.encode_plain_ext if lazy else C.encode_plain
    diag_pt = {}
    flat = []
    for b in range(desc.n_out):
        for p in range(desc.n2):
            for u in range(desc.n_in):
                for q in range(desc.n1):
                    pt = encode(P, diag_slots(b, p, u, q), scale_d, level)
                    diag_pt[(b, p, u, q)] = pt
                    flat.append(to_dev(pt))
    step(f"matvec plan n_in={desc.n_in} n_out={desc.n_out} n1={desc.n1} n2={desc.n2}")
    args = (desc.level, desc.n_in, desc.n_out, desc.n1, desc.n2, desc.unit, desc.real_extract,
            desc.rescale)
    cp = desc.complex_pair
    plan = F.MatvecPlan(S.ctx, *args, diags=flat, complex_pair=cp, lazy_moddown=lazy)
    out_level = level - 1 if desc.rescale else level
    outs_d = [torch.zeros(out_level * 2 * P.n, dtype=torch.int64, device="cuda")
              for _ in range(desc.n_out // 2 if cp else desc.n_out)]
    step("matvec run")
    plan(ins_d, outs_d)
    # the same diagonals through a diagonal bank give the same residues; the
    # bank starts with every bit set and is packed in reverse order, so each
    # diagonal must clear its own bits of the words it shares with others
    fd = F.matvec_desc(*args, cp, lazy)
    bank = torch.full((F.matvec_bank_words(S.ctx, fd),), -1, dtype=torch.int64, device="cuda")
    for t in reversed(range(len(flat))):
        F.matvec_bank_pack(S.ctx, fd, bank, t, flat[t])
    plan_b = F.MatvecPlan(S.ctx, *args, bank=bank, complex_pair=cp, lazy_moddown=lazy)
    outs_b = [torch.zeros_like(o) for o in outs_d]
    step("matvec run (bank)")
    plan_b(ins_d, outs_b)
    for ob, od in zip(outs_b, outs_d):
        assert torch.equal(ob, od)
    outs_o = OW.bsgs_matvec(P, desc, ins_o, lambda b, p, u, q: diag_pt[(b, p, u, q)], S.keys)
    assert keys_needed <= {r for r in range(P.n // 2)}
    return outs_o, outs_d


@pytest.mark.parametrize("lazy", [False, True])
def test_cfg1_diagonal_matvec(lazy):
    """N = 2^12, q0..q2 + one special prime, 64 x 64 U[-1,1] matrix at scale
    2^30 times x replicated to 2048 slots (ciphertext at scale q_2); also
    double-hoisted (63 baby steps left over Q u P, one ModDown)."""
    P = C.params_p12()
    U, x = WL.cfg1_values()
    d = WL.CFG1["dim"]
    n_slots = P.n // 2
    desc = OW.MatvecDesc(3, 1, 1, d, 1, 1, False, True, lazy_moddown=lazy)
    S = Setup(P, WL.CFG1["seed"], rot_steps=list(range(1, d)))
    xs = [np.tile(x, n_slots // d).astype(complex)]
    diag = lambda b, p, u, q: OW.bsgs_diagonal_slots(U.T, n_slots, 1, d, d, b, p, u, q, False)
    outs_o, outs_d = _run(P, S, desc, xs, float(P.q[2]), diag, 2.0 ** 30, "cfg1")
    got = to_host(outs_d[0]).reshape(outs_o[0].shape)
    assert np.array_equal(got, outs_o[0]), first_mismatch(got, outs_o[0])
    dec = C.decrypt(P, S.sk, outs_o[0], 2.0 ** 30)
    err = np.max(np.abs(dec - np.tile(U @ x, n_slots // d)))
    print(f"cfg1 max |decoded - fp64| = {err:.3e} (2^{np.log2(err):.1f})")
    assert err <= 2.0 ** -15


def test_bank_partial_output_groups():
    """19 outputs (b, p) per term: one full group of 16 and a partial group of
    3, an odd last pair of 16-bit fields and a second word of top bits; the
    bank plan, the table plan and the oracle agree on every residue."""
    P = C.params_p12()
    n_slots = P.n // 2
    desc = OW.MatvecDesc(3, 1, 1, 2, 19, 1, False, True)
    S = Setup(P, 31, rot_steps=sorted(OW.required_rotations(desc, n_slots)))
    xs = [synth.uniform_pm1(31, "x", (n_slots,)).astype(complex)]
    diag = lambda b, p, u, q: synth.uniform_pm1(31, "diag", (n_slots,), b, p, u, q).astype(complex)
    outs_o, outs_d = _run(P, S, desc, xs, float(P.q[2]), diag, 2.0 ** 30, "groups")
    got = to_host(outs_d[0]).reshape(outs_o[0].shape)
    assert np.array_equal(got, outs_o[0]), first_mismatch(got, outs_o[0])


@pytest.mark.parametrize("lazy", [False, True])
def test_bank_pack_many_matches_single_packs(lazy):
    """36 diagonals (9 outputs x 4 terms: a partial hi pair and a partly used
    top word) packed one at a time, in two batched calls, and in batched
    calls in reverse order give the same bank word for word; out-of-range
    slots and a short plaintext stride are refused before any launch."""
    import ctypes
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 4, 2)
    ctx = F.Context(P.log_n, P.q, P.p)
    level = 3
    fd = F.matvec_desc(level, 2, 3, 2, 3, 1, False, True, False, lazy)
    mods = P.qs(level) + (list(P.p) if lazy else [])
    n_diag = 36
    pts = torch.stack([to_dev(synth.uniform_residues(41, "bank", mods, P.n, t)).reshape(-1)
                       for t in range(n_diag)])
    words = F.matvec_bank_words(ctx, fd)
    banks = [torch.full((words,), -1, dtype=torch.int64, device="cuda") for _ in range(3)]
    for t in range(n_diag):
        F.matvec_bank_pack(ctx, fd, banks[0], t, pts[t])
    F.matvec_bank_pack_many(ctx, fd, banks[1], 0, pts[:20])
    F.matvec_bank_pack_many(ctx, fd, banks[1], 20, pts[20:])
    for c0 in reversed(range(0, n_diag, 7)):
        F.matvec_bank_pack_many(ctx, fd, banks[2], c0, pts[c0:c0 + 7])
    F.matvec_bank_pack_many(ctx, fd, banks[2], 0, pts[:0])  # empty: nothing
    torch.cuda.synchronize()
    assert torch.equal(banks[1], banks[0])
    assert torch.equal(banks[2], banks[0])
    with pytest.raises(RuntimeError):
        F.matvec_bank_pack_many(ctx, fd, banks[1], 30, pts[:7])
    rc = F._lib.fesc_matvec_bank_pack_many(ctx._h, ctypes.byref(fd), banks[1].data_ptr(), 0, 2,
                                           pts.data_ptr(), len(mods) * P.n - 1,
                                           torch.cuda.current_stream().cuda_stream)
    assert rc == -1
    torch.cuda.synchronize()
    assert torch.equal(banks[1], banks[0])
    ctx.close()


@pytest.mark.parametrize("lazy", [False, True])
def test_paired_bsgs_small(lazy):
    P = C.params_small(12, 50, 5, 2)
    n_slots, seg_len, Cc = P.n // 2, 64, 32
    T, d_in, d_out, n1, n2 = 64, 128, 64, 8, 4
    level = 4
    X = synth.normal(21, "X", (T, d_in))
    Wm = synth.normal(21, "W", (d_in, d_out), 0.02)
    desc = OW.MatvecDesc(level, d_in // Cc // 2, d_out // Cc, n1, n2, seg_len, True, True,
                         lazy_moddown=lazy)
    S = Setup(P, 21, rot_steps=sorted(OW.required_rotations(desc, n_slots)), conj=True)
    xs = [OW.pack_input(X, n_slots, seg_len, Cc, 2 * u)
          + 1j * OW.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1) for u in range(desc.n_in)]
    diag = lambda b, p, u, q: OW.bsgs_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, b, p, u, q,
                                                     True)
    outs_o, outs_d = _run(P, S, desc, xs, 2.0 ** 40, diag, float(P.q[level - 1]), "bsgs")
    Y = X @ Wm
    r, s = OW.segment_indices(n_slots, seg_len, Cc)
    for b in range(desc.n_out):
        got = to_host(outs_d[b]).reshape(outs_o[b].shape)
        assert np.array_equal(got, outs_o[b]), f"block {b}: {first_mismatch(got, outs_o[b])}"
        dec = C.decrypt(P, S.sk, outs_o[b], 2.0 ** 40)
        assert np.max(np.abs(dec.real - Y[r, b * Cc + s])) <= 2.0 ** -15


def test_cfg4_full_size_projection():
    """The 768 x 1536 projection at full size (N = 2^16, 16 limbs at input,
    12 paired input ciphertexts of 1024 tokens, 48 output ciphertexts, BSGS
    n1 = 16, n2 = 2) in the launch configuration the benchmark times: all
    18,432 diagonals in one tiled bank.  Output blocks 0 and 47 (47 lies in
    the second, partial group of 32 batched giant-step key switches) are
    compared residue by residue with the oracle; every output block is
    decrypted and compared with X W in fp64 within 2^-15."""
    import concurrent.futures as cf
    import os

    from paper_2608_17442_amd import fesc as F
    from paper_2608_17442_amd import packing as PK
    cfg = WL.CFG4
    P = C.params_p16()
    level, seg = cfg["level"], cfg["tokens"]
    n_slots = P.n // 2
    Cc = n_slots // seg
    n1, n2 = cfg["n1"], cfg["n2"]
    n_in, n_out = cfg["d_in"] // Cc // 2, cfg["d_out"] // Cc
    desc = OW.MatvecDesc(level, n_in, n_out, n1, n2, seg, True, True)
    S = Setup(P, cfg["seed"], rot_steps=sorted(OW.required_rotations(desc, n_slots)), conj=True)
    X, Wm = WL.cfg4_values()
    ins_o, ins_d = [], []
    for u in range(n_in):
        z = OW.pack_input(X, n_slots, seg, Cc, 2 * u) + 1j * OW.pack_input(X, n_slots, seg, Cc,
                                                                            2 * u + 1)
        co, cd = S.encrypt(z, 2.0 ** 40, level, 3000 + u)
        ins_o.append(co)
        ins_d.append(cd)
    check = (0, n_out - 1)
    scale = float(P.q[level - 1])
    index = [(b, p, u, q) for b in range(n_out) for p in range(n2) for u in range(n_in)
             for q in range(n1)]
    fd = F.matvec_desc(level, n_in, n_out, n1, n2, seg, True, True)
    bank = torch.zeros(F.matvec_bank_words(S.ctx, fd), dtype=torch.int64, device="cuda")
    stage = torch.empty(level * P.n, dtype=torch.int64, device="cuda")
    oracle_pt = {}

    def prepare(t):
        b, p, u, q = index[t]
        if b in check:   # oracle encoding of the diagonals of the compared blocks
            v = OW.bsgs_diagonal_slots(Wm, n_slots, seg, Cc, n1, b, p, u, q, True)
            oracle_pt[index[t]] = C.encode_plain(P, v, scale, level)
            return None
        return F.encode(P.log_n, PK.diagonal_slots(Wm, b, p, u, q, n1, n_slots, seg, Cc, True),
                        scale)

    step(f"cfg4 bank: {len(index)} diagonals")
    with cf.ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
        for c0 in range(0, len(index), 512):
            ids = list(range(c0, min(c0 + 512, len(index))))
            for t, coeffs in zip(ids, ex.map(prepare, ids)):
                if coeffs is None:
                    F.matvec_bank_pack(S.ctx, fd, bank, t, to_dev(oracle_pt[index[t]]))
                else:
                    S.ctx.plain_from_coeffs(torch.from_numpy(coeffs).cuda(), stage, level)
                    F.matvec_bank_pack(S.ctx, fd, bank, t, stage)
    torch.cuda.synchronize()
    plan = F.MatvecPlan(S.ctx, level, n_in, n_out, n1, n2, seg, True, True, bank=bank)
    outs_d = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
              for _ in range(n_out)]
    step("cfg4 matvec run")
    plan(ins_d, outs_d)
    torch.cuda.synchronize()
    del bank
    step("cfg4 oracle blocks")
    outs_o = OW.bsgs_matvec(P, desc, ins_o, lambda b, p, u, q: oracle_pt[(b, p, u, q)], S.keys,
                            blocks=check)
    for b, want in zip(check, outs_o):
        got = to_host(outs_d[b]).reshape(want.shape)
        assert np.array_equal(got, want), f"block {b}: {first_mismatch(got, want)}"
    Y = X @ Wm
    r, s = OW.segment_indices(n_slots, seg, Cc)
    worst = 0.0
    for b in range(n_out):
        ct = to_host(outs_d[b]).reshape(level - 1, 2, P.n)
        dec = C.decrypt(P, S.sk, ct, 2.0 ** 40)
        worst = max(worst, float(np.max(np.abs(dec.real - Y[r, b * Cc + s]))))
    print(f"cfg4 max |decoded - fp64| over 48 blocks = {worst:.3e} (2^{np.log2(worst):.1f})")
    assert worst <= 2.0 ** -15


def _slot_fn(mode, Wm, n_slots, seg, Cc, n1):
    if mode == "pair":
        return lambda b, p, u, q: OW.bsgs_pair_diagonal_slots(Wm, n_slots, seg, Cc, n1, b, p, u, q)
    return lambda b, p, u, q: OW.bsgs_diagonal_slots(Wm, n_slots, seg, Cc, n1, b, p, u, q,
                                                     mode == "paired")


@pytest.mark.parametrize("mode,segs", [("plain", 32), ("paired", 32), ("pair", 32),
                                       ("plain", 16)])
def test_bsgs_diagonal_slots_on_device(mode, segs):
    """fesc_bsgs_diagonal_slots against the oracle's slot vectors, every
    diagonal of a small projection, bit for bit (segs = 16 < (N/2)/unit: a
    repeated shorter vector)."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_small(12, 50, 3, 1)
    ctx = F.Context(P.log_n, P.q, P.p)
    n_slots, seg = P.n // 2, 64
    n1, n2 = 8, 4
    gin = 2 if mode != "plain" else 1
    n_in, n_out = 2, 4
    d_in, d_out = gin * n_in * segs - 5, n_out * segs - 3      # ragged: W shorter than blocks
    Wm = synth.normal(23, "W", (d_in, d_out), 0.1)
    desc = F.matvec_desc(2, n_in, n_out, n1, n2, seg, mode == "paired", True, mode == "pair")
    total = n_out * n2 * n_in * n1
    z = torch.zeros((total, n_slots), dtype=torch.complex128, device="cuda")
    Wd = torch.from_numpy(Wm).cuda()
    step(f"bsgs slots {mode} segs={segs}")
    F.bsgs_diagonal_slots(ctx, desc, Wd, segs, 0, 7, z)
    F.bsgs_diagonal_slots(ctx, desc, Wd, segs, 7, total - 7, z[7:])
    got = z.cpu().numpy()
    fn = _slot_fn(mode, Wm, n_slots, seg, segs, n1)
    t = 0
    for b in range(n_out):
        for p in range(n2):
            for u in range(n_in):
                for q in range(n1):
                    want = fn(b, p, u, q)
                    assert np.array_equal(got[t], want), (mode, t, b, p, u, q)
                    t += 1
    with pytest.raises(F.FescError):
        F.bsgs_diagonal_slots(ctx, desc, Wd, segs, total - 1, 2, z)
    with pytest.raises(F.FescError):
        F.bsgs_diagonal_slots(ctx, desc, Wd, 48, 0, 1, z)          # 48 does not divide 32


@pytest.mark.parametrize("lazy", [False, True])
def test_complex_paired_outputs_small(lazy):
    """Complex-paired outputs on a small ring (n_out = 4 diagonal sets -> 2
    output ciphertexts, n2 = 4 giant steps), table and bank plans, bit-exact
    against the oracle, also double-hoisted; the real and imaginary parts
    decode to blocks 2P and 2P + 1 of X W within 2^-15."""
    P = C.params_small(12, 50, 5, 2)
    n_slots, seg_len, Cc = P.n // 2, 64, 32
    T, d_in, d_out, n1, n2 = 64, 128, 128, 8, 4
    level = 4
    X = synth.normal(24, "X", (T, d_in))
    Wm = synth.normal(24, "W", (d_in, d_out), 0.02)
    desc = OW.MatvecDesc(level, d_in // Cc // 2, d_out // Cc, n1, n2, seg_len, False, True,
                         complex_pair=True, lazy_moddown=lazy)
    S = Setup(P, 24, rot_steps=sorted(OW.required_rotations(desc, n_slots)), conj=True)
    xs = [OW.pack_input(X, n_slots, seg_len, Cc, 2 * u)
          + 1j * OW.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1) for u in range(desc.n_in)]
    diag = _slot_fn("pair", Wm, n_slots, seg_len, Cc, n1)
    outs_o, outs_d = _run(P, S, desc, xs, 2.0 ** 40, diag, float(P.q[level - 1]), "pair")
    assert len(outs_o) == len(outs_d) == desc.n_out // 2
    Y = X @ Wm
    r, s = OW.segment_indices(n_slots, seg_len, Cc)
    for pair in range(desc.n_out // 2):
        got = to_host(outs_d[pair]).reshape(outs_o[pair].shape)
        assert np.array_equal(got, outs_o[pair]), f"pair {pair}: {first_mismatch(got, outs_o[pair])}"
        dec = C.decrypt(P, S.sk, outs_o[pair], 2.0 ** 40)
        assert np.max(np.abs(dec.real - Y[r, 2 * pair * Cc + s])) <= 2.0 ** -15
        assert np.max(np.abs(dec.imag - Y[r, (2 * pair + 1) * Cc + s])) <= 2.0 ** -15


def test_cfg4_full_size_complex_paired_outputs():
    """The 768 x 1536 projection with complex-paired outputs, as the benchmark
    runs it: 18,432 diagonals (48 sets = 24 output pairs) whose slot vectors
    come from the device generator and are encoded on the device, one tiled
    bank, 24 output ciphertexts (48 giant-step and 24 conjugation key
    switches).  Pairs 0 and 23 (output blocks 0, 1, 46, 47) are compared
    residue by residue with the oracle (their diagonals encoded by the
    oracle); all 24 outputs decode to X W within 2^-15 (real part block 2P,
    imaginary part block 2P + 1)."""
    from paper_2608_17442_amd import fesc as F
    cfg = WL.CFG4
    P = C.params_p16()
    level, seg = cfg["level"], cfg["tokens"]
    n_slots = P.n // 2
    Cc = n_slots // seg
    n1, n2 = cfg["n1"], cfg["n2"]
    n_in, n_out = cfg["d_in"] // Cc // 2, cfg["d_out"] // Cc
    desc = OW.MatvecDesc(level, n_in, n_out, n1, n2, seg, False, True, complex_pair=True)
    S = Setup(P, cfg["seed"], rot_steps=sorted(OW.required_rotations(desc, n_slots)), conj=True)
    X, Wm = WL.cfg4_values()
    ins_o, ins_d = [], []
    for u in range(n_in):
        z = OW.pack_input(X, n_slots, seg, Cc, 2 * u) + 1j * OW.pack_input(X, n_slots, seg, Cc,
                                                                            2 * u + 1)
        co, cd = S.encrypt(z, 2.0 ** 40, level, 3000 + u)
        ins_o.append(co)
        ins_d.append(cd)
    n_pairs = n_out // 2
    check = (0, n_pairs - 1)
    scale = float(P.q[level - 1])
    index = [(b, p, u, q) for b in range(n_out) for p in range(n2) for u in range(n_in)
             for q in range(n1)]
    fd = F.matvec_desc(level, n_in, n_out, n1, n2, seg, False, True, True)
    bank = torch.zeros(F.matvec_bank_words(S.ctx, fd), dtype=torch.int64, device="cuda")
    Wd = torch.from_numpy(Wm).cuda()
    chunk = 128
    zs = torch.empty((chunk, n_slots), dtype=torch.complex128, device="cuda")
    pts = torch.empty((chunk, level * P.n), dtype=torch.int64, device="cuda")
    step(f"cfg4 paired-output bank: {len(index)} diagonals, slots and encoding on the device")
    for c0 in range(0, len(index), chunk):
        m = min(chunk, len(index) - c0)
        F.bsgs_diagonal_slots(S.ctx, fd, Wd, Cc, c0, m, zs)
        S.ctx.encode_plain(zs[:m], scale, pts[:m], level)
        for j in range(m):
            F.matvec_bank_pack(S.ctx, fd, bank, c0 + j, pts[j])
    # the compared pairs' diagonals from the oracle's encoder (the device
    # encoder may round a near-tie coefficient differently)
    oracle_pt = {}
    step("cfg4 oracle diagonals of the compared pairs")
    for t, (b, p, u, q) in enumerate(index):
        if b // 2 in check:
            v = OW.bsgs_pair_diagonal_slots(Wm, n_slots, seg, Cc, n1, b, p, u, q)
            oracle_pt[(b, p, u, q)] = C.encode_plain(P, v, scale, level)
            F.matvec_bank_pack(S.ctx, fd, bank, t, to_dev(oracle_pt[(b, p, u, q)]))
    torch.cuda.synchronize()
    plan = F.MatvecPlan(S.ctx, level, n_in, n_out, n1, n2, seg, False, True, bank=bank,
                        complex_pair=True)
    outs_d = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
              for _ in range(n_pairs)]
    step("cfg4 paired-output matvec run")
    plan(ins_d, outs_d)
    torch.cuda.synchronize()
    del bank
    step("cfg4 oracle pairs")
    outs_o = OW.bsgs_matvec(P, desc, ins_o, lambda b, p, u, q: oracle_pt[(b, p, u, q)], S.keys,
                            blocks=check)
    for pair, want in zip(check, outs_o):
        got = to_host(outs_d[pair]).reshape(want.shape)
        assert np.array_equal(got, want), f"pair {pair}: {first_mismatch(got, want)}"
    Y = X @ Wm
    r, s = OW.segment_indices(n_slots, seg, Cc)
    worst = 0.0
    for pair in range(n_pairs):
        ct = to_host(outs_d[pair]).reshape(level - 1, 2, P.n)
        dec = C.decrypt(P, S.sk, ct, 2.0 ** 40)
        worst = max(worst, float(np.max(np.abs(dec.real - Y[r, 2 * pair * Cc + s]))),
                    float(np.max(np.abs(dec.imag - Y[r, (2 * pair + 1) * Cc + s]))))
    print(f"cfg4 paired outputs: max |decoded - fp64| over 48 blocks = {worst:.3e}")
    assert worst <= 2.0 ** -15


@pytest.mark.parametrize("log_n,L,alpha,level", [(12, 5, 2, 4), (16, 24, 8, 16)])
def test_encode_plain_ext(log_n, L, alpha, level):
    """Device encoding over the extended basis: the level rows equal
    fesc_encode_plain's residue for residue, and every special-prime row is
    the transform of the same integer coefficients modulo that prime."""
    from paper_2608_17442_amd import fesc as F
    P = C.params_p16(L) if log_n == 16 else C.params_small(log_n, 50, L, alpha)
    ctx = F.Context(log_n, P.q, P.p)
    n, count = P.n, 3
    z = np.stack([synth.uniform_pm1(80 + b, "ext-re", n // 2)
                  + 1j * synth.uniform_pm1(80 + b, "ext-im", n // 2) for b in range(count)])
    zd = torch.from_numpy(z).cuda()
    pq = torch.zeros(count * level * n, dtype=torch.int64, device="cuda")
    pe = torch.zeros(count * (level + P.alpha) * n, dtype=torch.int64, device="cuda")
    step(f"encode_plain(_ext) N=2^{log_n} level={level}")
    ctx.encode_plain(zd, 2.0 ** 40, pq, level)
    ctx.encode_plain_ext(zd, 2.0 ** 40, pe, level)
    gq = to_host(pq).reshape(count, level, n)
    ge = to_host(pe).reshape(count, level + P.alpha, n)
    qs = P.qs(level)
    for b in range(count):
        assert np.array_equal(ge[b, :level], gq[b])
        m = [int(v) - qs[0] if int(v) > qs[0] // 2 else int(v)
             for v in C.intt(P, gq[b, :1], qs[:1])[0]]
        want = C.ntt(P, C.lift(np.array(m, dtype=np.int64), P.p), P.p)
        assert np.array_equal(ge[b, level:], want)
