"""GPU parity of the homomorphic slot maps that realise the HEScan broadcasts
br^(kappa) (Appendix "HEScan Kernel Packing and Correctness") against the
oracle:

* bit-exact on small rings (N = 2^12, 2^13): every factor kind, B/C with the
  chunk inside one group and over two groups, a ragged baby-step split (6
  terms over 4 x 2), an offset of zero, the decay placed at two positions per
  head (giant steps over heads with their own stride), and the output written
  over the input;
* the device's mask slot vectors equal the oracle's exactly;
* the batched map (several tokens under one plan, each with its own first
  rotation) bit-exact against the oracle's map of each token;
* at N = 2^16, 23 limbs and the Mamba-2 base shape (24 heads of 64, d_s = 128,
  128 channels per chunk), with masks generated and encoded on the device,
  every output decrypts to the plain broadcast within 2^-15 (a property that
  holds at any size; the oracle's key generation at this size would take
  minutes)."""
import numpy as np
import pytest
import torch

import synth
from oracle import broadcast as BR
from oracle import ckks as C
from paper_2608_17442_amd import fesc as F
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_dev, to_host
from tests.test_gpu_ckks import Setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _oracle_map(d):
    """The library's descriptor as the oracle's SlotMap."""
    return BR.SlotMap(d.level, d.offset, d.stride, d.terms, d.n1, d.giant_stride, d.dst0,
                      d.dst_stride, d.dst_giant, d.width, d.rep_count, d.rep_stride)


SHAPE_A = BR.Dims(H=8, P=8, G=2, d_s=16, c_state=16, n_slots=2048)   # chunk inside a group
SHAPE_B = BR.Dims(H=8, P=2, G=4, d_s=8, c_state=8, n_slots=2048)     # chunk over two groups
SHAPE_C = BR.Dims(H=3, P=4, G=1, d_s=8, c_state=6, n_slots=2048)     # 6 terms: ragged split
SHAPE_D = BR.Dims(H=4, P=4, G=2, d_s=8, c_state=8, n_slots=4096)
SHAPE_E = BR.Dims(H=2, P=64, G=1, d_s=16, c_state=128, n_slots=2048)  # decay: 2 positions/head
SHAPE_F = BR.Dims(H=4, P=32, G=2, d_s=32, c_state=64, n_slots=4096)

CASES = [(12, 6, 2, SHAPE_A, kind, 3, 2, 6) for kind in BR.KINDS] + [
    (12, 6, 2, SHAPE_B, "B", 5, 1, 5),
    (12, 6, 2, SHAPE_B, "C", 0, 0, 3),       # offset 0: no first rotation
    (12, 6, 2, SHAPE_C, "x", 7, 1, 4),
    (13, 5, 3, SHAPE_D, "a", 9, 1, 5),
    (13, 5, 3, SHAPE_D, "x", 2, 0, 2),       # down to level 1
    (12, 6, 2, SHAPE_E, "a", 11, 0, 6),      # 2 x 2 terms, 512 copies
    (13, 5, 3, SHAPE_F, "a", 6, 1, 4),
    (13, 5, 3, SHAPE_F, "B", 6, 1, 4),
]


@pytest.mark.parametrize("log_n,L,alpha,D,kind,k,kappa,level", CASES,
                         ids=[f"n{c[0]}-{c[4]}-k{c[5]}-c{c[6]}-H{c[3].H}G{c[3].G}-l{c[7]}"
                              for c in CASES])
def test_broadcast_small(log_n, L, alpha, D, kind, k, kappa, level):
    P = C.params_small(log_n, 50, L, alpha)
    ns = P.n // 2
    assert D.n_slots == ns
    d = F.br_desc(P.log_n, D.H, D.P, D.G, D.d_s, D.c_state, kind, k, kappa, level)
    M = _oracle_map(d)
    S = Setup(P, 71, rot_steps=sorted(BR.slot_map_rotations(M, ns)))
    v = synth.normal(71, "brv" + kind, ns, 1.0, k) + 1j * synth.normal(71, "brw" + kind, ns, 1.0, k)
    ct_o, ct_d = S.encrypt(v, 2.0 ** 40, level, 7000 + k)
    ql = float(P.q[level - 1])
    masks_o = {(p, q): C.encode_plain(P, BR.mask_slots(M, ns, p, q), ql, level)
               for p in range(M.n2) for q in range(M.n1)}
    masks_d = [to_dev(masks_o[divmod(t, M.n1)]) for t in range(M.n)]
    plan = F.SlotMapPlan(S.ctx, d, masks_d)
    out = torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
    step(f"slot map {kind} log_n={log_n} k={k} kappa={kappa} level={level} terms={d.terms}")
    plan(ct_d, out)
    want = BR.slot_map_ct(P, ct_o, M, lambda p, q: masks_o[(p, q)], S.keys)
    got = to_host(out).reshape(want.shape)
    assert np.array_equal(got, want), f"{kind}: {first_mismatch(got, want)}"
    dec = C.decrypt(P, S.sk, want, 2.0 ** 40)
    np.testing.assert_allclose(dec, BR.br(D, kind, v, k, kappa), atol=2.0 ** -15)
    # output over the input
    x = ct_d.clone()
    step(f"slot map {kind} in place")
    plan(x, x)
    got = to_host(x)[: want.size].reshape(want.shape)
    assert np.array_equal(got, want), f"{kind} in place: {first_mismatch(got, want)}"
    # the device's mask slot vectors
    cnt = M.n1 * M.n2
    z = torch.empty((cnt, ns), dtype=torch.complex128, device="cuda")
    step(f"mask slots {kind} count={cnt}")
    F.slot_map_mask_slots(S.ctx, d, 0, cnt, z)
    zh = z.cpu().numpy()
    for t in range(cnt):
        assert np.array_equal(zh[t], BR.mask_slots(M, ns, *divmod(t, M.n1))), f"mask {t}"


BATCH_CASES = [(12, 6, 2, SHAPE_A, kind, 1, 6) for kind in ("x", "a", "B")] + [
    (13, 5, 3, SHAPE_D, "a", 1, 5),
    (12, 6, 2, SHAPE_B, "C", 0, 3),
]


@pytest.mark.parametrize("log_n,L,alpha,D,kind,kappa,level", BATCH_CASES,
                         ids=[f"n{c[0]}-{c[4]}-c{c[5]}-H{c[3].H}G{c[3].G}-l{c[6]}"
                              for c in BATCH_CASES])
def test_broadcast_batch_small(log_n, L, alpha, D, kind, kappa, level):
    """fesc_slot_map_batch over tokens 0, 1, 2 and 4 (token 0: an offset that
    may be zero) under the plan of token 1, each item with its own offset:
    every output bit-exact against the oracle's map of its own token, also
    written over the inputs."""
    P = C.params_small(log_n, 50, L, alpha)
    ns = P.n // 2
    toks = [0, 1, 2, 4]
    ds = {k: F.br_desc(P.log_n, D.H, D.P, D.G, D.d_s, D.c_state, kind, k, kappa, level)
          for k in toks}
    Ms = {k: _oracle_map(d) for k, d in ds.items()}
    rots = set()
    for M in Ms.values():
        rots |= BR.slot_map_rotations(M, ns)
    S = Setup(P, 74, rot_steps=sorted(rots))
    ql = float(P.q[level - 1])
    M1 = Ms[1]
    masks_o = {(p, q): C.encode_plain(P, BR.mask_slots(M1, ns, p, q), ql, level)
               for p in range(M1.n2) for q in range(M1.n1)}
    masks_d = [to_dev(masks_o[divmod(t, M1.n1)]) for t in range(M1.n)]
    plan = F.SlotMapPlan(S.ctx, ds[1], masks_d)
    cts_o, cts_d = [], []
    for k in toks:
        v = synth.normal(74, "bbv" + kind, ns, 1.0, k) + 1j * synth.normal(74, "bbw" + kind, ns,
                                                                          1.0, k)
        o, d = S.encrypt(v, 2.0 ** 40, level, 7400 + k)
        cts_o.append(o)
        cts_d.append(d)
    outs = [torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda") for _ in toks]
    step(f"slot map batch {kind} log_n={log_n} kappa={kappa} tokens={toks}")
    plan.batch(cts_d, [ds[k].offset for k in toks], outs)
    wants = [BR.slot_map_ct(P, o, Ms[k], lambda p, q: masks_o[(p, q)], S.keys)
             for k, o in zip(toks, cts_o)]
    for k, out, want in zip(toks, outs, wants):
        got = to_host(out).reshape(want.shape)
        assert np.array_equal(got, want), f"{kind} token {k}: {first_mismatch(got, want)}"
    step(f"slot map batch {kind} in place")
    xs = [c.clone() for c in cts_d]
    plan.batch(xs, [ds[k].offset for k in toks], xs)
    for k, x, want in zip(toks, xs, wants):
        got = to_host(x)[: want.size].reshape(want.shape)
        assert np.array_equal(got, want), f"{kind} token {k} in place: {first_mismatch(got, want)}"


def test_slot_map_errors():
    P = C.params_small(12, 50, 6, 2)
    S = Setup(P, 72)
    D = SHAPE_A
    d = F.br_desc(P.log_n, D.H, D.P, D.G, D.d_s, D.c_state, "x", 1, 1, 5)
    pts = [torch.zeros(5 * P.n, dtype=torch.int64, device="cuda") for _ in range(d.terms)]
    with pytest.raises(F.FescError) as ex:          # no rotation keys loaded
        F.SlotMapPlan(S.ctx, d, pts)
    assert ex.value.code == -3
    bad = F.SlotMapDesc(5, 0, 1, 2, 4, 2, 0, 1, 2, 2, 1, 1)   # width 2 at stride 1: overlap
    with pytest.raises(F.FescError, match="overlap"):
        F.SlotMapPlan(S.ctx, bad, pts[:4])
    bad = F.SlotMapDesc(5, 0, 1, 2, 4, 2, 0, 4, 4, 1, 1, 1)   # row 1 starts inside row 0
    with pytest.raises(F.FescError, match="overlap"):
        F.SlotMapPlan(S.ctx, bad, pts[:4])
    bad = F.SlotMapDesc(5, 0, 1, 1, 1, 1, 0, 0, 0, 1, 1, 3)   # replication count 3
    with pytest.raises(F.FescError, match="power of two"):
        F.SlotMapPlan(S.ctx, bad, pts[:1])
    bad = F.SlotMapDesc(1, 0, 1, 1, 1, 1, 0, 0, 0, 1, 1, 1)   # level 1: no rescale
    with pytest.raises(F.FescError) as ex:
        F.SlotMapPlan(S.ctx, bad, pts[:1])
    assert ex.value.code == -2
    bad = F.SlotMapDesc(5, 0, 1, 1, 2, 1, 2040, 0, 8, 1, 1, 1)  # 2nd run past the slots
    with pytest.raises(F.FescError, match="leave"):
        F.SlotMapPlan(S.ctx, bad, pts[:2])
    z = torch.empty((2, P.n // 2), dtype=torch.complex128, device="cuda")
    with pytest.raises(F.FescError, match="mask range"):
        F.slot_map_mask_slots(S.ctx, d, d.n1 * d.n2 - 1, 2, z)
    # a batch whose offset has no key: refused before any launch
    rots = BR.slot_map_rotations(_oracle_map(d), P.n // 2)
    S2 = Setup(P, 72, rot_steps=sorted(rots))
    plan = F.SlotMapPlan(S2.ctx, d, pts[:d.terms])
    ct = torch.zeros(5 * 2 * P.n, dtype=torch.int64, device="cuda")
    out = torch.full((4 * 2 * P.n,), 7, dtype=torch.int64, device="cuda")
    keyless = next(o for o in range(1, P.n // 2) if o not in rots)
    with pytest.raises(F.FescError) as ex:
        plan.batch([ct, ct], [d.offset, keyless], [out, out])
    assert ex.value.code == -3
    assert bool((out == 7).all())
    with pytest.raises(F.FescError):
        plan.batch([], [], [])


def test_broadcast_full_size():
    """N = 2^16, 24 primes, dnum 3, 8 special primes; the Mamba-2 base packing
    (E = 1536, d_s = 128, 12 chunks of 128 channels, G = 1); token 3, chunk 7,
    input level 23; seed-expanded keys; masks from fesc_slot_map_mask_slots
    encoded by fesc_encode_plain."""
    P = C.params_p16(24)
    D = BR.Dims(H=24, P=64, G=1, d_s=128, c_state=128, n_slots=P.n // 2)
    ns, level, k, kappa, seed = P.n // 2, 23, 3, 7, 73
    descs = {kind: F.br_desc(P.log_n, D.H, D.P, D.G, D.d_s, D.c_state, kind, k, kappa, level)
             for kind in BR.KINDS}
    steps = set()
    for d in descs.values():
        steps |= BR.slot_map_rotations(_oracle_map(d), ns)
    ctx = F.Context(P.log_n, P.q, P.p)
    s = synth.secret(seed, P.n)
    sk = C.secret_key(P, s)
    s_dev = torch.from_numpy(s).cuda()
    for r in sorted(steps):
        g = P.galois_elt(r)
        w, e = synth.switch_key_seed_draws(seed, P.ext(P.L), P.n, P.dnum, g)
        step(f"keygen_seeded g={g} (rotation {r})")
        ctx.keygen_seeded(g, s_dev, w, torch.from_numpy(e).cuda())
    v = synth.normal(seed, "full-v", ns) + 1j * synth.normal(seed, "full-w", ns)
    m = C.enc.encode(v, 2.0 ** 40, P.n)
    a, e = synth.encrypt_draws(seed, P.qs(level), P.n, "full", 0)
    ct = torch.zeros(level * 2 * P.n, dtype=torch.int64, device="cuda")
    step("encrypt full size")
    ctx.encrypt_sk(s_dev, torch.from_numpy(m).cuda(), to_dev(a), torch.from_numpy(e).cuda(), ct,
                   level)
    ql = float(P.q[level - 1])
    errs = {}
    for kind, d in descs.items():
        cnt = d.n1 * d.n2
        z = torch.empty((cnt, ns), dtype=torch.complex128, device="cuda")
        pts = torch.empty(cnt * level * P.n, dtype=torch.int64, device="cuda")
        step(f"masks {kind}: {cnt} slot vectors, device encoding")
        F.slot_map_mask_slots(ctx, d, 0, cnt, z)
        ctx.encode_plain(z, ql, pts, level)
        masks = [pts[t * level * P.n:(t + 1) * level * P.n] for t in range(d.terms)]
        plan = F.SlotMapPlan(ctx, d, masks)
        out = torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
        step(f"slot map {kind} full size: terms {d.terms}, n1 {d.n1}, x{d.rep_count}")
        plan(ct, out)
        dec = C.decrypt(P, sk, to_host(out).reshape(level - 1, 2, P.n), 2.0 ** 40)
        errs[kind] = float(np.abs(dec - BR.br(D, kind, v, k, kappa)).max())
        plan.close()
    step(f"max errors {errs}")
    assert max(errs.values()) < 2.0 ** -15, errs
