"""Pins of the oracle's broadcast maps (Appendix "HEScan Kernel Packing and
Correctness", paragraph "Exact State and Slot Maps") and of their homomorphic
realisation:

* br^(kappa) against the state tensor of the grouped Mamba-2 recurrence built
  by array reshapes (no slot formula), for the paper's toy packing (Figure
  "Factorized HEScan dataflow": H = 2, P = 4, G = 1, d_s = 2, K_s = 2), grouped
  shapes and the Mamba-2 base shape;
* the recurrence and contraction run on broadcast slot vectors chunk by chunk
  equal Eqs. "fesc_recurrence" and "fesc_contract" evaluated on tensors (the
  chunks partition the channels);
* product preservation br(a * a') = br(a) * br(a');
* the slot-map decomposition reproduces br exactly, its masked baby-step /
  giant-step sum equals the unsplit diagonal sum, and the encrypted
  realisation decrypts to br within 2^-15 on a small ring."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import broadcast as BR
from oracle import ckks as C

TOY = BR.Dims(H=2, P=4, G=1, d_s=2, c_state=4, n_slots=64)
SHAPES = [
    TOY,
    BR.Dims(H=4, P=2, G=2, d_s=4, c_state=4, n_slots=128),    # chunk = one group
    BR.Dims(H=8, P=2, G=4, d_s=2, c_state=8, n_slots=128),    # chunk = two groups
    BR.Dims(H=8, P=2, G=2, d_s=4, c_state=4, n_slots=256),    # chunk inside a group
    BR.Dims(H=24, P=64, G=1, d_s=128, c_state=128, n_slots=32768),  # Mamba-2 base
]


def _factors(D, L, tag):
    x = synth.normal(7, tag + "x", (L, D.H, D.P))
    a = 0.5 + 0.5 * synth.uniform_pm1(7, tag + "a", (L, D.H)) ** 2
    B = synth.normal(7, tag + "B", (L, D.G, D.d_s))
    Cf = synth.normal(7, tag + "C", (L, D.G, D.d_s))
    return x, a, B, Cf


def _groups(D):
    return np.repeat(np.arange(D.G), D.H // D.G)     # head -> group, contiguous


def _chunk_of(D, T, kappa):
    """Chunk kappa of a state-shaped tensor T[h, p, i]: channels e = h P + p
    in order, d_s entries each, padded with zeros to the slot count."""
    flat = T.reshape(D.E, D.d_s)[kappa * D.c_state:(kappa + 1) * D.c_state].reshape(-1)
    out = np.zeros(D.n_slots, np.complex128)
    out[:flat.size] = flat
    return out


@pytest.mark.parametrize("D", SHAPES, ids=lambda D: f"H{D.H}P{D.P}G{D.G}d{D.d_s}c{D.c_state}")
def test_broadcast_is_the_state_tensor(D):
    L = min(3, D.n_slots // max(D.E, D.H, D.G * D.d_s))
    x, a, B, Cf = _factors(D, L, "st")
    va, vx, vb, vc = BR.compact_a(D, a), BR.compact_x(D, x), BR.compact_bc(D, B), \
        BR.compact_bc(D, Cf)
    g = _groups(D)
    kappas = range(D.K_s) if D.K_s <= 4 else [0, 5, D.K_s - 1]
    for k in range(L):
        state_a = np.broadcast_to(a[k][:, None, None], (D.H, D.P, D.d_s))
        state_b = np.broadcast_to(B[k][g][:, None, :], (D.H, D.P, D.d_s))
        state_c = np.broadcast_to(Cf[k][g][:, None, :], (D.H, D.P, D.d_s))
        update = x[k][:, :, None] * B[k][g][:, None, :]      # x_k (x)_g B_k
        for kappa in kappas:
            assert np.array_equal(BR.br(D, "a", va, k, kappa), _chunk_of(D, state_a, kappa))
            assert np.array_equal(BR.br(D, "B", vb, k, kappa), _chunk_of(D, state_b, kappa))
            assert np.array_equal(BR.br(D, "C", vc, k, kappa), _chunk_of(D, state_c, kappa))
            s = BR.br(D, "x", vx, k, kappa) * BR.br(D, "B", vb, k, kappa)
            assert np.array_equal(s, _chunk_of(D, update, kappa))


def test_toy_packing_slots():
    """The toy packing: chunk 1 holds head 1 (channels 4..7), channel e at
    slots 2(e - 4), 2(e - 4) + 1; token 2's x_2[1, 3] lands at slots 6, 7."""
    D = TOY
    assert D.E == 8 and D.K_s == 2
    assert list(BR.chunk_channels(D, 1)) == [4, 5, 6, 7]
    x = np.arange(3 * 8, dtype=float).reshape(3, 2, 4)
    v = BR.br(D, "x", BR.compact_x(D, x), 2, 1)
    assert v[6] == v[7] == x[2, 1, 3] == 23
    assert np.count_nonzero(v[8:]) == 0


@pytest.mark.parametrize("D", SHAPES[:4], ids=lambda D: f"H{D.H}P{D.P}G{D.G}")
def test_recurrence_and_contraction_on_chunks(D):
    """h_k = br(a_k) h_{k-1} + br(x_k) br(B_k) per chunk, m_k = sum over
    chunks of Sigma(h_k br(C_k)): equal to the tensor recurrence and
    contraction of Eqs. "fesc_recurrence" and "fesc_contract"."""
    L = D.n_slots // max(D.E, D.H, D.G * D.d_s)
    x, a, B, Cf = _factors(D, L, "rec")
    va, vx, vb, vc = BR.compact_a(D, a), BR.compact_x(D, x), BR.compact_bc(D, B), \
        BR.compact_bc(D, Cf)
    g = _groups(D)
    h_t = np.zeros((D.H, D.P, D.d_s))
    h_c = [np.zeros(D.n_slots, np.complex128) for _ in range(D.K_s)]
    for k in range(L):
        h_t = a[k][:, None, None] * h_t + x[k][:, :, None] * B[k][g][:, None, :]
        m_t = np.einsum("hpi,hi->hp", h_t, Cf[k][g]).reshape(-1)
        m_c = np.zeros(D.E, np.complex128)
        for kappa in range(D.K_s):
            h_c[kappa] = BR.br(D, "a", va, k, kappa) * h_c[kappa] + \
                BR.br(D, "x", vx, k, kappa) * BR.br(D, "B", vb, k, kappa)
            part = BR.sigma(D, h_c[kappa] * BR.br(D, "C", vc, k, kappa), kappa)
            ch = BR.chunk_channels(D, kappa)
            assert not np.any(m_c[ch.start:ch.stop])          # chunks are disjoint
            m_c[ch.start:ch.stop] = part
        np.testing.assert_allclose(m_c.real, m_t, rtol=1e-12, atol=1e-12)


def test_product_preservation():
    D = SHAPES[2]
    _, a, _, _ = _factors(D, 4, "pp")
    _, a2, _, _ = _factors(D, 4, "pq")
    va, va2 = BR.compact_a(D, a), BR.compact_a(D, a2)
    for k in range(4):
        for kappa in range(D.K_s):
            assert np.array_equal(BR.br(D, "a", va * va2, k, kappa),
                                  BR.br(D, "a", va, k, kappa) * BR.br(D, "a", va2, k, kappa))


@pytest.mark.parametrize("D", SHAPES, ids=lambda D: f"H{D.H}P{D.P}G{D.G}d{D.d_s}c{D.c_state}")
def test_slot_map_reproduces_br(D):
    rng = np.random.default_rng(11)
    v = rng.standard_normal(D.n_slots) + 1j * rng.standard_normal(D.n_slots)
    L = D.n_slots // max(D.E, D.H, D.G * D.d_s)
    for kind in BR.KINDS:
        for k in sorted({0, L - 1}):
            for kappa in sorted({0, D.K_s - 1}):
                M = BR.br_slot_map(D, kind, k, kappa, 3)
                assert np.array_equal(BR.slot_map_plain(M, v), BR.br(D, kind, v, k, kappa)), \
                    (kind, k, kappa)


def _rot(v, r):
    return np.roll(v, -r)                       # rho(v; r)[j] = v[j + r]


@pytest.mark.parametrize("D", SHAPES[1:], ids=lambda D: f"H{D.H}P{D.P}G{D.G}")
def test_masked_bsgs_is_the_diagonal_sum(D):
    """sum_{p,q} rho(M'_{p,q} * rho(v; q d); p g) = sum_t M_t * rho(v; q d + p g)
    with the pre-rotated masks, and equals the first two steps of the map."""
    rng = np.random.default_rng(12)
    v = rng.standard_normal(D.n_slots)
    for kind in BR.KINDS:
        M = BR.br_slot_map(D, kind, 1, D.K_s - 1, 3)
        v0 = _rot(v, M.r0)
        got = np.zeros(D.n_slots, np.complex128)
        for p in range(M.n2):
            acc = sum(BR.mask_slots(M, D.n_slots, p, q) * _rot(v0, q * M.d) for q in range(M.n1))
            got += _rot(acc, p * M.g)
        y = BR.slot_map_plain(dataclasses.replace(M, R=1), v)
        np.testing.assert_allclose(got, y, atol=1e-12)


def test_slot_map_rejects_uncovered_shapes():
    with pytest.raises(ValueError, match="a"):   # 6 channels per chunk: not whole heads of 4
        BR.br_slot_map(BR.Dims(3, 4, 1, 2, 6, 64), "a", 0, 0, 3)
    with pytest.raises(ValueError, match="B/C"):  # 12-channel groups, 16-channel chunks
        BR.br_slot_map(BR.Dims(24, 2, 4, 2, 16, 2048), "B", 0, 1, 3)
    with pytest.raises(ValueError):        # d_s = 3 cannot be replicated by doubling
        BR.br_slot_map(BR.Dims(2, 4, 1, 3, 4, 64), "x", 0, 0, 3)
    with pytest.raises(ValueError):        # token 8 of x does not fit 64 slots
        BR.br_slot_map(TOY, "x", 8, 0, 3)


@pytest.mark.parametrize("kind", BR.KINDS)
def test_encrypted_broadcast_decrypts_to_br(kind):
    """N = 2^10 (512 slots), H = 4, P = 4, G = 2, d_s = 8, 8 channels per
    chunk: br^(1) of token 2's factor, encrypted at level 4."""
    P = C.params_small(10, 50, 4, 2)
    D = BR.Dims(H=4, P=4, G=2, d_s=8, c_state=8, n_slots=P.n // 2)
    sk = C.secret_key(P, synth.secret(13, P.n))
    level, k, kappa = 4, 2, 1
    M = BR.br_slot_map(D, kind, k, kappa, level)
    keys = {P.galois_elt(r): C.keygen_from_seed(P, sk, 13, P.galois_elt(r))
            for r in BR.slot_map_rotations(M, D.n_slots)}
    v = synth.normal(13, "br" + kind, D.n_slots) + 1j * synth.normal(13, "bi" + kind, D.n_slots)
    a, e = synth.encrypt_draws(13, P.qs(level), P.n, "br", 0)
    ct = C.encrypt(P, sk, C.encode_plain(P, v, 2.0 ** 40, level), level, a, e)
    ql = float(P.q[level - 1])
    masks = {(p, q): C.encode_plain(P, BR.mask_slots(M, D.n_slots, p, q), ql, level)
             for p in range(M.n2) for q in range(M.n1)}
    out = BR.slot_map_ct(P, ct, M, lambda p, q: masks[(p, q)], keys)
    assert out.shape[0] == level - 1
    dec = C.decrypt(P, sk, out, 2.0 ** 40)
    want = BR.br(D, kind, v, k, kappa)
    np.testing.assert_allclose(dec, want, atol=2.0 ** -15)


def test_encrypted_decay_broadcast_over_positions():
    """A head span of P d_s = 1024 slots is placed at two positions per head
    and replicated 512 times (terms (p, q): two heads x two positions):
    N = 2^12, H = 2, P = 64, d_s = 16, one chunk of 128 channels."""
    P = C.params_small(12, 50, 4, 2)
    D = BR.Dims(H=2, P=64, G=1, d_s=16, c_state=128, n_slots=P.n // 2)
    M = BR.br_slot_map(D, "a", 5, 0, 4)
    assert (M.n1, M.n2, M.R, M.d, M.g) == (2, 2, 512, -512, 1 - 1024)
    sk = C.secret_key(P, synth.secret(14, P.n))
    keys = {P.galois_elt(r): C.keygen_from_seed(P, sk, 14, P.galois_elt(r))
            for r in BR.slot_map_rotations(M, D.n_slots)}
    v = synth.normal(14, "dr", D.n_slots) + 1j * synth.normal(14, "di", D.n_slots)
    a, e = synth.encrypt_draws(14, P.qs(4), P.n, "dec", 0)
    ct = C.encrypt(P, sk, C.encode_plain(P, v, 2.0 ** 40, 4), 4, a, e)
    ql = float(P.q[3])
    masks = {(p, q): C.encode_plain(P, BR.mask_slots(M, D.n_slots, p, q), ql, 4)
             for p in range(M.n2) for q in range(M.n1)}
    out = BR.slot_map_ct(P, ct, M, lambda p, q: masks[(p, q)], keys)
    dec = C.decrypt(P, sk, out, 2.0 ** 40)
    np.testing.assert_allclose(dec, BR.br(D, "a", v, 5, 0), atol=2.0 ** -15)
