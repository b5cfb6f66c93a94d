"""Pins of the oracle's compositions: the decrypted projection equals the fp64
matrix product and the decrypted scan-contract slice equals the fp64
contraction, on small rings; the diagonal construction is checked in the slot
domain against the matrix product with no encryption at all."""
import numpy as np
import pytest

import synth
from oracle import ckks as C
from oracle import workloads as W


def _keys(P, sk, seed, rots, conj=False):
    elts = {P.galois_elt(r) for r in rots if r % (P.n // 2)}
    if conj:
        elts.add(P.conj_elt)
    return {g: C.keygen_from_seed(P, sk, seed, g) for g in elts}


def _slot_matvec(Wm, X, n_slots, seg_len, Cc, n1, n2, paired):
    """The BSGS algebra evaluated on plain slot vectors."""
    G = -(-Wm.shape[0] // Cc)
    B = -(-Wm.shape[1] // Cc)
    n_in = G // 2 if paired else G
    xs = []
    for u in range(n_in):
        if paired:
            xs.append(W.pack_input(X, n_slots, seg_len, Cc, 2 * u)
                      + 1j * W.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1))
        else:
            xs.append(W.pack_input(X, n_slots, seg_len, Cc, u).astype(complex))
    ys = []
    for b in range(B):
        y = 0
        for p in range(n2):
            acc = 0
            for u in range(n_in):
                for q in range(n1):
                    acc = acc + W.shift_segments(xs[u], q, seg_len) * W.bsgs_diagonal_slots(
                        Wm, n_slots, seg_len, Cc, n1, b, p, u, q, paired)
            y = y + W.shift_segments(acc, p * n1, seg_len)
        if paired:
            y = y + np.conj(y)
        ys.append(y)
    return ys


@pytest.mark.parametrize("paired", [False, True])
def test_bsgs_slot_algebra_is_the_matrix_product(paired):
    n_slots, seg_len, Cc = 256, 8, 32
    T, d_in, d_out = 8, 128, 64
    X = synth.normal(1, "X", (T, d_in))
    Wm = synth.normal(1, "W", (d_in, d_out), 0.1)
    Y = X @ Wm
    for n1, n2 in [(8, 4), (32, 1), (4, 8)]:
        ys = _slot_matvec(Wm, X, n_slots, seg_len, Cc, n1, n2, paired)
        for b, y in enumerate(ys):
            r, s = W.segment_indices(n_slots, seg_len, Cc)
            np.testing.assert_allclose(y.real, Y[r, b * Cc + s], atol=1e-12)
            np.testing.assert_allclose(y.imag, 0, atol=1e-12)


def test_bsgs_complex_paired_outputs_slot_algebra():
    """Complex-paired outputs: set 2P accumulates alpha, set 2P+1 conj(beta),
    and y_2P + conj(y_2P+1) carries output blocks 2P and 2P+1 as its real and
    imaginary parts (checked on plain slot vectors against X W in fp64)."""
    n_slots, seg_len, Cc = 256, 8, 32
    T, d_in, d_out = 8, 128, 128
    X = synth.normal(5, "X", (T, d_in))
    Wm = synth.normal(5, "W", (d_in, d_out), 0.1)
    Y = X @ Wm
    n_in, n_out = d_in // Cc // 2, d_out // Cc
    xs = [W.pack_input(X, n_slots, seg_len, Cc, 2 * u)
          + 1j * W.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1) for u in range(n_in)]
    r, s = W.segment_indices(n_slots, seg_len, Cc)
    for n1, n2 in [(8, 4), (32, 1), (4, 8)]:
        ys = []
        for v in range(n_out):
            y = 0
            for p in range(n2):
                acc = 0
                for u in range(n_in):
                    for q in range(n1):
                        acc = acc + W.shift_segments(xs[u], q, seg_len) * \
                            W.bsgs_pair_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, v, p, u, q)
                y = y + W.shift_segments(acc, p * n1, seg_len)
            ys.append(y)
        for pair in range(n_out // 2):
            out = ys[2 * pair] + np.conj(ys[2 * pair + 1])
            np.testing.assert_allclose(out.real, Y[r, 2 * pair * Cc + s], atol=1e-12)
            np.testing.assert_allclose(out.imag, Y[r, (2 * pair + 1) * Cc + s], atol=1e-12)


def test_replicated_diagonal_method_slot_algebra():
    """cfg1 shape: U x with x replicated to fill the slots, n1 = d, n2 = 1."""
    d, n_slots = 16, 128
    U = synth.uniform_pm1(2, "U", (d, d))
    x = synth.uniform_pm1(2, "x", d)
    ys = _slot_matvec(U.T, x[None, :], n_slots, 1, d, d, 1, False)
    np.testing.assert_allclose(ys[0].real, np.tile(U @ x, n_slots // d), atol=1e-12)


def test_encrypted_bsgs_matvec_paired():
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(3, P.n))
    n_slots, seg_len, Cc = P.n // 2, 16, 32
    T, d_in, d_out = 16, 128, 64
    n1, n2 = 8, 4
    level = 4
    X = synth.normal(3, "X", (T, d_in))
    Wm = synth.normal(3, "W", (d_in, d_out), 0.02)
    desc = W.MatvecDesc(level, d_in // Cc // 2, -(-d_out // Cc), n1, n2, seg_len, True, True)
    keys = _keys(P, sk, 3, W.required_rotations(desc, n_slots), conj=True)
    ins = []
    for u in range(desc.n_in):
        z = (W.pack_input(X, n_slots, seg_len, Cc, 2 * u)
             + 1j * W.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1))
        a, e = synth.encrypt_draws(3, P.qs(level), P.n, "x", u)
        ins.append(C.encrypt(P, sk, C.encode_plain(P, z, 2.0 ** 40, level), level, a, e))
    ql = float(P.q[level - 1])
    diag = lambda b, p, u, q: C.encode_plain(
        P, W.bsgs_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, b, p, u, q, True), ql, level)
    outs = W.bsgs_matvec(P, desc, ins, diag, keys)
    Y = X @ Wm
    r, s = W.segment_indices(n_slots, seg_len, Cc)
    for b, y in enumerate(outs):
        assert y.shape[0] == level - 1
        dec = C.decrypt(P, sk, y, 2.0 ** 40)
        np.testing.assert_allclose(dec.real, Y[r, b * Cc + s], atol=2.0 ** -15)
        np.testing.assert_allclose(dec.imag, 0, atol=2.0 ** -15)


def test_encrypted_bsgs_matvec_complex_paired_outputs():
    """The encrypted projection with complex-paired outputs decodes to output
    blocks 2P (real part) and 2P+1 (imaginary part) within 2^-15."""
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(3, P.n))
    n_slots, seg_len, Cc = P.n // 2, 16, 32
    T, d_in, d_out = 16, 128, 128
    n1, n2 = 8, 4
    level = 4
    X = synth.normal(6, "X", (T, d_in))
    Wm = synth.normal(6, "W", (d_in, d_out), 0.02)
    desc = W.MatvecDesc(level, d_in // Cc // 2, d_out // Cc, n1, n2, seg_len, False, True,
                        complex_pair=True)
    keys = _keys(P, sk, 3, W.required_rotations(desc, n_slots), conj=True)
    ins = []
    for u in range(desc.n_in):
        z = (W.pack_input(X, n_slots, seg_len, Cc, 2 * u)
             + 1j * W.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1))
        a, e = synth.encrypt_draws(3, P.qs(level), P.n, "xp", u)
        ins.append(C.encrypt(P, sk, C.encode_plain(P, z, 2.0 ** 40, level), level, a, e))
    ql = float(P.q[level - 1])
    diag = lambda v, p, u, q: C.encode_plain(
        P, W.bsgs_pair_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, v, p, u, q), ql, level)
    outs = W.bsgs_matvec(P, desc, ins, diag, keys)
    assert len(outs) == desc.n_out // 2
    Y = X @ Wm
    r, s = W.segment_indices(n_slots, seg_len, Cc)
    for pair, y in enumerate(outs):
        assert y.shape[0] == level - 1
        dec = C.decrypt(P, sk, y, 2.0 ** 40)
        np.testing.assert_allclose(dec.real, Y[r, 2 * pair * Cc + s], atol=2.0 ** -15)
        np.testing.assert_allclose(dec.imag, Y[r, (2 * pair + 1) * Cc + s], atol=2.0 ** -15)


@pytest.mark.parametrize("paired", [False, True])
def test_encrypted_bsgs_matvec_double_hoisted(paired):
    """Double hoisting (baby steps left in Q u P, the plaintext MAC over
    Q u P with diagonals encoded there, one ModDown per giant step's inner
    sum) decodes to X W within 2^-15, with real extraction or with
    complex-paired outputs, and within 2^-20 of the ordinary projection (the
    two differ only in where the ModDown rounds)."""
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(3, P.n))
    n_slots, seg_len, Cc = P.n // 2, 16, 32
    T, d_in, d_out = 16, 128, 128
    n1, n2 = 8, 4
    level = 4
    X = synth.normal(8, "X", (T, d_in))
    Wm = synth.normal(8, "W", (d_in, d_out), 0.02)
    args = (level, d_in // Cc // 2, d_out // Cc, n1, n2, seg_len, not paired, True)
    desc = W.MatvecDesc(*args, complex_pair=paired, lazy_moddown=True)
    plain = W.MatvecDesc(*args, complex_pair=paired)
    keys = _keys(P, sk, 3, W.required_rotations(desc, n_slots), conj=True)
    ins = []
    for u in range(desc.n_in):
        z = (W.pack_input(X, n_slots, seg_len, Cc, 2 * u)
             + 1j * W.pack_input(X, n_slots, seg_len, Cc, 2 * u + 1))
        a, e = synth.encrypt_draws(3, P.qs(level), P.n, "xdh", u)
        ins.append(C.encrypt(P, sk, C.encode_plain(P, z, 2.0 ** 40, level), level, a, e))
    ql = float(P.q[level - 1])

    def slots(b, p, u, q):
        if paired:
            return W.bsgs_pair_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, b, p, u, q)
        return W.bsgs_diagonal_slots(Wm, n_slots, seg_len, Cc, n1, b, p, u, q, True)

    blocks = [0, desc.n_out // 2 - 1] if paired else [0, desc.n_out - 1]
    outs = W.bsgs_matvec(P, desc, ins,
                         lambda b, p, u, q: C.encode_plain_ext(P, slots(b, p, u, q), ql, level),
                         keys, blocks)
    ref = W.bsgs_matvec(P, plain, ins,
                        lambda b, p, u, q: C.encode_plain(P, slots(b, p, u, q), ql, level),
                        keys, blocks)
    Y = X @ Wm
    r, s = W.segment_indices(n_slots, seg_len, Cc)
    for blk, y, y0 in zip(blocks, outs, ref):
        assert y.shape[0] == level - 1
        assert not np.array_equal(y, y0)
        dec = C.decrypt(P, sk, y, 2.0 ** 40)
        re_blk, im_blk = (2 * blk, 2 * blk + 1) if paired else (blk, None)
        np.testing.assert_allclose(dec.real, Y[r, re_blk * Cc + s], atol=2.0 ** -15)
        if paired:
            np.testing.assert_allclose(dec.imag, Y[r, im_blk * Cc + s], atol=2.0 ** -15)
        np.testing.assert_allclose(dec, C.decrypt(P, sk, y0, 2.0 ** 40), atol=2.0 ** -20)


def test_scan_contract_slice_small():
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(4, P.n))
    n_slots = P.n // 2
    d_s, head_dim, K = 8, 16, 4
    c_state = n_slots // d_s                      # channels per chunk
    E = K * c_state
    level = 4
    z = synth.normal(4, "z", E // head_dim)
    a = 1.0 / (1.0 + np.exp(z))                   # exp(-softplus(z))
    Cv = synth.normal(4, "C", d_s)
    H = synth.normal(4, "h", (E, d_s))
    want = (a[np.arange(E) // head_dim][:, None] * H * Cv[None, :]).sum(axis=1)
    rlk = C.keygen_from_seed(P, sk, 4, 0)
    keys = _keys(P, sk, 4, [1, 2, 4], conj=True)
    hs, ds, cs = [], [], []
    j = np.arange(n_slots)
    for k in range(K):
        e_idx = k * c_state + j // d_s
        i_idx = j % d_s
        enc = lambda vals, scale, tag: C.encrypt(
            P, sk, C.encode_plain(P, vals.astype(complex), scale, level), level,
            *synth.encrypt_draws(4, P.qs(level), P.n, tag, k))
        hs.append(enc(H[e_idx, i_idx], 2.0 ** 40, "h"))
        ds.append(enc(a[e_idx // head_dim], float(P.q[3]), "a"))
        cs.append(enc(Cv[i_idx], float(P.q[2]), "C"))
    outs = W.scan_contract_token(P, hs, ds, cs, rlk, keys, d_s)
    assert len(outs) == K
    for l in range(K // 2):
        for half in range(2):
            k = 2 * l + half
            dec = C.decrypt(P, sk, outs[2 * l + half], 2.0 * 2.0 ** 40)
            assert outs[2 * l + half].shape[0] == 2
            got = dec.real[:: d_s]
            np.testing.assert_allclose(got, want[k * c_state:(k + 1) * c_state], atol=2.0 ** -15)


def test_scan_contract_contraction_only_odd_chunks():
    """decay None: t = h * C alone (one level), three chunks: one complex
    pair (outputs 2 Sigma) and an odd chunk reduced alone (Sigma)."""
    P = C.params_small(10, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(5, P.n))
    n_slots, d_s, K, level = P.n // 2, 8, 3, 3
    c_state = n_slots // d_s
    Cv = synth.normal(5, "C", d_s)
    H = synth.normal(5, "h", (K * c_state, d_s))
    want = (H * Cv[None, :]).sum(axis=1)
    rlk = C.keygen_from_seed(P, sk, 5, 0)
    keys = _keys(P, sk, 5, [1, 2, 4], conj=True)
    j = np.arange(n_slots)
    hs, cs = [], []
    for k in range(K):
        enc = lambda vals, scale, tag: C.encrypt(
            P, sk, C.encode_plain(P, vals.astype(complex), scale, level), level,
            *synth.encrypt_draws(5, P.qs(level), P.n, tag, k))
        hs.append(enc(H[k * c_state + j // d_s, j % d_s], 2.0 ** 40, "h"))
        cs.append(enc(Cv[j % d_s], float(P.q[level - 1]), "C"))
    outs = W.scan_contract_token(P, hs, None, cs, rlk, keys, d_s)
    assert len(outs) == K and all(o.shape[0] == level - 1 for o in outs)
    for k in range(K):
        factor = 2.0 if k < K - 1 else 1.0
        got = C.decrypt(P, sk, outs[k], factor * 2.0 ** 40).real[::d_s]
        np.testing.assert_allclose(got, want[k * c_state:(k + 1) * c_state], atol=2.0 ** -15)


def hescan_packets(P, seed, L, K, d_s, head_dim):
    """Mamba-2 factor packets of L tokens (Sec. "HEScan": x_k over E = HP
    channels, a_k over heads, B_k and C_k over d_state, one group), the
    decay exp(-softplus(z)) and the rest N(0, 1), and their broadcasts into K
    chunks of c_state = n_slots / d_s channels (chunk slot j holds channel
    kappa c_state + j // d_s and state index j % d_s)."""
    n_slots = P.n // 2
    c_state = n_slots // d_s
    E = K * c_state
    x = synth.normal(seed, "hx", (L, E))
    z = synth.normal(seed, "hz", (L, E // head_dim))
    a = 1.0 / (1.0 + np.exp(z))
    Bv = synth.normal(seed, "hB", (L, d_s))
    Cv = synth.normal(seed, "hC", (L, d_s))
    j = np.arange(n_slots)

    def br(k, t):
        e, i = k * c_state + j // d_s, j % d_s
        return x[t, e], a[t, e // head_dim], Bv[t, i], Cv[t, i]
    return (x, a, Bv, Cv), br


def hescan_reference(vals, head_dim):
    """Eqs. "fesc_recurrence" and "fesc_contract" in fp64: h_k = a_k h_{k-1}
    + x_k (x) B_k, m_k = sum_i h_k[., i] C_k[i]; returns m [L][E]."""
    x, a, Bv, Cv = vals
    L, E = x.shape
    h = np.zeros((E, Bv.shape[1]))
    out = []
    for t in range(L):
        h = a[t][np.arange(E) // head_dim][:, None] * h + x[t][:, None] * Bv[t][None, :]
        out.append(h @ Cv[t])
    return np.array(out)


@pytest.mark.parametrize("L,block,low", [(4, None, False), (5, 2, False), (4, None, True)])
def test_hescan_layer_follows_the_recurrence(L, block, low):
    """Update construction, the encrypted scan (Brent-Kung or resident) and
    the contraction of every token decode to the fp64 recurrence; with `low`
    the contraction runs under a parameter set over the chain prefix
    q_0..q_4 with one special prime instead of two (five one-prime digits at
    the contraction's level 5, each switched with the smaller special modulus)."""
    from oracle import scan as OS
    P = C.params_small(10, 50, 8, 2)
    seed, d_s, head_dim, K, level = 6, 8, 16, 2, 8
    sk = C.secret_key(P, synth.secret(seed, P.n))
    rlk = C.keygen_from_seed(P, sk, seed, 0)
    keys = _keys(P, sk, seed, [1, 2, 4], conj=True)
    vals, br = hescan_packets(P, seed, L, K, d_s, head_dim)
    lo = {(4, None): 5, (5, 2): 4}[(L, block)]      # states' level: 8 - 1 - depth
    contract = None
    if low:
        Pc = C.Params(P.log_n, P.q[:lo], P.p[:1])
        skc = C.secret_key(Pc, synth.secret(seed, P.n))
        contract = (Pc, C.keygen_from_seed(Pc, skc, seed, 0),
                    _keys(Pc, skc, seed, [1, 2, 4], conj=True))
        assert Pc.alpha == 1 and Pc.dnum == lo

    def enc(v, scale, lvl, tag, idx):
        return C.encrypt(P, sk, C.encode_plain(P, v.astype(complex), scale, lvl), lvl,
                         *synth.encrypt_draws(seed, P.qs(lvl), P.n, tag, idx))
    X, Bc, A, Cc = [], [], [], []
    for k in range(K):
        cols = [br(k, t) for t in range(L)]
        X.append([enc(c[0], 2.0 ** 40, level, "hx", k * L + t) for t, c in enumerate(cols)])
        A.append([enc(c[1], float(P.q[level - 2]), level - 1, "ha", k * L + t)
                  for t, c in enumerate(cols)])
        Bc.append([enc(c[2], float(P.q[level - 1]), level, "hB", k * L + t)
                   for t, c in enumerate(cols)])
        Cc.append([enc(c[3], float(P.q[lo - 1]), lo, "hC", k * L + t)
                   for t, c in enumerate(cols)])
    outs = OS.hescan(P, X, Bc, A, Cc, rlk, keys, d_s, block, contract)
    want = hescan_reference(vals, head_dim)
    c_state = P.n // 2 // d_s
    for t in range(L):
        assert [o.shape[0] for o in outs[t]] == [lo - 1] * K
        for k in range(K):
            got = C.decrypt(P, sk, outs[t][k], 2.0 * 2.0 ** 40).real[::d_s]
            np.testing.assert_allclose(got, want[t, k * c_state:(k + 1) * c_state],
                                       atol=2.0 ** -15, err_msg=f"token {t} chunk {k}")


# ------------------------------------------------- small kernels (HEConv etc.)


def _enc_ct(P, sk, vals, scale, level, tag, idx=0):
    return C.encrypt(P, sk, C.encode_plain(P, np.asarray(vals, dtype=complex), scale, level),
                     level, *synth.encrypt_draws(6, P.qs(level), P.n, tag, idx))


def conv_inputs(P, T, d_conv, seed=6):
    """Channels on segments of T token slots (slot c*T + k); taps r = 0..d-1 at
    offset -r with the causal boundary (k >= r) in the mask."""
    n_slots = P.n // 2
    Cn = n_slots // T
    qv = synth.normal(seed, "conv-q", (Cn, T))
    w = synth.normal(seed, "conv-w", (Cn, d_conv), 0.5)
    b = synth.normal(seed, "conv-b", Cn)
    k = np.arange(T)
    masks = [np.where(k[None, :] >= r, w[:, r:r + 1], 0.0).reshape(-1) for r in range(d_conv)]
    return qv, w, b, masks


def test_heconv_decodes_to_the_depthwise_causal_convolution():
    P = C.params_small(12, 50, 4, 2)
    sk = C.secret_key(P, synth.secret(6, P.n))
    T, d_conv, level = 64, 4, 3
    deltas = [-r for r in range(d_conv)]
    keys = _keys(P, sk, 6, deltas)
    qv, w, b, masks = conv_inputs(P, T, d_conv)
    Cn = qv.shape[0]
    ql = float(P.q[level - 1])
    q = _enc_ct(P, sk, qv.reshape(-1), 2.0 ** 40, level, "q")
    pts = [C.encode_plain(P, m.astype(complex), ql, level) for m in masks]
    bias = C.encode_plain(P, np.repeat(b, T).astype(complex), 2.0 ** 40, level)
    out = W.heconv(P, q, deltas, pts, bias, keys)
    assert out.shape[0] == level - 1
    got = C.decrypt(P, sk, out, 2.0 ** 40).real.reshape(Cn, T)
    # Eq. "conv1d_depthwise": eta_k[c] = b_c + sum_r w_{c,r} q_{k-r}[c], q_t = 0 for t < 0
    want = np.tile(b[:, None], (1, T))
    for r in range(d_conv):
        shifted = np.zeros_like(qv)
        shifted[:, r:] = qv[:, :T - r]
        want += w[:, r:r + 1] * shifted
    np.testing.assert_allclose(got, want, atol=2.0 ** -15)


def test_post_ssm_decodes_to_gated_skip():
    P = C.params_small(12, 50, 5, 2)
    sk = C.secret_key(P, synth.secret(6, P.n))
    rlk = C.keygen_from_seed(P, sk, 6, 0)
    level, n_slots = 4, P.n // 2
    mv = synth.normal(6, "ps-m", n_slots)
    xv = synth.normal(6, "ps-x", n_slots)
    dv = synth.normal(6, "ps-D", n_slots)
    gv = synth.uniform_pm1(6, "ps-g", n_slots)
    m = _enc_ct(P, sk, mv, 2.0 ** 40, level, "m")
    x = _enc_ct(P, sk, xv, 2.0 ** 40, level, "x")
    g = _enc_ct(P, sk, gv, float(P.q[level - 2]), level, "g")
    D = C.encode_plain(P, dv.astype(complex), float(P.q[level - 1]), level)
    out = W.post_ssm(P, m, x, D, g, rlk)
    assert out.shape[0] == level - 2
    got = C.decrypt(P, sk, out, 2.0 ** 40).real
    np.testing.assert_allclose(got, (mv + dv * xv) * gv, atol=2.0 ** -15)


def test_c2m_level_is_the_shortest_admissible_modulus():
    P = C.params_p16(24)
    # 50-bit primes: ell + sigma + 1 = 64 + 40 + 1 = 105 bits need three primes
    assert W.c2m_level(P, 24, 64, 40, 2.0 ** 40, 2.0 ** 10) == 3
    # a large boundary magnitude: Q / 2 > 2^40 * 2^70 = 2^110 needs three primes too,
    # 2^160 needs four
    assert W.c2m_level(P, 24, 16, 40, 2.0 ** 40, 2.0 ** 120) == 4
    # below the requirement at the available level: none
    assert W.c2m_level(P, 2, 64, 40, 2.0 ** 40, 1.0) is None
    # brute force over every level
    for ell, sig, bm in [(32, 40, 2.0 ** 8), (48, 40, 2.0 ** 60), (20, 20, 1.0)]:
        want = None
        for lp in range(1, 25):
            Q = int(np.prod([P.q[i] for i in range(lp)], dtype=object))
            if Q.bit_length() - 1 >= ell + sig + 1 and Q > 2 * 2.0 ** 40 * bm:
                want = lp
                break
        assert W.c2m_level(P, 24, ell, sig, 2.0 ** 40, bm) == want


def test_c2m_mask_shares_reconstruct_the_message():
    """Dec(<m> + r_hat) - r_hat = Dec(<m>) exactly on the coefficients (the two
    shares of Algorithm "Complex CKKS-to-MPC conversion" reconstruct)."""
    P = C.params_small(12, 50, 3, 1)
    sk = C.secret_key(P, synth.secret(6, P.n))
    level = 2
    ct = _enc_ct(P, sk, synth.normal(6, "c2m", P.n // 2), 2.0 ** 40, level, "c2m")
    rhat = synth.uniform_residues(6, "rhat", P.qs(level), P.n)
    d = W.c2m_mask(P, ct, rhat)
    qs = P.qs(level)
    share0 = C.intt(P, C.padd(d[:, 0], C.pmul(d[:, 1], sk.ntt_ext[:level], qs), qs), qs)
    share1 = C.intt(P, C.psub(np.zeros_like(rhat), rhat, qs), qs)
    dec = C.intt(P, C.padd(ct[:, 0], C.pmul(ct[:, 1], sk.ntt_ext[:level], qs), qs), qs)
    assert np.array_equal(C.padd(share0, share1, qs), dec)
