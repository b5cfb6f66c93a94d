"""Compositions of the oracle's CKKS operations (test infrastructure only):
the plaintext-matrix x ciphertext projection and the scan-contract slice.

Projection (Appendix "Projection Kernel Breakdown"): slots are viewed as
segments, idx(r, s) = s * seg_len + r; the whole-segment shift Phi^delta is
one rotation by delta * seg_len.  Input block g packs X[r, g*C + c] at
idx(r, c); with complex pairing the ciphertext carries x^(2u) + i x^(2u+1).
For output block b, giant step p and baby step q,

    c~_p = sum_u sum_q Phi^q(x~_u) * D~_{b,u,p,q},     y = sum_p Phi^(p n1)(c~_p),

and the real lane is extracted as c + conj(c) (or, with complex-paired
outputs, two real blocks leave as one ciphertext y_2P + conj(y_2P+1); see
bsgs_pair_diagonal_slots).  The paper leaves the content
of D~ implicit ("the two real weight slices"); the reading used here is

    diag_t^(g,b)[idx(r, s)] = W[g*C + (s + t) mod C, b*C + s]   (0 if out of range)
    D~_{b,u,p,q} = Phi^(-p n1)( (diag_{p n1 + q}^(2u,b) - i diag_{p n1 + q}^(2u+1,b)) / 2 )

so that Re(x~ * D~) is the paired sum and one extraction c + conj(c) of the
sum over giant steps yields the real projection (extraction is linear, so one
conjugation per output block replaces one per giant step).  Without pairing
D_{b,g,p,q} = Phi^(-p n1)(diag_{p n1+q}^(g,b)) and no extraction is done.
When the slot count exceeds the packed width (n_slots > C * seg_len) the
segment index is taken modulo C, i.e. the vector is replicated, which is how a
short vector is made rotation-periodic.

Small kernels on the same primitives: HEConv (Sec. "Causal Depthwise
Convolution"), the fused post-SSM path (Appendix "Fused Post-SSM Path"),
modulus trimming before the CKKS-to-MPC conversion (Appendix "Adopted Modulus
Trimming") and the server's conversion mask (Algorithm "Complex CKKS-to-MPC
conversion", first two steps).

Scan-contract slice (Eq. "hescan-contract-output" and Appendix "Complex-Packed
Reduction Accounting"): per token and state chunk, t1 = RS(relin(a * h)),
t2 = RS(relin(t1 * C)); chunks (2l, 2l+1) are packed as chi = t2^(2l) + i
t2^(2l+1) (i = X^(N/2), exact), reduced over the d_s axis by a rotate-and-add
tree with steps d_s/2, ..., 1, and split by one conjugation:
Re = Xi + conj(Xi) = 2 Sigma(v0), Im = -i (Xi - conj(Xi)) = 2 Sigma(v1).  The
factor 2 is carried in the tracked scale (no constant multiplication).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import ckks as C


@dataclass
class MatvecDesc:
    level: int
    n_in: int
    n_out: int
    n1: int
    n2: int
    unit: int            # slots per segment (Phi^1 = rotation by `unit`)
    real_extract: bool
    rescale: bool
    # outputs in pairs: the n_out diagonal sets are taken as (2P, 2P+1) and
    # output P is y_2P + conj(y_2P+1) (n_out / 2 output ciphertexts)
    complex_pair: bool = False
    # double hoisting: baby steps stay in the extended basis Q u P (no
    # ModDown), the plaintext MAC runs there with diagonals encoded over
    # Q u P, and each giant step's inner sum takes one ModDown
    lazy_moddown: bool = False

    def baby_steps(self):
        return [q * self.unit for q in range(self.n1)]

    def giant_steps(self):
        return [p * self.n1 * self.unit for p in range(self.n2)]


def required_rotations(desc: MatvecDesc, n_slots: int) -> set:
    r = {s % n_slots for s in desc.baby_steps() + desc.giant_steps()}
    r.discard(0)
    return r


def bsgs_matvec(P: C.Params, desc: MatvecDesc, ins: list, diag, keys: dict,
                blocks=None) -> list:
    """``diag(b, p, u, q)`` returns the evaluation-form plaintext D~_{b,u,p,q}
    (``u64[level][N]``; with lazy_moddown over Q u P, ``u64[level+alpha][N]``).
    Baby steps are hoisted (one ModUp per input); with lazy_moddown they are
    also left in Q u P and each inner sum over (u, q) takes one ModDown
    (double hoisting).  Giant steps and the conjugation are ordinary key
    switches."""
    assert len(ins) == desc.n_in
    lazy = desc.lazy_moddown
    hoist = C.rotate_hoisted_ext if lazy else C.rotate_hoisted
    baby = [hoist(P, x, desc.baby_steps(), keys) for x in ins]

    def giant_sum(b):
        y = None
        for p in range(desc.n2):
            acc = None
            for u in range(desc.n_in):
                for q in range(desc.n1):
                    if lazy:
                        t = C.mul_plain_ext(P, baby[u][q], diag(b, p, u, q))
                        acc = t if acc is None else C.ext_add(P, acc, t)
                    else:
                        t = C.mul_plain(P, baby[u][q], diag(b, p, u, q))
                        acc = t if acc is None else C.ct_add(P, acc, t)
            if lazy:
                acc = C.moddown_ct(P, acc, desc.level)
            acc = C.rotate(P, acc, desc.giant_steps()[p], keys)
            y = acc if y is None else C.ct_add(P, y, acc)
        return y

    outs = []
    if desc.complex_pair:
        # output P = y_2P + conj(y_2P+1); `blocks` names pairs P
        for pair in (range(desc.n_out // 2) if blocks is None else blocks):
            y = C.ct_add(P, giant_sum(2 * pair), C.conjugate(P, giant_sum(2 * pair + 1), keys))
            outs.append(C.rescale(P, y) if desc.rescale else y)
        return outs
    for b in (range(desc.n_out) if blocks is None else blocks):
        y = giant_sum(b)
        if desc.real_extract:
            y = C.ct_add(P, y, C.conjugate(P, y, keys))
        if desc.rescale:
            y = C.rescale(P, y)
        outs.append(y)
    return outs


# ---------------------------------------------------- slot-domain packing


def segment_indices(n_slots: int, seg_len: int, C_: int):
    """(r, s) of every slot: r = j mod seg_len, s = (j div seg_len) mod C."""
    j = np.arange(n_slots)
    return j % seg_len, (j // seg_len) % C_


def pack_input(X: np.ndarray, n_slots: int, seg_len: int, C_: int, g: int) -> np.ndarray:
    """x^(g)[idx(r, c)] = X[r, g*C + c] (zero outside X)."""
    T, d_in = X.shape
    r, s = segment_indices(n_slots, seg_len, C_)
    col = g * C_ + s
    ok = (r < T) & (col < d_in)
    out = np.zeros(n_slots)
    out[ok] = X[r[ok], col[ok]]
    return out


def diagonal(W: np.ndarray, n_slots: int, seg_len: int, C_: int, g: int, b: int,
             t: int) -> np.ndarray:
    """diag_t^(g,b)[idx(r, s)] = W[g*C + (s + t) mod C, b*C + s]."""
    d_in, d_out = W.shape
    _, s = segment_indices(n_slots, seg_len, C_)
    row = g * C_ + (s + t) % C_
    col = b * C_ + s
    ok = (row < d_in) & (col < d_out)
    out = np.zeros(n_slots)
    out[ok] = W[row[ok], col[ok]]
    return out


def shift_segments(v: np.ndarray, delta: int, seg_len: int) -> np.ndarray:
    """Phi^delta in slots: left rotation by delta * seg_len."""
    return np.roll(v, -delta * seg_len)


def bsgs_diagonal_slots(W, n_slots, seg_len, C_, n1, b, p, u, q, paired: bool):
    t = p * n1 + q
    if paired:
        d = 0.5 * (diagonal(W, n_slots, seg_len, C_, 2 * u, b, t)
                   - 1j * diagonal(W, n_slots, seg_len, C_, 2 * u + 1, b, t))
    else:
        d = diagonal(W, n_slots, seg_len, C_, u, b, t).astype(np.complex128)
    return shift_segments(d, -p * n1, seg_len)


def bsgs_pair_diagonal_slots(W, n_slots, seg_len, C_, n1, v, p, u, q):
    """Diagonal set v = 2P + e of complex-paired outputs (paired inputs).

    Output pair P carries real blocks b = 2P (real part) and b' = 2P + 1
    (imaginary part).  Per slot, with x~ = x0 + i x1 the paired input and
    a = diag^(2u,b), c = diag^(2u+1,b), d = diag^(2u,b'), f = diag^(2u+1,b'),
    the wanted S_b + i S_b' = (a x0 + c x1) + i (d x0 + f x1) equals
    alpha x~ + beta conj(x~) with alpha = ((a + f) + i (d - c)) / 2 and
    beta = ((a - f) + i (d + c)) / 2.  Rotations commute with conjugation, so
    the beta part is the conjugate of a second accumulation over the same
    baby steps with conj(beta): set e = 0 holds alpha, set e = 1 holds
    conj(beta), and output P = y_2P + conj(y_2P+1).  With b' = b this is the
    real extraction (alpha = conj(beta))."""
    t = p * n1 + q
    pair, e = v // 2, v % 2
    a = diagonal(W, n_slots, seg_len, C_, 2 * u, 2 * pair, t)
    c = diagonal(W, n_slots, seg_len, C_, 2 * u + 1, 2 * pair, t)
    d = diagonal(W, n_slots, seg_len, C_, 2 * u, 2 * pair + 1, t)
    f = diagonal(W, n_slots, seg_len, C_, 2 * u + 1, 2 * pair + 1, t)
    if e == 0:
        z = 0.5 * (a + f) + 1j * (0.5 * (d - c))
    else:
        z = 0.5 * (a - f) - 1j * (0.5 * (d + c))
    return shift_segments(z, -p * n1, seg_len)


# -------------------------------------------------- scan-contract slice


def reduce_axis(P: C.Params, ct: np.ndarray, d: int, keys: dict) -> np.ndarray:
    """Rotate-and-add over a contiguous axis of length d (a power of two):
    slot e*d then holds sum_i v[e*d + i]."""
    step = d // 2
    while step >= 1:
        ct = C.ct_add(P, ct, C.rotate(P, ct, step, keys))
        step //= 2
    return ct


def scan_contract_token(P: C.Params, h: list, decay, cfac: list, rlk, keys: dict,
                        d_s: int) -> list:
    """One token of the scan-contract slice.  h, decay, cfac: per-chunk
    ciphertexts at the same level (decay None: the contraction alone,
    t = h * C).  Every relinearised product is rescaled in the same division
    (ckks.mul_relin_rescale, the reading the scan takes).  Returns
    [Re_0, Im_0, Re_1, Im_1, ...] (each twice the reduced sum of its chunk;
    an odd last chunk reduced alone)."""
    K = len(h)
    t2 = []
    for k in range(K):
        t1 = h[k] if decay is None else C.mul_relin_rescale(P, decay[k], h[k], rlk)
        c = cfac[k][: t1.shape[0]]
        t2.append(C.mul_relin_rescale(P, t1, c, rlk))
    outs = []
    for l in range(K // 2):
        chi = C.ct_add(P, t2[2 * l], C.mul_monomial(P, t2[2 * l + 1], P.n // 2))
        xi = reduce_axis(P, chi, d_s, keys)
        xc = C.conjugate(P, xi, keys)
        outs.append(C.ct_add(P, xi, xc))
        outs.append(C.mul_monomial(P, C.ct_sub(P, xi, xc), 3 * P.n // 2))
    if K % 2:
        outs.append(reduce_axis(P, t2[-1], d_s, keys))
    return outs


# ------------------------------------------ small kernels on the same primitives


def heconv(P: C.Params, q: np.ndarray, deltas, masks, bias, keys: dict) -> np.ndarray:
    """HEConv: eta = RS(sum_r M_r (.) rho(q; delta_r)) + b.  q: ciphertext at
    level l; masks: plaintexts (tap weights fused with the causal boundary
    mask), encoded at the scale of q_{l-1} so that the rescale returns q's
    scale; bias: plaintext at that output scale (>= l - 1 limbs), or None;
    deltas: public rotation offsets (negative: rotation to the right).  Output
    at level l - 1."""
    acc = None
    for d, m in zip(deltas, masks):
        t = C.mul_plain(P, C.rotate(P, q, d, keys), m)
        acc = t if acc is None else C.ct_add(P, acc, t)
    out = C.rescale(P, acc)
    if bias is not None:
        out = C.add_plain(P, out, bias)
    return out


def post_ssm(P: C.Params, m: np.ndarray, x_skip: np.ndarray, d_skip: np.ndarray,
             g: np.ndarray, rlk) -> np.ndarray:
    """Fused post-SSM path: y = m + D (.) x_skip, then y (.) g.  m, x_skip, g
    at level l; D a plaintext (at the scale of q_{l-1}); g at the scale of
    q_{l-2}.  y = RS(D (.) x_skip) + m at level l - 1; the gate product is
    relinearised and rescaled in one division (as in the scan) -> level l - 2."""
    level = m.shape[0]
    y = C.ct_add(P, C.rescale(P, C.mul_plain(P, x_skip, d_skip)), m[:level - 1])
    return C.mul_relin_rescale(P, y, g[:level - 1], rlk)


def c2m_level(P: C.Params, level: int, ell: int, sigma: int, delta: float, bmax: float):
    """Modulus trimming before CKKS-to-MPC conversion: the smallest level
    l' <= level whose modulus Q = q_0 ... q_{l'-1} has log2 Q >= ell + sigma + 1
    and Q / 2 > delta * bmax (the ciphertext is then its first l' limbs); None
    if no level qualifies."""
    Q = 1
    for lp in range(1, level + 1):
        Q *= P.q[lp - 1]
        if Q >= 1 << (ell + sigma + 1) and Q > 2 * delta * bmax:  # exact int/float compare
            return lp
    return None


def c2m_mask(P: C.Params, ct: np.ndarray, rhat: np.ndarray) -> np.ndarray:
    """The server's conversion mask: <d> = <m> + r_hat, r_hat a uniform
    polynomial (evaluation form, drawn by the caller) added to the message."""
    return C.add_plain(P, ct, rhat)
