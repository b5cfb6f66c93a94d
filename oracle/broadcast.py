"""Public broadcast and reduction slot maps of HEScan, and a homomorphic
realisation of a broadcast (test infrastructure only: the tests, the smoke
check and the benchmark's CPU baseline use this module; the library never
does).

Plain maps (Sec. "Factorized HEScan Kernel", paragraph "State-Chunk Packing"
with Eq. "hescan-chunk-map"; Appendix "HEScan Kernel Packing and Correctness",
paragraph "Exact State and Slot Maps").  E = H P expanded channels e = h P + p
with h(e) = floor(e / P), p(e) = e mod P; chunk kappa owns the channels
kappa c <= e < (kappa + 1) c (c = c_state) and keeps state coordinate (e, i),
i < d_s, at slot lambda_kappa(e, i) = (e - kappa c) d_s + i.  The compact
factors of a sequence block sit at

    a: k H + h,      x: k E + e,      B, C: k G d_s + g d_s + i,

and br^(kappa) of token k's factor holds, at slot lambda_kappa(e, i),
a_k[h(e)], x_k[h(e), p(e)], B_k[g(h(e)), i] or C_k[g(h(e)), i]; every other
slot is zero.  Sigma_{d_s} sums the d_s slots of each channel of a chunk.

Reading (the paper names the group map g(h) without giving it): the heads
form G contiguous groups of H / G, g(h) = floor(h G / H) (0-based), as in
Mamba-2's grouped heads.

Homomorphic realisation (the paper gives the maps, not their CKKS form; this
is the reading the library implements).  A broadcast is one *slot map* over
terms t = p n1 + q < n (q < n1 baby index, p giant index):

    y[j]   = v[j + r0 + q d + p g]   for j in run_t = [j0 + q J + p Jg, ... + w),
    y[j]   = 0                       elsewhere,
    out[j] = sum_{u < R} y[j - u S]

(indices mod n_slots; runs disjoint; R a power of two), evaluated in three
steps:
    1. rho(v; r0), one key switch (a copy when r0 = 0 mod n_slots);
    2. the diagonal method sum_t M_t (.) rho(.; q d + p g), M_t = 1 on run_t,
       baby-step/giant-step: the baby steps rho(.; q d) share one ModUp, the
       giant steps are rho(.; p g), each mask is rotated by -p g before
       encoding; the masks are encoded at the scale of q_{l-1} and the sum is
       rescaled once (level l -> l - 1);
    3. log2 R doublings out <- out + rho(out; -2^s S).
Replication by doubling adds the key-switching noise of every slot of R
shifted copies, so the error of an output slot grows as sqrt(R); the decay's
broadcast, whose natural replication is the P d_s slots of a head, places
each head at P d_s / R_a positions and replicates R_a = min(P d_s, 512)
times (512 keeps the decoded error below 2^-15 at N = 2^16 and scale 2^40:
about 8e-6 was measured at R = 128 and 4e-5 at R = 8192).
Per factor (c channels per chunk, Eg = P H / G channels per group, n1 the
smallest power of two whose square reaches n unless stated, g = n1 d and
Jg = n1 J unless stated):
    x:  r0 = k E + kappa c, d = 1 - d_s, n = c, J = d_s, w = 1, R = d_s, S = 1;
    a:  r0 = k H + kappa c / P, n1 = P d_s / R_a positions per head (d = -R_a,
        J = R_a), n2 = c / P heads (g = 1 - P d_s, Jg = P d_s), w = 1, R = R_a,
        S = 1 (P divides c);
    B, C, chunk inside group g0: r0 = k G d_s + g0 d_s, n = 1, run_0 = [0, d_s),
        R = c, S = d_s;
    B, C, chunk over whole groups g0, g0 + 1, ...: r0 = k G d_s + g0 d_s,
        d = d_s - Eg d_s, n = c / Eg, J = Eg d_s, w = d_s, R = Eg, S = d_s.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import ckks as C

KINDS = ("a", "x", "B", "C")


@dataclass(frozen=True)
class Dims:
    H: int          # heads
    P: int          # head width
    G: int          # groups of B and C
    d_s: int        # state size per channel
    c_state: int    # expanded channels per chunk
    n_slots: int

    @property
    def E(self) -> int:
        return self.H * self.P

    @property
    def K_s(self) -> int:
        return -(-self.E // self.c_state)


def group(D: Dims, h: int) -> int:
    """g(h): contiguous groups of H / G heads (reading)."""
    return h * D.G // D.H


def chunk_channels(D: Dims, kappa: int) -> range:
    """E_kappa of Eq. "hescan-chunk-map"."""
    return range(kappa * D.c_state, min((kappa + 1) * D.c_state, D.E))


def chunk_slot(D: Dims, kappa: int, e: int, i: int) -> int:
    """lambda_kappa(e, i) = (e - kappa c_state) d_s + i."""
    return (e - kappa * D.c_state) * D.d_s + i


def compact_a(D: Dims, a: np.ndarray) -> np.ndarray:
    """a[k][h] at slot k H + h (lambda_a)."""
    v = np.zeros(D.n_slots, np.complex128)
    for k in range(a.shape[0]):
        for h in range(D.H):
            v[k * D.H + h] = a[k, h]
    return v


def compact_x(D: Dims, x: np.ndarray) -> np.ndarray:
    """x[k][h][p] at slot k E + h P + p (lambda_x)."""
    v = np.zeros(D.n_slots, np.complex128)
    for k in range(x.shape[0]):
        for h in range(D.H):
            for p in range(D.P):
                v[k * D.E + h * D.P + p] = x[k, h, p]
    return v


def compact_bc(D: Dims, b: np.ndarray) -> np.ndarray:
    """B[k][g][i] (or C) at slot k G d_s + g d_s + i (lambda_B, lambda_C)."""
    v = np.zeros(D.n_slots, np.complex128)
    for k in range(b.shape[0]):
        for g in range(D.G):
            for i in range(D.d_s):
                v[k * D.G * D.d_s + g * D.d_s + i] = b[k, g, i]
    return v


def br(D: Dims, kind: str, v: np.ndarray, k: int, kappa: int) -> np.ndarray:
    """br^(kappa) of token k's factor from its compact slot vector v."""
    out = np.zeros(D.n_slots, np.complex128)
    for e in chunk_channels(D, kappa):
        h = e // D.P
        for i in range(D.d_s):
            if kind == "a":
                src = k * D.H + h
            elif kind == "x":
                src = k * D.E + e
            else:
                src = k * D.G * D.d_s + group(D, h) * D.d_s + i
            out[chunk_slot(D, kappa, e, i)] = v[src]
    return out


def sigma(D: Dims, u: np.ndarray, kappa: int) -> np.ndarray:
    """Sigma_{d_s} over chunk kappa: entry e - kappa c is sum_i u[lambda(e, i)]."""
    return np.array([sum(u[chunk_slot(D, kappa, e, i)] for i in range(D.d_s))
                     for e in chunk_channels(D, kappa)])


# ------------------------------------------------------------ realisation


@dataclass(frozen=True)
class SlotMap:
    level: int
    r0: int
    d: int       # rotation per baby step
    n: int       # terms
    n1: int      # baby steps
    g: int       # rotation per giant step
    j0: int
    J: int       # run offset per baby step
    Jg: int      # run offset per giant step
    w: int
    R: int
    S: int

    @property
    def n2(self) -> int:
        return -(-self.n // self.n1)

    def terms(self):
        """(p, q) of every term t = p n1 + q < n."""
        return [divmod(t, self.n1) for t in range(self.n)]


R_MAX_DECAY = 512


def _pow2(x: int) -> bool:
    return x > 0 and x & (x - 1) == 0


def _baby(n: int) -> int:
    """Baby steps: the power of two nearest above sqrt(n)."""
    n1 = 1
    while n1 * n1 < n:
        n1 *= 2
    return n1


def _progression(level, r0, d, n, J, w, R, S) -> SlotMap:
    n1 = _baby(n)
    return SlotMap(level, r0, d, n, n1, n1 * d, 0, J, n1 * J, w, R, S)


def br_slot_map(D: Dims, kind: str, k: int, kappa: int, level: int) -> SlotMap:
    """The slot map that realises br^(kappa) of token k's factor (module
    docstring); ValueError where the reading does not cover the shape."""
    c = D.c_state
    if D.E % c or not 0 <= kappa < D.E // c or c * D.d_s > D.n_slots:
        raise ValueError("chunking")
    if kind == "x":
        if not _pow2(D.d_s) or (k + 1) * D.E > D.n_slots:
            raise ValueError("x")
        return _progression(level, k * D.E + kappa * c, 1 - D.d_s, c, D.d_s, 1, D.d_s, 1)
    if kind == "a":
        if c % D.P or not _pow2(D.P * D.d_s) or (k + 1) * D.H > D.n_slots:
            raise ValueError("a")
        heads, span = c // D.P, D.P * D.d_s
        R = min(span, R_MAX_DECAY)
        pos = span // R
        return SlotMap(level, k * D.H + kappa * heads, -R, heads * pos, pos, 1 - span, 0, R,
                       span, 1, R, 1)
    if kind not in ("B", "C") or D.H % D.G or (k + 1) * D.G * D.d_s > D.n_slots:
        raise ValueError("B/C")
    Eg = D.P * D.H // D.G
    lo, hi = kappa * c // Eg, (kappa * c + c - 1) // Eg
    if lo == hi:
        if not _pow2(c):
            raise ValueError("B/C")
        return _progression(level, k * D.G * D.d_s + lo * D.d_s, 0, 1, 0, D.d_s, c, D.d_s)
    if c % Eg or not _pow2(Eg):
        raise ValueError("B/C")
    return _progression(level, k * D.G * D.d_s + lo * D.d_s, D.d_s - Eg * D.d_s, c // Eg,
                        Eg * D.d_s, D.d_s, Eg, D.d_s)


def _run_start(M: SlotMap, p: int, q: int) -> int:
    return M.j0 + q * M.J + p * M.Jg


def slot_map_plain(M: SlotMap, v: np.ndarray) -> np.ndarray:
    """The slot map's action on a plain slot vector (the definition above)."""
    ns = len(v)
    y = np.zeros(ns, np.complex128)
    for p, q in M.terms():
        for o in range(M.w):
            j = (_run_start(M, p, q) + o) % ns
            y[j] = v[(j + M.r0 + q * M.d + p * M.g) % ns]
    out = np.zeros(ns, np.complex128)
    for u in range(M.R):
        out += np.roll(y, u * M.S)          # out[j] += y[j - u S]
    return out


def mask_slots(M: SlotMap, n_slots: int, p: int, q: int) -> np.ndarray:
    """Mask of term (p, q) rotated by -p g (zero past the last term): entry j
    is 1 where j - p g falls in the term's run."""
    z = np.zeros(n_slots, np.complex128)
    if p * M.n1 + q >= M.n:
        return z
    for o in range(M.w):
        j = (_run_start(M, p, q) + o) % n_slots
        z[(j + p * M.g) % n_slots] = 1.0
    return z


def slot_map_rotations(M: SlotMap, n_slots: int) -> set:
    """Rotation steps (mod n_slots, nonzero) the realisation key-switches by."""
    r = {M.r0 % n_slots}
    r |= {(q * M.d) % n_slots for q in range(M.n1)}
    r |= {(p * M.g) % n_slots for p in range(M.n2)}
    s = 1
    while s < M.R:
        r.add((-s * M.S) % n_slots)
        s *= 2
    r.discard(0)
    return r


def slot_map_ct(P: C.Params, ct: np.ndarray, M: SlotMap, masks, keys: dict) -> np.ndarray:
    """The three steps on a ciphertext at level M.level; masks(p, q) gives the
    encoded mask of term (p, q) (scale q_{l-1}; zero past the last term).
    Output at level - 1."""
    v = C.rotate(P, ct, M.r0, keys)
    baby = C.rotate_hoisted(P, v, [q * M.d for q in range(M.n1)], keys)
    y = None
    for p in range(M.n2):
        acc = None
        for q in range(M.n1):
            t = C.mul_plain(P, baby[q], masks(p, q))
            acc = t if acc is None else C.ct_add(P, acc, t)
        acc = C.rotate(P, acc, p * M.g, keys)
        y = acc if y is None else C.ct_add(P, y, acc)
    y = C.rescale(P, y)
    s = 1
    while s < M.R:
        y = C.ct_add(P, y, C.rotate(P, y, -s * M.S, keys))
        s *= 2
    return y
