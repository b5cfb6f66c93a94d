"""Encrypted affine prefix scan of HEScan (test infrastructure only).

Follows Sec. "Parallel Prefix Scans", the paragraph "Affine Prefix
Composition" with Eq. "compact_affine_compose", Sec. "Resident Block Schedule"
with Eq. "resident-block-schedule", and the Brent-Kung network of Appendix
"Prefix-Network Selection".

A token-local map is the tuple (a, s) standing for F(z) = a * z + s; when R
follows L the composition is

    T_R o T_L = (a_R * a_L,  a_R * s_L + s_R),

and the inclusive prefix T_1 o ... o T_k applied to the zero state is the
state h_k, i.e. the s part of the prefix.

Readings taken where the paper is silent or inconsistent:

* br^(kappa) is the identity: the decay arrives already broadcast into the
  chunk's packing (as in the scan-contract slice), so every state chunk runs an
  independent scan over (a^(kappa), s^(kappa)), two relinearised products per
  composition, which is the per-chunk count 2 K_s BK(L) of Table
  "real-phantom-scan".
* A ciphertext product is relinearised and rescaled in one division by
  P q_{l-1} (ckks.mul_relin_rescale: the ModDown conversion takes q_{l-1}
  together with the special primes; the paper fixes neither operation); the
  addend s_R is brought to the product's level by dropping its trailing limbs
  (modulus switching without division: message and scale unchanged).
* Operands at different levels (the down-sweep combines prefixes of unequal
  depth) are composed at the lower level, the higher one dropped to it.
* Down-sweep: at stage s every multiple k of 2^s passes its prefix to
  k + 2^(s-1).  The printed side condition (k not a multiple of 2^(s+1))
  contradicts the stated count L' - 1 - log2 L' and would leave, for L' = 8,
  position 5 without its prefix; the count and the classical network agree
  with the reading used here.
* Positions past L (the padding to L' = 2^ceil(log2 L)) are not computed: a
  node only reads positions below its destination, so the prefixes of valid
  positions do not depend on them.  The same holds for the identity padding
  of a final partial block in the resident schedule.
* Outputs are returned at one level, the lowest any prefix reaches (the
  others are dropped to it).  For L = 2^m >= 4 this is 2m - 2 levels below
  the inputs; the paper's "depth 2 ceil(log2 L') - 1" counts network stages.
* The exclusive scan over block summaries (left open by the paper) is the
  same Brent-Kung network over S_0 .. S_{K-2}; the carry G_j is its (j-1)-th
  prefix, and the corrected state of token (j, t) is the s part of
  P_{j,t} o G_j, one relinearised product.
"""
from __future__ import annotations

import math

from . import ckks as C


def brent_kung(items: list, op) -> tuple[list, int, int]:
    """Inclusive prefix t_1 op ... op t_k for k = 1..L by the Brent-Kung
    network over L' = 2^ceil(log2 L) positions.  op(left, right) combines the
    earlier element `left` with the later `right`.  Returns (prefixes, number
    of op applications, number of network stages)."""
    L = len(items)
    if L == 0:
        return [], 0, 0
    m = math.ceil(math.log2(L)) if L > 1 else 0
    Lp = 1 << m
    t = [None] + list(items)  # 1-based positions as in the paper
    nodes = stages = 0
    # up-sweep: every 2^s-aligned position takes the one 2^(s-1) to its left
    for s in range(1, m + 1):
        for k in range(1 << s, Lp + 1, 1 << s):
            if k <= L:
                t[k] = op(t[k - (1 << (s - 1))], t[k])
                nodes += 1
        stages += 1
    # down-sweep: each multiple k of 2^s passes its prefix to k + 2^(s-1)
    for s in range(m - 1, 0, -1):
        for k in range(1 << s, Lp + 1, 1 << s):
            j = k + (1 << (s - 1))
            if j <= L:
                t[j] = op(t[k], t[j])
                nodes += 1
        stages += 1
    return t[1:], nodes, stages


def bk_count(Lp: int) -> int:
    """Closed form of the Brent-Kung composition count for L' = 2^m."""
    return 2 * (Lp - 1) - int(math.log2(Lp))


def bk_stages(Lp: int) -> int:
    """Closed form of the Brent-Kung stage count for L' = 2^m >= 2."""
    return 2 * int(math.log2(Lp)) - 1


def _drop(ct, level):
    return ct[:level]


def compose(P: C.Params, left: tuple, right: tuple, rlk) -> tuple:
    """T_right o T_left (Eq. "compact_affine_compose") at the lower of the two
    levels; the result is one level lower."""
    aL, sL = left
    aR, sR = right
    lvl = min(aL.shape[0], aR.shape[0])
    aL, sL, aR, sR = (_drop(x, lvl) for x in (aL, sL, aR, sR))
    a = C.mul_relin_rescale(P, aR, aL, rlk)
    s = C.ct_add(P, C.mul_relin_rescale(P, aR, sL, rlk), _drop(sR, lvl - 1))
    return a, s


def apply_to_state(P: C.Params, prefix: tuple, carry_s, rlk):
    """s part of prefix o G for a carry G with state part carry_s: the state
    prefix(G(0)) = a_P * s_G + s_P."""
    aP, sP = prefix
    lvl = min(aP.shape[0], carry_s.shape[0])
    prod = C.mul_relin_rescale(P, _drop(aP, lvl), _drop(carry_s, lvl), rlk)
    return C.ct_add(P, prod, _drop(sP, lvl - 1))


def resident_schedule(items: list, block: int, op, state, inject) -> list:
    """Two-pass resident schedule over `items` with blocks of `block` tokens
    (Eq. "resident-block-schedule"): pass 1 keeps the summary S_j (last local
    prefix) of every block but the last, an exclusive scan over the summaries
    gives the carries G_j, and pass 2 replays each block's local prefixes
    P_{j,t}.  state(P) is the state of block 0's prefixes; inject(P, G) that of
    the corrected prefix P o G.  Returns one state per item."""
    L = len(items)
    K = -(-L // block)
    blocks = [items[j * block:(j + 1) * block] for j in range(K)]
    summaries = [brent_kung(blocks[j], op)[0][-1] for j in range(K - 1)]
    carries = brent_kung(summaries, op)[0]  # carries[j-1] = G_j
    out = []
    for j in range(K):
        for pre in brent_kung(blocks[j], op)[0]:
            out.append(state(pre) if j == 0 else inject(pre, carries[j - 1]))
    return out


def _to_one_level(cts: list) -> list:
    lvl = min(c.shape[0] for c in cts)
    return [c[:lvl].copy() for c in cts]


def affine_scan(P: C.Params, a: list, s: list, rlk) -> tuple[list, list]:
    """Inclusive encrypted scan of one chunk's tuples (a_k, s_k), all at one
    level.  Returns the prefixes (A_k, S_k) at one common level; S_k = h_k."""
    pre, _, _ = brent_kung(list(zip(a, s)), lambda l, r: compose(P, l, r, rlk))
    lvl = min(x.shape[0] for x, _ in pre)
    return [x[:lvl].copy() for x, _ in pre], [y[:lvl].copy() for _, y in pre]


def resident_scan(P: C.Params, a: list, s: list, block: int, rlk) -> list:
    """States h_k of one chunk by the resident schedule, at one common level."""
    states = resident_schedule(list(zip(a, s)), block, lambda l, r: compose(P, l, r, rlk),
                               lambda pre: pre[1],
                               lambda pre, g: apply_to_state(P, pre, g[1], rlk))
    return _to_one_level(states)


def hescan(P: C.Params, x: list, B: list, a: list, cfac: list, rlk, keys: dict, d_s: int,
           block: int | None = None, contract: tuple | None = None) -> list:
    """HEScan of one sequence over K state chunks (Sec. "On-Demand
    Construction and Contraction", Eqs. "fesc_recurrence", "fesc_contract" and
    "hescan-contract-output").  x, B, a, cfac: [K][L] ciphertexts, broadcast
    into each chunk's packing; x and B at one level l, a at >= l - 1 limbs,
    cfac at >= the states' level.  Per chunk: the update s_k = RS(relin(x_k B_k))
    (level l - 1), the states h_k by the Brent-Kung scan (block None) or the
    resident schedule, at one common level; then per token the contraction
    (the scan-contract slice without the decay product).  Returns per token
    the slice's outputs.

    contract = (P_c, rlk_c, keys_c) runs the contraction under another
    parameter set whose ciphertext chain begins with the states' primes (the
    same residues then denote the same ciphertexts), typically with fewer
    special primes, so that its key switches work over a smaller extended
    basis; the contraction's arithmetic is otherwise unchanged."""
    from . import workloads as W
    K, L = len(x), len(x[0])
    H = []
    for k in range(K):
        s = [C.mul_relin_rescale(P, x[k][t], B[k][t], rlk) for t in range(L)]
        lvl = s[0].shape[0]
        ak = [_drop(a[k][t], lvl) for t in range(L)]
        H.append(affine_scan(P, ak, s, rlk)[1] if block is None
                 else resident_scan(P, ak, s, block, rlk))
    Pc, rlk_c, keys_c = contract if contract is not None else (P, rlk, keys)
    if contract is not None:
        lvl = max(H[0][0].shape[0], cfac[0][0].shape[0])
        assert list(Pc.q[:lvl]) == list(P.q[:lvl]), "contraction chain must extend the states'"
    return [W.scan_contract_token(Pc, [H[k][t] for k in range(K)], None,
                                  [cfac[k][t] for k in range(K)], rlk_c, keys_c, d_s)
            for t in range(L)]

