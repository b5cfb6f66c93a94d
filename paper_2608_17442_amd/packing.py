"""Offline preparation of projection inputs (host side, numpy): the segment
packing of an activation block and the slot vectors of the BSGS plaintext
diagonals (paper Appendix "Projection Kernel Breakdown").

Slots are viewed as segments, slot j = s * seg_len + r; the projection
Y = X W packs X[r, g*C + c] at segment c of input block g.  For output block b
and diagonal t the weights W[g*C + (c + t) mod C, b*C + c] fill segment c
(constant over its positions r).  With complex pairing an input ciphertext
carries blocks (2u, 2u+1) as real and imaginary parts, and its diagonal
carries (w_2u - i w_{2u+1}) / 2, so that the real part of the product is the
paired sum.  A giant step p pre-rotates the diagonal right by p*n1 segments.
These vectors are then encoded (fesc_encode) and transformed on the device.
"""
from __future__ import annotations

import numpy as np


def segment_of_slot(n_slots: int, seg_len: int, C: int):
    """(position r, segment c) of every slot; segments repeat with period C."""
    j = np.arange(n_slots)
    return j % seg_len, (j // seg_len) % C


def input_block(X: np.ndarray, g: int, n_slots: int, seg_len: int, C: int) -> np.ndarray:
    r, c = segment_of_slot(n_slots, seg_len, C)
    col = g * C + c
    keep = (r < X.shape[0]) & (col < X.shape[1])
    v = np.zeros(n_slots)
    v[keep] = X[r[keep], col[keep]]
    return v


def paired_input(X, u, n_slots, seg_len, C) -> np.ndarray:
    return input_block(X, 2 * u, n_slots, seg_len, C) + 1j * input_block(X, 2 * u + 1, n_slots,
                                                                         seg_len, C)


def _weight_diagonal(W, g, b, t, n_slots, seg_len, C) -> np.ndarray:
    _, c = segment_of_slot(n_slots, seg_len, C)
    row, col = g * C + (c + t) % C, b * C + c
    keep = (row < W.shape[0]) & (col < W.shape[1])
    v = np.zeros(n_slots)
    v[keep] = W[row[keep], col[keep]]
    return v


def diagonal_slots(W, b, p, u, q, n1, n_slots, seg_len, C, paired: bool) -> np.ndarray:
    """Slot vector of D~[b][p][u][q]."""
    t = p * n1 + q
    if paired:
        v = 0.5 * (_weight_diagonal(W, 2 * u, b, t, n_slots, seg_len, C)
                   - 1j * _weight_diagonal(W, 2 * u + 1, b, t, n_slots, seg_len, C))
    else:
        v = _weight_diagonal(W, u, b, t, n_slots, seg_len, C).astype(np.complex128)
    return np.roll(v, p * n1 * seg_len)
