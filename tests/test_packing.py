"""CPU checks of the library's host-side slot packing (paper_2608_17442_amd.
packing) against the oracle's definitions: the token-major input blocks and
the generalised BSGS diagonals of the projection (Sec. 4.1 packing), on the
full 768 x 1536 shape and on a ragged one."""
import numpy as np
import pytest

import synth
from oracle import workloads as OW
from paper_2608_17442_amd import packing as PK


@pytest.mark.parametrize("T,d_in,d_out,n_slots,seg,n1", [(1024, 768, 1536, 32768, 1024, 16),
                                                         (50, 70, 40, 2048, 64, 4)])
def test_packing_matches_oracle(T, d_in, d_out, n_slots, seg, n1):
    Cc = n_slots // seg
    X = synth.normal(7, "pk-X", (T, d_in))
    W = synth.normal(7, "pk-W", (d_in, d_out), 0.02)
    n_in, n_out = -(-d_in // Cc // 2), -(-d_out // Cc)
    n2 = -(-Cc // n1)
    for u in range(n_in):
        want = OW.pack_input(X, n_slots, seg, Cc, 2 * u) + 1j * OW.pack_input(X, n_slots, seg, Cc,
                                                                               2 * u + 1)
        assert np.array_equal(PK.paired_input(X, u, n_slots, seg, Cc), want)
    rng = np.random.default_rng(0)
    for _ in range(12):
        b, p, u, q = (int(rng.integers(n_out)), int(rng.integers(n2)), int(rng.integers(n_in)),
                      int(rng.integers(n1)))
        want = OW.bsgs_diagonal_slots(W, n_slots, seg, Cc, n1, b, p, u, q, True)
        got = PK.diagonal_slots(W, b, p, u, q, n1, n_slots, seg, Cc, True)
        assert np.array_equal(got, want), (b, p, u, q)
