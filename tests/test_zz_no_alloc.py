"""The rotation batch that allocates nothing (fesc_rotate_batch_noalloc)
against the batch that uses the context's scratch (fesc_rotate_batch): equal
residue for residue on two calls in a row, the second with a smaller input,
on a small ring (one group of up to 32 rotations), with seed-expanded keys,
and at N = 2^16 with 24 limbs (two rotations per group of the 256 MiB static
array), and the oracle confirms one output.  A level whose single rotation exceeds the array is
refused before any launch."""
import numpy as np
import pytest
import torch

from oracle import ckks as C
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_host
from tests.test_gpu_ckks import Setup, _z

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _both(S, cts, steps, level, tag):
    """Run the batch through both entry points; return the no-alloc outputs."""
    outs_a = [torch.full_like(c, -1) for c in cts]
    outs_b = [torch.full_like(c, -1) for c in cts]
    step(f"{tag}: rotate_batch (context scratch), {len(cts)} ciphertexts at level {level}")
    S.ctx.rotate_batch(cts, steps, outs_a, level)
    step(f"{tag}: rotate_batch_noalloc (static scratch)")
    S.ctx.rotate_batch_noalloc(cts, steps, outs_b, level)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(outs_a, outs_b)):
        assert torch.equal(a, b), f"{tag} item {i}: " + first_mismatch(
            to_host(b), to_host(a))
    return outs_b


def test_rotate_batch_noalloc_small_ring_two_calls():
    from paper_2608_17442_amd.fesc import CONJ
    P = C.params_small(13, 45, 4, 3)
    base = [1, 2, -3, 5, 0]
    S = Setup(P, 18, rot_steps=base, conj=True)
    # first call: 37 rotations at the top level (two groups of 32)
    level = P.L
    cts = [S.encrypt(_z(500 + i, P.n // 2), 2.0 ** 30, level, 500 + i) for i in range(37)]
    steps = [base[i % len(base)] if i % 7 else CONJ for i in range(37)]
    outs = _both(S, [d for _, d in cts], steps, level, "small call 1")
    want = C.rotate(P, cts[1][0], steps[1], S.keys)
    got = to_host(outs[1]).reshape(want.shape)
    assert np.array_equal(got, want), first_mismatch(got, want)
    # second call: fewer, smaller ciphertexts (level 2); the array keeps the
    # first call's contents, which nothing reads
    cts2 = [S.encrypt(_z(600 + i, P.n // 2), 2.0 ** 30, 2, 600 + i) for i in range(5)]
    outs2 = _both(S, [d for _, d in cts2], [1, CONJ, -3, 0, 2], 2, "small call 2")
    want = C.conjugate(P, cts2[1][0], S.keys)
    got = to_host(outs2[1]).reshape(want.shape)
    assert np.array_equal(got, want), first_mismatch(got, want)


def test_rotate_batch_noalloc_full_size_two_calls():
    P = C.params_p16()
    steps = [1, 32, 4096]
    S = Setup(P, 19, rot_steps=steps)
    cts = [S.encrypt(_z(700 + i, P.n // 2), 2.0 ** 40, 24, 700 + i) for i in range(3)]
    outs = _both(S, [d for _, d in cts], steps, 24, "full size call 1")
    want = C.rotate(P, cts[2][0], steps[2], S.keys)
    got = to_host(outs[2]).reshape(want.shape)
    assert np.array_equal(got, want), first_mismatch(got, want)
    cts2 = [S.encrypt(_z(800 + i, P.n // 2), 2.0 ** 40, 16, 800 + i) for i in range(2)]
    _both(S, [d for _, d in cts2], [32, 1], 16, "full size call 2")


def test_rotate_batch_noalloc_with_seed_expanded_keys():
    """The same comparison with seed-expanded keys (the inner product
    regenerates each key's uniform half in the static scratch's key
    switches as well), two calls, the oracle confirming one output."""
    from tests.test_gpu_seeded_keys import SeededSetup
    P = C.params_small(12, 50, 5, 2)
    base = [1, 3, -2]
    S = SeededSetup(P, 20, [P.galois_elt(r) for r in base])
    level = P.L
    cts = [S.encrypt(_z(900 + i, P.n // 2), 2.0 ** 30, level, 900 + i) for i in range(6)]
    steps = [base[i % len(base)] for i in range(6)]
    outs = _both(S, [d for _, d in cts], steps, level, "seeded call 1")
    want = C.rotate(P, cts[4][0], steps[4], S.keys)
    got = to_host(outs[4]).reshape(want.shape)
    assert np.array_equal(got, want), first_mismatch(got, want)
    cts2 = [S.encrypt(_z(950 + i, P.n // 2), 2.0 ** 30, 3, 950 + i) for i in range(2)]
    _both(S, [d for _, d in cts2], [3, -2], 3, "seeded call 2")


def test_rotate_batch_noalloc_refuses_a_level_beyond_the_array():
    """N = 2^16 with 60 ciphertext primes and 4 special primes: one rotation
    at level 60 needs 634 MiB (> 256 MiB) and is refused before any launch;
    level 8 fits."""
    from paper_2608_17442_amd import fesc as F
    pr = F.find_primes(16, 50, 64)
    ctx = F.Context(16, pr[4:], pr[:4])
    ct = torch.zeros(60 * 2 * ctx.n, dtype=torch.int64, device="cuda")
    out = torch.zeros_like(ct)
    with pytest.raises(F.FescError) as e:
        ctx.rotate_batch_noalloc([ct], [1], [out], 60)
    assert e.value.code == -1 and "static scratch" in str(e.value)
    with pytest.raises(F.FescError) as e:       # fits; no key loaded
        ctx.rotate_batch_noalloc([ct[: 8 * 2 * ctx.n]], [1], [out[: 8 * 2 * ctx.n]], 8)
    assert e.value.code == -3
    assert torch.count_nonzero(out).item() == 0
