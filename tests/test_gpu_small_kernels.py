"""GPU parity of the small kernels on the same primitives against the oracle
(every residue): HEConv (hoisted taps, fused accumulation, rescale with the
bias), the fused post-SSM path and the plaintext (conversion-mask) add.  A
small ring, and HEConv and the post-SSM path at N = 2^16 with the projection's
packing (32 channel segments of 1024 token slots, 16 limbs)."""
import numpy as np
import pytest
import torch

import synth
from oracle import ckks as C
from oracle import workloads as OW
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_dev, to_host
from tests.test_gpu_ckks import Setup
from tests.test_oracle_workloads import conv_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def _eq(dev, want, what):
    got = to_host(dev)[: want.size].reshape(want.shape)
    assert np.array_equal(got, want), f"{what}: {first_mismatch(got, want)}"


def _pt(P, vals, scale, level):
    pt = C.encode_plain(P, np.asarray(vals, dtype=complex), scale, level)
    return pt, to_dev(pt)


def _heconv(P, seed, T, d_conv, level, with_bias):
    deltas = [-r for r in range(d_conv)]
    S = Setup(P, seed, rot_steps=deltas)
    qv, w, b, masks = conv_inputs(P, T, d_conv, seed)
    ql = float(P.q[level - 1])
    q_o, q_d = S.encrypt(qv.reshape(-1), 2.0 ** 40, level, 1)
    pts = [_pt(P, m, ql, level) for m in masks]
    bias = _pt(P, np.repeat(b, T), 2.0 ** 40, level) if with_bias else (None, None)
    out = torch.zeros((level - 1) * 2 * P.n, dtype=torch.int64, device="cuda")
    step(f"heconv N={P.n} taps={d_conv} level={level}")
    S.ctx.heconv(q_d, deltas, [d for _, d in pts], bias[1], out, level)
    want = OW.heconv(P, q_o, deltas, [o for o, _ in pts], bias[0], S.keys)
    _eq(out, want, "heconv")


@pytest.mark.parametrize("with_bias,level", [(True, 3), (False, 3), (True, 2)])
def test_heconv_small(with_bias, level):
    _heconv(C.params_small(12, 50, 4, 2), 61, 64, 4, level, with_bias)


def test_heconv_full_size():
    _heconv(C.params_p16(24), 62, 1024, 4, 16, True)


def _post_ssm(P, seed, level):
    S = Setup(P, seed, relin=True)
    n_slots = P.n // 2
    mv = synth.normal(seed, "ps-m", n_slots)
    xv = synth.normal(seed, "ps-x", n_slots)
    dv = synth.normal(seed, "ps-D", n_slots)
    gv = synth.uniform_pm1(seed, "ps-g", n_slots)
    m = S.encrypt(mv, 2.0 ** 40, level, 1)
    x = S.encrypt(xv, 2.0 ** 40, level, 2)
    g = S.encrypt(gv, float(P.q[level - 2]), level, 3)
    D = _pt(P, dv, float(P.q[level - 1]), level)
    out = torch.zeros((level - 2) * 2 * P.n, dtype=torch.int64, device="cuda")
    step(f"post_ssm N={P.n} level={level}")
    S.ctx.post_ssm(m[1], x[1], D[1], g[1], out, level)
    want = OW.post_ssm(P, m[0], x[0], D[0], g[0], S.keys[0])
    _eq(out, want, "post_ssm")


@pytest.mark.parametrize("level", [4, 3])
def test_post_ssm_small(level):
    _post_ssm(C.params_small(12, 50, 5, 2), 63, level)


def test_post_ssm_full_size():
    _post_ssm(C.params_p16(24), 64, 16)


def test_add_plain_is_the_conversion_mask():
    P = C.params_small(12, 50, 3, 1)
    S = Setup(P, 65)
    level = 2
    ct_o, ct_d = S.encrypt(synth.normal(65, "c2m", P.n // 2), 2.0 ** 40, level, 1)
    rhat = synth.uniform_residues(65, "rhat", P.qs(level), P.n)
    out = torch.zeros(level * 2 * P.n, dtype=torch.int64, device="cuda")
    step("add_plain")
    S.ctx.add_plain(ct_d, to_dev(rhat), out, level)
    _eq(out, OW.c2m_mask(P, ct_o, rhat), "mask add")
    S.ctx.add_plain(ct_d, to_dev(rhat), ct_d, level)      # in place
    _eq(ct_d, OW.c2m_mask(P, ct_o, rhat), "mask add in place")
