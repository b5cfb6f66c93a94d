"""GPU parity of the scan-contract slice against the oracle: a small ring with
five chunks, blocks of tokens, one full-size Mamba-2-base token (N = 2^16,
12 state chunks of 128 channels x d_state 128, level 20 -> 18), also run as a
16-token block of copies that must all equal it, and the benchmark's pool of
16 distinct tokens in one call (tokens 0, 7 and 15 compared)."""
import numpy as np
import pytest
import torch

import synth
import synth.workloads as WL
from oracle import ckks as C
from oracle import workloads as OW
from tests.gpu_helpers import first_mismatch, need_gpu, step, to_host
from tests.test_gpu_ckks import Setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    need_gpu()


def chunk_slots(z, cvec, H, K, n_slots, d_s, head_dim, s_state=None):
    """Slot vectors of the state-chunk packing: chunk k holds channels
    [k*c, (k+1)*c), c = s_state / d_s, channel e at slots (e - k*c)*d_s + i;
    slots from s_state on are zero.  Returns per chunk (h, decay, C)."""
    s_state = s_state or n_slots
    c_state = s_state // d_s
    j = np.arange(n_slots)
    out = []
    decay = 1.0 / (1.0 + np.exp(z))          # exp(-softplus(z))
    for k in range(K):
        e = k * c_state + j // d_s
        i = j % d_s
        ok = (e < H.shape[0]) & (j < s_state)
        hv = np.where(ok, H[np.minimum(e, H.shape[0] - 1), i], 0.0)
        dv = np.where(ok, decay[np.minimum(e, H.shape[0] - 1) // head_dim], 0.0)
        cv = np.where(ok, cvec[i], 0.0)
        out.append((hv, dv, cv))
    return out


def _run(P, S, chunks, level, d_s, tag, block=0):
    hs_o, ds_o, cs_o, hs_d, ds_d, cs_d = [], [], [], [], [], []
    for k, (hv, dv, cv) in enumerate(chunks):
        for vals, scale, lo, ld, role in [(hv, 2.0 ** 40, hs_o, hs_d, 0),
                                          (dv, float(P.q[level - 1]), ds_o, ds_d, 1),
                                          (cv, float(P.q[level - 2]), cs_o, cs_d, 2)]:
            co, cd = S.encrypt(vals.astype(complex), scale, level, 10 * k + role)
            lo.append(co)
            ld.append(cd)
    outs_d = [torch.zeros((level - 2) * 2 * P.n, dtype=torch.int64, device="cuda")
              for _ in chunks]
    step(f"scan_contract {tag} chunks={len(chunks)}")
    S.ctx.scan_contract(hs_d, ds_d, cs_d, d_s, outs_d, level)
    outs_o = OW.scan_contract_token(P, hs_o, ds_o, cs_o, S.keys[0], S.keys, d_s)
    for k, (od, oo) in enumerate(zip(outs_d, outs_o)):
        got = to_host(od).reshape(oo.shape)
        assert np.array_equal(got, oo), f"{tag} output {k}: {first_mismatch(got, oo)}"
    if block:
        # the launch configuration of a token block: `block` tokens per call
        # (copies of this token's inputs), every token equal to the one above
        K = len(chunks)
        outs_b = [torch.zeros((level - 2) * 2 * P.n, dtype=torch.int64, device="cuda")
                  for _ in range(K * block)]
        step(f"scan_contract {tag} block of {block} tokens")
        S.ctx.scan_contract(hs_d * block, ds_d * block, cs_d * block, d_s, outs_b, level,
                            tokens=block)
        for u in range(block):
            for k in range(K):
                got = to_host(outs_b[u * K + k]).reshape(outs_o[k].shape)
                assert np.array_equal(got, outs_o[k]), \
                    f"{tag} block token {u} output {k}: {first_mismatch(got, outs_o[k])}"
    return outs_o


def test_scan_contract_small():
    P = C.params_small(12, 50, 5, 2)
    d_s, head_dim, K, level = 8, 16, 5, 4       # odd K exercises the lone last chunk
    n_slots = P.n // 2
    S = Setup(P, 31, rot_steps=[1, 2, 4], relin=True, conj=True)
    E = K * (n_slots // d_s) - 40               # ragged: last chunk partly empty
    z = synth.normal(31, "z", -(-E // head_dim))
    cvec = synth.normal(31, "C", d_s)
    H = synth.normal(31, "h", (E, d_s))
    outs = _run(P, S, chunk_slots(z, cvec, H, K, n_slots, d_s, head_dim), level, d_s, "small")
    decay = 1.0 / (1.0 + np.exp(z))
    want = (decay[np.arange(E) // head_dim][:, None] * H * cvec[None, :]).sum(axis=1)
    c_state = n_slots // d_s
    for l in range(K // 2):
        for half in range(2):
            k = 2 * l + half
            dec = C.decrypt(P, S.sk, outs[k], 2.0 * 2.0 ** 40).real[::d_s]
            ref = np.zeros(c_state)
            seg = want[k * c_state:(k + 1) * c_state]
            ref[:len(seg)] = seg
            assert np.max(np.abs(dec - ref)) <= 2.0 ** -15


def test_cfg5_one_token_full_size():
    P = C.params_p16(24)
    cfg = WL.CFG5
    d_s, head_dim, level = cfg["d_state"], cfg["head_dim"], cfg["level"]
    n_slots = P.n // 2
    s_state = 16384
    K = cfg["heads"] * head_dim * d_s // s_state          # 12 chunks
    steps = [d_s >> k for k in range(1, 8)]               # 64 .. 1
    S = Setup(P, cfg["seed"], rot_steps=steps, relin=True, conj=True)
    z, cvec, H = WL.cfg5_token(0)
    chunks = chunk_slots(z, cvec, H, K, n_slots, d_s, head_dim, s_state)
    outs = _run(P, S, chunks, level, d_s, "cfg5", block=cfg["pool"])
    decay = 1.0 / (1.0 + np.exp(z))
    want = (decay[np.arange(H.shape[0]) // head_dim][:, None] * H * cvec[None, :]).sum(axis=1)
    c_state = s_state // d_s
    for k in [0, 1, K - 1]:
        dec = C.decrypt(P, S.sk, outs[k], 2.0 * 2.0 ** 40).real[:s_state:d_s]
        err = np.max(np.abs(dec - want[k * c_state:(k + 1) * c_state]))
        print(f"cfg5 chunk {k}: max |decoded - fp64| = {err:.3e}")
        assert err <= 2.0 ** -15


def test_cfg5_pool_of_distinct_tokens():
    """The benchmark's launch configuration with its real inputs: the 16
    distinct tokens of the cfg5 pool (N = 2^16, 12 state chunks, level
    20 -> 18) in ONE fesc_scan_contract call, token-major.  Tokens 0, 7 and 15
    are compared with the oracle's one-token slice on every residue of all 12
    chunk outputs, so a token-index mix-up in the batched products, the
    rotation batches over all tokens or the pairing kernel would show."""
    P = C.params_p16(24)
    cfg = WL.CFG5
    d_s, head_dim, level, T = cfg["d_state"], cfg["head_dim"], cfg["level"], cfg["pool"]
    n_slots, s_state = P.n // 2, 16384
    K = cfg["heads"] * head_dim * d_s // s_state
    S = Setup(P, cfg["seed"], rot_steps=[d_s >> k for k in range(1, 8)], relin=True, conj=True)
    check = (0, 7, T - 1)
    dev = ([], [], [])
    orc = {u: ([], [], []) for u in check}
    for u in range(T):
        z, cvec, H = WL.cfg5_token(u)
        for k, vals in enumerate(chunk_slots(z, cvec, H, K, n_slots, d_s, head_dim, s_state)):
            scales = (2.0 ** 40, float(P.q[level - 1]), float(P.q[level - 2]))
            for r in range(3):
                co, cd = S.encrypt(vals[r].astype(complex), scales[r], level,
                                   9000 + 3 * (u * K + k) + r, oracle=u in check)
                dev[r].append(cd)
                if u in check:
                    orc[u][r].append(co)
    outs = [torch.zeros((level - 2) * 2 * P.n, dtype=torch.int64, device="cuda")
            for _ in range(K * T)]
    step(f"scan_contract cfg5 pool: {T} distinct tokens x {K} chunks")
    S.ctx.scan_contract(dev[0], dev[1], dev[2], d_s, outs, level, tokens=T)
    torch.cuda.synchronize()
    for u in check:
        want = OW.scan_contract_token(P, *orc[u], S.keys[0], S.keys, d_s)
        for k in range(K):
            got = to_host(outs[u * K + k]).reshape(want[k].shape)
            assert np.array_equal(got, want[k]), \
                f"pool token {u} chunk {k}: {first_mismatch(got, want[k])}"


@pytest.mark.parametrize("K,T", [(4, 3), (5, 2), (2, 17), (2, 65)])
def test_scan_contract_token_block(K, T):
    """Several tokens per call (the reduction batched over all of them, the
    outputs used as its workspace): every token equals the oracle's
    one-token slice.  K = 2, T = 17 puts 17 pairs in each rotation batch;
    T = 65 crosses the 64-pair batches of the pairing kernel."""
    P = C.params_small(12, 50, 5, 2)
    d_s, head_dim, level = 8, 16, 4
    n_slots = P.n // 2
    S = Setup(P, 37, rot_steps=[1, 2, 4], relin=True, conj=True)
    E = K * (n_slots // d_s)
    hs_o, ds_o, cs_o, hs_d, ds_d, cs_d = [], [], [], [], [], []
    for u in range(T):
        z = synth.normal(37 + u, "z", -(-E // head_dim))
        cvec = synth.normal(37 + u, "C", d_s)
        H = synth.normal(37 + u, "h", (E, d_s))
        for k, (hv, dv, cv) in enumerate(chunk_slots(z, cvec, H, K, n_slots, d_s, head_dim)):
            i = 3 * (u * K + k)
            for vals, scale, lo, ld, j in [(hv, 2.0 ** 40, hs_o, hs_d, 0),
                                           (dv, float(P.q[level - 1]), ds_o, ds_d, 1),
                                           (cv, float(P.q[level - 2]), cs_o, cs_d, 2)]:
                co, cd = S.encrypt(vals.astype(complex), scale, level, 5000 + i + j)
                lo.append(co)
                ld.append(cd)
    outs_d = [torch.zeros((level - 2) * 2 * P.n, dtype=torch.int64, device="cuda")
              for _ in range(K * T)]
    step(f"scan_contract token block K={K} T={T}")
    S.ctx.scan_contract(hs_d, ds_d, cs_d, d_s, outs_d, level, tokens=T)
    for u in range(T):
        sl = slice(u * K, (u + 1) * K)
        want = OW.scan_contract_token(P, hs_o[sl], ds_o[sl], cs_o[sl], S.keys[0], S.keys, d_s)
        for k, (od, oo) in enumerate(zip(outs_d[sl], want)):
            got = to_host(od).reshape(oo.shape)
            assert np.array_equal(got, oo), f"token {u} output {k}: {first_mismatch(got, oo)}"
