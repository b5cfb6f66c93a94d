"""Seeded raw draws of the five benchmark workloads (no CKKS arithmetic).

cfg1  N=2^12 diagonal matvec:     U (64x64) and x (64) ~ U[-1,1], seed 0.
cfg2  NTT microbench:             64 polynomials x 24 limbs of uniform
                                  residues (A) and 64 more (B), seed 1.
cfg3  rotation / key switch:      32 slot vectors ~ U[-1,1], seed 2.
cfg4  768x1536 projection:        X (1024x768) ~ N(0,1), W ~ N(0, 0.02^2),
                                  seed 3.
cfg5  scan-contract slice:        decay logits z ~ N(0,1) per head, C ~ N(0,1)
                                  per state index, states h ~ N(0,1), seed 4.
"""
from __future__ import annotations

import numpy as np

from . import normal, uniform_pm1, uniform_residues

CFG1 = dict(seed=0, log_n=12, dim=64)
CFG2 = dict(seed=1, log_n=16, limbs=24, batch=64)
CFG3 = dict(seed=2, log_n=16, limbs=24, count=32, scale_bits=40)
CFG4 = dict(seed=3, log_n=16, tokens=1024, d_in=768, d_out=1536, level=16, n1=16, n2=2)
CFG5 = dict(seed=4, log_n=16, L=2048, heads=24, head_dim=64, d_state=128, chunk=256,
            level=20, pool=16)


def cfg1_values():
    s = CFG1["seed"]
    return uniform_pm1(s, "cfg1-U", (CFG1["dim"], CFG1["dim"])), uniform_pm1(s, "cfg1-x",
                                                                             CFG1["dim"])


def cfg2_polys(tag: str, moduli, n: int, batch: int, seed: int = CFG2["seed"]) -> np.ndarray:
    """u64[batch][len(moduli)][n] uniform residues; tag 'A' or 'B'."""
    out = np.empty((batch, len(moduli), n), dtype=np.uint64)
    for b in range(batch):
        out[b] = uniform_residues(seed, "cfg2-" + tag, moduli, n, b)
    return out


def cfg3_slots(i: int, n_slots: int) -> np.ndarray:
    return uniform_pm1(CFG3["seed"], "cfg3-z", n_slots, i)


def cfg3_steps() -> list:
    """Ciphertext i rotates left by 2^(i mod 16)."""
    return [1 << (i % 16) for i in range(CFG3["count"])]


def cfg4_values():
    s = CFG4["seed"]
    X = normal(s, "cfg4-X", (CFG4["tokens"], CFG4["d_in"]))
    W = normal(s, "cfg4-W", (CFG4["d_in"], CFG4["d_out"]), 0.02)
    return X, W


def cfg5_token(k: int):
    """Raw values of pool token k: decay logits z[heads], C[d_state],
    states h[heads*head_dim][d_state]."""
    s = CFG5["seed"]
    z = normal(s, "cfg5-z", CFG5["heads"], 1.0, k)
    c = normal(s, "cfg5-C", CFG5["d_state"], 1.0, k)
    h = normal(s, "cfg5-h", (CFG5["heads"] * CFG5["head_dim"], CFG5["d_state"]), 1.0, k)
    return z, c, h
