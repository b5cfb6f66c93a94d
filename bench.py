"""Benchmark of the RNS-CKKS linear hot path on one MI355X.

Workload (the metric's headline configuration): batched negacyclic NTT at
N = 2^16 over 24 limbs of ~50-bit primes = 1 mod 2N, 64 polynomials with
uniform residues, forward then inverse, and the limb-wise modular Hadamard
multiply-accumulate of 64 pairs (seed 1).

One step = forward NTT of A (64 x 24 x 2^16), 64-pair MAC with B, inverse NTT.
NTT GB/s = 2 * 8 * N * limbs * batch / t per direction (one read and one
write of the data; twiddles excluded), over the forward + inverse time.

Prints ONE JSON line.  --gpus > 1 is refused (single-GPU build).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "keyswitch/s + NTT GB/s at N=2^16, 24 limbs; encrypted 768×1536 matvec ms"
HBM_PEAK_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(n_polys: int = 8):
    """The CPU reference timed on a bounded sample of the same workload:
    forward + inverse NTT of n_polys x 24 limbs at N = 2^16."""
    import numpy as np

    import synth.workloads as WL
    from oracle import ckks as C

    P = C.params_p16()
    mods = P.q
    A = WL.cfg2_polys("A", mods, P.n, n_polys).reshape(-1, P.n)
    rows = mods * n_polys
    t0 = time.perf_counter()
    f = C.ntt(P, A, rows)
    C.intt(P, f, rows)
    dt = time.perf_counter() - t0
    gbs = 2 * (2 * 8 * P.n * len(rows)) / dt / 1e9
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(gbs, 3), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"forward+inverse NTT of {n_polys} polys x 24 limbs at N=2^16 "
                      f"({2 * len(rows)} limb transforms, {dt:.2f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (no multi-GPU path); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth.workloads as WL
    from paper_2608_17442_amd import fesc as F

    torch.cuda.set_device(0)
    log_n, limbs, batch = WL.CFG2["log_n"], WL.CFG2["limbs"], WL.CFG2["batch"]
    n = 1 << log_n
    primes = F.find_primes(log_n, 50, 8 + limbs)
    ctx = F.Context(log_n, primes[8:], primes[:8])
    mods = primes[8:]
    log("generating inputs")
    A = torch.from_numpy(WL.cfg2_polys("A", mods, n, batch).view(np.int64)).cuda()
    B = torch.from_numpy(WL.cfg2_polys("B", mods, n, batch).view(np.int64)).cuda()
    M = torch.zeros(limbs * n, dtype=torch.int64, device="cuda")
    stride = limbs * n

    def step(ev=None):
        if ev:
            ev[0].record()
        ctx.ntt_fwd(A, batch, stride, limbs, n, 0)
        if ev:
            ev[1].record()
        ctx.mac(A, B, M, batch, stride, limbs, 0)
        if ev:
            ev[2].record()
        ctx.ntt_inv(A, batch, stride, limbs, n, 0)
        if ev:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd = np.mean([e[0].elapsed_time(e[1]) for e in evs])
    mac = np.mean([e[1].elapsed_time(e[2]) for e in evs])
    inv = np.mean([e[2].elapsed_time(e[3]) for e in evs])
    rows = limbs * batch
    bytes_dir = 2 * 8 * n * rows
    ntt_gbs = 2 * bytes_dir / ((fwd + inv) * 1e-3) / 1e9
    mac_bytes = 2 * 8 * n * rows + 8 * n * limbs
    ms_per_step = wall / args.steps * 1e3
    out = {
        "metric": METRIC,
        "value": round(ntt_gbs, 2),
        "unit": "GB/s (NTT, N=2^16, 24 limbs)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64 residues, fp64 modular arithmetic",
        "data": "synthetic (uniform residues, seed 1)",
        "config": {"workload": "NTT microbench: 64 polys x 24 limbs x N=2^16, forward + "
                               "inverse, then 64-pair limb-wise modular MAC",
                   "log_n": log_n, "limbs": limbs, "batch": batch, "parallelism": "single GPU"},
        "components": {
            "ntt_fwd_ms": round(fwd, 4), "ntt_inv_ms": round(inv, 4),
            "mac_ms": round(mac, 4),
            "mac_gbs": round(mac_bytes / (mac * 1e-3) / 1e9, 2),
        },
        "roofline": {
            "bound": "hbm", "kernel": "forward NTT (outer + inner pass)",
            "achieved": round(bytes_dir / (fwd * 1e-3) / 1e9, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(bytes_dir / (fwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": None,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU reference sample")
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
