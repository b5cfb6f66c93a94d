"""Benchmark of the RNS-CKKS linear hot path on one MI355X.

Metric (three workloads, all N = 2^16 with ~50-bit primes = 1 mod 2N; the
8 largest are the special primes, the next 24 the ciphertext primes):

  NTT    64 polynomials x 24 limbs of uniform residues (seed 1): forward
         NTT, 64-pair limb-wise modular multiply-accumulate, inverse NTT.
         NTT GB/s = 2 * 8 * N * limbs * batch / t per direction (one read and
         one write of the data; twiddles excluded) over forward + inverse.
  KS     32 fresh ciphertexts at 24 limbs (dnum 3, 8 special primes), U[-1,1]
         slots at scale 2^40, ciphertext i rotated left by 2^(i mod 16)
         (seed 2): 30 key switches + 2 identity copies.  keyswitch/s = 30 / t.
  MATVEC 768 x 1536 plaintext weight (N(0, 0.02^2)) times 1024 tokens x 768
         features (N(0,1)) packed as 12 complex-paired ciphertexts at 16 limbs,
         BSGS n1 = 16, n2 = 2 over 32 segments of 1024 slots, complex-paired
         outputs and rescale -> 24 ciphertexts carrying the 48 output blocks
         (seed 3); 18,432 pre-encoded diagonals resident in HBM (a 120.8 GB
         bank: 50 bits per residue).

  SCAN   scan-contract slice of a block of 16 distinct Mamba-base tokens (24
         heads x 64 channels x d_state 128 in 12 state chunks of 16,384 slots,
         level 20 -> 18, seed 4): products with decay and C, rotate-and-add
         over d_state, complex-paired conjugation split, every step batched
         over the block.  After the steps the whole 2048-token sequence (the
         16-token pool cycled, 128 calls) is timed as
         `components.scan_contract_sequence`.

One step runs all four.  `value` is the NTT GB/s (the headline
configuration); keyswitch/s, matvec ms and scan-contract ms are reported in
`components`.  After the steps, the HEScan affine prefix scan (Brent-Kung,
128 tokens x 12 state chunks at 16 limbs, uniform residues: the arithmetic
is data-oblivious) is timed on its own as `components.affine_scan`, and one
whole HEScan layer at the paper's long-sequence shape (L = 2048, 12 state
chunks, 23 limbs in: update construction, scan, contraction of every token;
full-length and two-pass schedules) as `components.hescan_layer`; then the
broadcasts br^(kappa) of one token's factors from their compact packings
(homomorphic slot maps) as `components.broadcast`.
Other modes: --affine-only, --scan-sweep (resident block sizes at L = 2048),
--hescan-sweep (the HEScan layer at L = 128 .. 2048).
Prints ONE JSON line on stdout.  --gpus > 1 is refused (single-GPU build).
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


# HBM traffic of the roofline kernel (k_ptmac) per launch, from the committed
# rocprofv3 FETCH_SIZE / WRITE_SIZE summary; valid only while the kernel's
# sources are byte-identical to those the counters were taken on.
PTMAC_PROFILE = os.path.join(ROOT, "profiles", "k_ptmac_projection_768x1536_n65536_l16.txt")
PTMAC_SOURCES = [os.path.join(ROOT, "paper_2608_17442_amd", "csrc", f)
                 for f in ("matvec.hip", "fesc_internal.hpp")]


def kernel_sources_sha256(paths) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# Per-kernel roofline of the key switch (each kernel's time at its own binding
# resource, HBM from the rocprofv3 counters or VALU from its work and the
# calibrated rates), from the committed profile of the rotation set; valid
# only while the pipeline's sources are unchanged.
KS_PROFILE = os.path.join(ROOT, "profiles", "keyswitch_rotation_set_n65536_l24_dnum3.txt")
KS_SOURCES = [os.path.join(ROOT, "paper_2608_17442_amd", "csrc", f)
              for f in ("ntt.hip", "keyswitch.hip", "butterfly.hpp", "fesc_internal.hpp",
                        "ops.cpp", "ops.hpp", "scratch.hpp")]


def profiled_fields(profile: str, sources) -> dict | None:
    """The '# key: value' lines of `profile`, or None if the file is missing
    or the kernel sources changed since it was taken."""
    if not os.path.exists(profile):
        return None
    fields = {}
    for line in open(profile):
        if ":" in line and line.startswith("# ") and not line.startswith("#   "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_sources_sha256") != kernel_sources_sha256(sources):
        return None
    return fields


def profiled_traffic(profile: str, sources) -> int | None:
    """Bytes per launch recorded in `profile`, or None if the file is missing
    or the kernel sources changed since the counters were taken."""
    fields = profiled_fields(profile, sources)
    if fields is None:
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# --------------------------------------------------------------- workloads

def keygen_into(W, ctx, elt, seed, moduli, dnum):
    """Switching key of `elt` in `ctx` from the synthetic draws: seed-expanded
    (W.seeded_keys) or stored."""
    if W.seeded_keys:
        w, e = W.synth.switch_key_seed_draws(seed, moduli, W.n, dnum, elt)
        ctx.keygen_seeded(elt, W.s_dev, w, W.dev(e))
    else:
        a, e = W.synth.switch_key_draws(seed, moduli, W.n, dnum, elt)
        ctx.keygen(elt, W.s_dev, W.dev(a), W.dev(e))


class Workloads:
    def __init__(self, F, torch, np, skip_matvec=False, affine_only=False, seeded_keys=True):
        import synth
        import synth.workloads as WL
        self.F, self.torch, self.np, self.WL, self.synth = F, torch, np, WL, synth
        self.log_n = 16
        self.n = 1 << 16
        primes = F.find_primes(self.log_n, 50, 32)
        self.q, self.p = primes[8:], primes[:8]
        self.alpha = len(self.p)
        self.ks_level = 24
        self.ctx = F.Context(self.log_n, self.q, self.p)
        self.s = synth.secret(WL.CFG3["seed"], self.n)
        self.s_dev = torch.from_numpy(self.s).cuda()
        self._keys = set()
        # switching keys seed-expanded (the context keeps the seed and the b
        # half; the key switch regenerates the uniform half) unless asked
        # for stored keys
        self.seeded_keys = seeded_keys
        if affine_only:
            return
        self.setup_ntt()
        self.setup_ks()
        self.skip_matvec = skip_matvec
        if not skip_matvec:
            self.setup_matvec()
        self.setup_scan_contract()

    def dev(self, a):
        a = self.np.ascontiguousarray(a)
        if a.dtype == self.np.uint64:
            a = a.view(self.np.int64)
        return self.torch.from_numpy(a).cuda()

    def keygen(self, elt, seed):
        if elt in self._keys:
            return
        keygen_into(self, self.ctx, elt, seed, self.q + self.p, 3)
        self._keys.add(elt)

    def encrypt(self, z, scale, level, seed, tag, idx):
        m = self.F.encode(self.log_n, z, scale)
        a, e = self.synth.encrypt_draws(seed, self.q[:level], self.n, tag, idx)
        ct = self.torch.empty(level * 2 * self.n, dtype=self.torch.int64, device="cuda")
        self.ctx.encrypt_sk(self.s_dev, self.dev(m), self.dev(a), self.dev(e), ct, level)
        return ct

    # ---- NTT + MAC
    def setup_ntt(self):
        WL, n = self.WL, self.n
        log("NTT inputs")
        self.batch, self.limbs = WL.CFG2["batch"], WL.CFG2["limbs"]
        self.A = self.dev(WL.cfg2_polys("A", self.q, n, self.batch))
        self.B = self.dev(WL.cfg2_polys("B", self.q, n, self.batch))
        self.M = self.torch.zeros(self.limbs * n, dtype=self.torch.int64, device="cuda")

    def run_ntt(self, ev):
        n, b, l = self.n, self.batch, self.limbs
        ev[0].record()
        self.ctx.ntt_fwd(self.A, b, l * n, l, n, 0)
        ev[1].record()
        self.ctx.mac(self.A, self.B, self.M, b, l * n, l, 0)
        ev[2].record()
        self.ctx.ntt_inv(self.A, b, l * n, l, n, 0)
        ev[3].record()

    # ---- rotations / key switching
    def setup_ks(self):
        WL = self.WL
        seed = WL.CFG3["seed"]
        self.ks_steps = WL.cfg3_steps()
        log("rotation keys and ciphertexts")
        for st in sorted(set(self.ks_steps)):
            g = self.ctx.galois_element(st)
            if g != 1:
                self.keygen(g, seed)
        self.ks_in = [self.encrypt(WL.cfg3_slots(i, self.n // 2), 2.0 ** 40, 24, seed, "cfg3", i)
                      for i in range(len(self.ks_steps))]
        self.ks_out = [self.torch.empty_like(c) for c in self.ks_in]
        self.n_ks = sum(1 for st in self.ks_steps if st % (self.n // 2))

    def run_ks(self, ev):
        ev[0].record()
        self.ctx.rotate_batch(self.ks_in, self.ks_steps, self.ks_out, 24)
        ev[1].record()

    # ---- BSGS projection
    def setup_matvec(self):
        from paper_2608_17442_amd import packing as PK
        np, torch, WL = self.np, self.torch, self.WL
        cfg = WL.CFG4
        seed, level = cfg["seed"], cfg["level"]
        n_slots, seg, Cc = self.n // 2, cfg["tokens"], (self.n // 2) // cfg["tokens"]
        n1, n2 = cfg["n1"], cfg["n2"]
        n_in, n_out = cfg["d_in"] // Cc // 2, cfg["d_out"] // Cc
        self.mv_level = level
        log("projection keys")
        for q in list(range(1, n1)) + [p * n1 for p in range(1, n2)]:
            self.keygen(self.ctx.galois_element(q * seg), seed)
        self.keygen(2 * self.n - 1, seed)
        X, W = WL.cfg4_values()
        self.mv_in = [self.encrypt(PK.paired_input(X, u, n_slots, seg, Cc), 2.0 ** 40, level,
                                   seed, "cfg4", u) for u in range(n_in)]
        # complex-paired outputs: 48 diagonal sets, output blocks (2P, 2P+1)
        # leave as the real and imaginary parts of output ciphertext P
        n_diag = n_out * n2 * n_in * n1
        desc = self.F.matvec_desc(level, n_in, n_out, n1, n2, seg, False, True, True)
        self.bank_bytes = 8 * self.F.matvec_bank_words(self.ctx, desc)
        log(f"encoding {n_diag} diagonals ({self.bank_bytes / 1e9:.1f} GB bank)")
        self.bank = torch.empty(self.bank_bytes // 8, dtype=torch.int64, device="cuda")
        scale = float(self.q[level - 1])
        # slot values, encoding, lift, NTT and packing all on the device
        t0 = time.perf_counter()
        chunk = 128
        Wd = torch.from_numpy(np.ascontiguousarray(W)).cuda()
        zs = torch.empty((chunk, n_slots), dtype=torch.complex128, device="cuda")
        pts = torch.empty((chunk, level * self.n), dtype=torch.int64, device="cuda")
        for c0 in range(0, n_diag, chunk):
            m = min(chunk, n_diag - c0)
            self.F.bsgs_diagonal_slots(self.ctx, desc, Wd, Cc, c0, m, zs)
            self.ctx.encode_plain(zs[:m], scale, pts[:m], level)
            self.F.matvec_bank_pack_many(self.ctx, desc, self.bank, c0, pts[:m])
        torch.cuda.synchronize()
        del Wd, zs, pts
        self.bank_build_s = time.perf_counter() - t0
        log(f"diagonals ready in {self.bank_build_s:.1f} s (all on the device)")
        self.mv_plan = self.F.MatvecPlan(self.ctx, level, n_in, n_out, n1, n2, seg, False, True,
                                         bank=self.bank, complex_pair=True)
        self.mv_out = [torch.empty((level - 1) * 2 * self.n, dtype=torch.int64, device="cuda")
                       for _ in range(n_out // 2)]
        self.mv_shape = dict(n_in=n_in, n_out=n_out, n1=n1, n2=n2, n_diag=n_diag)

    def run_matvec(self, ev):
        ev[0].record()
        self.mv_plan(self.mv_in, self.mv_out)
        ev[1].record()

    # ---- scan-contract slice: a block of 16 Mamba-base tokens, 12 state chunks each
    def setup_scan_contract(self):
        np, WL = self.np, self.WL
        cfg = WL.CFG5
        seed, level, d_s, hd = cfg["seed"], cfg["level"], cfg["d_state"], cfg["head_dim"]
        n_slots, s_state = self.n // 2, 16384
        log("scan-contract keys and ciphertexts")
        for st in [d_s >> k for k in range(1, 8)]:
            self.keygen(self.ctx.galois_element(st), seed)
        self.keygen(2 * self.n - 1, seed)
        self.keygen(0, seed)
        K = cfg["heads"] * hd * d_s // s_state
        c_state = s_state // d_s
        j = np.arange(n_slots)
        T = cfg["pool"]
        # a pool of 16 distinct tokens (token k of the sequence uses entry k mod 16),
        # token-major: index u*K + k
        self.sc_in = ([], [], [])
        for u in range(T):
            z, cvec, H = WL.cfg5_token(u)
            decay = 1.0 / (1.0 + np.exp(z))
            for k in range(K):
                # chunk k: channel e = k c_state + j // d_s at slots (j // d_s) d_s + j % d_s
                e, i = k * c_state + j // d_s, j % d_s
                ok = j < s_state
                e = np.minimum(e, H.shape[0] - 1)
                vals = (np.where(ok, H[e, i], 0.0), np.where(ok, decay[e // hd], 0.0),
                        np.where(ok, cvec[i], 0.0))
                scales = (2.0 ** 40, float(self.q[level - 1]), float(self.q[level - 2]))
                for r in range(3):
                    self.sc_in[r].append(self.encrypt(vals[r].astype(complex), scales[r], level,
                                                      seed, "cfg5", 3 * (u * K + k) + r))
        # two output sets: tokens 0-15 kept, the rest of a sequence to a ring
        self.sc_out = [[self.torch.empty((level - 2) * 2 * self.n, dtype=self.torch.int64,
                                         device="cuda") for _ in range(K * T)] for _ in range(2)]
        self.sc_shape = dict(chunks=K, tokens=T, d_state=d_s, level=level)

    def run_scan_contract(self, ev, ring=0):
        ev and ev[0].record()
        h, dec, cf_ = self.sc_in
        self.ctx.scan_contract(h, dec, cf_, self.sc_shape["d_state"], self.sc_out[ring],
                               self.sc_shape["level"], tokens=self.sc_shape["tokens"])
        ev and ev[1].record()

    def time_scan_contract_sequence(self):
        """The slice over a whole cfg5 sequence (2048 tokens: 128 calls over the
        16-token pool, outputs of tokens 0-15 kept, the rest to a ring)."""
        torch = self.torch
        L, T = self.WL.CFG5["L"], self.sc_shape["tokens"]
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for b in range(L // T):
            self.run_scan_contract(None, ring=min(b, 1))
        ev[1].record()
        torch.cuda.synchronize()
        t = ev[0].elapsed_time(ev[1]) / 1e3
        ks = L * (2 * self.sc_shape["chunks"] + (self.sc_shape["chunks"] // 2)
                  * (self.sc_shape["d_state"].bit_length() - 1 + 1))
        return {"tokens": L, "tokens_per_call": T, "s": round(t, 3),
                "ms_per_token": round(t * 1e3 / L, 3), "key_switches": ks,
                "keyswitch_per_s": round(ks / t, 1)}

    # ---- affine prefix scan (HEScan): Brent-Kung over 128 tokens x 12 chunks
    def setup_affine(self, L=128, chunks=12, level=16):
        torch = self.torch
        self.keygen(0, self.WL.CFG5["seed"])
        words = level * 2 * self.n
        log(f"affine-scan inputs ({2 * L * chunks * words * 8 / 1e9:.1f} GB)")
        # residues below 2^49 are valid for every prime here (all exceed 2^49);
        # the modular arithmetic is data-oblivious, so timing needs no encryption
        self.af_buf = torch.randint(0, 1 << 49, (2 * L * chunks, words), dtype=torch.int64,
                                    device="cuda")
        self.af_a = [self.af_buf[i] for i in range(L * chunks)]
        self.af_s = [self.af_buf[L * chunks + i] for i in range(L * chunks)]
        self.af_shape = dict(L=L, chunks=chunks, level=level)

    def run_affine(self, ev):
        sh = self.af_shape
        ev[0].record()
        lo = self.ctx.affine_scan(self.af_a, self.af_s, sh["chunks"], sh["level"],
                                  states_only=True)
        ev[1].record()
        return lo


def time_hescan(W, F, torch, np, L=2048, block=1024, level=23, chunks=12, d_s=128, pool=64,
                low_q=4, low_alpha=2):
    """One HEScan layer at the paper's long-sequence shape (L tokens, `chunks`
    state chunks of 128 channels x d_state 128, N = 2^16), chunk pair by chunk
    pair (2l, 2l+1): the on-demand update construction s = RS(relin(x B)) from
    `level` (23 limbs, the paper's chain of 23 ciphertext primes), the scan of
    the states from level - 1, and the contraction of every token
    (RS(relin(h C)), complex-paired rotate-and-add over d_state, one
    conjugation), in two schedules:
      full_length: the whole sequence as one Brent-Kung network, in place and
        states only, both chunks of the pair in one launch sequence;
      two_pass: the resident schedule with blocks of `block` tokens, one chunk
        at a time (the paper's schedule on a 40 GB device).
    Ciphertexts are uniform residues (the arithmetic is data-oblivious): x, a
    and C per (token, chunk) of the pair, B from a pool of `pool` (B is as
    large as x: holding both for 4,096 tuples next to a would exceed HBM);
    every pair reuses the buffers; one warm-up pair per schedule.
    The contraction runs in a second context over the chain prefix
    q_0..q_{low_q - 1} with the first `low_alpha` special primes: the states'
    buffers are valid there as they are (same primes, same layout), and its
    key switches at levels 2-3 work over 4-5 extended rows instead of 10-11.
    States above level low_q (short sequences, less scan depth) are
    contracted in the layer's own context."""
    for name in ("af_buf", "af_a", "af_s"):
        if hasattr(W, name):
            delattr(W, name)
    torch.cuda.empty_cache()
    seed = W.WL.CFG5["seed"]
    W.keygen(0, seed)
    for st in [d_s >> k for k in range(1, d_s.bit_length())]:
        W.keygen(W.ctx.galois_element(st), seed)
    W.keygen(2 * W.n - 1, seed)
    ctx, n = W.ctx, W.n
    # contraction context: chain prefix, fewer special primes, its own keys
    lq, lp = W.q[:low_q], W.p[:low_alpha]
    cctx = F.Context(W.log_n, lq, lp)
    for g in [0, 2 * n - 1] + [ctx.galois_element(d_s >> k) for k in range(1, d_s.bit_length())]:
        keygen_into(W, cctx, g, seed, lq + lp, -(-low_q // low_alpha))
    words = lambda lvl: lvl * 2 * n
    rnd = lambda rows, lvl: torch.randint(0, 1 << 49, (rows, words(lvl)), dtype=torch.int64,
                                          device="cuda")
    ev = lambda: torch.cuda.Event(enable_timing=True)
    out = {"tokens": L, "chunks": chunks, "d_state": d_s, "level_in": level,
           "paper_context": "HEScan 284.2 s/layer on one A100-40GB at this shape (two-pass, "
                            "blocks of 1024, chain of 23 ciphertext primes; construction, scan "
                            "and contraction; 372K key switches)",
           "contraction_context": {"ciphertext_primes": low_q, "special_primes": low_alpha,
                                   "note": "chain prefix q_0..q_%d of the layer's context "
                                           "(8 special primes), own keys" % (low_q - 1)}}
    pairs = chunks // 2
    red_ks = L * (d_s.bit_length() - 1) + L            # rotations + conjugations per pair

    def span(spans, key, fn):
        a, b = ev(), ev()
        a.record()
        fn()
        b.record()
        spans.append((key, a, b))

    def run(one_pair):
        one_pair([])                                    # warm-up
        torch.cuda.synchronize()
        spans = []
        for _ in range(pairs):
            one_pair(spans)
        torch.cuda.synchronize()
        r = {k: 0.0 for k in ("construct_s", "scan_s", "contract_s")}
        for k, a, b in spans:
            r[k] += a.elapsed_time(b) / 1e3
        r = {k: round(v, 3) for k, v in r.items()}
        r["s_per_layer"] = round(spans[0][1].elapsed_time(spans[-1][2]) / 1e3, 3)
        return r

    tm = lambda v, K: [v[k * L + t] for t in range(L) for k in range(K)]

    def ks_rates(r, layer_ks, contract_ks, prefix):
        """Key switches per context: construction and scan run in the layer's
        context (l + 8 extended rows); the contraction's run in the prefix
        context (l + 2 rows) when the states' level allows it, so their rates
        are reported apart (a combined rate would mix two key-switch sizes)."""
        d = {"key_switches": layer_ks + contract_ks,
             "layer_context": {"key_switches": layer_ks,
                               "keyswitch_per_s": round(
                                   layer_ks / (r["construct_s"] + r["scan_s"]), 1)},
             "contraction": {"key_switches": contract_ks,
                             "keyswitch_per_s": round(contract_ks / r["contract_s"], 1),
                             "context": "prefix context" if prefix else "layer context"}}
        if not prefix:
            d["keyswitch_per_s"] = round((layer_ks + contract_ks) / r["s_per_layer"], 1)
        return d
    # full length: both chunks of a pair in place
    lo, ks = ctx.affine_scan_info(L, level - 1, states_only=True)
    gb = (2 * L * (2 * level - 1 + 2 * lo - 1) + pool * level) * 16 * n / 1e9
    log(f"HEScan layer, full length: {gb:.1f} GB of ciphertexts")
    X, A, Cc, O, Bp = rnd(2 * L, level), rnd(2 * L, level - 1), rnd(2 * L, lo), \
        rnd(2 * L, lo - 1), rnd(pool, level)
    xs, as_, cs, os_ = list(X), list(A), list(Cc), list(O)
    bs = [Bp[i % pool] for i in range(2 * L)]

    def full_pair(spans):
        span(spans, "construct_s", lambda: ctx.mul_relin_rescale(xs, bs, xs, level))
        span(spans, "scan_s", lambda: ctx.affine_scan(as_, xs, 2, level - 1, states_only=True))
        span(spans, "contract_s", lambda: cc.scan_contract(tm(xs, 2), None, tm(cs, 2), d_s,
                                                           tm(os_, 2), lo, tokens=L))
    cc = cctx if lo <= low_q else ctx
    r = run(full_pair)
    r.update({"level_states": lo, "level_out": lo - 1})
    r.update(ks_rates(r, pairs * (2 * L + 2 * ks), pairs * (2 * L + red_ks), cc is cctx))
    out["full_length"] = r
    del X, A, Cc, O, Bp, xs, as_, cs, os_, bs
    torch.cuda.empty_cache()
    # two-pass resident schedule: one chunk at a time, the pair contracted together
    lo, ws_bytes, ks = ctx.affine_scan_resident_info(L, 1, block, level - 1)
    log(f"HEScan layer, two-pass: workspace {ws_bytes / 1e9:.1f} GB")
    X, A, H, Cc, O, Bp = rnd(L, level), rnd(L, level - 1), rnd(2 * L, lo), rnd(2 * L, lo), \
        rnd(2 * L, lo - 1), rnd(pool, level)
    ws = torch.empty(ws_bytes // 8 + 1, dtype=torch.int64, device="cuda")
    xs, as_, hs, cs, os_ = list(X), list(A), list(H), list(Cc), list(O)
    bs = [Bp[i % pool] for i in range(L)]

    def two_pass_pair(spans):
        for c in range(2):
            span(spans, "construct_s", lambda: ctx.mul_relin_rescale(xs, bs, xs, level))
            span(spans, "scan_s", lambda: ctx.affine_scan_resident(
                as_, xs, 1, block, hs[c * L:(c + 1) * L], level - 1, ws))
        span(spans, "contract_s", lambda: cc.scan_contract(tm(hs, 2), None, tm(cs, 2), d_s,
                                                           tm(os_, 2), lo, tokens=L))
    cc = cctx if lo <= low_q else ctx
    r = run(two_pass_pair)
    r.update({"block": block, "level_states": lo, "level_out": lo - 1})
    r.update(ks_rates(r, pairs * (2 * L + 2 * ks), pairs * (2 * L + red_ks), cc is cctx))
    out["two_pass"] = r
    del X, A, H, Cc, O, Bp, ws, xs, as_, hs, cs, os_, bs
    torch.cuda.empty_cache()
    return out


def scan_block_sweep(W, F, torch, np, L=2048, level=22, blocks=(64, 128, 256, 512, 1024, 2048)):
    """Resident-schedule block sizes at L tokens, one state chunk, inputs at
    `level` (the paper's sweep at L = 2048): output level (the depth the
    schedule needs), key switches, resident bytes and time per chunk.  A block
    of L is the full-length network (in place, states only)."""
    W.keygen(0, W.WL.CFG5["seed"])
    ctx, n = W.ctx, W.n
    words = level * 2 * n
    buf = torch.randint(0, 1 << 49, (2 * L, words), dtype=torch.int64, device="cuda")
    a = [buf[i] for i in range(L)]
    s = [buf[L + i] for i in range(L)]
    rows = []
    for B in blocks:
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        if B >= L:
            lo, ks = ctx.affine_scan_info(L, level, states_only=True)
            ctx.affine_scan(a, s, 1, level, states_only=True)          # warm-up
            torch.cuda.synchronize()
            ev[0].record()
            ctx.affine_scan(a, s, 1, level, states_only=True)
            ev[1].record()
            resident = 2 * L * words * 8
        else:
            lo, ws_bytes, ks = ctx.affine_scan_resident_info(L, 1, B, level)
            hb = torch.empty((L, lo * 2 * n), dtype=torch.int64, device="cuda")
            h = [hb[i] for i in range(L)]
            ws = torch.empty(ws_bytes // 8 + 1, dtype=torch.int64, device="cuda")
            ctx.affine_scan_resident(a, s, 1, B, h, level, ws)
            torch.cuda.synchronize()
            ev[0].record()
            ctx.affine_scan_resident(a, s, 1, B, h, level, ws)
            ev[1].record()
            resident = 2 * L * words * 8 + ws_bytes + L * lo * 2 * n * 8
        torch.cuda.synchronize()
        rows.append({"block": B, "level_out": lo, "depth": level - lo, "key_switches": ks,
                     "resident_gb": round(resident / 1e9, 1),
                     "ms_per_chunk": round(ev[0].elapsed_time(ev[1]), 1)})
        log(f"block {B}: {rows[-1]}")
        if B < L:
            del hb, h, ws
            torch.cuda.empty_cache()
    del buf, a, s
    torch.cuda.empty_cache()
    return {"tokens": L, "level_in": level, "chunk": "one state chunk (N=2^16, 12 per layer)",
            "rows": rows}


def modmul_probe(ctx, F) -> dict:
    """The residue product alone, fp64 (the library's form) against 64-bit
    integer Shoup, on every CU with no memory traffic (products per second)."""
    f = ctx.calib_valu(F.CALIB_MODMUL_F64)
    u = ctx.calib_valu(F.CALIB_MODMUL_U64)
    ph = ctx.calib_valu(F.CALIB_PHILOX, 1 << 12)
    return {"fp64_shoup_per_s": round(f, -9), "u64_shoup_per_s": round(u, -9),
            "fp64_over_u64": round(f / u, 2),
            "philox4x64_blocks_per_s": round(ph, -8),
            "kernels": "k_calib_modmul_f64 / k_calib_modmul_u64 / k_calib_philox "
                       "(fesc_calib_valu)"}


def matvec_double_hoisting(F, torch, np) -> dict:
    """The projection with and without double hoisting (lazy ModDown), timed
    on the diagonal-method workload (N = 2^12, 64 x 64, 63 hoisted rotations)
    and on the 768 x 1536 shape (N = 2^16, 16 limbs, complex-paired outputs,
    diagonal bank).  The modular arithmetic does not depend on the values, so
    the inputs are uniform residues and the banks random words (values below
    2^50); the two 2^16 banks (120.8 and 181.2 GB at 50 bits per residue) are
    built one after the other."""
    import synth
    import synth.workloads as WL

    def timed(plan, ins, outs, reps):
        plan(ins, outs)
        torch.cuda.synchronize()
        ts, ph = [], []
        for _ in range(reps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            plan(ins, outs)
            ev[1].record()
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
            ph.append(plan.phase_ms())
        med = lambda v: round(float(np.median(v)), 3)
        return {"ms": med(ts), "baby_ms": med([x[0] for x in ph]),
                "pt_mac_ms": med([x[1] for x in ph]), "tail_ms": med([x[2] for x in ph])}

    out = {}
    # diagonal method, N = 2^12
    pr = F.find_primes(12, 36, 4)
    q, p = pr[1:4], pr[0:1]
    n = 1 << 12
    ctx = F.Context(12, q, p)
    sd = torch.from_numpy(synth.secret(0, n)).cuda()
    for r in range(1, 64):
        g = ctx.galois_element(r)
        w, e = synth.switch_key_seed_draws(0, q + p, n, 3, g)
        ctx.keygen_seeded(g, sd, w, torch.from_numpy(e).cuda())
    ins = [torch.randint(0, 1 << 35, (3 * 2 * n,), dtype=torch.int64, device="cuda")]
    outs = [torch.empty(2 * 2 * n, dtype=torch.int64, device="cuda")]
    res = {}
    for lazy in (False, True):
        diags = [torch.randint(0, 1 << 35, ((3 + int(lazy)) * n,), dtype=torch.int64,
                               device="cuda") for _ in range(64)]
        plan = F.MatvecPlan(ctx, 3, 1, 1, 64, 1, 1, False, True, diags=diags,
                            lazy_moddown=lazy)
        res["double_hoisted" if lazy else "plain"] = timed(plan, ins, outs, 20)
        plan.close()
    out["n4096_64x64_diagonal_method"] = res
    del ctx
    # 768 x 1536, N = 2^16
    pr = F.find_primes(16, 50, 32)
    q, p = pr[8:], pr[:8]
    n = 1 << 16
    ctx = F.Context(16, q, p)
    cfg = WL.CFG4
    level, seg, n1, n2 = cfg["level"], cfg["tokens"], cfg["n1"], cfg["n2"]
    Cc = (n // 2) // seg
    n_in, n_out = cfg["d_in"] // Cc // 2, cfg["d_out"] // Cc
    sd = torch.from_numpy(synth.secret(3, n)).cuda()
    steps = [k * seg for k in range(1, n1)] + [k * n1 * seg for k in range(1, n2)]
    for g in sorted({ctx.galois_element(st) for st in steps} | {2 * n - 1}):
        w, e = synth.switch_key_seed_draws(3, q + p, n, 3, g)
        ctx.keygen_seeded(g, sd, w, torch.from_numpy(e).cuda())
    ins = [torch.randint(0, 1 << 49, (level * 2 * n,), dtype=torch.int64, device="cuda")
           for _ in range(n_in)]
    outs = [torch.empty((level - 1) * 2 * n, dtype=torch.int64, device="cuda")
            for _ in range(n_out // 2)]
    res = {}
    for lazy in (False, True):
        desc = F.matvec_desc(level, n_in, n_out, n1, n2, seg, False, True, True, lazy)
        words = F.matvec_bank_words(ctx, desc)
        bank = torch.empty(words, dtype=torch.int64, device="cuda")
        for o in range(0, words, 1 << 30):
            bank[o:o + (1 << 30)].random_(0, 1 << 49)
        plan = F.MatvecPlan(ctx, level, n_in, n_out, n1, n2, seg, False, True, bank=bank,
                            complex_pair=True, lazy_moddown=lazy)
        r = timed(plan, ins, outs, 5)
        r["bank_gb"] = round(words * 8 / 1e9, 1)
        res["double_hoisted" if lazy else "plain"] = r
        plan.close()
        del plan, bank
        torch.cuda.empty_cache()
    out["n65536_768x1536_complex_paired"] = res
    return out


def keyswitch_per_kernel():
    f = profiled_fields(KS_PROFILE, KS_SOURCES)
    if f is None or "keyswitch_bound_fraction" not in f:
        return None
    return {"bound": "hbm or alu per kernel",
            "frac": float(f["keyswitch_bound_fraction"].split()[0]),
            "source": os.path.relpath(KS_PROFILE, ROOT),
            "note": "sum over the key switch's kernels of max(HBM bytes / 8 TB/s, VALU work / "
                    "calibrated VALU rate), over the sum of their measured times"}


def time_affine(W, F, torch, np):
    """HEScan affine prefix scan: one warm-up, mean of two timed runs (in
    place; the arithmetic is data-oblivious, so reruns are timed alike)."""
    W.setup_affine()
    ev = lambda: [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    W.run_affine(ev())
    torch.cuda.synchronize()
    aev = [ev() for _ in range(2)]
    lo = [W.run_affine(e) for e in aev]
    torch.cuda.synchronize()
    af_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in aev]))
    sh = W.af_shape
    Lp, m = sh["L"], sh["L"].bit_length() - 1
    n_paper = 2 * sh["chunks"] * (2 * (Lp - 1) - m)     # two per composition node
    n_ks = sh["chunks"] * W.ctx.affine_scan_info(sh["L"], sh["level"], states_only=True)[1]
    return {"tokens": sh["L"], "chunks": sh["chunks"], "level_in": sh["level"],
            "level_out": lo[-1], "ms": round(af_ms, 2), "key_switches": n_ks,
            "key_switches_all_nodes": n_paper,
            "keyswitch_per_s": round(n_ks / (af_ms * 1e-3), 1),
            "network": "Brent-Kung, in place, states only (dead decay products skipped), "
                       "stages batched over chunks"}


def time_broadcast(W, F, torch, np, level=24, k=3, kappa=7, reps=3, batch=16):
    """The broadcasts br^(kappa) of one token's factors from their compact
    packings (Mamba-2 base: 24 heads of 64 channels, d_s = 128, 128 channels
    per chunk, one group), input level 24 -> 23, as homomorphic slot maps.
    Masks are generated and encoded on the device beforehand (offline, not
    timed); one warm-up, then the mean of `reps` runs (HIP events).  B and C
    share one map.  Each map is also timed over a block of `batch` tokens in
    one call (batched_ms_per_token)."""
    shape = dict(H=24, P=64, G=1, d_s=128, c_state=128)
    n, ns, seed = W.n, W.n // 2, 97
    z = W.synth.normal(seed, "br-re", ns) + 1j * W.synth.normal(seed, "br-im", ns)
    ct = W.encrypt(z, 2.0 ** 40, level, seed, "br", 0)
    ql = float(W.q[level - 1])
    res = {}
    for kind in ("x", "a", "B"):
        d = F.br_desc(W.log_n, shape["H"], shape["P"], shape["G"], shape["d_s"],
                      shape["c_state"], kind, k, kappa, level)
        n2 = d.n2
        steps = {d.offset} | {q * d.stride for q in range(1, d.n1)} | \
            {p * d.giant_stride for p in range(1, n2)}
        r = 1
        while r < d.rep_count:
            steps.add(-r * d.rep_stride)
            r *= 2
        for st in steps:
            g = W.ctx.galois_element(st % ns)
            if g != 1:
                W.keygen(g, seed)
        cnt = d.n1 * n2
        zs = torch.empty((cnt, ns), dtype=torch.complex128, device="cuda")
        pts = torch.empty(cnt * level * n, dtype=torch.int64, device="cuda")
        F.slot_map_mask_slots(W.ctx, d, 0, cnt, zs)
        W.ctx.encode_plain(zs, ql, pts, level)
        plan = F.SlotMapPlan(W.ctx, d, [pts[t * level * n:(t + 1) * level * n]
                                        for t in range(d.terms)])
        out = torch.empty((level - 1) * 2 * n, dtype=torch.int64, device="cuda")
        plan(ct, out)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            plan(ct, out)
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        n_ks = int(d.offset % ns != 0) + (d.n1 - 1) + (n2 - 1) + (d.rep_count.bit_length() - 1)
        res[kind] = {"ms": round(ms, 3), "key_switches": n_ks, "terms": d.terms, "n1": d.n1,
                     "n2": n2, "copies": d.rep_count}
        # the same map for a block of tokens 0 .. batch-1 of the chunk under one
        # plan (fesc_slot_map_batch), each with its own first rotation
        offs = [F.br_desc(W.log_n, shape["H"], shape["P"], shape["G"], shape["d_s"],
                          shape["c_state"], kind, kt, kappa, level).offset
                for kt in range(batch)]
        for st in offs:
            g = W.ctx.galois_element(st % ns)
            if g != 1:
                W.keygen(g, seed)
        outs = [torch.empty((level - 1) * 2 * n, dtype=torch.int64, device="cuda")
                for _ in range(batch)]
        plan.batch([ct] * batch, offs, outs)
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            plan.batch([ct] * batch, offs, outs)
        ev[1].record()
        torch.cuda.synchronize()
        res[kind]["batched_ms_per_token"] = round(ev[0].elapsed_time(ev[1]) / reps / batch, 3)
        del outs
        plan.close()
        del zs, pts
    L, K = 2048, 12
    layer_ms = L * K * (res["x"]["ms"] + res["a"]["ms"]) + 2 * L * res["B"]["ms"]
    layer_ms_b = L * K * (res["x"]["batched_ms_per_token"] + res["a"]["batched_ms_per_token"]) \
        + 2 * L * res["B"]["batched_ms_per_token"]
    return {"token": k, "chunk": kappa, "level_in": level, "maps": res,
            "layer_s_if_homomorphic": round(layer_ms / 1e3, 1),
            "layer_s_if_homomorphic_batched": round(layer_ms_b / 1e3, 1),
            "batch_tokens": batch,
            "layer_key_switches_if_homomorphic":
                L * K * (res["x"]["key_switches"] + res["a"]["key_switches"])
                + 2 * L * res["B"]["key_switches"],
            "note": "per layer (2048 tokens, 12 chunks): x and a per token and chunk, B and C "
                    "per token (one group: the same map for every chunk)"}


# ---------------------------------------------------------------- baseline

def _omp_threads() -> int:
    """Threads the oracle's OpenMP loops use in this process."""
    import ctypes
    try:
        return int(ctypes.CDLL("libgomp.so.1").omp_get_max_threads())
    except OSError:
        return int(os.environ.get("OMP_NUM_THREADS", "1"))


def cpu_sample(mode: str) -> dict:
    """The oracle (CPU reference, as it stands) on bounded samples of every
    configuration, in this process's OpenMP thread count.  mode "all": the
    all-core samples; "single": smaller samples for one thread.  Inputs,
    keys and diagonals are prepared outside the timed regions; every timed
    region runs the oracle's operations in the order the workload issues
    them.  Each entry gives the sample, its seconds, the factor that scales it
    to the whole configuration and the extrapolated seconds.  The modular
    arithmetic does not depend on the values, so the projection's sampled
    blocks multiply uniform random plaintexts in place of encoded diagonals,
    and the affine-scan-style inputs are not needed."""
    import numpy as np

    import synth
    import synth.workloads as WL
    from oracle import ckks as C
    from oracle import workloads as OW

    single = mode == "single"
    res = {"threads": _omp_threads()}
    tick = time.perf_counter

    def entry(sample, t, factor):
        return {"sample": sample, "sample_s": round(t, 3), "factor": factor,
                "extrapolated_s": round(t * factor, 3)}

    # cfg1: N = 2^12 diagonal matvec, in full on either thread count
    P = C.params_p12()
    U, x = WL.cfg1_values()
    d, ns = WL.CFG1["dim"], P.n // 2
    sk = C.secret_key(P, synth.secret(WL.CFG1["seed"], P.n))
    keys = {P.galois_elt(r): C.keygen_from_seed(P, sk, WL.CFG1["seed"], P.galois_elt(r))
            for r in range(1, d)}
    a, e = synth.encrypt_draws(WL.CFG1["seed"], P.qs(3), P.n, "cfg1", 0)
    ct = C.encrypt(P, sk, C.encode_plain(P, np.tile(x, ns // d), float(P.q[2]), 3), 3, a, e)
    desc = OW.MatvecDesc(3, 1, 1, d, 1, 1, False, True)
    dg = {q: C.encode_plain(P, OW.bsgs_diagonal_slots(U.T, ns, 1, d, d, 0, 0, 0, q, False),
                            2.0 ** 30, 3) for q in range(d)}
    t0 = tick()
    OW.bsgs_matvec(P, desc, [ct], lambda b, p_, u, q: dg[q], keys)
    res["cfg1"] = entry("the whole N=2^12 diagonal matvec (63 hoisted rotations, 64 ptmul, "
                        "rescale)", tick() - t0, 1)

    P = C.params_p16()
    n = P.n
    # cfg2: forward NTT, 64-pair MAC, inverse NTT of the 64 x 24 x 2^16 batch
    B = WL.CFG2["batch"]
    nb = 4 if single else 16
    A = WL.cfg2_polys("A", P.q, n, nb).reshape(-1, n)
    Bm = WL.cfg2_polys("B", P.q, n, nb).reshape(nb, len(P.q), n)
    rows = P.q * nb
    t0 = tick()
    f = C.ntt(P, A, rows)
    t1 = tick()
    fr = f.reshape(nb, len(P.q), n)
    acc = C.pmul(fr[0], Bm[0], P.q)
    for j in range(1, nb):
        acc = C.padd(acc, C.pmul(fr[j], Bm[j], P.q), P.q)
    t2 = tick()
    C.intt(P, f, rows)
    t3 = tick()
    res["cfg2"] = entry(f"forward NTT + {nb}-pair MAC + inverse NTT of {nb} of the 64 "
                        "polynomials x 24 limbs", t3 - t0, B // nb)
    res["cfg2"]["ntt_gbs"] = round(2 * 2 * 8 * n * len(rows) / (t1 - t0 + t3 - t2) / 1e9, 3)

    # cfg3: the 32-ciphertext rotation set (30 key switches)
    seed = WL.CFG3["seed"]
    sk = C.secret_key(P, synth.secret(seed, n))
    steps = WL.cfg3_steps()
    take = [0, 1] if single else list(range(len(steps)))
    keys = {}
    for i in take:
        g = P.galois_elt(steps[i])
        if steps[i] % (n // 2) and g not in keys:
            keys[g] = C.keygen_from_seed(P, sk, seed, g)
    cts = {}
    for i in take:
        a, e = synth.encrypt_draws(seed, P.qs(24), n, "cfg3", i)
        cts[i] = C.encrypt(P, sk, C.encode_plain(P, WL.cfg3_slots(i, n // 2), 2.0 ** 40, 24),
                           24, a, e)
    t0 = tick()
    for i in take:
        C.rotate(P, cts[i], steps[i], keys)
    t = tick() - t0
    n_ks = sum(1 for i in take if steps[i] % (n // 2))
    res["cfg3"] = entry(f"{n_ks} of the 30 key switches of the rotation set (24 limbs)", t,
                        30 / n_ks)
    res["cfg3"]["keyswitch_per_s"] = round(n_ks / t, 3)

    # cfg4: the 768 x 1536 projection at 16 limbs, n1 = 16, n2 = 2, 12 inputs,
    # 48 diagonal sets -> 24 complex-paired outputs: baby steps of one input
    # (x 12) plus whole output pairs (pt-MAC of both sets over all inputs and
    # baby steps, two giant steps, conjugation, rescale; x 12 for pairs
    # {0, 23}) -- one thread: 2 of the 15 baby rotations of one input (x 90),
    # the pt-MAC of one input into one set (x 576) and one pair's two giant
    # steps, conjugation and rescale (x 24)
    cfg = WL.CFG4
    seed, lvl, seg = cfg["seed"], cfg["level"], cfg["tokens"]
    n1, n2 = cfg["n1"], cfg["n2"]
    sk = C.secret_key(P, synth.secret(seed, n))
    baby = [q * seg for q in range(n1)]
    giant = [p * n1 * seg for p in range(n2)]
    bsteps = baby[1:3] if single else baby[1:]
    need = set(bsteps) | set(giant[1:])
    keys = {P.galois_elt(r): C.keygen_from_seed(P, sk, seed, P.galois_elt(r)) for r in need}
    keys[P.conj_elt] = C.keygen_from_seed(P, sk, seed, P.conj_elt)
    X, _ = WL.cfg4_values()
    Cc = (n // 2) // seg
    a, e = synth.encrypt_draws(seed, P.qs(lvl), n, "cfg4", 0)
    z0 = OW.pack_input(X, n // 2, seg, Cc, 0) + 1j * OW.pack_input(X, n // 2, seg, Cc, 1)
    x0 = C.encrypt(P, sk, C.encode_plain(P, z0, 2.0 ** 40, lvl), lvl, a, e)
    t0 = tick()
    bb = C.rotate_hoisted(P, x0, [0] + bsteps, keys)
    t_baby = tick() - t0
    n_in = cfg["d_in"] // Cc // 2
    rnd = synth.uniform_residues(seed, "cpu-diag", P.qs(lvl), n)

    def giant_sum(n_u):
        y = None
        for p_ in range(n2):
            acc = None
            for _u in range(n_u):
                for q in range(n1):
                    tq = C.mul_plain(P, bb[q % len(bb)], rnd)
                    acc = tq if acc is None else C.ct_add(P, acc, tq)
            if n_u == n_in:
                acc = C.rotate(P, acc, giant[p_], keys)
                y = acc if y is None else C.ct_add(P, y, acc)
        return y

    if single:
        t0 = tick()
        giant_sum(1)
        t_mac = tick() - t0
        t0 = tick()
        y1 = C.rotate(P, bb[0], giant[1], keys)
        y2 = C.rotate(P, bb[1], giant[1], keys)
        C.rescale(P, C.ct_add(P, y1, C.conjugate(P, y2, keys)))
        t_tail = tick() - t0
        res["cfg4"] = {"sample": "2 of the 15 hoisted baby rotations of one input (x 90); the "
                                 "pt-MAC of one input into one diagonal set (x 576); one output "
                                 "pair's two giant steps, conjugation and rescale (x 24)",
                       "sample_s": round(t_baby + t_mac + t_tail, 3),
                       "factors": [90, 576, 24],
                       "extrapolated_s": round(90 * t_baby + 576 * t_mac + 24 * t_tail, 3)}
    else:
        t0 = tick()
        for _pair in (0, 1):
            y = C.ct_add(P, giant_sum(n_in), C.conjugate(P, giant_sum(n_in), keys))
            C.rescale(P, y)
        t_pairs = tick() - t0
        res["cfg4"] = {"sample": "the hoisted baby steps of one input (15 key switches, x 12); "
                                 "output pairs 0 and 23 whole (pt-MAC of both diagonal sets over "
                                 "12 inputs x 32 baby/giant terms, two giant steps, "
                                 "conjugation, rescale; x 12)",
                       "sample_s": round(t_baby + t_pairs, 3), "factors": [12, 12],
                       "extrapolated_s": round(12 * t_baby + 12 * t_pairs, 3)}

    # cfg5: the scan-contract slice of one Mamba-base token (pool entry 0);
    # the 2048-token sequence is 2048 such tokens -- one thread: the two
    # products of one chunk (x 12) and the reduction of one chunk pair (x 6)
    cfg = WL.CFG5
    seed, lvl, d_s, hd = cfg["seed"], cfg["level"], cfg["d_state"], cfg["head_dim"]
    s_state = 16384
    K = cfg["heads"] * hd * d_s // s_state
    sk = C.secret_key(P, synth.secret(seed, n))
    rlk = C.keygen_from_seed(P, sk, seed, 0)
    keys = {P.galois_elt(d_s >> k): C.keygen_from_seed(P, sk, seed, P.galois_elt(d_s >> k))
            for k in range(1, 8)}
    keys[P.conj_elt] = C.keygen_from_seed(P, sk, seed, P.conj_elt)
    z, cvec, H = WL.cfg5_token(0)
    decay = 1.0 / (1.0 + np.exp(z))
    j = np.arange(n // 2)
    kk = 1 if single else K
    ins = ([], [], [])
    for k in range(kk):
        e_idx = np.minimum(k * (s_state // d_s) + j // d_s, H.shape[0] - 1)
        ok = j < s_state
        vals = (np.where(ok, H[e_idx, j % d_s], 0.0), np.where(ok, decay[e_idx // hd], 0.0),
                np.where(ok, cvec[j % d_s], 0.0))
        scales = (2.0 ** 40, float(P.q[lvl - 1]), float(P.q[lvl - 2]))
        for r in range(3):
            a, e = synth.encrypt_draws(seed, P.qs(lvl), n, "cfg5", 3 * k + r)
            ins[r].append(C.encrypt(P, sk, C.encode_plain(P, vals[r].astype(complex), scales[r],
                                                          lvl), lvl, a, e))
    if single:
        t0 = tick()
        t1 = C.mul_relin_rescale(P, ins[1][0], ins[0][0], rlk)
        t2 = C.mul_relin_rescale(P, t1, ins[2][0][:t1.shape[0]], rlk)
        t_prod = tick() - t0
        t0 = tick()
        chi = C.ct_add(P, t2, C.mul_monomial(P, t2, n // 2))
        xi = OW.reduce_axis(P, chi, d_s, keys)
        C.conjugate(P, xi, keys)
        t_red = tick() - t0
        res["cfg5"] = {"sample": "the two relinearised products of one state chunk (x 12 "
                                 "chunks x 2048 tokens) and the reduction of one chunk pair "
                                 "(7 rotations + conjugation; x 6 pairs x 2048 tokens)",
                       "sample_s": round(t_prod + t_red, 3), "factors": [12 * 2048, 6 * 2048],
                       "extrapolated_s": round(2048 * (12 * t_prod + 6 * t_red), 3)}
    else:
        t0 = tick()
        OW.scan_contract_token(P, ins[0], ins[1], ins[2], rlk, keys, d_s)
        res["cfg5"] = entry("the slice of one token (12 chunks: 24 products, 6 complex-paired "
                            "reductions; 72 key switches), x 2048 tokens", tick() - t0, 2048)
    return res


def cpu_baseline() -> dict:
    """The oracle timed on this host on bounded samples (about 30 s of CPU
    work in all), in two child processes: all cores (the OpenMP default of
    the environment) and one thread (OMP_NUM_THREADS=1; OpenMP fixes its
    thread count per process)."""
    import subprocess
    out = {"kind": "oracle"}
    for mode in ("all", "single"):
        env = dict(os.environ)
        if mode == "single":
            env["OMP_NUM_THREADS"] = "1"
        t0 = time.perf_counter()
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-sample", mode],
                           capture_output=True, text=True, timeout=900, env=env)
        if r.returncode != 0:
            out[mode] = f"not measured: {r.stderr.strip().splitlines()[-1:]}"
            continue
        out[mode] = json.loads(r.stdout.strip().splitlines()[-1])
        out[mode]["wall_s"] = round(time.perf_counter() - t0, 1)
    allc = out.get("all")
    if isinstance(allc, dict):
        out["value"] = allc["cfg2"]["ntt_gbs"]
        out["unit"] = "GB/s"
        out["cores"] = allc["threads"]
        out["keyswitch_per_s"] = allc["cfg3"]["keyswitch_per_s"]
        out["matvec_ms"] = round(allc["cfg4"]["extrapolated_s"] * 1e3, 1)
        out["sample"] = ("bounded samples of all five configurations (see all / single: "
                         "sample, seconds, factor to the whole configuration)")
    out["nproc"] = len(os.sched_getaffinity(0))
    try:
        lscpu = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=30).stdout
        fields = dict(l.split(":", 1) for l in lscpu.splitlines() if ":" in l)
        fields = {k.strip(): v.strip() for k, v in fields.items()}
        out["cpu_model"] = fields.get("Model name")
        # the model string can be generic under virtualisation: keep the
        # identifying fields lscpu reports next to it
        out["lscpu"] = {k: fields[k] for k in (
            "Architecture", "Vendor ID", "Model name", "CPU family", "Model", "Stepping",
            "CPU(s)", "Thread(s) per core", "Core(s) per socket", "Socket(s)", "CPU max MHz",
            "L3 cache", "Hypervisor vendor", "Virtualization type") if k in fields}
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    return out


# -------------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-affine", action="store_true",
                    help="skip the components timed after the steps (whole-sequence "
                         "scan-contract, affine prefix scan, HEScan layer)")
    ap.add_argument("--no-hescan", action="store_true",
                    help="skip the HEScan layer component (L=2048: construction, scan, "
                         "contraction)")
    ap.add_argument("--hescan-sweep", action="store_true",
                    help="only the HEScan layer at L = 128 .. 2048 (blocks of min(1024, L))")
    ap.add_argument("--scan-sweep", action="store_true",
                    help="only the resident-schedule block-size sweep at L=2048 (one chunk)")
    ap.add_argument("--affine-only", action="store_true",
                    help="set up and time only the affine prefix scan component (profiling)")
    ap.add_argument("--calibrate-only", action="store_true",
                    help="only the register-resident VALU calibrations and the fp64 / int64 "
                         "modular-product probe (one JSON line)")
    ap.add_argument("--cpu-sample", choices=("all", "single"),
                    help="(internal) time the oracle's bounded samples in this process and "
                         "print them as JSON; no GPU is used")
    ap.add_argument("--matvec-double-hoisting", action="store_true",
                    help="only the projection with and without double hoisting (lazy "
                         "ModDown), at N = 2^12 (64 x 64) and at the 768 x 1536 shape")
    ap.add_argument("--stored-keys", action="store_true",
                    help="switching keys stored whole (both halves read by every key switch) "
                         "instead of seed-expanded")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one 1 GiB device-to-device copy, the reference kernel for "
                         "scaling hardware traffic counters")
    args = ap.parse_args()
    if args.cpu_sample:
        print(json.dumps(cpu_sample(args.cpu_sample)), flush=True)
        return
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU per process and has no multi-GPU path; use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_17442_amd import fesc as F

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.ones(1 << 27, dtype=torch.int64, device="cuda")   # 1 GiB
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.matvec_double_hoisting:
        print(json.dumps({"matvec_double_hoisting": matvec_double_hoisting(F, torch, np)}),
              flush=True)
        return
    if args.calibrate_only:
        pr = F.find_primes(16, 50, 32)
        ctx = F.Context(16, pr[8:], pr[:8])
        out = {"valu_peaks_per_s": {k: round(ctx.calib_valu(v), -9) for k, v in (
            ("ct_butterflies", F.CALIB_CT), ("gs_butterflies", F.CALIB_GS),
            ("mod_macs", F.CALIB_MAC))}, "modmul_probe": modmul_probe(ctx, F),
            "hbm_measured_ceilings_gbs": {
                "read": round(ctx.calib_hbm(F.CALIB_HBM_READ) / 1e9, 1),
                "copy": round(ctx.calib_hbm(F.CALIB_HBM_COPY) / 1e9, 1)}}
        print(json.dumps(out), flush=True)
        return
    if args.hescan_sweep:
        W = Workloads(F, torch, np, affine_only=True, seeded_keys=not args.stored_keys)
        sweep = {}
        for L in (128, 256, 512, 1024, 2048):
            log(f"HEScan layer sweep: L = {L}")
            sweep[L] = time_hescan(W, F, torch, np, L=L, block=min(1024, L))
        print(json.dumps({"hescan_layer_sweep": sweep}), flush=True)
        return
    if args.scan_sweep:
        W = Workloads(F, torch, np, affine_only=True, seeded_keys=not args.stored_keys)
        print(json.dumps({"scan_block_sweep": scan_block_sweep(W, F, torch, np)}), flush=True)
        return
    if args.affine_only:
        W = Workloads(F, torch, np, affine_only=True, seeded_keys=not args.stored_keys)
        comp = {"affine_scan": time_affine(W, F, torch, np)}
        if not args.no_hescan:
            comp["hescan_layer"] = time_hescan(W, F, torch, np)
        print(json.dumps({"components": comp}), flush=True)
        return
    W = Workloads(F, torch, np, seeded_keys=not args.stored_keys)
    torch.cuda.synchronize()
    # the device's practical streaming ceilings (8 GiB read; 8 GiB copied)
    hbm = {"read_gbs": round(W.ctx.calib_hbm(F.CALIB_HBM_READ) / 1e9, 1),
           "copy_gbs": round(W.ctx.calib_hbm(F.CALIB_HBM_COPY) / 1e9, 1)}
    # register-resident arithmetic peaks of this device (VALU roof)
    peak = {k: W.ctx.calib_valu(v) for k, v in (("ct", F.CALIB_CT), ("gs", F.CALIB_GS),
                                                 ("mac", F.CALIB_MAC))}
    modmul = modmul_probe(W.ctx, F)

    def new_events(k):
        return [torch.cuda.Event(enable_timing=True) for _ in range(k)]

    def step(ev):
        W.run_ntt(ev["ntt"])
        W.run_ks(ev["ks"])
        W.run_matvec(ev["mv"])
        W.run_scan_contract(ev["sc"])

    def step_events():
        return {"ntt": new_events(4), "ks": new_events(2), "mv": new_events(2),
                "sc": new_events(2)}

    for _ in range(args.warmup):
        step(step_events())
    torch.cuda.synchronize()
    evs = [step_events() for _ in range(args.steps)]
    phases = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
        if k == args.steps - 1:
            pass
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    phases.append(W.mv_plan.phase_ms())

    el = lambda e, i, j: e[i].elapsed_time(e[j])
    fwd = float(np.mean([el(e["ntt"], 0, 1) for e in evs]))
    mac = float(np.mean([el(e["ntt"], 1, 2) for e in evs]))
    inv = float(np.mean([el(e["ntt"], 2, 3) for e in evs]))
    ks = float(np.mean([el(e["ks"], 0, 1) for e in evs]))
    mv = float(np.median([el(e["mv"], 0, 1) for e in evs]))
    sc = float(np.median([el(e["sc"], 0, 1) for e in evs]))
    baby_ms, ptmac_ms, tail_ms = phases[-1]
    # HEScan affine prefix scan, timed after the steps with the projection's
    # diagonal bank released (its 128 x 12 x 2 ciphertexts take 51.5 GB)
    affine = hescan = sc_seq = broadcast = None
    if not args.no_affine:
        sc_seq = W.time_scan_contract_sequence()
        del W.mv_plan, W.bank, W.sc_in, W.sc_out
        torch.cuda.empty_cache()
        affine = time_affine(W, F, torch, np)
        if not args.no_hescan:
            hescan = time_hescan(W, F, torch, np)
        broadcast = time_broadcast(W, F, torch, np)
    n, rows = W.n, W.limbs * W.batch
    bytes_dir = 2 * 8 * n * rows
    ntt_gbs = 2 * bytes_dir / ((fwd + inv) * 1e-3) / 1e9
    mac_bytes = 2 * 8 * n * rows + 8 * n * W.limbs
    s = W.mv_shape
    lv = W.mv_level
    ct_bytes = 2 * lv * n * 8
    ptmac_bytes = W.bank_bytes + s["n_in"] * s["n1"] * ct_bytes \
        + s["n_out"] * s["n2"] * ct_bytes
    ptmac_gbs = ptmac_bytes / (ptmac_ms * 1e-3) / 1e9
    # VALU work: a limb transform is (N/2) log N butterflies; a key switch at
    # level l with alpha special primes and beta digits transforms l + 2 alpha
    # rows inversely (c1, the P-rows of both components) and beta(l + alpha) - l
    # + 2 l rows forward (extended digits, y), and spends sum_j alpha_j (l +
    # alpha - alpha_j) + 2 alpha l basis-conversion and 2 beta (l + alpha)
    # inner-product multiply-accumulates per coefficient.
    half_logn = n // 2 * W.log_n
    ntt_bfly = rows * half_logn
    ntt_valu_frac = (ntt_bfly / peak["ct"] + ntt_bfly / peak["gs"]) / ((fwd + inv) * 1e-3)
    lv, al = W.ks_level, W.alpha
    beta = -(-lv // al)
    digits = [min(al, lv - j * al) for j in range(beta)]
    inv_rows, fwd_rows = lv + 2 * al, beta * (lv + al) - lv + 2 * lv
    ks_bfly = (inv_rows + fwd_rows) * half_logn
    ks_macs = (sum(a * (lv + al - a) for a in digits) + 2 * al * lv + 2 * beta * (lv + al)) * n
    ks_valu_frac = ((inv_rows * half_logn / peak["gs"] + fwd_rows * half_logn / peak["ct"]
                     + ks_macs / peak["mac"]) * W.n_ks / (ks * 1e-3))
    # whole-operation fractions against the benchmark spec's target (>= 60% of the
    # HBM or VALU roofline for the N = 2^16 NTT and for key switching): NTT
    # bytes = one read + one write of the data per direction; a key switch's
    # bytes = its key 2 beta (l + alpha) 8N plus the ciphertext read and
    # written 2 * 2l * 8N (151 MB at 24 limbs; keys shared by two jobs of the
    # set make the set's own minimum lower, so this fraction is generous)
    ks_bytes = (2 * beta * (lv + al) + 2 * 2 * lv) * 8 * n
    ks_hbm_frac = ks_bytes * W.n_ks / (ks * 1e-3) / (HBM_PEAK_GBS * 1e9)
    targets = {
        "target_frac": 0.6,
        "ntt": {"hbm_frac": round(ntt_gbs / HBM_PEAK_GBS, 4),
                "valu_frac": round(ntt_valu_frac, 4),
                "met": bool(max(ntt_gbs / HBM_PEAK_GBS, ntt_valu_frac) >= 0.6)},
        "keyswitch": {"valu_frac": round(ks_valu_frac, 4), "hbm_frac": round(ks_hbm_frac, 4),
                      "bytes_per_key_switch": ks_bytes,
                      "us_per_key_switch": round(ks * 1e3 / W.n_ks, 2),
                      "met": bool(max(ks_valu_frac, ks_hbm_frac) >= 0.6),
                      "valu_work": "83.9 M butterflies + 75.5 M modular MACs per key switch "
                                   "(the conversions' MACs counted as VALU MACs); the "
                                   "conversions run as int8 matrix-core products, which leaves "
                                   "about 27 us of VALU work per key switch: the pipeline is "
                                   "bound by the bytes its kernels move"},
        "note": "whole operations timed with HIP events in the step; the per-kernel key-switch "
                "fraction in rooflines_other is a diagnostic (it scores each kernel against "
                "its own floor, so intermediate round trips count as useful work)",
    }
    out = {
        "metric": METRIC,
        "value": round(ntt_gbs, 2),
        "unit": "GB/s (NTT, N=2^16, 24 limbs)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64 residues, fp64 modular arithmetic",
        "data": "synthetic (uniform residues seed 1; U[-1,1] slots seed 2; N(0,1) x N(0,0.02^2) "
                "projection seed 3; N(0,1) Mamba-base token seed 4; uniform residues for the "
                "affine scan)",
        "config": {"workload": "N=2^16, 24 limbs: NTT microbench (64 polys fwd + 64-pair MAC + "
                               "inv) + 32-ciphertext rotation set (30 key switches, dnum 3, 8 "
                               "special primes) + 768x1536 BSGS projection (12 -> 24 cts, "
                               "16 limbs) + scan-contract slice of a block of 16 Mamba-base "
                               "tokens (12 state chunks each, 20 -> 18 limbs)",
                   "log_n": 16, "limbs": 24, "special_primes": 8, "parallelism": "single GPU",
                   "switching_keys": "seed-expanded (seed and b half stored, a regenerated "
                                     "in the key switch)" if W.seeded_keys else "stored whole"},
        "components": {
            "ntt_gbs": round(ntt_gbs, 2),
            "ntt_fwd_ms": round(fwd, 4), "ntt_inv_ms": round(inv, 4),
            "mac_ms": round(mac, 4), "mac_gbs": round(mac_bytes / (mac * 1e-3) / 1e9, 2),
            "keyswitch_per_s": round(W.n_ks / (ks * 1e-3), 1),
            "keyswitch_set_ms": round(ks, 4), "key_switches": W.n_ks,
            "matvec_ms": round(mv, 3),
            "matvec_phases_ms": {"baby_steps": round(baby_ms, 3), "pt_mac": round(ptmac_ms, 3),
                                 "giant_conj_rescale": round(tail_ms, 3)},
            "scan_contract_ms_per_token": round(sc / W.sc_shape["tokens"], 3),
            "scan_contract_tokens_per_call": W.sc_shape["tokens"],
            "scan_contract_sequence": sc_seq,
            "matvec_outputs": {"ciphertexts": W.mv_shape["n_out"] // 2,
                               "blocks": W.mv_shape["n_out"],
                               "packing": "complex-paired outputs: block 2P real part, "
                                          "2P+1 imaginary part of output P",
                               "tail_key_switches": W.mv_shape["n_out"] * (W.mv_shape["n2"] - 1)
                               + W.mv_shape["n_out"] // 2},
            "diagonal_bank_build_s": {"total": round(W.bank_build_s, 2),
                                      "host_slot_values": 0.0,
                                      "diagonals": W.mv_shape["n_diag"],
                                      "note": "offline, all on the device: slot values "
                                              "(fesc_bsgs_diagonal_slots), encoding, lift, NTT, "
                                              "bank packing"},
            "affine_scan": affine,
            "hescan_layer": hescan,
            "broadcast": broadcast,
        },
        "roofline": {
            "bound": "hbm", "kernel": "k_ptmac (projection plaintext-diagonal MAC)",
            "achieved": round(ptmac_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ptmac_gbs / HBM_PEAK_GBS, 4),
            "traffic": profiled_traffic(PTMAC_PROFILE, PTMAC_SOURCES),
            "algorithmic_bytes": ptmac_bytes,
            "frac_of_measured_read_ceiling": round(ptmac_gbs / hbm["read_gbs"], 4),
        },
        "targets": targets,
        "rooflines_other": {
            "hbm_measured_ceilings": dict(hbm, note="fesc_calib_hbm: a streaming read with "
                                          "16-byte non-temporal loads and a 16-byte copy "
                                          "(read + write), "
                                          "8 GiB each; the practical ceilings of HBM-bound "
                                          "kernels on this device, against the 8 TB/s peak"),
            "ntt_valu": {"bound": "alu",
                         "achieved": round(2 * ntt_bfly / ((fwd + inv) * 1e-3) / 1e12, 4),
                         "peak": round(2 / (1 / peak["ct"] + 1 / peak["gs"]) / 1e12, 4),
                         "unit": "T butterflies/s", "frac": round(ntt_valu_frac, 4),
                         "peak_source": "fesc_calib_valu (register-resident CT/GS butterflies)"},
            "ntt_hbm_hardware": {"bound": "hbm", "achieved": round(2 * ntt_gbs, 1),
                                 "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                 "frac": round(2 * ntt_gbs / HBM_PEAK_GBS, 4),
                                 "note": "two passes each read and write the data once"},
            "keyswitch_per_kernel_diagnostic": keyswitch_per_kernel(),
            "keyswitch_valu": {"bound": "alu", "frac": round(ks_valu_frac, 4),
                               "per_key_switch": {"butterflies": ks_bfly, "mod_macs": ks_macs},
                               "peak_butterflies_per_s": round(peak["ct"], -9),
                               "peak_macs_per_s": round(peak["mac"], -9)},
            "ntt_fwd_two_pass": {"bound": "hbm", "achieved": round(bytes_dir / (fwd * 1e-3) / 1e9,
                                                                   1),
                                 "peak": HBM_PEAK_GBS, "unit": "GB/s"},
            "mac": {"bound": "hbm", "achieved": round(mac_bytes / (mac * 1e-3) / 1e9, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s"},
            "modmul_probe": modmul,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU reference sample")
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
