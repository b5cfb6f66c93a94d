"""CPU reference ("the oracle") for FESC's RNS-CKKS linear hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import, call or link anything in this
package.  It shares no code with the GPU library (``paper_2608_17442_amd``)
and neither imports the other; both take their random draws from ``synth``.

Layout of the package:
  ckks_oracle.c  exact modular arithmetic in C (128-bit products, '%'):
                 primes, roots, radix-2 NTT, basis conversion, automorphism;
  encoding.py    slot encoding / decoding (numpy FFT) and exact CRT lift;
  ckks.py        keys, encryption, and every CKKS operation of the path;
  workloads.py   the matvec and scan-contract compositions.

Parity status of every function is listed in the module that defines it; all
of them are pinned by tests under ``tests/`` (test_oracle_*.py).
"""
