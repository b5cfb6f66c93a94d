"""MI355X (gfx950) RNS-CKKS linear hot path of FESC (arXiv 2608.17442).

``libfesc.so`` (built from ``csrc/`` by ``build.py``) holds the HIP kernels
and the C ABI declared in ``include/fesc.h``; ``fesc`` is its ctypes binding.
"""
