"""MI355X-native (gfx950) MoE-layer hot path: HIP kernels behind a C ABI.

The kernels and the C ABI live in ``csrc/`` and ``include/moe.h``; ``moe``
is the ctypes binding (argument marshalling only), ``inputs`` the seeded
workload generator. Importing the package does not load the library; the
binding loads it on first use and fails loudly if it is missing.
"""
__version__ = "0.1.0"
