"""CPU oracle for the MoE-layer hot path (test infrastructure only).

Importable only from the test suite, the smoke check and the benchmark's
CPU-baseline leg; the product path never touches it.
"""
