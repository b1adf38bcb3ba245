"""fp64 CPU oracle for factorized sparse causal attention.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
CPU-baseline leg of bench.py.  The GPU library never imports it.
"""
